// Host-side repair metrics (paper Section 3, "What counts as repaired";
// Eq. 2 and Eq. 3), computed from the outputs of kvr_score and kvr_generate.
#include <cstdint>

#include "../../include/kvr.h"

namespace kvr {
void set_global_error(const char *msg);
}

namespace {

// Whether `sub` occurs in `seq` as a contiguous run (an empty run always does).
bool occurs(const int32_t *seq, int32_t n, const int32_t *sub, int32_t k) {
    if (k == 0) return true;
    for (int32_t i = 0; i + k <= n; ++i) {
        int32_t j = 0;
        while (j < k && seq[i + j] == sub[j]) ++j;
        if (j == k) return true;
    }
    return false;
}

}  // namespace

extern "C" kvr_status kvr_answer_logprob(const float *h_logprob, int32_t n_logprob, int32_t query_len,
                                         int32_t answer_len, double *out) {
    if (!h_logprob || !out) {
        kvr::set_global_error("kvr_answer_logprob: NULL argument");
        return KVR_E_ARG;
    }
    // entry j of kvr_score's output predicts appended token j + 1, so the
    // answer's tokens are predicted by entries query_len-1 .. query_len+answer_len-2
    if (query_len < 1 || answer_len < 1 || (int64_t)query_len - 1 + answer_len > n_logprob) {
        kvr::set_global_error("kvr_answer_logprob: the scored block does not hold the whole answer");
        return KVR_E_RANGE;
    }
    double s = 0.0;
    for (int32_t j = 0; j < answer_len; ++j) s += (double)h_logprob[query_len - 1 + j];
    *out = s / answer_len;
    return KVR_OK;
}

extern "C" kvr_status kvr_margin_recovery(double m_repaired, double m_stale, double m_oracle, double *out,
                                          int32_t *defined) {
    if (!out || !defined) {
        kvr::set_global_error("kvr_margin_recovery: NULL output");
        return KVR_E_ARG;
    }
    const double gap = m_oracle - m_stale;
    *defined = gap != 0.0;
    *out = *defined ? (m_repaired - m_stale) / gap : 0.0;
    return KVR_OK;
}

extern "C" kvr_status kvr_flipped(const int32_t *h_continuation, int32_t n_continuation, const int32_t *h_a_new,
                                  int32_t n_new, const int32_t *h_a_old, int32_t n_old, int32_t *out) {
    if (!out || n_continuation < 0 || n_new < 0 || n_old < 0 || (n_continuation > 0 && !h_continuation) ||
        (n_new > 0 && !h_a_new) || (n_old > 0 && !h_a_old)) {
        kvr::set_global_error("kvr_flipped: NULL or negative-length argument");
        return KVR_E_ARG;
    }
    *out = occurs(h_continuation, n_continuation, h_a_new, n_new) &&
           !occurs(h_continuation, n_continuation, h_a_old, n_old);
    return KVR_OK;
}
