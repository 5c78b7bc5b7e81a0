// Host-side position selection (paper Table 1): EditLocal and Random over the
// downstream pool D = [edit_end, n - 1).
#include <algorithm>
#include <cstdint>
#include <vector>

#include "../../include/kvr.h"

namespace kvr {
void set_global_error(const char *msg);
}

namespace {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the state advances by the
// golden-ratio increment and each output is the state run through the
// variant-13 mixing function.
struct SplitMix64 {
    uint64_t state;
    explicit SplitMix64(uint64_t seed) : state(seed) {}
    uint64_t next() {
        state += 0x9E3779B97F4A7C15ull;
        uint64_t z = state;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
};

}  // namespace

extern "C" kvr_status kvr_select(kvr_policy policy, int32_t n, int32_t edit_start, int32_t edit_end,
                                 int32_t K, uint64_t seed, int32_t *h_out, int32_t *n_out) {
    if (!n_out || (K > 0 && !h_out) || K < 0) {
        kvr::set_global_error("kvr_select: NULL output or negative K");
        return KVR_E_ARG;
    }
    if (policy != KVR_EDIT_LOCAL && policy != KVR_RANDOM) {
        kvr::set_global_error("kvr_select: unknown policy");
        return KVR_E_ARG;
    }
    if (n < 1 || edit_start < 0 || edit_start > edit_end || edit_end > n) {
        kvr::set_global_error("kvr_select: need n >= 1 and 0 <= edit_start <= edit_end <= n");
        return KVR_E_RANGE;
    }
    const int64_t pool_begin = edit_end;
    const int64_t pool_size = std::max<int64_t>(0, (int64_t)(n - 1) - pool_begin);
    const int64_t k = std::min<int64_t>(K, pool_size);
    *n_out = (int32_t)k;
    if (k == 0) return KVR_OK;
    if (policy == KVR_EDIT_LOCAL) {
        for (int64_t i = 0; i < k; ++i) h_out[i] = (int32_t)(pool_begin + i);
        return KVR_OK;
    }
    std::vector<int32_t> pool((size_t)pool_size);
    for (int64_t i = 0; i < pool_size; ++i) pool[(size_t)i] = (int32_t)(pool_begin + i);
    SplitMix64 rng(seed);
    for (int64_t i = 0; i < k; ++i) {
        const uint64_t span = (uint64_t)(pool_size - i);
        const int64_t j = i + (int64_t)(rng.next() % span);
        std::swap(pool[(size_t)i], pool[(size_t)j]);
    }
    std::sort(pool.begin(), pool.begin() + k);
    std::copy(pool.begin(), pool.begin() + k, h_out);
    return KVR_OK;
}

extern "C" kvr_status kvr_select_to_boundary(int32_t n, int32_t edit_start, int32_t edit_end, int32_t boundary,
                                             int32_t capacity, int32_t *h_out, int32_t *n_out) {
    if (!n_out || capacity < 0 || (capacity > 0 && !h_out)) {
        kvr::set_global_error("kvr_select_to_boundary: NULL output or negative capacity");
        return KVR_E_ARG;
    }
    if (n < 1 || edit_start < 0 || edit_start > edit_end || edit_end > n || boundary < edit_end) {
        kvr::set_global_error("kvr_select_to_boundary: need n >= 1, 0 <= edit_start <= edit_end <= n, "
                              "boundary >= edit_end");
        return KVR_E_RANGE;
    }
    const int64_t end = std::min<int64_t>(boundary, (int64_t)n - 1);
    const int64_t k = std::max<int64_t>(0, end - edit_end);
    if (k > capacity) {
        kvr::set_global_error("kvr_select_to_boundary: more positions than the output capacity");
        return KVR_E_RANGE;
    }
    for (int64_t i = 0; i < k; ++i) h_out[i] = (int32_t)(edit_end + i);
    *n_out = (int32_t)k;
    return KVR_OK;
}
