// Row kernels of the scoring forward: hidden rows -> LM-head operand, and the
// log-softmax over the vocabulary with the teacher-forced target gather and
// the greedy argmax.
#include <math.h>

#include <algorithm>

#include "common.h"

namespace kvr {

namespace {

// X = Y rows [0, R) (fp32, row stride d) as the LM head's operand: a
// compensated bf16 pair in operand order (PERM) or row-major, or fp32.
template <typename TO, bool PERM>
__global__ __launch_bounds__(256) void to_operand_kernel(const float *Y, int d, TO *X, TO *X_lo) {
    const int r = blockIdx.x;
    for (int c = threadIdx.x; c < d; c += 256)
        store_operand(X, X_lo, PERM ? perm_offset(r, c, d) : (size_t)r * d + c, Y[(size_t)r * d + c]);
}

// Log-softmax in two stages so that a few rows still spread over the chip.
// The logits of row r are z[v] = sum of the `nsplit` fp32 tiles part[s][r][V]
// (fixed order).  Stage 1: block (chunk c, row r) reduces the vocabulary slice
// c to (max, sum of exp(z - max), lowest index of the max).  Stage 2: one
// wavefront per row merges the chunks in a fixed tree and writes
//   argmax[r] = the lowest index of max z,
//   lp[r]     = z[target[r]] - max z - log(sum exp(z - max z))   (r < n_targets)
// and, when `next` is given, next[0] = argmax of the block's last row.
struct LsmStat {
    float m, s;
    int32_t idx, pad;
};

__device__ __forceinline__ float z_at(const float *part, int nsplit, int R, int V, int r, int v) {
    float z = part[(size_t)r * V + v];
    for (int q = 1; q < nsplit; ++q) z += part[((size_t)q * R + r) * V + v];
    return z;
}

// (m, s, i) <- merge of two partial reductions; an empty one has m = -inf, s = 0.
__device__ __forceinline__ void lsm_merge(float &m, float &s, int &i, float m2, float s2, int i2) {
    const float M = fmaxf(m, m2);
    if (M == -INFINITY) return;
    s = (m == -INFINITY ? 0.f : s * __expf(m - M)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - M));
    if (m2 > m || (m2 == m && i2 < i)) i = i2;
    m = M;
}

__device__ __forceinline__ void lsm_wave(float &m, float &s, int &i) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o), s2 = __shfl_xor(s, o);
        const int i2 = __shfl_xor(i, o);
        lsm_merge(m, s, i, m2, s2, i2);
    }
}

__global__ __launch_bounds__(256) void logsoftmax_chunk_kernel(const float *part, int nsplit, int R, int V, int C,
                                                               LsmStat *st) {
    __shared__ LsmStat red[4];
    const int c = blockIdx.x, r = blockIdx.y;
    const int chunk = (V + C - 1) / C;
    const int v0 = c * chunk, v1 = min(V, v0 + chunk);
    float m = -INFINITY, sum = 0.f;
    int mi = 0x7fffffff;
    for (int v = v0 + (int)threadIdx.x; v < v1; v += 256) {  // ascending v: the first maximum is kept
        const float z = z_at(part, nsplit, R, V, r, v);
        if (z > m) {
            sum = (m == -INFINITY ? 0.f : sum * __expf(m - z)) + 1.f;
            m = z;
            mi = v;
        } else {
            sum += __expf(z - m);
        }
    }
    lsm_wave(m, sum, mi);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[w] = LsmStat{m, sum, mi, 0};
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int q = 1; q < 4; ++q) lsm_merge(m, sum, mi, red[q].m, red[q].s, red[q].idx);
        st[(size_t)r * C + c] = LsmStat{m, sum, mi, 0};
    }
}

__global__ __launch_bounds__(64) void logsoftmax_final_kernel(const float *part, int nsplit, int R, int V, int C,
                                                              const LsmStat *st, const int32_t *target, int n_targets,
                                                              float *lp, int32_t *argmax, int32_t *next) {
    const int r = blockIdx.x, lane = threadIdx.x;
    float m = -INFINITY, s = 0.f;
    int mi = 0x7fffffff;
    for (int c = lane; c < C; c += 64) {
        const LsmStat q = st[(size_t)r * C + c];
        lsm_merge(m, s, mi, q.m, q.s, q.idx);
    }
    lsm_wave(m, s, mi);
    if (lane == 0) {
        if (argmax) argmax[r] = mi;
        if (r < n_targets) {
            const int tg = target[r];
            lp[r] = (tg >= 0 && tg < V) ? z_at(part, nsplit, R, V, r, tg) - m - logf(s) : NAN;
        }
        if (next && r == R - 1) next[0] = mi;
    }
}

constexpr int LSM_CHUNK = 2048;  // target vocabulary entries per stage-1 block
constexpr int LSM_MAXC = 64;     // chunks per row at most

int lsm_chunks(int V) { return std::min(LSM_MAXC, std::max(1, (V + LSM_CHUNK - 1) / LSM_CHUNK)); }

}  // namespace

hipError_t launch_to_operand(bool bf16, bool perm, const float *Y, int R, int d, void *X, void *X_lo, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (bf16 && perm) kvr_launch((to_operand_kernel<bf16_t, true>), dim3(R), dim3(256), 0, s, Y, d, (bf16_t *)X, (bf16_t *)X_lo);
    else if (bf16) kvr_launch((to_operand_kernel<bf16_t, false>), dim3(R), dim3(256), 0, s, Y, d, (bf16_t *)X, (bf16_t *)X_lo);
    else kvr_launch((to_operand_kernel<float, false>), dim3(R), dim3(256), 0, s, Y, d, (float *)X, (float *)nullptr);
    return hipGetLastError();
}

size_t logsoftmax_ws_bytes(int R, int V) { return (size_t)R * lsm_chunks(V) * sizeof(LsmStat); }

hipError_t launch_logsoftmax(const float *part, int nsplit, int R, int V, const int32_t *target, int n_targets,
                             float *lp, int32_t *argmax, int32_t *next, void *ws, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (nsplit < 1 || !ws || (n_targets > 0 && (!target || !lp))) return hipErrorInvalidValue;
    const int C = lsm_chunks(V);
    kvr_launch(logsoftmax_chunk_kernel, dim3(C, R), dim3(256), 0, s, part, nsplit, R, V, C, (LsmStat *)ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    kvr_launch(logsoftmax_final_kernel, dim3(R), dim3(64), 0, s, part, nsplit, R, V, C, (const LsmStat *)ws, target,
               n_targets, lp, argmax, next);
    return hipGetLastError();
}

}  // namespace kvr
