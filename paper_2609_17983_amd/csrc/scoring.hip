// Row kernels of the scoring forward: hidden rows -> LM-head operand, and the
// log-softmax over the vocabulary with the teacher-forced target gather and
// the greedy argmax.
#include <math.h>

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

// One block per row r: z = sum of the `nsplit` fp32 logit tiles part[s][r][V]
// (fixed order), then
//   argmax[r] = the lowest index of max z,
//   lp[r]     = z[target[r]] - max z - log(sum exp(z - max z))   (r < n_targets)
// and, when `next` is given, next[0] = argmax of the block's last row.
__global__ __launch_bounds__(1024) void logsoftmax_kernel(const float *part, int nsplit, int R, int V,
                                                          const int32_t *target, int n_targets, float *lp,
                                                          int32_t *argmax, int32_t *next) {
    __shared__ float smax[16];
    __shared__ int sidx[16];
    __shared__ float ssum[16];
    const int r = blockIdx.x;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    auto z_at = [&](int v) {
        float z = part[(size_t)r * V + v];
        for (int s = 1; s < nsplit; ++s) z += part[((size_t)s * R + r) * V + v];
        return z;
    };
    float m = -INFINITY;
    int mi = 0x7fffffff;
    for (int v = threadIdx.x; v < V; v += 1024) {
        const float z = z_at(v);
        if (z > m) { m = z; mi = v; }  // ascending v per thread: the first maximum is kept
    }
    // max with the lowest index among equal maxima
    for (int o = 32; o > 0; o >>= 1) {
        const float m2 = __shfl_xor(m, o);
        const int i2 = __shfl_xor(mi, o);
        if (m2 > m || (m2 == m && i2 < mi)) { m = m2; mi = i2; }
    }
    if (lane == 0) { smax[w] = m; sidx[w] = mi; }
    __syncthreads();
    m = smax[0];
    mi = sidx[0];
    for (int q = 1; q < 16; ++q)
        if (smax[q] > m || (smax[q] == m && sidx[q] < mi)) { m = smax[q]; mi = sidx[q]; }
    float s = 0.f;
    for (int v = threadIdx.x; v < V; v += 1024) s += __expf(z_at(v) - m);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) ssum[w] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.f;
        for (int q = 0; q < 16; ++q) t += ssum[q];
        if (argmax) argmax[r] = mi;
        if (r < n_targets) {
            const int tg = target[r];
            lp[r] = (tg >= 0 && tg < V) ? z_at(tg) - m - logf(t) : NAN;
        }
        if (next && r == R - 1) next[0] = mi;
    }
}

}  // namespace

hipError_t launch_to_operand(bool bf16, bool perm, const float *Y, int R, int d, void *X, void *X_lo, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (bf16 && perm) kvr_launch((to_operand_kernel<bf16_t, true>), dim3(R), dim3(256), 0, s, Y, d, (bf16_t *)X, (bf16_t *)X_lo);
    else if (bf16) kvr_launch((to_operand_kernel<bf16_t, false>), dim3(R), dim3(256), 0, s, Y, d, (bf16_t *)X, (bf16_t *)X_lo);
    else kvr_launch((to_operand_kernel<float, false>), dim3(R), dim3(256), 0, s, Y, d, (float *)X, (float *)nullptr);
    return hipGetLastError();
}

hipError_t launch_logsoftmax(const float *part, int nsplit, int R, int V, const int32_t *target, int n_targets,
                             float *lp, int32_t *argmax, int32_t *next, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (nsplit < 1 || (n_targets > 0 && (!target || !lp))) return hipErrorInvalidValue;
    kvr_launch(logsoftmax_kernel, dim3(R), dim3(1024), 0, s, part, nsplit, R, V, target, n_targets, lp, argmax, next);
    return hipGetLastError();
}

}  // namespace kvr
