// Device side of the CacheBlend selector (Table 1: top-K positions by the
// key/value deviation of one layer): per-position deviation between freshly
// computed and stale keys/values, and a block-wide top-K.
#include <math.h>

#include "common.h"

namespace kvr {

namespace {

// One wavefront per position p in [p0, p1):
//   dev[p - p0] = || K_fresh[p] - K_stale[p] ||_2 + || V_fresh[p] - V_stale[p] ||_2
// with the norms over all kv heads and dimensions of layer `fl` of the fresh
// cache and layer `sl` of the stale one.
template <typename T>
__global__ __launch_bounds__(256) void kv_deviation_kernel(const T *fresh, int fresh_ncap, int fl, const T *stale,
                                                           int stale_ncap, int sl, int Hkv, int hd, int p0, int p1,
                                                           float *dev) {
    const int lane = threadIdx.x & 63;
    const int p = p0 + blockIdx.x * 4 + (threadIdx.x >> 6);
    if (p >= p1) return;
    float sk = 0.f, sv = 0.f;
    for (int g = 0; g < Hkv; ++g)
        for (int i = lane; i < hd; i += 64) {
            const size_t fk = (((size_t)fl * 2 + 0) * Hkv + g) * fresh_ncap * hd + (size_t)p * hd + i;
            const size_t fv = (((size_t)fl * 2 + 1) * Hkv + g) * fresh_ncap * hd + (size_t)p * hd + i;
            const size_t sk_i = (((size_t)sl * 2 + 0) * Hkv + g) * stale_ncap * hd + (size_t)p * hd + i;
            const size_t sv_i = (((size_t)sl * 2 + 1) * Hkv + g) * stale_ncap * hd + (size_t)p * hd + i;
            const float a = to_f32(fresh[fk]) - to_f32(stale[sk_i]);
            const float b = to_f32(fresh[fv]) - to_f32(stale[sv_i]);
            sk += a * a;
            sv += b * b;
        }
    for (int o = 32; o > 0; o >>= 1) {
        sk += __shfl_xor(sk, o);
        sv += __shfl_xor(sv, o);
    }
    if (lane == 0) dev[p - p0] = sqrtf(sk) + sqrtf(sv);
}

__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // monotone map of floats to unsigned
}

// Exclusive scan over the block of per-thread counts (thread order).
__device__ __forceinline__ int block_exclusive_scan(int c, int *buf) {
    buf[threadIdx.x] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int q = 0; q < 1024; ++q) { const int v = buf[q]; buf[q] = acc; acc += v; }
    }
    __syncthreads();
    const int r = buf[threadIdx.x];
    __syncthreads();
    return r;
}

// The K largest of m deviations (ties: lower position first), written as
// ascending positions p0 + i.  One 1024-thread block.  A radix select over the
// order-preserving 32-bit keys finds the K-th largest key T (four 8-bit
// passes with a 256-bucket histogram); every key above T is taken, and of the
// keys equal to T the lowest positions fill the rest.  Positions are emitted
// in ascending order with block scans over contiguous per-thread chunks.
__global__ __launch_bounds__(1024) void topk_kernel(const float *dev, int m, int K, int p0, int32_t *out) {
    __shared__ int hist[256];
    __shared__ int scan[1024];
    __shared__ uint32_t s_prefix, s_mask;
    __shared__ int s_left;
    if (threadIdx.x == 0) { s_prefix = 0; s_mask = 0; s_left = K; }
    __syncthreads();
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = threadIdx.x; i < 256; i += 1024) hist[i] = 0;
        __syncthreads();
        const uint32_t prefix = s_prefix, mask = s_mask;
        for (int i = threadIdx.x; i < m; i += 1024) {
            const uint32_t k = order_key(dev[i]);
            if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255], 1);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int left = s_left, b = 255;
            for (; b > 0 && hist[b] < left; --b) left -= hist[b];
            s_left = left;  // keys still needed from bucket b
            s_prefix = prefix | ((uint32_t)b << shift);
            s_mask = mask | (255u << shift);
        }
        __syncthreads();
    }
    const uint32_t T = s_prefix;
    const int ties = s_left;  // keys equal to T to take, lowest positions first
    const int chunk = (m + 1023) / 1024;
    const int b0 = min(m, threadIdx.x * chunk), b1 = min(m, b0 + chunk);
    int eq = 0;
    for (int i = b0; i < b1; ++i) eq += order_key(dev[i]) == T;
    int eq_before = block_exclusive_scan(eq, scan);
    int sel = 0;
    {
        int e = eq_before;
        for (int i = b0; i < b1; ++i) {
            const uint32_t k = order_key(dev[i]);
            sel += k > T || (k == T && e++ < ties);
        }
    }
    int o = block_exclusive_scan(sel, scan);
    int e = eq_before;
    for (int i = b0; i < b1; ++i) {
        const uint32_t k = order_key(dev[i]);
        if (k > T || (k == T && e++ < ties)) out[o++] = p0 + i;
    }
}

}  // namespace

hipError_t launch_kv_deviation(bool bf16, const void *fresh, int fresh_ncap, int fl, const void *stale, int stale_ncap,
                               int sl, int Hkv, int hd, int p0, int p1, float *dev, hipStream_t s) {
    if (p1 <= p0) return hipSuccess;
    const dim3 grid((p1 - p0 + 3) / 4);
    if (bf16)
        kvr_launch(kv_deviation_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t *)fresh, fresh_ncap, fl,
                   (const bf16_t *)stale, stale_ncap, sl, Hkv, hd, p0, p1, dev);
    else
        kvr_launch(kv_deviation_kernel<float>, grid, dim3(256), 0, s, (const float *)fresh, fresh_ncap, fl,
                   (const float *)stale, stale_ncap, sl, Hkv, hd, p0, p1, dev);
    return hipGetLastError();
}

hipError_t launch_topk(const float *dev, int m, int K, int p0, int32_t *out, hipStream_t s) {
    if (K <= 0 || m <= 0) return hipSuccess;
    if (K > m) return hipErrorInvalidValue;
    kvr_launch(topk_kernel, dim3(1), dim3(1024), 0, s, dev, m, K, p0, out);
    return hipGetLastError();
}

}  // namespace kvr
