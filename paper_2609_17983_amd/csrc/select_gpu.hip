// Device side of the forward-based selectors of Table 1: the CacheBlend
// per-position deviation between freshly computed and stale keys/values, the
// Attention selector's per-position attention mass from the query rows, and a
// block-wide top-K.
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

// ---- Attention selector: attention probability that the query rows place on
// each stale key, summed over the query rows and heads of one kv head group.
//
// For kv head g, key p < n and query row r, head j of the group:
//   prob = 2^(q_rj . k_p * log2(e)/sqrt(hd) - lse[r * Hq + j])
// where lse is the row's base-2 log-sum-exp written by the attention pass of
// the same layer.  part[g * n + p] receives the sum (accumulate = 0) or has it
// added (accumulate = 1: later layers), so every entry is owned by one block
// and the sum over layers runs in layer order.

constexpr int MASS_KT = 64;             // keys per block
constexpr int MASS_WAVES = 8;
constexpr int MASS_HD = 128;
constexpr int MASS_STRIDE = MASS_HD + 8;  // LDS row stride of the key tile (bf16)

__device__ __forceinline__ bf16x8 ld16(const bf16_t *p) { return *reinterpret_cast<const bf16x8 *>(p); }

// bf16, head_dim 128.  Block = (64-key tile, kv head).  The key tile is staged
// in LDS and held as MFMA A operands; the (query head, 16-row tile) pairs of
// the group are dealt to the eight wavefronts.  S^T = K Q^T with
// v_mfma_f32_16x16x32_bf16 (Q a compensated pair, two MFMAs per k-step): lane
// l holds query row l%16 and keys 16*nt + 4*(l/16) + e, so each lane adds its
// probabilities for fixed keys over all of its pairs; the 16 lanes of a key
// slot and then the wavefronts are summed in a fixed order.
__global__ __launch_bounds__(64 * MASS_WAVES) void attn_mass_mfma_kernel(const bf16_t *Q, const bf16_t *Q_lo,
                                                                         const float *lse, int q, const bf16_t *cache,
                                                                         int n_cap, int layer, int Hq, int Hkv, int n,
                                                                         float *part, int accumulate) {
    __shared__ __attribute__((aligned(16))) bf16_t Ks[MASS_KT * MASS_STRIDE];
    __shared__ float red[MASS_WAVES][MASS_KT];
    const int tid = threadIdx.x, lane = tid & 63, g4 = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int k0 = blockIdx.x * MASS_KT, kvh = blockIdx.y;
    const bf16_t *Kg = cache + (((size_t)layer * 2 + 0) * Hkv + kvh) * (size_t)n_cap * MASS_HD;
    // 64 keys x 128 dims = 1024 chunks of 16 bytes; keys past n read key n - 1 (never summed)
    for (int i = tid; i < MASS_KT * MASS_HD / 8; i += 64 * MASS_WAVES) {
        const int key = min(k0 + (i >> 4), n - 1);
        *reinterpret_cast<u32x4 *>(&Ks[(i >> 4) * MASS_STRIDE + (i & 15) * 8]) =
            *reinterpret_cast<const u32x4 *>(Kg + (size_t)key * MASS_HD + (i & 15) * 8);
    }
    __syncthreads();
    bf16x8 kb[4][4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) kb[nt][ks] = ld16(&Ks[(nt * 16 + (lane & 15)) * MASS_STRIDE + ks * 32 + 8 * g4]);

    const int G = Hq / Hkv, MTq = (q + 15) >> 4, npairs = G * MTq, qd = Hq * MASS_HD;
    const float sc = 1.4426950408889634f / sqrtf((float)MASS_HD);
    f32x4 acc[4];
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int p = w; p < npairs; p += MASS_WAVES) {
        const int j = kvh * G + p / MTq;
        const int row = (p % MTq) * 16 + (lane & 15);
        const int qrow = min(row, q - 1);
        bf16x8 qv[4], ql[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            qv[ks] = ld16(Q + (size_t)qrow * qd + j * MASS_HD + ks * 32 + 8 * g4);
            ql[ks] = ld16(Q_lo + (size_t)qrow * qd + j * MASS_HD + ks * 32 + 8 * g4);
        }
        const float L = lse[(size_t)qrow * Hq + j];
        const bool valid = row < q;
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            f32x4 sv = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[nt][ks], qv[ks], sv, 0, 0, 0);
                sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[nt][ks], ql[ks], sv, 0, 0, 0);
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[nt][e] += valid ? exp2f(sv[e] * sc - L) : 0.f;
        }
    }
    // sum over the 16 query-row lanes of each key slot, then over the wavefronts
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float v = acc[nt][e];
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o);
            if ((lane & 15) == 0) red[w][nt * 16 + 4 * g4 + e] = v;
        }
    __syncthreads();
    if (tid < MASS_KT && k0 + tid < n) {
        float t = 0.f;
#pragma unroll
        for (int u = 0; u < MASS_WAVES; ++u) t += red[u][tid];
        float *o = part + (size_t)kvh * n + k0 + tid;
        *o = accumulate ? *o + t : t;
    }
}

// Any supported head_dim (<= 128), fp32 or bf16 operands.  One wavefront per
// (key, kv head); lanes take the (query row, head) pairs of the group in turn.
template <typename T>
__global__ __launch_bounds__(64) void attn_mass_simple_kernel(const T *Q, const T *Q_lo, const float *lse, int q,
                                                              const T *cache, int n_cap, int layer, int Hq, int Hkv,
                                                              int hd, int n, float *part, int accumulate) {
    __shared__ float kr[128];
    const int key = blockIdx.x, kvh = blockIdx.y, lane = threadIdx.x;
    const T *Kp = cache + (((size_t)layer * 2 + 0) * Hkv + kvh) * (size_t)n_cap * hd + (size_t)key * hd;
    for (int i = lane; i < hd; i += 64) kr[i] = to_f32(Kp[i]);
    __syncthreads();
    const int G = Hq / Hkv, qd = Hq * hd;
    const float sc = 1.4426950408889634f / sqrtf((float)hd);
    float acc = 0.f;
    for (int pr = lane; pr < q * G; pr += 64) {
        const int r = pr / G, j = kvh * G + pr % G;
        float dot = 0.f;
        for (int i = 0; i < hd; ++i) dot += load_operand(Q, Q_lo, (size_t)r * qd + j * hd + i) * kr[i];
        acc += exp2f(dot * sc - lse[(size_t)r * Hq + j]);
    }
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) {
        float *o = part + (size_t)kvh * n + key;
        *o = accumulate ? *o + acc : acc;
    }
}

// mass[p] = sum over kv heads g (ascending) of part[g * n + p].
__global__ __launch_bounds__(256) void mass_reduce_kernel(const float *part, int Hkv, int n, float *mass) {
    const int p = blockIdx.x * 256 + threadIdx.x;
    if (p >= n) return;
    float t = 0.f;
    for (int g = 0; g < Hkv; ++g) t += part[(size_t)g * n + p];
    mass[p] = t;
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

bool attn_mass_mfma_ok(bool bf16, int hd) { return bf16 && hd == MASS_HD; }

hipError_t launch_attn_mass(bool bf16, const void *Q, const void *Q_lo, const float *lse, int q, const void *cache,
                            int n_cap, int layer, int Hq, int Hkv, int hd, int n, float *part, bool accumulate,
                            hipStream_t s) {
    if (n <= 0) return hipSuccess;
    if (q < 1 || !lse || !part || hd > 128 || (bf16 && !Q_lo)) return hipErrorInvalidValue;
    if (attn_mass_mfma_ok(bf16, hd))
        kvr_launch(attn_mass_mfma_kernel, dim3((n + MASS_KT - 1) / MASS_KT, Hkv), dim3(64 * MASS_WAVES), 0, s,
                   (const bf16_t *)Q, (const bf16_t *)Q_lo, lse, q, (const bf16_t *)cache, n_cap, layer, Hq, Hkv, n,
                   part, (int)accumulate);
    else if (bf16)
        kvr_launch(attn_mass_simple_kernel<bf16_t>, dim3(n, Hkv), dim3(64), 0, s, (const bf16_t *)Q,
                   (const bf16_t *)Q_lo, lse, q, (const bf16_t *)cache, n_cap, layer, Hq, Hkv, hd, n, part,
                   (int)accumulate);
    else
        kvr_launch(attn_mass_simple_kernel<float>, dim3(n, Hkv), dim3(64), 0, s, (const float *)Q,
                   (const float *)nullptr, lse, q, (const float *)cache, n_cap, layer, Hq, Hkv, hd, n, part,
                   (int)accumulate);
    return hipGetLastError();
}

hipError_t launch_mass_reduce(const float *part, int Hkv, int n, float *mass, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    kvr_launch(mass_reduce_kernel, dim3((n + 255) / 256), dim3(256), 0, s, part, Hkv, n, mass);
    return hipGetLastError();
}

hipError_t launch_topk(const float *dev, int m, int K, int p0, int32_t *out, hipStream_t s) {
    if (K <= 0 || m <= 0) return hipSuccess;
    if (K > m) return hipErrorInvalidValue;
    kvr_launch(topk_kernel, dim3(1), dim3(1024), 0, s, dev, m, K, p0, out);
    return hipGetLastError();
}

}  // namespace kvr
