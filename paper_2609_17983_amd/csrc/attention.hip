// Causal grouped-query attention of a set of rows over a KV cache, bf16 MFMA,
// head_dim 128.
//
// A work item is (document, kv head, up to 16 consecutive rows of that
// document, key range [k0, k1)).  The G = Hq/Hkv query heads that share the kv
// head each form one 16-row MFMA tile, so one K/V tile staged in LDS serves
// 16*G query rows.  Per 64-key tile: S = Q K^T (v_mfma_f32_16x16x32_bf16, K
// row-major in LDS), causal mask against each row's own position, online
// softmax in the exp2 domain (row max / sum over the 16 lanes of a row group
// by cross-lane shuffles), P rounded to bf16 and re-read from LDS in operand
// layout, O += P V with V stored transposed in LDS.  When the key range of a
// row block is split over several items (few rows, long contexts) each item
// writes (m, l, unnormalised O) partials and a combine pass merges them with
// the usual log-sum-exp rescaling.
#include <math.h>

#include "common.h"

namespace kvr {

namespace {

constexpr int HD = ATT_HD;
constexpr int KT = ATT_KT;
constexpr int KS_STRIDE = HD + 8;  // keys tile row stride (bf16)
constexpr int VT_STRIDE = KT + 8;  // transposed values row stride (bf16)
constexpr int PS_STRIDE = KT + 8;
constexpr int MAXH = 2;            // query heads per wavefront (G <= 8)
constexpr int PART_ROW = HD + 4;   // floats per (head, row) partial: O[128], m, l

__device__ __forceinline__ bf16x8 lds16(const bf16_t *p) { return *reinterpret_cast<const bf16x8 *>(p); }

__device__ __forceinline__ float group16_max(float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    return v;
}
__device__ __forceinline__ float group16_sum(float v) {
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__global__ __launch_bounds__(256) void attention_mfma_kernel(const bf16_t *Q, const RowInfo *rows,
                                                             const DocInfo *docs, const AttnItem *items, int layer,
                                                             int Hq, int Hkv, float *part, bf16_t *O) {
    __shared__ __attribute__((aligned(16))) bf16_t Ks[KT * KS_STRIDE];
    __shared__ __attribute__((aligned(16))) bf16_t Vt[HD * VT_STRIDE];
    __shared__ __attribute__((aligned(16))) bf16_t Ps[4][16 * PS_STRIDE];

    const AttnItem it = items[blockIdx.x];
    const DocInfo dc = docs[it.doc];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int G = Hq / Hkv;
    const int qd = Hq * HD;
    const size_t head_stride = (size_t)dc.n_cap * HD;
    const bf16_t *Kg = (const bf16_t *)dc.cache + (((size_t)layer * 2 + 0) * Hkv + it.kvh) * head_stride;
    const bf16_t *Vg = (const bf16_t *)dc.cache + (((size_t)layer * 2 + 1) * Hkv + it.kvh) * head_stride;

    // rows 4*(lane/16)+e of the accumulator tiles: their positions (-1 = padding)
    int prow[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int i = 4 * (lane >> 4) + e;
        prow[e] = i < it.nrows ? rows[it.row0 + i].pos : -1;
    }

    // Q operands of this wavefront's heads: lane holds row lane%16, dims 32*ks + 8*(lane/16)
    const int qrow = it.row0 + min(lane & 15, it.nrows - 1);
    bf16x8 qv[MAXH][4];
    bool hvalid[MAXH];
#pragma unroll
    for (int h = 0; h < MAXH; ++h) {
        const int t = w + 4 * h;
        hvalid[h] = t < G;
        const int j = it.kvh * G + (hvalid[h] ? t : 0);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            qv[h][ks] = lds16(Q + (size_t)qrow * qd + j * HD + ks * 32 + 8 * (lane >> 4));
    }

    f32x4 oacc[MAXH][8];
    float m[MAXH][4], l[MAXH][4];
#pragma unroll
    for (int h = 0; h < MAXH; ++h) {
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) oacc[h][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) { m[h][e] = -INFINITY; l[h][e] = 0.f; }
    }
    const float sc = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)

    for (int kt = it.k0; kt < it.k1; kt += KT) {
        __syncthreads();
        // K tile: thread covers keys tid/16 + 16*i, dims (tid%16)*8 .. +8
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int key = (tid >> 4) + 16 * i;
            const int src = min(kt + key, it.k1 - 1);
            const uint4 u = *reinterpret_cast<const uint4 *>(Kg + (size_t)src * HD + (tid & 15) * 8);
            *reinterpret_cast<uint4 *>(&Ks[key * KS_STRIDE + (tid & 15) * 8]) = u;
        }
        // V tile, stored transposed: thread covers key tid%64, dims 8*(tid/64 + 4*i) .. +8
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int key = tid & 63;
            const int d0 = 8 * ((tid >> 6) + 4 * i);
            const int src = min(kt + key, it.k1 - 1);
            const uint4 u = *reinterpret_cast<const uint4 *>(Vg + (size_t)src * HD + d0);
            const bf16_t *pv = reinterpret_cast<const bf16_t *>(&u);
#pragma unroll
            for (int e = 0; e < 8; ++e) Vt[(d0 + e) * VT_STRIDE + key] = pv[e];
        }
        __syncthreads();

#pragma unroll
        for (int h = 0; h < MAXH; ++h) {
            if (!hvalid[h]) continue;  // uniform per wavefront
            f32x4 s[4];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                s[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const bf16x8 kb = lds16(&Ks[(nt * 16 + (lane & 15)) * KS_STRIDE + ks * 32 + 8 * (lane >> 4)]);
                    s[nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qv[h][ks], kb, s[nt], 0, 0, 0);
                }
            }
            // mask + scale; per-row max over the tile
            float mx[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) mx[e] = -INFINITY;
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                const int key = kt + nt * 16 + (lane & 15);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const bool ok = key < it.k1 && key <= prow[e];
                    const float v = ok ? s[nt][e] * sc : -INFINITY;
                    s[nt][e] = v;
                    mx[e] = fmaxf(mx[e], v);
                }
            }
            float corr[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const float mt = group16_max(mx[e]);
                const float mnew = fmaxf(m[h][e], mt);
                const float muse = mnew == -INFINITY ? 0.f : mnew;
                corr[e] = exp2f(m[h][e] - muse);
                m[h][e] = mnew;
                float rs = 0.f;
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) {
                    const float p = exp2f(s[nt][e] - muse);
                    s[nt][e] = p;
                    rs += p;
                }
                l[h][e] = l[h][e] * corr[e] + group16_sum(rs);
            }
#pragma unroll
            for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                for (int e = 0; e < 4; ++e) oacc[h][nt][e] *= corr[e];
            // P (bf16) -> LDS, row-major [16 rows][64 keys]
            bf16_t *ps = Ps[w];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    ps[(4 * (lane >> 4) + e) * PS_STRIDE + nt * 16 + (lane & 15)] = f32_to_bf16(s[nt][e]);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            bf16x8 pa[2];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) pa[ks] = lds16(&ps[(lane & 15) * PS_STRIDE + ks * 32 + 8 * (lane >> 4)]);
#pragma unroll
            for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const bf16x8 vb = lds16(&Vt[(nt * 16 + (lane & 15)) * VT_STRIDE + ks * 32 + 8 * (lane >> 4)]);
                    oacc[h][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[ks], vb, oacc[h][nt], 0, 0, 0);
                }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
    }

    // write out: accumulator rows 4*(lane/16)+e, dims nt*16 + lane%16
#pragma unroll
    for (int h = 0; h < MAXH; ++h) {
        if (!hvalid[h]) continue;
        const int t = w + 4 * h;
        const int j = it.kvh * G + t;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int i = 4 * (lane >> 4) + e;
            if (i >= it.nrows) continue;
            if (it.part < 0) {
                const float inv = 1.0f / l[h][e];
                bf16_t *o = O + (size_t)(it.row0 + i) * qd + j * HD + (lane & 15);
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) o[nt * 16] = f32_to_bf16(oacc[h][nt][e] * inv);
            } else {
                float *p = part + ((size_t)(it.part * G + t) * 16 + i) * PART_ROW;
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) p[nt * 16 + (lane & 15)] = oacc[h][nt][e];
                if ((lane & 15) == 0) { p[HD] = m[h][e]; p[HD + 1] = l[h][e]; }
            }
        }
    }
}

// One block per (combine item, query head of the group): merge the split
// partials of up to 16 rows.
__global__ __launch_bounds__(128) void attention_combine_kernel(const CombineItem *items, const float *part, int Hq,
                                                                int Hkv, bf16_t *O) {
    const CombineItem it = items[blockIdx.x];
    const int t = blockIdx.y;
    const int G = Hq / Hkv;
    const int j = it.kvh * G + t;
    const int d = threadIdx.x;  // 0..127
    for (int i = 0; i < it.nrows; ++i) {
        float M = -INFINITY;
        for (int q = 0; q < it.nparts; ++q)
            M = fmaxf(M, part[((size_t)((it.part0 + q) * G + t) * 16 + i) * PART_ROW + HD]);
        float L = 0.f, acc = 0.f;
        for (int q = 0; q < it.nparts; ++q) {
            const float *p = part + ((size_t)((it.part0 + q) * G + t) * 16 + i) * PART_ROW;
            const float mq = p[HD];
            const float f = mq == -INFINITY ? 0.f : exp2f(mq - M);
            L += p[HD + 1] * f;
            acc += p[d] * f;
        }
        O[(size_t)(it.row0 + i) * Hq * HD + j * HD + d] = f32_to_bf16(acc / L);
    }
}

}  // namespace

hipError_t launch_attention_mfma(const bf16_t *Q, const RowInfo *rows, const DocInfo *docs, const AttnItem *items,
                                 int n_items, int layer, int Hq, int Hkv, float *part, bf16_t *O, hipStream_t s) {
    if (n_items <= 0) return hipSuccess;
    hipLaunchKernelGGL(attention_mfma_kernel, dim3(n_items), dim3(256), 0, s, Q, rows, docs, items, layer, Hq, Hkv,
                       part, O);
    return hipGetLastError();
}

hipError_t launch_attention_combine(const CombineItem *items, int n_items, const float *part, int Hq, int Hkv,
                                    bf16_t *O, hipStream_t s) {
    if (n_items <= 0) return hipSuccess;
    hipLaunchKernelGGL(attention_combine_kernel, dim3(n_items, Hq / Hkv), dim3(128), 0, s, items, part, Hq, Hkv, O);
    return hipGetLastError();
}

}  // namespace kvr
