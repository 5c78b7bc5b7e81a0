// Causal grouped-query attention of a set of rows over a KV cache, bf16 MFMA,
// head_dim 128.
//
// A work item is (document, kv head, up to 16*MT consecutive rows of that
// document, key range [k0, k1)).  The G = Hq/Hkv query heads sharing the kv
// head times the item's 16-row tiles give (head, row tile) pairs, dealt
// round-robin to the eight wavefronts of the block (two per SIMD); every
// 64-key K/V tile staged in LDS serves all of them, so the cache is read once
// per item.  Scores are computed transposed, S^T = K Q^T
// (v_mfma_f32_16x16x32_bf16 with the key tile as A operand; Q is a compensated
// bf16 pair hi + lo, so two MFMAs per k-step), so that each lane
// owns one query row: the row max and sum of a tile are 16 in-lane values plus
// two cross-lane steps.  The probabilities go straight from the S^T
// accumulator into the B operand of O^T += V^T P^T (as a compensated pair, two
// MFMAs per k-step): both operands enumerate the
// 32 keys of a k-step in the same permuted order (slot j of lane group g <->
// key 16*(j/4) + 4*g + j%4), so P never leaves registers.  V is staged in LDS
// in its own [key][dim] layout (16-byte stores) and the V^T operand is read
// with gfx950's transposing LDS load (ds_read_b64_tr_b16: in each 16-lane
// group, lane i receives element i%4 of the 8-byte chunks that lanes
// 4m + i/4 address, m = 0..3), so each lane gets four keys of one dimension
// per load.  Softmax runs in the exp2 domain; the running max is only
// raised (and the accumulators rescaled) when a row's tile max exceeds it by
// more than 2^8, which keeps every probability below 256.  The causal mask is
// applied only on tiles that reach a row's own position.  The next K/V tile is
// fetched into registers while the current one is used.  The output is written
// as a compensated pair.  When the key range of a row block is split over
// several items (few rows, long contexts) each item writes (m, l, unnormalised
// O) partials and a combine pass merges them with log-sum-exp rescaling.
// When `lse` is given, the row's softmax normaliser is also written there:
// lse[r * Hq + j] = log2 of the sum over its keys of 2^(q.k * log2(e)/sqrt(hd)).
#include <math.h>

#include <algorithm>

#include "common.h"

namespace kvr {

namespace {

constexpr int HD = ATT_HD;
constexpr int KT = ATT_KT;
constexpr int WAVES = 8;           // wavefronts per block
constexpr int NLD = 16 / WAVES;    // 16-byte K (and V) loads per thread per tile
constexpr int KS_STRIDE = HD + 8;   // key tile row stride (bf16): rows 4 banks apart, so the 16
                                    // rows of a key fragment read fall on distinct banks
constexpr int VS_STRIDE = HD + 16;  // value tile row stride: rows 8 banks apart, so the four rows
                                    // a transposing read takes per 16 lanes fall on distinct banks
constexpr int PART_ROW = HD + 4;   // floats per (head, row) partial: O[128], m, l
constexpr float RESCALE_SLACK = 8.0f;  // log2 headroom before the running max is raised
constexpr int COMBINE_NP = 16;         // partials per row loaded in one round by the combine

typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Transposing LDS load (see above): four 16-bit values from the chunks that
// the lane's 16-lane group addresses.
__device__ __forceinline__ i16x4 lds_read_tr16(const bf16_t *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4 *)p);
}
typedef __attribute__((ext_vector_type(2))) float f32x2;

__device__ __forceinline__ bf16x8 ld16(const bf16_t *p) { return *reinterpret_cast<const bf16x8 *>(p); }

// Reductions over the four lanes l, l^16, l^32, l^48 that hold one query row.
// v_permlane16_swap (v_permlane32_swap) run with both operands equal to v hand
// every lane the pair {v[l], v[l^16]} ({v[l], v[l^32]}), in an order that is the
// same for both lanes of the pair, so one VALU op per step completes each
// butterfly without an LDS round trip and all four lanes end bit-identical.
__device__ __forceinline__ float xmax4(float v) {
    unsigned u = __float_as_uint(v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    u = __float_as_uint(v);
    const auto b = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xsum4(float v) {
    unsigned u = __float_as_uint(v);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    u = __float_as_uint(v);
    const auto b = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// PPW: (head, row tile) pairs per wavefront; MT: row tiles of a full item.
template <int PPW, int KG>
__global__ __launch_bounds__(64 * WAVES) void attention_mfma_kernel(const bf16_t *Q, const bf16_t *Q_lo,
                                                                    const RowInfo *rows,
                                                                    const AttnItem *items, int layer, int Hq, int Hkv,
                                                                    int MT, float *part, bf16_t *O, bf16_t *O_lo,
                                                                    int o_perm, float *lse) {
    // KG 64-key K tiles, then KG V tiles (one per key group); after the key
    // loop the same memory takes the second key group's softmax state
    __shared__ __attribute__((aligned(16))) bf16_t kv_lds[KG * KT * (KS_STRIDE + VS_STRIDE)];
    bf16_t *Ks = kv_lds, *Vs = kv_lds + KG * KT * KS_STRIDE;

    const AttnItem it = items[blockIdx.x];
    const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront index (uniform)
    const int G = Hq / Hkv;
    const int qd = Hq * HD;
    const int MTi = (it.nrows + 15) >> 4;  // row tiles this item has
    const int npairs = G * MTi;
    // KG = 2: the wavefronts form two key groups that take alternate 64-key
    // tiles (each pair is worked by two wavefronts, one per group) and merge
    // their softmax states at the end (items of at most four pairs).
    static_assert(KG == 1 || KG == 2, "key groups");
    constexpr int WG = WAVES / KG;
    const int kg = w / WG, lw = w - kg * WG;
    const size_t head_stride = (size_t)it.n_cap * HD;
    const bf16_t *Kg = (const bf16_t *)it.cache + (((size_t)layer * 2 + 0) * Hkv + it.kvh) * head_stride;
    const bf16_t *Vg = (const bf16_t *)it.cache + (((size_t)layer * 2 + 1) * Hkv + it.kvh) * head_stride;

    // this wavefront's pairs: p = w + WAVES*i -> head t = p / MTi, row tile p % MTi
    bool pvalid[PPW];
    int pt[PPW], pm[PPW], prow[PPW];
    bf16x8 qv[PPW][4], ql[PPW][4];
    f32x4 oacc[PPW][8];
    float m[PPW], l[PPW];
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        const int p = lw + WG * i;
        pvalid[i] = p < npairs;
        pt[i] = pvalid[i] ? p / MTi : 0;
        pm[i] = pvalid[i] ? p % MTi : 0;
        const int r = pm[i] * 16 + (lane & 15);  // this lane's query row within the item
        prow[i] = (pvalid[i] && r < it.nrows) ? rows[it.row0 + r].pos : -1;
        const int qrow = it.row0 + min(r, it.nrows - 1);
        const int j = it.kvh * G + pt[i];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            qv[i][ks] = ld16(Q + (size_t)qrow * qd + j * HD + ks * 32 + 8 * g);
            ql[i][ks] = ld16(Q_lo + (size_t)qrow * qd + j * HD + ks * 32 + 8 * g);
        }
#pragma unroll
        for (int nt = 0; nt < 8; ++nt) oacc[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
        m[i] = -INFINITY;
        l[i] = 0.f;
    }
    const float sc = 1.4426950408889634f / sqrtf((float)HD);  // log2(e) / sqrt(hd)
    const int minpos = rows[it.row0].pos;  // rows ascend: every row sees all keys <= minpos

    // the next KG key tiles are fetched into registers while the current ones are used
    u32x4 kreg[KG][NLD], vreg[KG][NLD];
#define KVR_ATT_FETCH(kb_)                                                                                  \
    _Pragma("clang loop unroll(full)") for (int q = 0; q < KG; ++q) {                                       \
        _Pragma("clang loop unroll(full)") for (int i = 0; i < NLD; ++i) {                                 \
            /* K and V: key (tid + 64*WAVES*i)/16 of tile q, dims (tid%16)*8 */                             \
            const int ksrc = min((kb_) + q * KT + ((tid + 64 * WAVES * i) >> 4), it.k1 - 1);                \
            kreg[q][i] = *reinterpret_cast<const u32x4 *>(Kg + (size_t)ksrc * HD + (tid & 15) * 8);         \
            vreg[q][i] = *reinterpret_cast<const u32x4 *>(Vg + (size_t)ksrc * HD + (tid & 15) * 8);         \
        }                                                                                                   \
    }
    KVR_ATT_FETCH(it.k0)
    for (int kb0 = it.k0; kb0 < it.k1; kb0 += KG * KT) {
        __syncthreads();
#pragma clang loop unroll(full)
        for (int q = 0; q < KG; ++q) {
#pragma clang loop unroll(full)
            for (int i = 0; i < NLD; ++i) {
                const int key = q * KT + ((tid + 64 * WAVES * i) >> 4);
                *reinterpret_cast<u32x4 *>(&Ks[key * KS_STRIDE + (tid & 15) * 8]) = kreg[q][i];
                *reinterpret_cast<u32x4 *>(&Vs[key * VS_STRIDE + (tid & 15) * 8]) = vreg[q][i];
            }
        }
        __syncthreads();
        if (kb0 + KG * KT < it.k1) {
            KVR_ATT_FETCH(kb0 + KG * KT)
        }
        const int kt = kb0 + kg * KT;  // this key group's tile
        if (kt >= it.k1) continue;
        const bf16_t *Kt = Ks + kg * KT * KS_STRIDE, *Vt = Vs + kg * KT * VS_STRIDE;
        const bool full = kt + KT <= it.k1 && kt + KT - 1 <= minpos;  // no key of the tile is masked

        // S^T = K Q^T: lane holds query row lane%16, keys 16*nt + 4*g + e of the
        // tile.  The key fragments are read from LDS first, then the MFMAs run
        // k-step-major over the accumulators, so that no MFMA waits for an LDS
        // round trip or for the one before it in its chain (read, wait, two
        // dependent MFMAs per fragment made the tile a chain of LDS latencies).
        // With two pairs per wavefront the registers hold one column tile's
        // four fragments at a time (more would spill: the two pairs' Q fragments and
        // output accumulators take 128 registers).  Each accumulator still sums
        // hi, lo of k-step 0, then of k-step 1, ...
        constexpr int NTH = PPW == 1 ? 4 : 1;  // key fragments' column tiles held at once
        f32x4 s[PPW][4];
#pragma unroll
        for (int i = 0; i < PPW; ++i)
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) s[i][nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int n0 = 0; n0 < 4; n0 += NTH) {
            bf16x8 kb[NTH][4];
#pragma unroll
            for (int nt = 0; nt < NTH; ++nt)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    kb[nt][ks] = ld16(&Kt[((n0 + nt) * 16 + (lane & 15)) * KS_STRIDE + ks * 32 + 8 * g]);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
#pragma unroll
                for (int i = 0; i < PPW; ++i) {
                    if (!pvalid[i]) continue;
#pragma unroll
                    for (int nt = 0; nt < NTH; ++nt)
                        s[i][n0 + nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[nt][ks], qv[i][ks], s[i][n0 + nt], 0, 0, 0);
#pragma unroll
                    for (int nt = 0; nt < NTH; ++nt)
                        s[i][n0 + nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kb[nt][ks], ql[i][ks], s[i][n0 + nt], 0, 0, 0);
                }
        }
        // online softmax, one query row per lane column
        bf16x8 pb[PPW][2], pl[PPW][2];
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            if (!pvalid[i]) continue;
            float mx = -INFINITY;
            if (full) {
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) mx = fmaxf(mx, s[i][nt][e]);
            } else {
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int key = kt + nt * 16 + 4 * g + e;
                        const float v = (key < it.k1 && key <= prow[i]) ? s[i][nt][e] : -INFINITY;
                        s[i][nt][e] = v;
                        mx = fmaxf(mx, v);
                    }
            }
            mx = xmax4(mx) * sc;
            if (__any(mx > m[i] + RESCALE_SLACK)) {
                const float mnew = fmaxf(m[i], mx);
                const float corr = m[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[i] - mnew);
                m[i] = mnew;
                l[i] *= corr;
#pragma unroll
                for (int nt = 0; nt < 8; ++nt) oacc[i][nt] *= corr;
            }
            const float muse = m[i] == -INFINITY ? 0.f : m[i];
            float rs = 0.f;
#pragma unroll
            for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p = __builtin_amdgcn_exp2f(s[i][nt][e] * sc - muse);
                    s[i][nt][e] = p;
                    rs += p;
                }
            l[i] += xsum4(rs);
            // B operand P^T for 32-key step ks: slot j <-> key 32*ks + 16*(j/4) + 4*g + j%4
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                u32x4 u, v;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x2 f = {s[i][2 * ks + q / 2][2 * (q % 2)], s[i][2 * ks + q / 2][2 * (q % 2) + 1]};
                    const bf16x2 h = __builtin_convertvector(f, bf16x2);
                    u[q] = __builtin_bit_cast(unsigned int, h);
                    v[q] = __builtin_bit_cast(unsigned int, __builtin_convertvector(f - __builtin_convertvector(h, f32x2), bf16x2));
                }
                pb[i][ks] = __builtin_bit_cast(bf16x8, u);
                pl[i][ks] = __builtin_bit_cast(bf16x8, v);
            }
        }
        // O^T += V^T P^T: A operand = V^T rows (dims 16*nt + lane%16) over the
        // same key slots; as above, the fragments are read first (half of them
        // at a time with two pairs per wavefront, for the same reason) and the MFMAs of the
        // accumulators then interleave (same per-accumulator order)
        constexpr int NVH = PPW == 1 ? 8 : 4;  // value fragments' column tiles held at once
#pragma unroll
        for (int n0 = 0; n0 < 8; n0 += NVH) {
            bf16x8 va[NVH][2];
#pragma unroll
            for (int nt = 0; nt < NVH; ++nt)
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    // this lane addresses key ks*32 + 4g + m (then + 16), dims
                    // 16 nt + 4q .. +3, for m = (lane%16)/4, q = lane%4; it receives
                    // dim 16 nt + lane%16 of keys ks*32 + 4g + 0..3 and + 16 + 0..3
                    const bf16_t *vr =
                        &Vt[(ks * 32 + 4 * g + ((lane & 15) >> 2)) * VS_STRIDE + (n0 + nt) * 16 + 4 * (lane & 3)];
                    const i16x4 lo = lds_read_tr16(vr);
                    const i16x4 hi = lds_read_tr16(vr + 16 * VS_STRIDE);
                    va[nt][ks] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int i = 0; i < PPW; ++i) {
                    if (!pvalid[i]) continue;
#pragma unroll
                    for (int nt = 0; nt < NVH; ++nt)
                        oacc[i][n0 + nt] =
                            __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[nt][ks], pb[i][ks], oacc[i][n0 + nt], 0, 0, 0);
#pragma unroll
                    for (int nt = 0; nt < NVH; ++nt)
                        oacc[i][n0 + nt] =
                            __builtin_amdgcn_mfma_f32_16x16x32_bf16(va[nt][ks], pl[i][ks], oacc[i][n0 + nt], 0, 0, 0);
                }
        }
    }
#undef KVR_ATT_FETCH

    if constexpr (KG == 2) {
        // the second key group hands its state (per lane: O^T 32 values, m, l)
        // to the wavefront of the first group that holds the same pairs
        constexpr int ST = 34;
        static_assert(WG * PPW * 64 * ST * 4 <= KG * KT * (KS_STRIDE + VS_STRIDE) * 2, "merge area");
        float *mg = reinterpret_cast<float *>(kv_lds);
        __syncthreads();  // every wavefront is done with the K/V tiles
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < PPW; ++i) {
                float *q = mg + ((lw * PPW + i) * 64 + lane) * ST;
#pragma unroll
                for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) q[nt * 4 + e] = oacc[i][nt][e];
                q[32] = m[i];
                q[33] = l[i];
            }
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const float *q = mg + ((lw * PPW + i) * 64 + lane) * ST;
            const float m1 = q[32], l1 = q[33];
            const float M = fmaxf(m[i], m1);
            const float a0 = m[i] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[i] - M);
            const float a1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
            m[i] = M;
            l[i] = l[i] * a0 + l1 * a1;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt)
#pragma unroll
                for (int e = 0; e < 4; ++e) oacc[i][nt][e] = oacc[i][nt][e] * a0 + q[nt * 4 + e] * a1;
        }
    }

    // O^T accumulator: lane holds query row lane%16, dims 16*nt + 4*g + e
    const int rows_item = 16 * MT;
#pragma unroll
    for (int i = 0; i < PPW; ++i) {
        if (!pvalid[i]) continue;
        const int ri = pm[i] * 16 + (lane & 15);
        if (ri >= it.nrows) continue;
        const int t = pt[i];
        const int j = it.kvh * G + t;
        if (it.part < 0) {
            const float inv = 1.0f / l[i];
            const int r = it.row0 + ri;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) {
                const int c = j * HD + nt * 16 + 4 * g;  // 4 consecutive columns, 8-byte aligned
                const size_t off = o_perm ? perm_offset(r, c, qd) : (size_t)r * qd + c;
                uint32_t hi[2], lo[2];
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const f32x2 x = {oacc[i][nt][2 * q] * inv, oacc[i][nt][2 * q + 1] * inv};
                    const bf16x2 h = __builtin_convertvector(x, bf16x2);
                    const f32x2 back = __builtin_convertvector(h, f32x2);
                    hi[q] = __builtin_bit_cast(unsigned int, h);
                    lo[q] = __builtin_bit_cast(unsigned int, __builtin_convertvector(x - back, bf16x2));
                }
                *reinterpret_cast<uint2 *>(O + off) = make_uint2(hi[0], hi[1]);
                *reinterpret_cast<uint2 *>(O_lo + off) = make_uint2(lo[0], lo[1]);
            }
            if (lse && g == 0) lse[(size_t)r * Hq + j] = m[i] + log2f(l[i]);
        } else {
            float *p = part + ((size_t)(it.part * G + t) * rows_item + ri) * PART_ROW;
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) *reinterpret_cast<f32x4 *>(p + nt * 16 + 4 * g) = oacc[i][nt];
            if (g == 0) { p[HD] = m[i]; p[HD + 1] = l[i]; }
        }
    }
}

// One wavefront per (combine item, query head of the group, two rows): each
// half-wavefront takes one row, a lane four consecutive head dimensions.  The
// split partials of the row are merged with log-sum-exp weights (exp2
// domain), the parts summed in ascending order.  With at most NP parts every
// partial of the row is loaded in one round (clamped indexes, so the loads
// are unconditional and all in flight together); longer lists take batches
// of NP.  `lse` as above.
template <int NP>
__global__ __launch_bounds__(64) void attention_combine_kernel(const CombineItem *items, const float *part, int Hq,
                                                               int Hkv, int MT, bf16_t *O, bf16_t *O_lo, int o_perm,
                                                               float *lse) {
    static_assert(HD == 128, "a half-wavefront covers one head row");
    const CombineItem it = items[blockIdx.x];
    const int t = blockIdx.y;
    const int lane = threadIdx.x;
    const int i = 2 * blockIdx.z + (lane >> 5);
    if (i >= it.nrows) return;
    const int G = Hq / Hkv;
    const int rows_item = 16 * MT;
    const int j = it.kvh * G + t;
    const int d = 4 * (lane & 31);
    const size_t qstride = (size_t)G * rows_item * PART_ROW;
    const float *base = part + ((size_t)(it.part0 * G + t) * rows_item + i) * PART_ROW;
    const int np = it.nparts;
    float M = -INFINITY, L = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int q0 = 0; q0 < np; q0 += NP) {
        float mm[NP], ll[NP];
        f32x4 oo[NP];
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const float *p = base + (size_t)min(q0 + u, np - 1) * qstride;
            mm[u] = p[HD];
            ll[u] = p[HD + 1];
            oo[u] = *reinterpret_cast<const f32x4 *>(p + d);
        }
        float Mb = M;
#pragma unroll
        for (int u = 0; u < NP; ++u) Mb = fmaxf(Mb, mm[u]);  // clamped duplicates do not change the max
        const float r = M == -INFINITY ? 0.f : exp2f(M - Mb);  // rescale what earlier batches summed
        acc *= r;
        L *= r;
#pragma unroll
        for (int u = 0; u < NP; ++u) {
            const float wq = (q0 + u >= np || mm[u] == -INFINITY) ? 0.f : exp2f(mm[u] - Mb);
            acc += oo[u] * wq;
            L += ll[u] * wq;
        }
        M = Mb;
    }
    const int r = it.row0 + i, c = j * HD + d;  // four consecutive columns (adjacent in operand order too)
    const size_t off = o_perm ? perm_offset(r, c, Hq * HD) : (size_t)r * Hq * HD + c;
    const f32x4 y = acc / L;
    uint32_t hi[2], lo[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const bf16_t h0 = f32_to_bf16(y[2 * q]), h1 = f32_to_bf16(y[2 * q + 1]);
        const bf16_t l0 = f32_to_bf16(y[2 * q] - bf16_to_f32(h0)), l1 = f32_to_bf16(y[2 * q + 1] - bf16_to_f32(h1));
        hi[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        lo[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    *reinterpret_cast<uint2 *>(O + off) = make_uint2(hi[0], hi[1]);
    *reinterpret_cast<uint2 *>(O_lo + off) = make_uint2(lo[0], lo[1]);
    if (lse && d == 0) lse[(size_t)r * Hq + j] = M + log2f(L);
}

}  // namespace

int attention_max_row_tiles(int Hq, int Hkv) {
    const int G = Hq / Hkv;
    return G >= 16 ? 1 : std::min(4, std::max(1, 16 / G));
}

hipError_t launch_attention_mfma(const bf16_t *Q, const bf16_t *Q_lo, const RowInfo *rows,
                                 const AttnItem *items, int n_items, int MT, int layer, int Hq, int Hkv, float *part,
                                 bf16_t *O, bf16_t *O_lo, bool o_perm, float *lse, hipStream_t s) {
    if (n_items <= 0) return hipSuccess;
    if (!Q_lo || !O_lo || MT < 1 || MT > attention_max_row_tiles(Hq, Hkv)) return hipErrorInvalidValue;
    // at most four pairs per item: two key groups of four wavefronts, one pair
    // each; otherwise one group, pairs dealt round-robin to the eight wavefronts
    const int npairs = (Hq / Hkv) * MT;
    if (2 * npairs <= WAVES)
        kvr_launch(attention_mfma_kernel<1, 2>, dim3(n_items), dim3(64 * WAVES), 0, s, Q, Q_lo, rows, items, layer, Hq,
                   Hkv, MT, part, O, O_lo, (int)o_perm, lse);
    else if (npairs <= WAVES)
        kvr_launch(attention_mfma_kernel<1, 1>, dim3(n_items), dim3(64 * WAVES), 0, s, Q, Q_lo, rows, items, layer, Hq,
                   Hkv, MT, part, O, O_lo, (int)o_perm, lse);
    else if (npairs <= 2 * WAVES)
        kvr_launch(attention_mfma_kernel<2, 1>, dim3(n_items), dim3(64 * WAVES), 0, s, Q, Q_lo, rows, items, layer, Hq,
                   Hkv, MT, part, O, O_lo, (int)o_perm, lse);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_attention_combine(const CombineItem *items, int n_items, int MT, const float *part, int Hq,
                                    int Hkv, bf16_t *O, bf16_t *O_lo, bool o_perm, float *lse, hipStream_t s) {
    if (n_items <= 0) return hipSuccess;
    if (MT < 1 || MT > attention_max_row_tiles(Hq, Hkv)) return hipErrorInvalidValue;
    kvr_launch(attention_combine_kernel<COMBINE_NP>, dim3(n_items, Hq / Hkv, 8 * MT), dim3(64), 0, s, items, part,
               Hq, Hkv, MT, O, O_lo, (int)o_perm, lse);
    return hipGetLastError();
}

}  // namespace kvr
