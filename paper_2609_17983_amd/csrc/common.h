// Internal declarations shared by the library's HIP sources.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvr {

typedef uint16_t bf16_t;  // raw bf16 bits in memory

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) unsigned int u32x4;

// "Operand order" of an activation matrix [rows][K] (rows padded to a multiple
// of 16, K a multiple of 32): the 16-byte A operand of v_mfma_f32_16x16x32_bf16
// for 16-row tile t and k-step s (32 columns) is stored for the 64 lanes
// contiguously, lane l holding row 16t + l%16, columns 32s + 8*(l/16) .. +8.
__host__ __device__ __forceinline__ size_t perm_offset(int r, int c, int K) {
    return ((size_t)((r >> 4) * (K >> 5) + (c >> 5)) * 64 + (r & 15) + 16 * ((c & 31) >> 3)) * 8 + (c & 7);
}

// Packed weights (pack.hip): the matrix is a sequence of 16-row tiles; each
// tile's k-step is one 1 KB operand fragment.  The tiles are stored in groups
// of `grp` consecutive tiles (the last group may be shorter), k-step major
// within a group, so a block that streams the tiles of one group reads one
// contiguous range.  Element offset of tile t's fragment at k-step 0; the
// fragment of k-step s is `*kstride` elements further on.  grp <= 1 is
// tile-major (each tile's k-steps adjacent).
__host__ __device__ __forceinline__ size_t packed_tile_offset(int t, int ntiles, int ksteps, int grp, int *kstride) {
    const int g = grp > 1 ? grp : 1;
    const int g0 = (t / g) * g;
    const int gl = ntiles - g0 < g ? ntiles - g0 : g;
    *kstride = gl * 512;
    return ((size_t)g0 * ksteps + (t - g0)) * 512;
}

__device__ __forceinline__ float bf16_to_f32(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp32 -> bf16, round to nearest, ties to even (NaN kept quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// Matrix operands of the bf16 path are compensated pairs: x = hi + lo with
// hi = bf16(x) and lo = bf16(x - hi), which carries x to about 16 significant
// bits; a product with an exact bf16 weight is then two MFMAs into one fp32
// accumulator.  For fp32 operands there is no low part (lo == nullptr).
template <typename T>
__device__ __forceinline__ void store_operand(T *hi, T *lo, size_t i, float x) {
    if constexpr (sizeof(T) == 4) {
        hi[i] = x;
    } else {
        const bf16_t h = f32_to_bf16(x);
        hi[i] = h;
        if (lo) lo[i] = f32_to_bf16(x - bf16_to_f32(h));
    }
}
template <typename T>
__device__ __forceinline__ float load_operand(const T *hi, const T *lo, size_t i) {
    return lo ? to_f32(hi[i]) + to_f32(lo[i]) : to_f32(hi[i]);
}

// One repaired (or prefilled) row: its document, absolute position, and the row
// index of its final hidden state inside the document's output buffer.
struct RowInfo {
    int32_t pos;
    int32_t doc;
    int32_t out;
    int32_t pad;
};

// One document of a pass.
struct DocInfo {
    void *cache;            // [L][2][Hkv][n_cap][hd]
    const int32_t *tokens;  // C' (device)
    float *hidden_out;      // [rows][d] or null
    int32_t n, n_cap;
    int32_t row0, nrows;    // rows of this document in the pass's row table
};

// One attention work item: up to 16 consecutive rows of one document, one kv
// head group, keys [k0, k1).  part < 0: the item covers all keys its rows need
// and writes the normalised output; otherwise it writes split partials at slot
// `part` of the partial buffer.
struct AttnItem {
    int32_t doc;
    int32_t row0, nrows;
    int32_t kvh;
    int32_t k0, k1;
    int32_t part;
    int32_t n_cap;        // the document's cache (copied from its DocInfo so
    const void *cache;    // that the key/value loads need no second lookup)
};

// Combine step for rows whose keys were split over several items.
struct CombineItem {
    int32_t row0, nrows;  // rows of the block
    int32_t kvh;
    int32_t part0, nparts;  // consecutive partial slots
    int32_t pad[3];
};

enum Epi { EPI_STORE = 0, EPI_RESID = 1, EPI_SWIGLU = 2 };

// A linear layer Y[r][n] = sum_k X[r][k] * W[n][k] whose weight is the
// concatenation of up to three row blocks (Q, K, V), or for SWIGLU the pair
// (gate, up) with output A[r][f] = silu(gate) * up.
struct LinearArgs {
    const void *x;        // [R][K] operand (bf16 or fp32), row stride ldx
    const void *x_lo;     // low part of a compensated bf16 operand, or null
    int32_t ldx;
    int32_t R, K, N;      // N: output columns (SWIGLU: number of features f)
    const void *w[3];     // row-major row blocks of W (simple kernel)
    int32_t seg_end[3];   // cumulative output-column boundaries of the blocks
    const void *wp;       // W packed in operand order (tiled kernel; pack.hip)
    int32_t grp;          // tile group of the packed layout (packed_tile_offset)
    void *out;            // STORE: float [R][ldo]; RESID: float [R][ldo] (+=);
                          // SWIGLU: operand type [R][ldo]
    void *out_lo;         // SWIGLU: low part of the compensated output, or null
    int32_t ldo;
    int32_t split;        // tiled STORE only: K cut into `split` slices, partial
                          // tiles out[s][R][ldo] summed by the consumer (<= 1: none)
    int32_t group_all;    // tiled: at most this many row blocks form one group of the tile order (set by the launcher)
    int32_t tpb;          // tall kernel: weight tiles per block (0: not the tall kernel)
    // tall kernel: RMS scale of the rows (resid_gain), as in SkinnyArgs: when
    // rs_ssq is set, output row r is multiplied by
    // rsqrt((rs_ssq[0][r] + ... + rs_ssq[rs_nb-1][r]) / rs_d + rs_eps)
    const float *rs_ssq;
    int32_t rs_nb, rs_d;
    float rs_eps;
};

// Skinny (R <= 64) linear layer: X in operand order, W packed in operand order
// with ntiles 16-row tiles (SWIGLU: gate/up interleaved, 2N virtual rows);
// STORE writes fp32 partial tiles [split][R][N]; SWIGLU (split 1) writes
// silu(gate)*up in operand order.
struct SkinnyArgs {
    const void *x, *x_lo;  // compensated operand (hi, lo), both in operand order
    int32_t R, K, N;      // N: output columns (SWIGLU: number of features)
    const void *w;         // packed weight
    int32_t ntiles;
    int32_t grp;           // tile group of the packed layout (packed_tile_offset)
    void *out, *out_lo;    // SWIGLU writes a compensated pair
    int32_t split;
    // RMS scale of the rows (resid_gain): when rs_ssq is set, output row r is
    // multiplied by rsqrt((rs_ssq[0][r] + ... + rs_ssq[rs_nb-1][r]) / rs_d + rs_eps)
    const float *rs_ssq;
    int32_t rs_nb, rs_d;
    float rs_eps;
};

// ---- kernel launch with optional execution timing
//
// While launch_timer() holds events (the context's step profiler arms it
// before a launcher call), the next launch records them at the start and the
// end of the kernel's execution (hipExtLaunchKernel), which excludes the
// dispatch gap in front of the kernel; the launch disarms the timer.
struct LaunchTimer {
    hipEvent_t start = nullptr, stop = nullptr;
};
LaunchTimer &launch_timer();

template <typename... KArgs, typename... Args>
inline void kvr_launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, uint32_t shmem, hipStream_t s,
                       Args... args) {
    LaunchTimer &t = launch_timer();
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, t.start, t.stop, 0, static_cast<KArgs>(args)...);
    t.start = t.stop = nullptr;
}

// ---- launchers (each enqueues one kernel on `stream`; return hipSuccess or the launch error)

hipError_t launch_embed(bool bf16, const RowInfo *rows, const DocInfo *docs, int R, const void *embed,
                        int d, int vocab, float *H, hipStream_t s);
// RMSNorm of the residual rows.  First H[r] += sum of `nsplit` fp32 partial
// tiles part[s][R][d] (the split-K outputs of the projection that produced the
// residual update; nsplit 0 = none), then X = H * rsqrt(mean(H^2)+eps) * gain,
// row-major with stride ldx, or in operand order when `perm`.
hipError_t launch_rmsnorm(bool bf16_out, bool bf16_gain, float *H, const float *part, int nsplit, const void *gain,
                          int R, int d, float eps, void *X, void *X_lo, int ldx, bool perm, hipStream_t s);
// Residual update + gain for the skinny path (see resid_gain_kernel): H[r] +=
// partials, X = H * gain (compensated, operand order), ssq[b][r] per 1024-column
// block b; resid_gain_blocks(d) blocks per row.
int resid_gain_blocks(int d);
hipError_t launch_resid_gain(bool bf16_gain, float *H, const float *part, int nsplit, const void *gain, int R, int d,
                             void *X, void *X_lo, float *ssq, hipStream_t s);
hipError_t launch_final_norm(bool bf16_gain, float *H, const float *part, int nsplit, const void *gain,
                             const RowInfo *rows, const DocInfo *docs, int R, int d, float eps, hipStream_t s);
// qkv: `nsplit` fp32 tiles [nsplit][R][qd+2kd] summed in order.
hipError_t launch_rope_scatter(bool bf16, const float *qkv, int nsplit, const void *bq, const void *bk,
                               const void *bv, const RowInfo *rows, const DocInfo *docs, int R, int layer, int Hq,
                               int Hkv, int hd, const float *rope_cos, const float *rope_sin, void *Q, void *Q_lo,
                               hipStream_t s);
// O is written row-major [R][Hq*hd], or in operand order when o_perm.  The
// attention launchers also write, when lse is not null, each (row, query head)
// softmax normaliser as a base-2 log-sum-exp of the scores q.k*log2(e)/sqrt(hd):
// lse[r * Hq + j].
hipError_t launch_attention_simple(bool bf16, const void *Q, const void *Q_lo, const RowInfo *rows,
                                   const DocInfo *docs, int R, int layer, int Hq, int Hkv, int hd, void *O, void *O_lo,
                                   bool o_perm, float *lse, hipStream_t s);
// Largest number of 16-row tiles an attention work item may carry for a head
// grouping.  A pass's items all carry at most MT tiles (1 <= MT <= this), the
// same MT for the MFMA kernel and the combine (it sets the partials' layout).
int attention_max_row_tiles(int Hq, int Hkv);
hipError_t launch_attention_mfma(const bf16_t *Q, const bf16_t *Q_lo, const RowInfo *rows,
                                 const AttnItem *items, int n_items, int MT, int layer, int Hq, int Hkv,
                                 float *part, bf16_t *O, bf16_t *O_lo, bool o_perm, float *lse, hipStream_t s);
hipError_t launch_attention_combine(const CombineItem *items, int n_items, int MT, const float *part, int Hq,
                                    int Hkv, bf16_t *O, bf16_t *O_lo, bool o_perm, float *lse, hipStream_t s);
hipError_t launch_linear_simple(bool bf16, int epi, const LinearArgs &a, hipStream_t s);
// Skinny MFMA path (R <= 64); nt = 16-row weight tiles per block (1..8).
hipError_t launch_linear_skinny(int epi, const SkinnyArgs &a, int nt, hipStream_t s);
// Tiled MFMA path for many rows (packed weight, K a multiple of 32,
// activations in operand order).
hipError_t launch_linear_tiled(int epi, const LinearArgs &a, hipStream_t s);
// Tall MFMA path for 64 < R <= 16 * TALL_MT_MAX rows (packed weight,
// activations in operand order): a block holds every row; a.tpb weight tiles
// per block and a.split K slices come from plan_tall.
constexpr int TALL_MT_MAX = 12;    // 16-row tiles a block holds (its activation ring: four stages of 2 MT KB)
constexpr int TALL_TPB = 12;       // weight tiles per block at most (three per wavefront)
constexpr int TALL_TPB_WIDE = 20;  // ... for STORE launches (five per wavefront)
constexpr int TALL_SPLIT_MAX = 32;
constexpr int TALL_GU_SPLIT_MAX = 2;  // K slices of a split gate/up projection
// tpb weight tiles per block, split K slices.  For the SwiGLU projection a
// split > 1 means: the gate/up columns go to fp32 partial tiles (a STORE
// launch over 2 N virtual columns) and launch_swiglu_partials finishes them.
struct TallPlan { int tpb, split; };
bool tall_rows_ok(int R);
// store_tpb_max: widest block a STORE plan may take (TALL_TPB .. TALL_TPB_WIDE)
TallPlan plan_tall(int R, int vrows, int K, bool swiglu, size_t p_floats, int store_tpb_max);
hipError_t launch_linear_tall(int epi, const LinearArgs &a, hipStream_t s);
// A[r][f] = silu(g) * u with g, u the sums over `nsplit` fp32 partial tiles
// part[s][R][2F] of the gate/up-interleaved columns (column 16t + j: gate of
// feature 8t + j for j < 8, up of feature 8t + j - 8 otherwise); A is written
// as a compensated pair in operand order ([R][F], F a multiple of 32).
hipError_t launch_swiglu_partials(const float *part, int nsplit, int R, int F, bf16_t *A, bf16_t *A_lo, hipStream_t s);
// Output-tile blocks the tiled kernel launches for R rows and vrows weight
// rows (before any K split), and how many of them the chip runs at once.
int tiled_blocks(int R, int vrows, int *slots);
// Repack up to three row-major bf16 matrices (rows [0,e0), [e0,e1), [e1,V) of
// the virtual matrix; interleave: w0 = gate, w1 = up, tile t = gate rows
// 8t..8t+7 then up rows 8t..8t+7) of K columns into operand order at dst.
hipError_t launch_pack_weight(const void *w0, const void *w1, const void *w2, int e0, int e1, bool interleave,
                              int V, int K, int grp, void *dst, hipStream_t s);

// Scoring rows: hidden rows Y [R][d] fp32 -> LM-head operand (compensated
// bf16 pair, operand order or row-major, or fp32 row-major).
hipError_t launch_to_operand(bool bf16, bool perm, const float *Y, int R, int d, void *X, void *X_lo, hipStream_t s);
// Log-softmax of R rows of V logits (sum of nsplit fp32 tiles part[s][R][V]):
// lp[r] = log p(target[r]) for r < n_targets, argmax[r] (lowest index among
// maxima; argmax may be null), next[0] = argmax of row R-1 when next is given.
hipError_t launch_logsoftmax(const float *part, int nsplit, int R, int V, const int32_t *target, int n_targets,
                             float *lp, int32_t *argmax, int32_t *next, void *ws, hipStream_t s);
// Device scratch the log-softmax of R rows of V logits needs (ws above).
size_t logsoftmax_ws_bytes(int R, int V);

// CacheBlend selector: dev[p - p0] = ||K_fresh[p] - K_stale[p]|| + ||V_fresh[p] -
// V_stale[p]|| over layer fl of `fresh` and layer sl of `stale` (cache
// layouts with their own n_cap), p in [p0, p1).
hipError_t launch_kv_deviation(bool bf16, const void *fresh, int fresh_ncap, int fl, const void *stale, int stale_ncap,
                               int sl, int Hkv, int hd, int p0, int p1, float *dev, hipStream_t s);
// Attention selector, one layer: part[g * n + p] (=, or += when accumulate)
// the attention probability that the q query rows (row-major Q [q][Hq*hd],
// compensated pair in bf16; lse from the same layer's attention launch) place
// on stale key p < n of kv head g, summed over the rows and the group's heads.
bool attn_mass_mfma_ok(bool bf16, int hd);
hipError_t launch_attn_mass(bool bf16, const void *Q, const void *Q_lo, const float *lse, int q, const void *cache,
                            int n_cap, int layer, int Hq, int Hkv, int hd, int n, float *part, bool accumulate,
                            hipStream_t s);
// mass[p] = sum over g of part[g * n + p], p < n.
hipError_t launch_mass_reduce(const float *part, int Hkv, int n, float *mass, hipStream_t s);
// The K largest of dev[0, m) (ties: lower index), as ascending positions p0 + i.
hipError_t launch_topk(const float *dev, int m, int K, int p0, int32_t *out, hipStream_t s);

// Attention item geometry shared by the planner and the kernels.
constexpr int ATT_KT = 64;     // keys per LDS tile
constexpr int ATT_HD = 128;    // head_dim of the MFMA attention kernel

}  // namespace kvr
