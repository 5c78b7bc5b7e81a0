// Tiled bf16 MFMA linear layer for many rows (prefill, batched repair).
//
// Y[r][n] = sum_k X[r][k] * W[n][k].  Both operands arrive in MFMA operand
// order: the activations X (a compensated pair hi + lo, written so by their
// producers) and the packed weight W (pack.hip) are sequences of 1 KB
// fragments, one per 16-row tile and 32-wide k-step, that a wavefront loads
// with one 16-byte access per lane.  A block computes a 128 x 256 output tile
// (8 row tiles x 16 weight tiles); its four wavefronts own 64 x 128 sub-tiles
// (4 x 8 v_mfma_f32_16x16x32_bf16 tiles, two MFMAs per product for hi and lo).
// When 128-row blocks would not give every compute unit two of them, the
// launch takes 64 x 256 tiles (four wavefronts of 64 x 64), three per unit.
// A STORE launch may also cut K into `split` slices (grid dimension y), each
// writing an fp32 partial tile that the consumer sums in a fixed order: the
// way a few hundred rows still fill the chip.
//
// The fragments go from memory straight into LDS (global_load_lds_dwordx4:
// lane l's 16 bytes land at the destination + 16 l, so a fragment keeps its
// layout and no registers stage it).  LDS holds a ring of STAGES k-steps of
// 32 fragments each (32 KB); the loads for k-step kk + STAGES - 1 are issued
// while k-step kk is multiplied, and each wavefront waits only for its own
// loads of k-step kk before the block barrier.  The barrier is a bare
// s_barrier: the compiler's workgroup fence would also wait for the loads
// still in flight for the later stages.  Two stages (64 KB) let two blocks
// share a compute unit, so that one block's MFMAs run while the other waits
// for its next k-step (the register budget is set for two waves per SIMD);
// measured on the 8B shape at 5000 rows, this beats four stages with one
// block per unit by 20 % (gate/up 1.73 ms against 2.21 ms).  Row tiles past the last one and
// weight tiles past the last one re-read the last tile; their results are
// not stored.
//
// Tile order.  Workgroups are handed to the eight XCDs in turn (workgroup b to
// XCD b % 8), and each XCD has its own L2.  The output tiles are therefore
// numbered in groups of row blocks (within a group: column block outer, row
// block inner), the numbering is cut into eight contiguous ranges, and XCD x
// runs range x in order, so the blocks that read one weight slab run at the
// same time on one XCD and share its L2.  Up to GROUP_ALL row blocks form one
// group (a repair of a few hundred rows: every weight slab is fetched from
// HBM about once; with groups of four, 528 rows fetched 3.6 times the
// gate/up weights); more (prefill, batches) are grouped by four.
#include <stdlib.h>

#include <algorithm>

#include "common.h"

namespace kvr {

namespace {

constexpr int WT = 16;          // 16-row weight tiles per block (256 output columns)
constexpr int FRAG = 512;       // bf16 elements of one 16 x 32 operand fragment
constexpr int XCDS = 8;         // L2 domains the workgroups are dealt to in turn
constexpr int GROUP_M = 4;      // row blocks per group of the tile order (many row blocks)
constexpr int GROUP_ALL = 12;   // up to this many row blocks, one group holds them all

// Block shape for RT 16-row activation tiles: wavefronts in WM rows x WN
// columns, each owning 4 row tiles x JT weight tiles (64 x 128 or 64 x 64).
//   RT = 16: 256 rows, eight wavefronts, three LDS stages (144 KB), one block
//            per compute unit: the weight tile of a k-step serves 256 rows;
//   RT = 8:  128 rows, four wavefronts, two stages, two blocks per unit;
//   RT = 4:  64 rows, four wavefronts, two stages, three blocks per unit, for
//            grids that would otherwise not fill the chip.
template <int RT>
struct TileShape {
    static constexpr int NW = RT == 16 ? 8 : 4;      // wavefronts per block
    static constexpr int STAGES = RT == 16 ? 3 : 2;  // k-steps held in the LDS ring
    static constexpr int NFRAG = 2 * RT + WT;        // fragments per k-step: X hi, X lo, W
    static constexpr int STAGE = NFRAG * FRAG;
    static constexpr int FPW = NFRAG / NW;           // fragments each wavefront loads per k-step
    static constexpr int WM = RT / 4, WN = NW / WM, JT = WT / WN;
    static constexpr int BLOCKS_PER_CU = RT == 16 ? 1 : (RT == 8 ? 2 : 3);
    static_assert(NFRAG % NW == 0 && WM * WN == NW && FPW <= 8, "block shape");
    static_assert(STAGES * STAGE * 2 <= 160 * 1024, "LDS");
};

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

// Block barrier that orders LDS accesses for the compiler without waiting for
// outstanding vector-memory loads.  The LDS wait is the builtin (not part of
// the asm) so that the compiler knows every earlier LDS read has completed.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
    asm volatile("s_barrier" ::: "memory");
}

// Wait until none of this wavefront's vector-memory loads is in flight
// (expcnt and lgkmcnt left unconstrained).
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x70 | 0xF00); }

// Wait until at most n of this wavefront's vector-memory loads are in flight
// (n a compile-time count below 16).
template <int N>
__device__ __forceinline__ void wait_loads_upto() {
    static_assert(N >= 0 && N < 16, "vmcnt immediate");
    __builtin_amdgcn_s_waitcnt(0x70 | 0xF00 | N);
}

template <int EPI, int RT>
__global__ __launch_bounds__(64 * TileShape<RT>::NW, TileShape<RT>::BLOCKS_PER_CU) void linear_tiled_kernel(
    LinearArgs a) {
    using S = TileShape<RT>;
    constexpr int STAGE = S::STAGE, FPW = S::FPW, JT = S::JT, STAGES = S::STAGES;
    __shared__ __attribute__((aligned(16))) bf16_t lds[STAGES * STAGE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = w / S::WN, wn = w % S::WN;
    const int ksteps = a.K >> 5;   // k-steps of the whole row (operand strides)
    const int split = EPI == EPI_STORE ? max(1, a.split) : 1;
    const int sp = blockIdx.y;    // this block's K slice: k-steps [k0, k0 + nk)
    const int k0 = (int)(((long long)ksteps * sp) / split);
    const int nk = (int)(((long long)ksteps * (sp + 1)) / split) - k0;
    const int ntiles = (a.N * (EPI == EPI_SWIGLU ? 2 : 1)) >> 4;
    const int rtiles = (a.R + 15) >> 4;
    // this workgroup's output tile (bm, bn) in the XCD-grouped order
    const int MB = (rtiles + RT - 1) / RT, NB = (ntiles + WT - 1) / WT;
    const int T = MB * NB, per = (T + XCDS - 1) / XCDS;
    const int tile = (blockIdx.x % XCDS) * per + blockIdx.x / XCDS;
    if (tile >= T) return;
    const int GM = MB <= a.group_all ? MB : GROUP_M;
    const int grp = tile / (GM * NB);
    const int gm = min(GM, MB - grp * GM);
    const int ti = tile - grp * GM * NB;
    const int bn = ti / gm, bm = grp * GM + ti % gm;

    // this wavefront's fragments of every k-step: f = FPW w + i (X hi row
    // tiles, X lo row tiles, then weight tiles).  The array has a fixed size:
    // a local array whose size depends on the template parameter, captured by
    // the lambda below, made the host compiler drop the kernel's launch stub.
    static_assert(FPW <= 8, "at most eight fragments per wavefront");
    const bf16_t *src[8];
    int kstride[8];  // elements between a fragment's k-steps
#pragma unroll
    for (int i = 0; i < FPW; ++i) {
        const int f = FPW * w + i;
        if (f < 2 * RT) {
            const int t = min(bm * RT + (f % RT), rtiles - 1);
            src[i] = (const bf16_t *)(f < RT ? a.x : a.x_lo) + ((size_t)t * ksteps * 64 + lane) * 8;
            kstride[i] = 512;
        } else {
            const int t = min(bn * WT + (f - 2 * RT), ntiles - 1);
            src[i] = (const bf16_t *)a.wp + packed_tile_offset(t, ntiles, ksteps, a.grp, &kstride[i]) + lane * 8;
        }
    }
    // k-steps are issued in order, so each fragment keeps a running pointer
    // (one add per k-step, no multiply by the stride in the loop)
#pragma unroll
    for (int i = 0; i < FPW; ++i) src[i] += (size_t)k0 * kstride[i];
    auto issue = [&](int kk) {
        bf16_t *st = lds + (kk % STAGES) * STAGE + FPW * w * FRAG;
#pragma unroll
        for (int i = 0; i < FPW; ++i) {
            __builtin_amdgcn_global_load_lds(src[i], st + i * FRAG, 16, 0, 0);
            src[i] += kstride[i];
        }
    };

    f32x4 acc[4][JT];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < JT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue(s);
    for (int kk = 0; kk < nk; ++kk) {
        // this wavefront's loads of k-step kk have landed (with three stages
        // the loads of kk + 1, issued later, may still be in flight)
        if (STAGES == 3 && kk + 1 < nk) wait_loads_upto<(STAGES == 3 ? FPW : 0)>();
        else wait_loads();
        lds_barrier();  // every wavefront's loads of kk have landed; all reads of kk - 1 are done
        if (kk + STAGES - 1 < nk) issue(kk + STAGES - 1);  // into the slot k-step kk - 1 used

        const bf16_t *st = lds + (kk % STAGES) * STAGE + lane * 8;
        bf16x8 av[4], al[4], bv[JT];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            av[i] = *reinterpret_cast<const bf16x8 *>(st + (wm * 4 + i) * FRAG);
            al[i] = *reinterpret_cast<const bf16x8 *>(st + (RT + wm * 4 + i) * FRAG);
        }
#pragma unroll
        for (int j = 0; j < JT; ++j) bv[j] = *reinterpret_cast<const bf16x8 *>(st + (2 * RT + wn * JT + j) * FRAG);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < JT; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], bv[j], acc[i][j], 0, 0, 0);
            }
    }

    // Epilogue through LDS.  The accumulators hold, per lane, one column and
    // four rows of each 16 x 16 tile, so stores straight from them write 2- or
    // 4-byte pieces scattered over rows (measured on the 5000-token prefill:
    // skipping every store of these kernels saved 8.5 of 126 ms).  Instead
    // each wavefront writes its results into its own 16 KB region of the LDS
    // ring (free once every wavefront has passed the last k-step) and copies
    // them out in whole pieces: a SwiGLU output fragment (16 rows x 32
    // features in operand order) as one contiguous 1 KB store of hi and one
    // of lo, fp32 partial rows in pieces of SC / 4 lanes x 16 bytes.  The
    // region is [64 rows][SC floats] (SC = 64, or 32 for the 64-row shape,
    // whose ring is smaller) with the 16-byte column index XORed with the
    // row, so the rows read by a fragment's lanes fall on distinct banks.
    constexpr int SC = S::NW * 64 * 64 * 4 <= STAGES * STAGE * 2 ? 64 : 32;
    static_assert(S::NW * 64 * SC * 4 <= STAGES * STAGE * 2 && 8 * JT <= SC, "epilogue staging fits in the LDS ring");
    __syncthreads();
    float *stg = reinterpret_cast<float *>(lds) + w * 64 * SC;
    auto sidx = [](int r, int c) { return r * SC + ((((c >> 2) ^ r) & (SC / 4 - 1)) << 2) + (c & 3); };
    const int lrow = 4 * (lane >> 4);  // accumulator layout: lane l holds tile column l%16, rows 4*(l/16)+e
    const int row0 = bm * 16 * RT + wm * 64;  // the wavefront's first row
    if (EPI == EPI_SWIGLU) {
        // gate/up interleaved: column j < 8 of weight tile t is the gate of
        // feature 8t+j, column j+8 its up (lane l+8 holds it); the output is
        // the down projection's operand, in operand order
        bf16_t *A = (bf16_t *)a.out;
        bf16_t *Alo = (bf16_t *)a.out_lo;
        constexpr int NFEAT = 8 * JT;  // features of the wavefront: 64 or 32
        const bool gate_lane = (lane & 8) == 0;
#pragma unroll
        for (int j = 0; j < JT; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float g = acc[i][j][e];
                    const float u = __shfl_xor(g, 8);
                    if (gate_lane) stg[sidx(16 * i + lrow + e, 8 * j + (lane & 7))] = silu_f(g) * u;
                }
        __syncthreads();
        const int f_base = 8 * (bn * WT + wn * JT);  // a multiple of 32: k-step aligned
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int ks = 0; ks < NFEAT / 32; ++ks) {
                const int lr = 16 * i + (lane & 15), c = 32 * ks + 8 * (lane >> 4);
                const int r = row0 + lr, f = f_base + c;
                if (r >= a.R || f >= a.N) continue;
                const f32x4 v0 = *reinterpret_cast<const f32x4 *>(&stg[sidx(lr, c)]);
                const f32x4 v1 = *reinterpret_cast<const f32x4 *>(&stg[sidx(lr, c + 4)]);
                const float y[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
                uint32_t hi[4], lo[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const bf16_t h0 = f32_to_bf16(y[2 * q]), h1 = f32_to_bf16(y[2 * q + 1]);
                    const bf16_t l0 = f32_to_bf16(y[2 * q] - bf16_to_f32(h0)), l1 = f32_to_bf16(y[2 * q + 1] - bf16_to_f32(h1));
                    hi[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
                    lo[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
                }
                const size_t off = perm_offset(r, f, a.N);
                *reinterpret_cast<u32x4 *>(A + off) = u32x4{hi[0], hi[1], hi[2], hi[3]};
                *reinterpret_cast<u32x4 *>(Alo + off) = u32x4{lo[0], lo[1], lo[2], lo[3]};
            }
        return;
    }
    // fp32 rows [R][ldo], SC / 16 weight tiles (SC columns) at a time
    constexpr int JC = SC / 16, LPR = SC / 4;  // tiles per pass, lanes per row
    float *out = (float *)a.out + (size_t)sp * a.R * a.ldo;
#pragma unroll
    for (int j0 = 0; j0 < JT; j0 += JC) {
        if (j0 > 0) __syncthreads();  // the previous pass's reads are done
#pragma unroll
        for (int j = 0; j < JC; ++j)
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) stg[sidx(16 * i + lrow + e, 16 * j + (lane & 15))] = acc[i][j0 + j][e];
        __syncthreads();
        const int c = 4 * (lane % LPR);        // this lane's four columns of the SC
        const int t = bn * WT + wn * JT + j0 + c / 16;
#pragma unroll
        for (int q = 0; q < 64 / (64 / LPR); ++q) {
            const int lr = (64 / LPR) * q + lane / LPR;
            const int r = row0 + lr;
            if (r >= a.R || t >= ntiles) continue;
            const f32x4 v = *reinterpret_cast<const f32x4 *>(&stg[sidx(lr, c)]);
            f32x4 *o = reinterpret_cast<f32x4 *>(out + (size_t)r * a.ldo + 16 * t + (c & 15));
            if (EPI == EPI_RESID) *o += v;
            else *o = v;
        }
    }
}

}  // namespace

template <int RT>
void launch_rt(int epi, const LinearArgs &a, int tiles, hipStream_t s) {
    dim3 grid((tiles + XCDS - 1) / XCDS * XCDS, epi == EPI_STORE ? std::max(1, (int)a.split) : 1);
    const dim3 block(64 * TileShape<RT>::NW);
    if (epi == EPI_STORE) kvr_launch(linear_tiled_kernel<EPI_STORE, RT>, grid, block, 0, s, a);
    else if (epi == EPI_RESID) kvr_launch(linear_tiled_kernel<EPI_RESID, RT>, grid, block, 0, s, a);
    else kvr_launch(linear_tiled_kernel<EPI_SWIGLU, RT>, grid, block, 0, s, a);
}

// Row tiles per block for R rows and vrows weight rows.  256-row blocks
// (one per compute unit) only when they make at least eight rounds: their
// last, partial round costs a whole one (8B gate/up at 5000 rows, 8.75
// rounds: prefill 132.1 -> 128.1 ms; at 3072 rows, 5.25 rounds: 33.0 ->
// 37.2 ms).  Else 128-row blocks when there is one per unit (a K split then
// brings them to two per unit: batched down 17.5 -> 15.8 ms against 64-row
// blocks), else 64-row blocks.  A larger block is taken only if it pads at
// most 5 % more row tiles than the next smaller one (144 rows are 9 row
// tiles: 16 in 128-row blocks against 12 in 64-row ones; Qwen gate/up 4.5
// against 3.0 ms).  KVR_TILED_RT (4, 8, 16) forces a shape.
static int tiled_rt(int R, int vrows) {
    const int rtiles = (R + 15) / 16, nb = (vrows / 16 + WT - 1) / WT;
    if (const char *e = getenv("KVR_TILED_RT")) {
        const int v = atoi(e);
        if (v == 4 || v == 8 || v == 16) return v;
    }
    auto padded = [&](int rt) { return (rtiles + rt - 1) / rt * rt; };
    const bool fits8 = 20 * padded(8) <= 21 * padded(4), fits16 = 20 * padded(16) <= 21 * padded(8);
    if (fits8 && fits16 && (rtiles + 15) / 16 * nb >= 8 * 256) return 16;
    if (fits8 && (rtiles + 7) / 8 * nb >= 256) return 8;
    return 4;
}

int tiled_blocks(int R, int vrows, int *slots) {
    const int rtiles = (R + 15) / 16, nb = (vrows / 16 + WT - 1) / WT;
    const int rt = tiled_rt(R, vrows);
    if (slots) *slots = (rt == 16 ? TileShape<16>::BLOCKS_PER_CU : rt == 8 ? TileShape<8>::BLOCKS_PER_CU
                                                                           : TileShape<4>::BLOCKS_PER_CU) * 256;
    return (rtiles + rt - 1) / rt * nb;
}

hipError_t launch_linear_tiled(int epi, const LinearArgs &a, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    if (!a.x_lo || !a.wp || (epi == EPI_SWIGLU && !a.out_lo)) return hipErrorInvalidValue;
    const int vrows = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    if (a.K % 32 != 0 || vrows % 16 != 0) return hipErrorInvalidValue;
    if (a.split > 1 && (epi != EPI_STORE || a.split > a.K / 32)) return hipErrorInvalidValue;
    const int rt = tiled_rt(a.R, vrows);
    const int blocks = tiled_blocks(a.R, vrows, nullptr);
    LinearArgs b = a;
    const char *ge = getenv("KVR_TILED_GROUP");  // tuning: row blocks that may form one group
    b.group_all = ge && *ge ? atoi(ge) : GROUP_ALL;
    if (rt == 16) launch_rt<16>(epi, b, blocks, s);
    else if (rt == 8) launch_rt<8>(epi, b, blocks, s);
    else launch_rt<4>(epi, b, blocks, s);
    return hipGetLastError();
}

}  // namespace kvr
