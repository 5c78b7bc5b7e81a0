// Linear layer for a mid-size number of rows (64 < R <= 192), bf16 MFMA.
//
// Between the skinny kernel (a few dozen rows: every weight element is read
// once and each wavefront streams its own activations) and the tiled kernel
// (hundreds of rows and more: both operands tiled through LDS, each weight
// slab re-read by every row block) lies the repair of one or two hundred
// rows.  There the tiled kernel's 64-row blocks re-read every weight slab once
// per row block and stream the whole compensated activation matrix once per
// 256-column block, so a compute unit waits on several megabytes of reads per
// projection while neither HBM nor the MFMA pipes are busy.  This kernel
// gives a block every row of the pass: each weight element is read from HBM
// once and multiplies all rows.
//
// A block owns up to TALL_TPB (STORE launches: TALL_TPB_WIDE) consecutive
// 16-row weight tiles and one of `split` slices of K.  Per k-step, the 2 MT activation fragments (hi and lo
// of every 16-row tile) and the block's weight fragments are copied straight
// from memory into a ring of LDS stages (global_load_lds_dwordx4; both
// operands are stored in operand order, so each 16 x 32 fragment is one
// contiguous 1 KB block, and lane l's 16 bytes land at byte 16 l), STAGES - 1
// k-steps ahead (three, or two where four stages do not fit in LDS).  The
// four wavefronts share the activation fragments; wavefront w owns the
// block's weight tiles w, w + 4, w + 8 (, w + 12, w + 16) and keeps their
// accumulators for all rows, so no reduction across wavefronts is needed.
// Each wavefront copies the same number of fragments per k-step (the short
// ones repeat their last fragment), so the count of its loads in flight is
// known exactly; only real k-steps are copied, and the wait at each k-step
// allows exactly the loads of the later k-steps already issued.
//
// What bounds it: a compute unit takes in about 30 GB/s of this mix of
// weight (HBM) and activation (L2) fragments, so a projection costs its bytes
// per unit at that rate.  A K split cuts each unit's share of the activation
// matrix.  The SwiGLU projection needs whole dot products: unsplit it runs
// with the SwiGLU in the epilogue, and at 144 rows its 2 MB of compensated
// activations per unit (beside 1 MB of weights) hold it at the tiled
// kernel's time; split in two it runs as a STORE launch of up to twenty
// tiles per block (1 MB of activations per unit) into fp32 partials that
// swiglu_partials_kernel sums, activates and writes as the down projection's
// operand.  Measured and rejected: a fifth stage (four k-steps in
// flight; Qwen2.5-7B shape, 144 rows: 6.93 against 6.80 ms per repair), and
// wavefronts 0-1 copying the activations with 2-3 copying the weights into a
// twice deeper ring (every projection about twice slower).
//
// Outputs as the tiled kernel: STORE writes fp32 partial tiles [split][R][ldo]
// that the next row-wise kernel sums in a fixed order; SWIGLU (unsplit)
// takes gate/up-interleaved tiles and writes silu(gate) * up in operand order.
#include <algorithm>

#include "common.h"

namespace kvr {

namespace {

constexpr int FRAG = 512;           // bf16 elements per fragment (1 KB)

// LDS ring stages for MT activation tiles and TPB weight tiles per k-step:
// four (three k-steps in flight) where they fit in 160 KB, else three.
template <int MT, int TPB>
constexpr int tall_stages() { return 4 * (2 * MT + TPB) * FRAG * 2 <= 160 * 1024 ? 4 : 3; }

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

__device__ __forceinline__ void copy_to_lds(const bf16_t *g, bf16_t *l) {
    __builtin_amdgcn_global_load_lds(g, l, 16, 0, 0);
}

// Block barrier for LDS hand-over that does not wait for vector-memory loads
// still in flight (the loads of later k-steps).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0) only
    asm volatile("s_barrier" ::: "memory");
}

// Wait until at most N of this wavefront's vector-memory loads are in flight
// (vmcnt is six bits: low four at [3:0], high two at [15:14]).
template <int N>
__device__ __forceinline__ void wait_loads_upto() {
    static_assert(N >= 0 && N < 64, "vmcnt immediate");
    __builtin_amdgcn_s_waitcnt(0x70 | 0xF00 | (N & 15) | ((N >> 4) << 14));
}

// Wait until the loads of `later` (<= L) k-steps issued after the one needed,
// PER loads each, are all that may still be in flight.
template <int PER, int L>
__device__ __forceinline__ void wait_later(int later) {
    if constexpr (L == 0) {
        wait_loads_upto<0>();
    } else {
        if (later >= L) wait_loads_upto<L * PER>();
        else wait_later<PER, L - 1>(later);
    }
}

template <int MT, int TPB, int EPI>
__global__ __launch_bounds__(256, 1) void linear_tall_kernel(LinearArgs a) {
    constexpr int NTW = TPB / 4;        // weight tiles per wavefront at most
    constexpr int STAGES = tall_stages<MT, TPB>();
    constexpr int NX = 2 * MT;          // activation fragments per k-step: hi row tiles, then lo
    constexpr int NF = NX + TPB;        // fragments per k-step in a stage
    constexpr int FPW = (NF + 3) / 4;   // fragments each wavefront copies per k-step
    static_assert(STAGES * NF * FRAG * 2 <= 160 * 1024, "LDS");
    __shared__ __attribute__((aligned(16))) bf16_t lds[STAGES * NF * FRAG];

    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wavefront index (uniform)
    const int split = a.split > 1 ? a.split : 1;
    const int tg = blockIdx.x / split, sp = blockIdx.x - tg * split;
    const int ksteps = a.K >> 5;
    const int s0 = (int)((long long)ksteps * sp / split), s1 = (int)((long long)ksteps * (sp + 1) / split);
    const int nk = s1 - s0;
    const int ntiles = (EPI == EPI_SWIGLU ? 2 * a.N : a.N) >> 4;
    const int t0 = tg * a.tpb, tend = min(t0 + a.tpb, ntiles);

    // this wavefront's fragments of a k-step: f = w + 4 i, the last one
    // repeated by the wavefronts that have fewer
    const bf16_t *src[FPW];
    int kst[FPW], dst[FPW];
#pragma unroll
    for (int i = 0; i < FPW; ++i) {
        const int f = w + 4 * min(i, (NF - 1 - w) / 4);
        dst[i] = f * FRAG;
        if (f < NX) {
            const int mt = f < MT ? f : f - MT;
            src[i] = (const bf16_t *)(f < MT ? a.x : a.x_lo) + ((size_t)mt * ksteps + s0) * FRAG + lane * 8;
            kst[i] = FRAG;
        } else {
            // weight tiles past the block's last one re-read it (never stored)
            const int t = min(t0 + (f - NX), tend - 1);
            src[i] = (const bf16_t *)a.wp + packed_tile_offset(t, ntiles, ksteps, a.grp, &kst[i]) + lane * 8;
            src[i] += (size_t)s0 * kst[i];
        }
    }
    int issued = 0;  // k-steps copied so far (k-steps 0 .. issued-1 of the slice)
    auto issue = [&]() {
        bf16_t *st = lds + (issued % STAGES) * NF * FRAG;
#pragma unroll
        for (int i = 0; i < FPW; ++i) {
            copy_to_lds(src[i], st + dst[i]);
            src[i] += kst[i];
        }
        ++issued;
    };

    f32x4 acc[MT][NTW];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int j = 0; j < NTW; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // row threadIdx.x's sums of squares (the first four column blocks),
    // loaded before the ring starts and first used in the epilogue; they are
    // older than every ring load, so the ring's exact waits cover them too
    const bool rs_row = a.rs_ssq && (int)threadIdx.x < a.R;
    float rs_pre[4] = {0.f, 0.f, 0.f, 0.f};
    if (rs_row) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (q < a.rs_nb) rs_pre[q] = a.rs_ssq[(size_t)q * a.R + threadIdx.x];
    }

    for (int j = 0; j < STAGES - 1 && j < nk; ++j) issue();
    for (int kk = 0; kk < nk; ++kk) {
        // k-step kk's fragments (this wavefront's) have landed: the k-steps
        // issued after it may stay in flight
        wait_later<FPW, STAGES - 2>(issued - 1 - kk);
        lds_barrier();  // everyone's fragments of kk have landed; all reads of kk - 1 are done
        if (issued < nk) issue();  // k-step kk + STAGES - 1, into the stage k-step kk - 1 used

        const bf16_t *st = lds + (kk % STAGES) * NF * FRAG + lane * 8;
        bf16x8 wf[NTW];
#pragma unroll
        for (int j = 0; j < NTW; ++j) wf[j] = *reinterpret_cast<const bf16x8 *>(st + (NX + w + 4 * j) * FRAG);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const bf16x8 xh = *reinterpret_cast<const bf16x8 *>(st + m * FRAG);
            const bf16x8 xl = *reinterpret_cast<const bf16x8 *>(st + (MT + m) * FRAG);
            // every slot, present tile or not (a missing one holds a copy of the
            // block's last tile and is never stored): the wavefronts run in
            // lockstep, so skipping would save no time, and branches around the
            // MFMAs would split the chain
#pragma unroll
            for (int j = 0; j < NTW; ++j) {
                acc[m][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xh, wf[j], acc[m][j], 0, 0, 0);
                acc[m][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl, wf[j], acc[m][j], 0, 0, 0);
            }
        }
    }

    bool tv[NTW];  // weight tile w + 4 j of the block exists
#pragma unroll
    for (int j = 0; j < NTW; ++j) tv[j] = t0 + w + 4 * j < tend;
    if (a.rs_ssq) {
        // RMS scales of the rows (the sums in column-block order, as the
        // skinny kernel takes them), handed over through LDS: the ring is no
        // longer read after the first barrier
        float *rsl = reinterpret_cast<float *>(lds);
        float sc = 1.f;
        if (rs_row) {
            float t = 0.f;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (q < a.rs_nb) t += rs_pre[q];
            for (int b = 4; b < a.rs_nb; ++b) t += a.rs_ssq[(size_t)b * a.R + threadIdx.x];
            sc = rsqrtf(t / (float)a.rs_d + a.rs_eps);
        }
        __syncthreads();
        if ((int)threadIdx.x < 16 * MT) rsl[threadIdx.x] = sc;
        __syncthreads();
    }
    // accumulator layout: lane l holds tile column l%16, rows 16 m + 4 (l/16) + e
    const int rq = 4 * (lane >> 4);
    // the scale of each of this lane's rows (1 without rs_ssq), applied as
    // the accumulators are stored
    float rsc[MT][4];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int e = 0; e < 4; ++e) rsc[m][e] = a.rs_ssq ? reinterpret_cast<const float *>(lds)[16 * m + rq + e] : 1.f;
    if (EPI == EPI_SWIGLU) {
        // column c < 8 of tile t is the gate of feature 8t + c, column c + 8
        // its up (held by lane l + 8)
        bf16_t *A = (bf16_t *)a.out;
        bf16_t *Alo = (bf16_t *)a.out_lo;
        const bool gate_lane = (lane & 8) == 0;
#pragma unroll
        for (int j = 0; j < NTW; ++j) {
            if (!tv[j]) continue;
            const int f = 8 * (t0 + w + 4 * j) + (lane & 7);
#pragma unroll
            for (int m = 0; m < MT; ++m)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float g = acc[m][j][e] * rsc[m][e];
                    const float u = __shfl_xor(g, 8);  // lane l + 8: the same row
                    const int r = 16 * m + rq + e;
                    if (gate_lane && r < a.R) store_operand(A, Alo, perm_offset(r, f, a.N), silu_f(g) * u);
                }
        }
        return;
    }
    float *out = (float *)a.out + (size_t)sp * a.R * a.ldo;
#pragma unroll
    for (int j = 0; j < NTW; ++j) {
        if (!tv[j]) continue;
        const int c = 16 * (t0 + w + 4 * j) + (lane & 15);
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = 16 * m + rq + e;
                if (r < a.R) out[(size_t)r * a.ldo + c] = acc[m][j][e] * rsc[m][e];
            }
    }
}

template <int MT>
hipError_t launch_mt(int epi, const LinearArgs &a, int blocks, hipStream_t s) {
    if (epi == EPI_SWIGLU) kvr_launch((linear_tall_kernel<MT, TALL_TPB, EPI_SWIGLU>), dim3(blocks), dim3(256), 0, s, a);
    else if (a.tpb <= TALL_TPB) kvr_launch((linear_tall_kernel<MT, TALL_TPB, EPI_STORE>), dim3(blocks), dim3(256), 0, s, a);
    else kvr_launch((linear_tall_kernel<MT, TALL_TPB_WIDE, EPI_STORE>), dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

// One thread per (row, eight features): the gate and up partials of the
// features' weight tile summed in split order, SwiGLU, and one 16-byte store
// each of the hi and lo parts (eight consecutive features are contiguous in
// operand order).  The 16 rows of a row tile are the fastest index, so that
// 16 neighbouring threads store 256 contiguous bytes of an operand fragment.
__global__ __launch_bounds__(256) void swiglu_partials_kernel(const float *part, int nsplit, int R, int F, bf16_t *A,
                                                               bf16_t *A_lo) {
    const int per_row = F >> 3;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    const int q = idx >> 4;
    const int rt = q / per_row, t = q - rt * per_row;
    const int r = rt * 16 + (idx & 15);
    if (r >= R) return;
    const size_t row = (size_t)2 * F;
    const float *p = part + (size_t)r * row + 16 * t;
    f32x4 g0 = *reinterpret_cast<const f32x4 *>(p), g1 = *reinterpret_cast<const f32x4 *>(p + 4);
    f32x4 u0 = *reinterpret_cast<const f32x4 *>(p + 8), u1 = *reinterpret_cast<const f32x4 *>(p + 12);
    for (int q = 1; q < nsplit; ++q) {
        const float *pq = p + (size_t)q * R * row;
        g0 += *reinterpret_cast<const f32x4 *>(pq);
        g1 += *reinterpret_cast<const f32x4 *>(pq + 4);
        u0 += *reinterpret_cast<const f32x4 *>(pq + 8);
        u1 += *reinterpret_cast<const f32x4 *>(pq + 12);
    }
    float y[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        y[e] = silu_f(g0[e]) * u0[e];
        y[4 + e] = silu_f(g1[e]) * u1[e];
    }
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const bf16_t h0 = f32_to_bf16(y[2 * e]), h1 = f32_to_bf16(y[2 * e + 1]);
        const bf16_t l0 = f32_to_bf16(y[2 * e] - bf16_to_f32(h0)), l1 = f32_to_bf16(y[2 * e + 1] - bf16_to_f32(h1));
        hi[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        lo[e] = (uint32_t)l0 | ((uint32_t)l1 << 16);
    }
    const size_t off = perm_offset(r, 8 * t, F);
    *reinterpret_cast<u32x4 *>(A + off) = u32x4{hi[0], hi[1], hi[2], hi[3]};
    *reinterpret_cast<u32x4 *>(A_lo + off) = u32x4{lo[0], lo[1], lo[2], lo[3]};
}

}  // namespace

bool tall_rows_ok(int R) { return R > 64 && R <= 16 * TALL_MT_MAX; }

// Weight tiles per block and K split: the plan (tiles per block that keep
// the grid within 256 blocks for each split) that minimises the bytes one
// block reads and writes: activations R x K/split x 4 bytes (a compensated
// pair), weights tiles x 16 x K/split x 2 bytes and, when split, its fp32
// partial tile; the partial buffer bounds the split.  A STORE projection
// takes blocks of up to store_tpb_max tiles and splits up to TALL_SPLIT_MAX.
// The SwiGLU projection runs unsplit (at most TALL_TPB tiles per block, the
// SwiGLU in the epilogue) or, split in two, as a STORE launch of up to
// TALL_TPB_WIDE tiles per block whose partials the SwiGLU pass finishes; its
// cost adds that pass's reads and writes spread over 256 compute units.  At
// 144 rows (Qwen2.5-7B shape) the unsplit block takes in 2 MB of
// activations beside its 1 MB of weights, the split one half of that.  With
// more than 256 x TALL_TPB tiles the grid takes several rounds of full blocks.
TallPlan plan_tall(int R, int vrows, int K, bool swiglu, size_t p_floats, int store_tpb_max) {
    const int ntiles = vrows / 16, ksteps = K / 32;
    const long long rows = (R + 15) / 16 * 16;
    TallPlan p{std::min(TALL_TPB, std::max(1, (ntiles + 255) / 256)), 1};
    const int spmax = swiglu ? TALL_GU_SPLIT_MAX : TALL_SPLIT_MAX;
    long long best = -1;
    for (int sp = 1; sp <= std::min(spmax, std::max(1, ksteps / 4)); ++sp) {
        if (sp > 1 && (size_t)sp * R * vrows > p_floats) break;
        const int cols = 256 / sp;
        if (cols < 1) break;
        const int tpb = (ntiles + cols - 1) / cols;
        const int cap = swiglu ? (sp == 1 ? TALL_TPB : TALL_TPB_WIDE) : store_tpb_max;
        if (tpb > cap) continue;
        const long long ks = (ksteps + sp - 1) / sp;
        long long bytes = ks * 32 * (rows * 4 + (long long)tpb * 16 * 2) + (sp > 1 ? rows * tpb * 16 * 4 : 0);
        if (swiglu && sp > 1) bytes += ((long long)sp * R * vrows * 4 + (long long)R * (vrows / 2) * 4) / 256;
        if (best < 0 || bytes < best) {
            best = bytes;
            p = TallPlan{tpb, sp};
        }
    }
    return p;
}

hipError_t launch_linear_tall(int epi, const LinearArgs &a, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    if (!tall_rows_ok(a.R) || !a.x_lo || !a.wp || (epi == EPI_SWIGLU && !a.out_lo)) return hipErrorInvalidValue;
    if (epi != EPI_STORE && epi != EPI_SWIGLU) return hipErrorInvalidValue;
    const int vrows = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    if (a.K % 32 != 0 || a.K < 32 || vrows % 16 != 0 || a.tpb < 1 ||
        a.tpb > (epi == EPI_SWIGLU ? TALL_TPB : TALL_TPB_WIDE))
        return hipErrorInvalidValue;
    const int split = a.split > 1 ? a.split : 1;
    if (split > a.K / 32 || (epi == EPI_SWIGLU && split != 1)) return hipErrorInvalidValue;
    const int blocks = (vrows / 16 + a.tpb - 1) / a.tpb * split;
    switch ((a.R + 15) / 16) {
        case 5: return launch_mt<5>(epi, a, blocks, s);
        case 6: return launch_mt<6>(epi, a, blocks, s);
        case 7: return launch_mt<7>(epi, a, blocks, s);
        case 8: return launch_mt<8>(epi, a, blocks, s);
        case 9: return launch_mt<9>(epi, a, blocks, s);
        case 10: return launch_mt<10>(epi, a, blocks, s);
        case 11: return launch_mt<11>(epi, a, blocks, s);
        default: return launch_mt<12>(epi, a, blocks, s);
    }
}

hipError_t launch_swiglu_partials(const float *part, int nsplit, int R, int F, bf16_t *A, bf16_t *A_lo,
                                  hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (!part || !A || !A_lo || nsplit < 1 || F % 32 != 0) return hipErrorInvalidValue;
    const long long items = (long long)((R + 15) / 16 * 16) * (F / 8);
    kvr_launch(swiglu_partials_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, part, nsplit, R, F, A,
               A_lo);
    return hipGetLastError();
}

}  // namespace kvr
