// Weight-streaming linear layer for few rows (R <= 64), bf16 MFMA.
//
// With a repair budget of a few dozen rows the projections are bound by
// reading the weights once from HBM: every weight element meets only R rows.
// The weights are packed in operand order (pack.hip), so a wavefront's load of
// one 16-row x 32-k weight tile is one contiguous 1 KB block that lands in the
// B-operand layout of v_mfma_f32_16x16x32_bf16 (lane l: weight row l%16, 8
// consecutive k at 8*(l/16)).  The activations X come in the same operand
// order, as compensated pairs (hi + lo), so every (row tile, weight tile)
// product is two MFMAs into one fp32 accumulator.
//
// A block owns NT consecutive 16-row weight tiles and one of `split` slices of
// K; its four wavefronts split that slice further and are summed through LDS
// at the end.  A wide block lets one X read serve NT tiles (X traffic from L2
// falls as 1/NT), and the planner sizes NT and split so that the grid is about
// one block per compute unit.  Each wavefront keeps a ring of D k-steps of
// loads in flight: it consumes one k-step and immediately refills that slot
// with the k-step D further on, so the memory pipe never drains between
// batches.
//
// The tiles may be stored in groups (packed_tile_offset): when a block's NT
// tiles form one group, its weight stream is one contiguous range.
//
// Blocks never exchange data: with split > 1 each block writes an fp32 partial
// tile [split][R][N] and the row-wise kernel that runs next sums the partials
// in a fixed order (deterministic, and free of device-wide fences).  The
// gate/up projection is never split; its weight is gate/up interleaved (tile t
// = gate rows 8t..8t+7, then up rows 8t..8t+7) and the epilogue applies
// SwiGLU, writing the down projection's operand.  When X is an unnormalised
// H * gain (skinny passes, resid_gain), the epilogue multiplies each output
// row by its RMSNorm scale first.
#include "common.h"

namespace kvr {

namespace {

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

__device__ __forceinline__ bf16x8 ld16(const bf16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}
// Weights are read exactly once per pass: stream them with the nontemporal
// hint so that they do not evict the activations, which every block re-reads.
__device__ __forceinline__ bf16x8 ld16_stream(const bf16_t *p) {
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p)));
}

template <int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void linear_skinny_kernel(SkinnyArgs a) {
    constexpr int FW = 16 * NT;          // virtual weight rows of a block
    constexpr int D = NT >= 6 ? 2 : 3;   // k-steps in flight per wavefront
    __shared__ __attribute__((aligned(16))) float red[4][MT * 16 * (FW + 4)];  // each wavefront's partial sums

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    // RMS row scale (see SkinnyArgs): the first four sums of squares of this
    // thread's row are loaded now, ahead of every weight load, so that they
    // have arrived when the epilogue adds them (R <= 16 MT, so these threads
    // hold rows of the output)
    const bool rs_row = a.rs_ssq && (int)threadIdx.x < a.R;
    float rs_pre[4] = {0.f, 0.f, 0.f, 0.f};
    if (rs_row) {
#pragma unroll
        for (int q = 0; q < 4; ++q) rs_pre[q] = a.rs_ssq[(size_t)min(q, a.rs_nb - 1) * a.R + threadIdx.x];
    }
    const int split = a.split;
    const int tg = blockIdx.x / split, sp = blockIdx.x - tg * split;
    const int ksteps = a.K >> 5;
    const int gw = sp * 4 + w, nw = split * 4;
    const int s0 = (int)(((long long)ksteps * gw) / nw);
    const int s1 = (int)(((long long)ksteps * (gw + 1)) / nw);

    // tiles past the end (last block of a ragged grid) re-read the last tile;
    // their results are never stored
    const bf16_t *wp[NT];
    int wstride[NT];  // elements between a tile's k-steps (packed_tile_offset)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
        wp[nt] = (const bf16_t *)a.w +
                 packed_tile_offset(min(tg * NT + nt, a.ntiles - 1), a.ntiles, ksteps, a.grp, &wstride[nt]) + lane * 8;
    const bf16_t *xp[MT], *xq[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        xp[mt] = (const bf16_t *)a.x + ((size_t)mt * ksteps * 64 + lane) * 8;
        xq[mt] = (const bf16_t *)a.x_lo + ((size_t)mt * ksteps * 64 + lane) * 8;
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    if (s0 < s1) {
        // With tile-major weights every block walks its K slice from a
        // different starting k-step (rotated by the block's index within its
        // XCD).  In lockstep the 32 blocks of an XCD ask for each activation
        // line at the same moment, and all of them wait for its first fetch;
        // rotated, one of them takes the miss and the others find the line in
        // L2 (8B shape, 48 rows: down 27.0 -> 25.8 us, QKV 15.8 -> 15.2 us).
        // Grouped weights (one contiguous range per block) are walked in
        // order: rotation split that range and cost gate/up 1 %.  Logical step
        // lg maps to k-step phys(lg); steps past the slice re-read its last one.
        const int nks = s1 - s0;
        const int rot = a.grp > 1 ? 0 : (int)((blockIdx.x >> 3) % (unsigned)nks);
        auto phys = [&](int lg) {
            lg = min(lg, s1 - 1);
            int q = lg - s0 + rot;
            if (q >= nks) q -= nks;
            return s0 + q;
        };
        bf16x8 wv[D][NT], xv[D][MT], xl[D][MT];
        // The ring loads are unconditional: a slot whose k-step lies past the
        // wavefront's range re-reads its last k-step (a cache hit), so that the
        // compiler can count outstanding loads exactly.
        auto load = [&](int j, int st) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) wv[j][nt] = ld16_stream(wp[nt] + (size_t)st * wstride[nt]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                xv[j][mt] = ld16(xp[mt] + (size_t)st * 512);
                xl[j][mt] = ld16(xq[mt] + (size_t)st * 512);
            }
        };
        auto mma = [&](int j) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[j][mt], wv[j][nt], acc[mt][nt], 0, 0, 0);
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl[j][mt], wv[j][nt], acc[mt][nt], 0, 0, 0);
                }
        };
#pragma unroll
        for (int j = 0; j < D; ++j) load(j, phys(s0 + j));
        int s = s0;
        // The scheduling barriers keep each slot's refill right behind its
        // MFMAs: left free, the compiler sank every refill below the MFMAs of
        // all slots and waited for nearly every load before issuing the next
        // batch, so the ring drained once per pass through it.
        for (; s + D <= s1; s += D) {
#pragma unroll
            for (int j = 0; j < D; ++j) {
                mma(j);
                __builtin_amdgcn_sched_barrier(0);
                load(j, phys(s + j + D));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // fewer than D k-steps remain, already in the ring
#pragma unroll
        for (int j = 0; j < D; ++j)
            if (s + j < s1) mma(j);
    }

    // every wavefront stores its partial sums (accumulator layout: lane l holds
    // column l%16, rows 4*(l/16)+e); after one barrier each output is the sum
    // over the four wavefronts in a fixed order
    constexpr int LD = FW + 4;  // padded row: the four row groups of a store fall on different banks
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int e = 0; e < 4; ++e) red[w][(mt * 16 + 4 * (lane >> 4) + e) * LD + nt * 16 + (lane & 15)] = acc[mt][nt][e];
    // row scales (RMSNorm applied to the output, see SkinnyArgs)
    __shared__ float rscale[MT * 16];
    if (threadIdx.x < MT * 16) {
        float sc = 1.f;
        if (rs_row) {
            float t = 0.f;  // the sums in slice order
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (q < a.rs_nb) t += rs_pre[q];
            for (int b = 4; b < a.rs_nb; ++b) t += a.rs_ssq[(size_t)b * a.R + threadIdx.x];
            sc = rsqrtf(t / (float)a.rs_d + a.rs_eps);
        }
        rscale[threadIdx.x] = sc;
    }
    __syncthreads();
    auto total4 = [&](int r, int c) {
        const int i = r * LD + c;
        const f32x4 v0 = *reinterpret_cast<const f32x4 *>(&red[0][i]), v1 = *reinterpret_cast<const f32x4 *>(&red[1][i]);
        const f32x4 v2 = *reinterpret_cast<const f32x4 *>(&red[2][i]), v3 = *reinterpret_cast<const f32x4 *>(&red[3][i]);
        return ((v0 + v1) + v2) + v3;
    };

    const int R = a.R;
    const int tiles_here = min(NT, a.ntiles - tg * NT);
    if (EPI == EPI_SWIGLU) {
        // item (r, nt): the 8 features of weight tile nt for row r (gate in
        // columns 0-7 of the tile, up in 8-15) are 16 contiguous bytes of the
        // operand-order output, hi and lo
        bf16_t *A = (bf16_t *)a.out;
        bf16_t *Al = (bf16_t *)a.out_lo;
        for (int i = threadIdx.x; i < MT * 16 * NT; i += 256) {
            const int r = i / NT, nt = i - r * NT;
            if (r >= R || nt >= tiles_here) continue;
            const float sc = rscale[r];
            const f32x4 g0 = total4(r, 16 * nt) * sc, g1 = total4(r, 16 * nt + 4) * sc;
            const f32x4 u0 = total4(r, 16 * nt + 8) * sc, u1 = total4(r, 16 * nt + 12) * sc;
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
            const size_t off = perm_offset(r, 8 * (tg * NT + nt), a.N);
            *reinterpret_cast<u32x4 *>(A + off) = u32x4{hi[0], hi[1], hi[2], hi[3]};
            *reinterpret_cast<u32x4 *>(Al + off) = u32x4{lo[0], lo[1], lo[2], lo[3]};
        }
    } else {
        float *out = (float *)a.out + (size_t)sp * R * a.N + tg * FW;
        constexpr int C4 = FW / 4;
        for (int i = threadIdx.x; i < MT * 16 * C4; i += 256) {
            const int r = i / C4, c = 4 * (i - r * C4);
            if (r >= R || c >= 16 * tiles_here) continue;
            *reinterpret_cast<f32x4 *>(out + (size_t)r * a.N + c) = total4(r, c) * rscale[r];
        }
    }
}

template <int MT, int NT>
hipError_t launch_mt_nt(int epi, const SkinnyArgs &a, hipStream_t s) {
    dim3 grid(((a.ntiles + NT - 1) / NT) * a.split);
    if (epi == EPI_SWIGLU) kvr_launch((linear_skinny_kernel<MT, NT, EPI_SWIGLU>), grid, dim3(256), 0, s, a);
    else kvr_launch((linear_skinny_kernel<MT, NT, EPI_STORE>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int NT>
hipError_t launch_nt(int epi, const SkinnyArgs &a, hipStream_t s) {
    switch ((a.R + 15) / 16) {
        case 1: return launch_mt_nt<1, NT>(epi, a, s);
        case 2: return launch_mt_nt<2, NT>(epi, a, s);
        case 3: return launch_mt_nt<3, NT>(epi, a, s);
        default: return launch_mt_nt<4, NT>(epi, a, s);
    }
}

// Blocks of more than eight tiles: at most 48 rows (the wavefronts' partial
// sums of 64 rows would not fit in LDS).
template <int NT>
hipError_t launch_nt_wide(int epi, const SkinnyArgs &a, hipStream_t s) {
    switch ((a.R + 15) / 16) {
        case 1: return launch_mt_nt<1, NT>(epi, a, s);
        case 2: return launch_mt_nt<2, NT>(epi, a, s);
        case 3: return launch_mt_nt<3, NT>(epi, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_linear_skinny(int epi, const SkinnyArgs &a, int nt, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    if (!a.x_lo || !a.w || (epi == EPI_SWIGLU && !a.out_lo)) return hipErrorInvalidValue;
    if (epi != EPI_STORE && epi != EPI_SWIGLU) return hipErrorInvalidValue;
    const int vrows = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    if (a.R > 64 || a.K % 32 != 0 || a.split < 1 || (epi == EPI_SWIGLU && a.split != 1) || vrows % 16 != 0 ||
        a.ntiles != vrows / 16)
        return hipErrorInvalidValue;
    // the epilogue stores 16 bytes at a time
    if (((uintptr_t)a.out & 15) != 0 || ((uintptr_t)a.out_lo & 15) != 0 || (epi == EPI_SWIGLU && a.N % 32 != 0))
        return hipErrorInvalidValue;
    switch (nt) {
        case 1: return launch_nt<1>(epi, a, s);
        case 2: return launch_nt<2>(epi, a, s);
        case 3: return launch_nt<3>(epi, a, s);
        case 4: return launch_nt<4>(epi, a, s);
        case 5: return launch_nt<5>(epi, a, s);
        case 6: return launch_nt<6>(epi, a, s);
        case 7: return launch_nt<7>(epi, a, s);
        case 8: return launch_nt<8>(epi, a, s);
        case 9: return launch_nt_wide<9>(epi, a, s);
        case 10: return launch_nt_wide<10>(epi, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace kvr
