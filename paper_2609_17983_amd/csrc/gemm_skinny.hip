// Weight-streaming linear layer for few rows (R <= 64), bf16 MFMA.
//
// With a repair budget of a few dozen rows the projections are bound by
// reading the weights once from HBM: every weight element meets only R rows.
// Each wavefront streams a 16*NT-row slab of W over a contiguous range of K
// directly into registers in the B-operand layout of v_mfma_f32_16x16x32_bf16
// (lane l: weight row l%16, 8 consecutive k at 8*(l/16)); a batch of k-steps
// of loads is issued before its MFMAs.  The activations X come in "operand
// order" (see perm_offset in common.h) so that each 16-row A-operand load is one
// contiguous 1 KB read; they are compensated pairs (hi + lo), so every
// (row tile, weight tile) product is two MFMAs into one fp32 accumulator.  The
// four wavefronts of a block split the block's K range and are summed through
// LDS.
//
// Blocks never exchange data with each other: when K is split over `split`
// blocks, each writes an fp32 partial tile [split][R][N] and the row-wise
// kernel that runs next sums the partials in a fixed order (deterministic, and
// free of device-wide fences).  The gate/up projection is never split; it
// applies SwiGLU in its epilogue and writes the down projection's operand.
#include "common.h"

namespace kvr {

namespace {

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

__device__ __forceinline__ bf16x8 ld16(const bf16_t *p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
}

template <int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void linear_skinny_kernel(SkinnyArgs a) {
    constexpr int FW = 16 * NT;  // output columns of a block
    constexpr int U = NT >= 8 ? 2 : 4;  // k-steps (of 32) per load batch
    __shared__ float red[MT * 16][FW];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int split = a.split;
    const int tile = blockIdx.x / split, sp = blockIdx.x - tile * split;
    const int K = a.K;
    const int ksteps = K >> 5;
    const int gw = sp * 4 + w, nw = split * 4;
    const int s0 = (int)(((long long)ksteps * gw) / nw);
    const int s1 = (int)(((long long)ksteps * (gw + 1)) / nw);

    const int koff = 8 * (lane >> 4);
    const bf16_t *wp[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int c = nt * 16 + (lane & 15);
        const bf16_t *base;
        int row;
        if (EPI == EPI_SWIGLU) {
            base = (const bf16_t *)a.w[nt < NT / 2 ? 0 : 1];
            row = tile * (FW / 2) + (c & (FW / 2 - 1));
        } else {
            const int n = tile * FW + c;
            if (n < a.seg_end[0]) { base = (const bf16_t *)a.w[0]; row = n; }
            else if (n < a.seg_end[1]) { base = (const bf16_t *)a.w[1]; row = n - a.seg_end[0]; }
            else { base = (const bf16_t *)a.w[2]; row = n - a.seg_end[1]; }
        }
        wp[nt] = base + (size_t)row * K + koff;
    }
    // operand-order X: tile mt, k-step s at ((mt * ksteps + s) * 64 + lane) * 8
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

    int s = s0;
    for (; s + U <= s1; s += U) {
        bf16x8 wv[U][NT], xv[U][MT], xl[U][MT];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) wv[u][nt] = ld16(wp[nt] + (s + u) * 32);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                xv[u][mt] = ld16(xp[mt] + (size_t)(s + u) * 512);
                xl[u][mt] = ld16(xq[mt] + (size_t)(s + u) * 512);
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[u][mt], wv[u][nt], acc[mt][nt], 0, 0, 0);
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl[u][mt], wv[u][nt], acc[mt][nt], 0, 0, 0);
                }
    }
    for (; s < s1; ++s) {
        bf16x8 wv[NT], xv[MT], xl[MT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) wv[nt] = ld16(wp[nt] + s * 32);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            xv[mt] = ld16(xp[mt] + (size_t)s * 512);
            xl[mt] = ld16(xq[mt] + (size_t)s * 512);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[mt], wv[nt], acc[mt][nt], 0, 0, 0);
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xl[mt], wv[nt], acc[mt][nt], 0, 0, 0);
            }
    }

    // sum the four wavefronts in a fixed order; accumulator layout: lane l holds
    // column l%16, rows 4*(l/16)+e
    for (int q = 0; q < 4; ++q) {
        if (w == q) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float &d = red[mt * 16 + 4 * (lane >> 4) + e][nt * 16 + (lane & 15)];
                        d = (q == 0 ? 0.f : d) + acc[mt][nt][e];
                    }
        }
        __syncthreads();
    }

    const int R = a.R;
    if (EPI == EPI_SWIGLU) {
        constexpr int FH = FW / 2;
        bf16_t *A = (bf16_t *)a.out;
        bf16_t *Al = (bf16_t *)a.out_lo;
        for (int i = threadIdx.x; i < R * FH; i += 256) {
            const int r = i / FH, f = i - r * FH;
            store_operand(A, Al, perm_offset(r, tile * FH + f, a.N), silu_f(red[r][f]) * red[r][FH + f]);
        }
    } else {
        float *out = (float *)a.out + (size_t)sp * R * a.N;
        for (int i = threadIdx.x; i < R * FW; i += 256) {
            const int r = i / FW, c = i - r * FW;
            out[(size_t)r * a.N + tile * FW + c] = red[r][c];
        }
    }
}

template <int MT, int NT>
hipError_t launch_mt_nt(int epi, const SkinnyArgs &a, hipStream_t s) {
    constexpr int FW = 16 * NT;
    const int tiles = epi == EPI_SWIGLU ? a.N / (FW / 2) : a.N / FW;
    dim3 grid(tiles * a.split);
    if (epi == EPI_SWIGLU) hipLaunchKernelGGL((linear_skinny_kernel<MT, NT, EPI_SWIGLU>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((linear_skinny_kernel<MT, NT, EPI_STORE>), grid, dim3(256), 0, s, a);
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

}  // namespace

hipError_t launch_linear_skinny(int epi, const SkinnyArgs &a, int nt, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    const int ncols = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    if (!a.x_lo || (epi == EPI_SWIGLU && !a.out_lo)) return hipErrorInvalidValue;
    if (a.R > 64 || a.K % 32 != 0 || a.split < 1 || (epi == EPI_SWIGLU && a.split != 1) ||
        (nt != 1 && nt != 2 && nt != 4 && nt != 8) || ncols % (16 * nt) != 0 || (epi == EPI_SWIGLU && nt < 2))
        return hipErrorInvalidValue;
    if (nt == 1) return launch_nt<1>(epi, a, s);
    if (nt == 2) return launch_nt<2>(epi, a, s);
    if (nt == 4) return launch_nt<4>(epi, a, s);
    return launch_nt<8>(epi, a, s);
}

}  // namespace kvr
