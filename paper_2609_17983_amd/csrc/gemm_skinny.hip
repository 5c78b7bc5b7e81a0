// Weight-streaming linear layer for few rows (R <= 64), bf16 MFMA.
//
// With a repair budget of a few dozen rows the projections are bound by
// reading the weights once from HBM: every weight element is used by R rows
// only.  Each wavefront streams a 16*NT-row slab of W over a contiguous range
// of K directly into registers in the operand layout of
// v_mfma_f32_16x16x32_bf16 (lane l: weight row l%16, 8 consecutive k at
// 8*(l/16)), the R activation rows (X, a few hundred KB, L2-resident) are read
// alongside, and the four wavefronts of a block split the block's K range.
// Blocks of one output tile may further split K; their fp32 partial tiles are
// summed in a fixed order by the last block to finish (deterministic), which
// also applies the epilogue (store, residual add, or SwiGLU).
#include "common.h"

namespace kvr {

namespace {

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

__device__ __forceinline__ bf16x8 ld16(const bf16_t *p) {
    uint4 u = *reinterpret_cast<const uint4 *>(p);
    return __builtin_bit_cast(bf16x8, u);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 ld16_stream(const bf16_t *p) {
    u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return __builtin_bit_cast(bf16x8, u);
}

template <int MT, int NT, int EPI>
__global__ __launch_bounds__(256) void linear_skinny_kernel(LinearArgs a, int split) {
    constexpr int FW = 16 * NT;  // output columns of a block
    constexpr int U = 4;         // k-steps (of 32) per load batch
    __shared__ float red[4][MT * 16][FW];
    __shared__ int last_flag;

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int tile = blockIdx.x / split, sp = blockIdx.x - tile * split;
    const int K = a.K;

    // this wavefront's K range, in steps of 32
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
    const bf16_t *xp[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int r = min(mt * 16 + (lane & 15), a.R - 1);
        xp[mt] = (const bf16_t *)a.x + (size_t)r * a.ldx + koff;
    }

    f32x4 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4{0.f, 0.f, 0.f, 0.f};

    int s = s0;
    for (; s + U <= s1; s += U) {
        bf16x8 wv[U][NT], xv[U][MT];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) wv[u][nt] = ld16_stream(wp[nt] + (s + u) * 32);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) xv[u][mt] = ld16(xp[mt] + (s + u) * 32);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[u][mt], wv[u][nt], acc[mt][nt], 0, 0, 0);
    }
    for (; s < s1; ++s) {
        bf16x8 wv[NT], xv[MT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) wv[nt] = ld16_stream(wp[nt] + s * 32);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) xv[mt] = ld16(xp[mt] + s * 32);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xv[mt], wv[nt], acc[mt][nt], 0, 0, 0);
    }

    // accumulator layout: lane l holds column l%16, rows 4*(l/16)+e
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int e = 0; e < 4; ++e) red[w][mt * 16 + 4 * (lane >> 4) + e][nt * 16 + (lane & 15)] = acc[mt][nt][e];
    __syncthreads();

    const int R = a.R;
    const int nel = R * FW;
    float *sum = &red[0][0][0];
    for (int i = threadIdx.x; i < nel; i += 256) {
        const int r = i / FW, c = i - r * FW;
        sum[r * FW + c] = red[0][r][c] + red[1][r][c] + red[2][r][c] + red[3][r][c];
    }

    if (split > 1) {
        float *mine = a.partial + ((size_t)tile * split + sp) * nel;
        __syncthreads();
        for (int i = threadIdx.x; i < nel; i += 256) mine[i] = sum[i];
        __threadfence();
        __syncthreads();
        if (threadIdx.x == 0) last_flag = (atomicAdd(&a.counters[tile], 1) == split - 1);
        __syncthreads();
        if (!last_flag) return;
        __threadfence();
        const float *all = a.partial + (size_t)tile * split * nel;
        for (int i = threadIdx.x; i < nel; i += 256) {
            float v = 0.f;
            for (int q = 0; q < split; ++q) v += all[(size_t)q * nel + i];
            sum[i] = v;
        }
        if (threadIdx.x == 0) a.counters[tile] = 0;
    }
    __syncthreads();

    if (EPI == EPI_SWIGLU) {
        constexpr int FH = FW / 2;
        bf16_t *A = (bf16_t *)a.out;
        for (int i = threadIdx.x; i < R * FH; i += 256) {
            const int r = i / FH, f = i - r * FH;
            A[(size_t)r * a.ldo + tile * FH + f] = f32_to_bf16(silu_f(sum[r * FW + f]) * sum[r * FW + FH + f]);
        }
    } else {
        float *out = (float *)a.out;
        for (int i = threadIdx.x; i < nel; i += 256) {
            const int r = i / FW, c = i - r * FW;
            float *o = out + (size_t)r * a.ldo + tile * FW + c;
            if (EPI == EPI_RESID) *o += sum[i];
            else *o = sum[i];
        }
    }
}

template <int MT, int NT>
hipError_t launch_mt_nt(int epi, const LinearArgs &a, int split, hipStream_t s) {
    constexpr int FW = 16 * NT;
    const int tiles = epi == EPI_SWIGLU ? a.N / (FW / 2) : a.N / FW;
    dim3 grid(tiles * split);
    if (epi == EPI_STORE) hipLaunchKernelGGL((linear_skinny_kernel<MT, NT, EPI_STORE>), grid, dim3(256), 0, s, a, split);
    else if (epi == EPI_RESID) hipLaunchKernelGGL((linear_skinny_kernel<MT, NT, EPI_RESID>), grid, dim3(256), 0, s, a, split);
    else hipLaunchKernelGGL((linear_skinny_kernel<MT, NT, EPI_SWIGLU>), grid, dim3(256), 0, s, a, split);
    return hipGetLastError();
}

template <int NT>
hipError_t launch_nt(int epi, const LinearArgs &a, int split, hipStream_t s) {
    const int mt = (a.R + 15) / 16;
    switch (mt) {
        case 1: return launch_mt_nt<1, NT>(epi, a, split, s);
        case 2: return launch_mt_nt<2, NT>(epi, a, split, s);
        case 3: return launch_mt_nt<3, NT>(epi, a, split, s);
        default: return launch_mt_nt<4, NT>(epi, a, split, s);
    }
}

}  // namespace

hipError_t launch_linear_skinny(int epi, const LinearArgs &a, int split, int nt, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    if (a.R > 64 || a.K % 32 != 0 || split < 1) return hipErrorInvalidValue;
    if (nt == 2) return launch_nt<2>(epi, a, split, s);
    return launch_nt<4>(epi, a, split, s);
}

}  // namespace kvr
