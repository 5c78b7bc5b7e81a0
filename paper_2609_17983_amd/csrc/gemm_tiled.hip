// Tiled bf16 MFMA linear layer for many rows (prefill, batched repair).
//
// Y[r][n] = sum_k X[r][k] * W[n][k].  A 128x128 output tile streams 64-wide K
// slabs of X and W through LDS, and each of the four wavefronts computes a
// 64x64 sub-tile as 4x4 v_mfma_f32_16x16x32_bf16 tiles.  X is row-major (rows
// padded to 144 B in LDS so that the 16-byte operand reads of a wavefront
// spread over the banks) and a compensated pair (hi + lo), so its slab is
// staged twice and every product is two MFMAs into one fp32 accumulator.  W is
// packed in operand order (pack.hip): the slab is eight 16-row tiles x two
// k-steps of contiguous 1 KB blocks, copied to LDS as they are and read back
// one lane-contiguous block per operand.  The next slab is fetched into
// registers while the current one is multiplied.  Column tiles past the last
// weight tile (N not a multiple of 128) re-read the last tile and are not
// stored.
#include "common.h"

namespace kvr {

namespace {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int LDS_STRIDE = BK + 8;  // bf16 elements per LDS row (144 B)

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + __expf(-z)); }

template <int EPI>
__global__ __launch_bounds__(256) void linear_tiled_kernel(LinearArgs a) {
    __shared__ __attribute__((aligned(16))) bf16_t As[BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) bf16_t Al[BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) bf16_t Bs[BN * BK];  // [tile 8][k-step 2][lane 64][8]

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int wm = w >> 1, wn = w & 1;
    const int bn = blockIdx.x, bm = blockIdx.y;
    const int K = a.K;

    // global -> register loader.  X: thread covers rows tid/8 + 32*i, 16 bytes at
    // k (tid%8)*8.  W: thread covers 16-byte chunk q = tid + 256*i of the slab,
    // i.e. tile q/128, k-step (q/64)%2, lane q%64.
    const int lrow = tid >> 3, lk = (tid & 7) * 8;
    const int ksteps = K >> 5, ntiles = (a.N * (EPI == EPI_SWIGLU ? 2 : 1)) >> 4;
    const bf16_t *ag[4], *al[4];
    const bf16_t *bg[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = min(bm * BM + lrow + 32 * i, a.R - 1);
        ag[i] = (const bf16_t *)a.x + (size_t)r * a.ldx + lk;
        al[i] = (const bf16_t *)a.x_lo + (size_t)r * a.ldx + lk;
        const int q = tid + 256 * i;
        const int t = min(bn * 8 + (q >> 7), ntiles - 1);
        bg[i] = (const bf16_t *)a.wp + (((size_t)t * ksteps + ((q >> 6) & 1)) * 64 + (q & 63)) * 8;
    }

    u32x4 ra[4], rl[4], rb[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        ra[i] = *reinterpret_cast<const u32x4 *>(ag[i]);
        rl[i] = *reinterpret_cast<const u32x4 *>(al[i]);
        rb[i] = *reinterpret_cast<const u32x4 *>(bg[i]);
    }

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int koff = 8 * (lane >> 4);
    for (int k0 = 0; k0 < K; k0 += BK) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            *reinterpret_cast<u32x4 *>(&As[(lrow + 32 * i) * LDS_STRIDE + lk]) = ra[i];
            *reinterpret_cast<u32x4 *>(&Al[(lrow + 32 * i) * LDS_STRIDE + lk]) = rl[i];
            *reinterpret_cast<u32x4 *>(&Bs[(tid + 256 * i) * 8]) = rb[i];
        }
        __syncthreads();
        if (k0 + BK < K) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                ra[i] = *reinterpret_cast<const u32x4 *>(ag[i] + k0 + BK);
                rl[i] = *reinterpret_cast<const u32x4 *>(al[i] + k0 + BK);
                rb[i] = *reinterpret_cast<const u32x4 *>(bg[i] + (size_t)(k0 + BK) * 16);
            }
        }
#pragma unroll
        for (int ks = 0; ks < BK / 32; ++ks) {
            bf16x8 av[4], avl[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                av[i] = *reinterpret_cast<const bf16x8 *>(&As[(wm * 64 + i * 16 + (lane & 15)) * LDS_STRIDE + ks * 32 + koff]);
                avl[i] = *reinterpret_cast<const bf16x8 *>(&Al[(wm * 64 + i * 16 + (lane & 15)) * LDS_STRIDE + ks * 32 + koff]);
                bv[i] = *reinterpret_cast<const bf16x8 *>(&Bs[(((wn * 4 + i) * 2 + ks) * 64 + lane) * 8]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(avl[i], bv[j], acc[i][j], 0, 0, 0);
                }
        }
    }

    // accumulator layout: lane l holds tile column l%16, rows 4*(l/16)+e
    const int rbase = bm * BM + wm * 64 + 4 * (lane >> 4);
    if (EPI == EPI_SWIGLU) {
        // gate/up interleaved: column j < 8 of weight tile t is the gate of
        // feature 8t+j, column j+8 its up (lane l+8 holds it)
        bf16_t *A = (bf16_t *)a.out;
        bf16_t *Alo = (bf16_t *)a.out_lo;
        const bool gate_lane = (lane & 8) == 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int t = bn * 8 + wn * 4 + j;
            const int f = 8 * t + (lane & 7);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float g = acc[i][j][e];
                    const float u = __shfl_xor(g, 8);
                    const int r = rbase + i * 16 + e;
                    if (gate_lane && t < ntiles && r < a.R)
                        store_operand(A, Alo, (size_t)r * a.ldo + f, silu_f(g) * u);
                }
        }
        return;
    }
    float *out = (float *)a.out;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (bn * 8 + wn * 4 + j >= ntiles) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = rbase + i * 16 + e;
                if (r >= a.R) continue;
                float *o = out + (size_t)r * a.ldo + bn * BN + wn * 64 + j * 16 + (lane & 15);
                if (EPI == EPI_RESID) *o += acc[i][j][e];
                else *o = acc[i][j][e];
            }
    }
}

}  // namespace

hipError_t launch_linear_tiled(int epi, const LinearArgs &a, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    if (!a.x_lo || !a.wp || (epi == EPI_SWIGLU && !a.out_lo)) return hipErrorInvalidValue;
    const int vrows = epi == EPI_SWIGLU ? 2 * a.N : a.N;
    if (a.K % BK != 0 || a.ldx % 8 != 0 || vrows % 16 != 0) return hipErrorInvalidValue;
    dim3 grid((vrows + BN - 1) / BN, (a.R + BM - 1) / BM);
    if (epi == EPI_STORE) kvr_launch(linear_tiled_kernel<EPI_STORE>, grid, dim3(256), 0, s, a);
    else if (epi == EPI_RESID) kvr_launch(linear_tiled_kernel<EPI_RESID>, grid, dim3(256), 0, s, a);
    else kvr_launch(linear_tiled_kernel<EPI_SWIGLU>, grid, dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace kvr
