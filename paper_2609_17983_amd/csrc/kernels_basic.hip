// Row-wise kernels of the decoder pass (embedding gather, RMSNorm, rotary
// embedding + cache scatter) and the straightforward attention / linear kernels
// used for fp32 models and for shapes the MFMA kernels do not cover.
#include <math.h>

#include "common.h"

namespace kvr {

namespace {

__device__ __forceinline__ float warp_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// Sum over a 256-thread block.
__device__ __forceinline__ float block_sum256(float v, float *red) {
    v = warp_sum(v);
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    if (l == 0) red[w] = v;
    __syncthreads();
    float t = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    return t;
}

// Token ids outside [0, vocab) are clamped into range rather than read out of
// bounds.  Rows are copied in 16-byte chunks when d allows it (the table and H
// are 16-byte aligned).
template <typename TW>
__global__ __launch_bounds__(256) void embed_kernel(const RowInfo *rows, const DocInfo *docs, const TW *embed,
                                                    int d, int vocab, float *H) {
    constexpr int V = 16 / sizeof(TW);  // table elements per chunk
    const int r = blockIdx.x;
    const RowInfo ri = rows[r];
    const int tok = min(max(docs[ri.doc].tokens[ri.pos], 0), vocab - 1);
    const TW *src = embed + (size_t)tok * d;
    float *dst = H + (size_t)r * d;
    if (d % V != 0) {
        for (int i = threadIdx.x; i < d; i += 256) dst[i] = to_f32(src[i]);
        return;
    }
    for (int i = threadIdx.x; i < d / V; i += 256) {
        const u32x4 u = *reinterpret_cast<const u32x4 *>(src + (size_t)i * V);
        if constexpr (sizeof(TW) == 2) {
            float4 *o = reinterpret_cast<float4 *>(dst + (size_t)i * V);
            o[0] = make_float4(__uint_as_float(u[0] << 16), __uint_as_float(u[0] & 0xffff0000u),
                               __uint_as_float(u[1] << 16), __uint_as_float(u[1] & 0xffff0000u));
            o[1] = make_float4(__uint_as_float(u[2] << 16), __uint_as_float(u[2] & 0xffff0000u),
                               __uint_as_float(u[3] << 16), __uint_as_float(u[3] & 0xffff0000u));
        } else {
            *reinterpret_cast<u32x4 *>(dst + (size_t)i * V) = u;
        }
    }
}

// Sum over a 1024-thread block.
__device__ __forceinline__ float block_sum1024(float v, float *red) {
    v = warp_sum(v);
    const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
    if (l == 0) red[w] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < 16; ++q) t += red[q];
    __syncthreads();
    return t;
}

// h4 = H[r][4i..4i+3] + the split-K partial tiles part[q][r][4i..] in order
// (batches of eight independent loads).
__device__ __forceinline__ float4 add_partials(float4 h, const float *part, int nsplit, int R, int r, int d, int i) {
    constexpr int B = 8;
    int q = 0;
    for (; q + B <= nsplit; q += B) {
        float4 p[B];
#pragma unroll
        for (int u = 0; u < B; ++u) p[u] = *reinterpret_cast<const float4 *>(part + ((size_t)(q + u) * R + r) * d + 4 * i);
#pragma unroll
        for (int u = 0; u < B; ++u) { h.x += p[u].x; h.y += p[u].y; h.z += p[u].z; h.w += p[u].w; }
    }
    if (q < nsplit) {
        float4 p[B];
#pragma unroll
        for (int u = 0; u < B; ++u)
            if (q + u < nsplit) p[u] = *reinterpret_cast<const float4 *>(part + ((size_t)(q + u) * R + r) * d + 4 * i);
#pragma unroll
        for (int u = 0; u < B; ++u)
            if (q + u < nsplit) { h.x += p[u].x; h.y += p[u].y; h.z += p[u].z; h.w += p[u].w; }
    }
    return h;
}

constexpr int NORM_V = 4;  // float4 per thread of the row kernels: d <= 16384

// Four consecutive outputs (columns c..c+3, c % 4 == 0) of an operand row;
// they are contiguous in both the row-major and the operand-order layout.
template <typename T>
__device__ __forceinline__ void store_operand4(T *hi, T *lo, size_t off, const float (&x)[4]) {
    if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<float4 *>(hi + off) = make_float4(x[0], x[1], x[2], x[3]);
    } else {
        uint32_t h[2], l[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const bf16_t h0 = f32_to_bf16(x[2 * q]), h1 = f32_to_bf16(x[2 * q + 1]);
            h[q] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            const bf16_t l0 = f32_to_bf16(x[2 * q] - bf16_to_f32(h0)), l1 = f32_to_bf16(x[2 * q + 1] - bf16_to_f32(h1));
            l[q] = (uint32_t)l0 | ((uint32_t)l1 << 16);
        }
        *reinterpret_cast<uint2 *>(hi + off) = make_uint2(h[0], h[1]);
        if (lo) *reinterpret_cast<uint2 *>(lo + off) = make_uint2(l[0], l[1]);
    }
}

// H[r] += sum of the split-K partial tiles (fixed order), then
// X = H * rsqrt(mean(H^2) + eps) * gain in the operand type (row-major or
// operand order).  One 1024-thread block per row; the row stays in registers
// between the two passes (four columns per thread per pass, d % 4 == 0).
template <typename TO, typename TG, bool PERM>
__global__ __launch_bounds__(1024) void rmsnorm_kernel(float *H, const float *part, int nsplit, int R,
                                                       const TG *gain, int d, float eps, TO *X, TO *X_lo, int ldx) {
    __shared__ float red[16];
    const int r = blockIdx.x;
    float *h = H + (size_t)r * d;
    float4 v[NORM_V];
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NORM_V; ++k) {
        const int i = threadIdx.x + 1024 * k;
        if (4 * i >= d) break;
        v[k] = *reinterpret_cast<const float4 *>(h + 4 * i);
        if (nsplit) {
            v[k] = add_partials(v[k], part, nsplit, R, r, d, i);
            *reinterpret_cast<float4 *>(h + 4 * i) = v[k];
        }
        ss += v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
    }
    ss = block_sum1024(ss, red);
    const float inv = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int k = 0; k < NORM_V; ++k) {
        const int i = threadIdx.x + 1024 * k;
        if (4 * i >= d) break;
        const int c = 4 * i;
        const float x[4] = {v[k].x * inv * to_f32(gain[c]), v[k].y * inv * to_f32(gain[c + 1]),
                            v[k].z * inv * to_f32(gain[c + 2]), v[k].w * inv * to_f32(gain[c + 3])};
        store_operand4(X, X_lo, PERM ? perm_offset(r, c, d) : (size_t)r * ldx + c, x);
    }
}

// The same for many rows with at most two partial tiles (prefill, batched
// repair): one wavefront per row, each lane holding NV float4 of it, so that
// the row and its partial tiles are loaded in one round (NV + NV loads in
// flight per lane) and no block barrier is needed.  A 1024-thread block per
// row keeps one load per thread in flight and waits at two barriers; at
// 5000 rows that kernel ran at 3.4 TB/s.  Results are bit-identical to it
// (d <= 4096, where it holds one float4 per thread).
template <typename TO, typename TG, bool PERM, int NV>
__global__ __launch_bounds__(512) void rmsnorm_wave_kernel(float *H, const float *part, int nsplit, int R,
                                                           const TG *gain, int d, float eps, TO *X, TO *X_lo,
                                                           int ldx) {
    const int lane = threadIdx.x & 63;
    const int r = blockIdx.x * 8 + (threadIdx.x >> 6);
    if (r >= R) return;
    float *h = H + (size_t)r * d;
    float4 v[NV], p[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int c = 4 * (lane + 64 * k);
        v[k] = c < d ? *reinterpret_cast<const float4 *>(h + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        if (nsplit > 0)
            p[k] = c < d ? *reinterpret_cast<const float4 *>(part + (size_t)r * d + c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int q = 0; q < nsplit; ++q) {  // partial tiles in order
        if (q > 0) {
#pragma unroll
            for (int k = 0; k < NV; ++k) {
                const int c = 4 * (lane + 64 * k);
                p[k] = c < d ? *reinterpret_cast<const float4 *>(part + ((size_t)q * R + r) * d + c)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
#pragma unroll
        for (int k = 0; k < NV; ++k) { v[k].x += p[k].x; v[k].y += p[k].y; v[k].z += p[k].z; v[k].w += p[k].w; }
    }
    // the sum of squares in the row kernel's order (float4 k of lane l is the
    // row kernel's thread 64 k + l): a wavefront sum per k, then the sums in
    // k order, so that both kernels normalise a row bit for bit alike (a row
    // must not depend on how many rows the pass has)
    float ss = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int c = 4 * (lane + 64 * k);
        float t = 0.f;
        if (c < d) {
            if (nsplit) *reinterpret_cast<float4 *>(h + c) = v[k];
            t = v[k].x * v[k].x + v[k].y * v[k].y + v[k].z * v[k].z + v[k].w * v[k].w;
        }
        ss += warp_sum(t);
    }
    const float inv = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int k = 0; k < NV; ++k) {
        const int c = 4 * (lane + 64 * k);
        if (c >= d) continue;
        const float x[4] = {v[k].x * inv * to_f32(gain[c]), v[k].y * inv * to_f32(gain[c + 1]),
                            v[k].z * inv * to_f32(gain[c + 2]), v[k].w * inv * to_f32(gain[c + 3])};
        store_operand4(X, X_lo, PERM ? perm_offset(r, c, d) : (size_t)r * ldx + c, x);
    }
}

template <typename TG>
__global__ __launch_bounds__(1024) void final_norm_kernel(float *H, const float *part, int nsplit, int R,
                                                          const TG *gain, const RowInfo *rows, const DocInfo *docs,
                                                          int d, float eps) {
    __shared__ float red[16];
    const int r = blockIdx.x;
    const RowInfo ri = rows[r];
    float *dst = docs[ri.doc].hidden_out;
    float *h = H + (size_t)r * d;
    float ss = 0.f;
    for (int i = threadIdx.x; 4 * i < d; i += 1024) {
        float4 v = *reinterpret_cast<const float4 *>(h + 4 * i);
        if (nsplit) {
            v = add_partials(v, part, nsplit, R, r, d, i);
            *reinterpret_cast<float4 *>(h + 4 * i) = v;
        }
        ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
    }
    ss = block_sum1024(ss, red);
    if (!dst) return;
    dst += (size_t)ri.out * d;
    const float inv = rsqrtf(ss / (float)d + eps);
    for (int i = threadIdx.x; 4 * i < d; i += 1024) {
        const float4 v = *reinterpret_cast<const float4 *>(h + 4 * i);
        float4 o;
        o.x = v.x * inv * to_f32(gain[4 * i]);
        o.y = v.y * inv * to_f32(gain[4 * i + 1]);
        o.z = v.z * inv * to_f32(gain[4 * i + 2]);
        o.w = v.w * inv * to_f32(gain[4 * i + 3]);
        *reinterpret_cast<float4 *>(dst + 4 * i) = o;
    }
}

// Adds the Q/K/V bias, rotates Q and K at the row's absolute position
// (rotate-half pairing) and scatters K and V into the row's cache slot; Q goes
// to the attention operand buffer [R][Hq*hd].
template <typename T>
__global__ __launch_bounds__(1024) void rope_scatter_kernel(const float *qkv, int nsplit, int R, const T *bq,
                                                           const T *bk, const T *bv, const RowInfo *rows,
                                                           const DocInfo *docs, int layer, int Hq, int Hkv, int hd,
                                                           const float *rcos, const float *rsin, T *Q, T *Q_lo) {
    const int r = blockIdx.x;
    const RowInfo ri = rows[r];
    const DocInfo dc = docs[ri.doc];
    const int half = hd >> 1;
    const int qd = Hq * hd, kd = Hkv * hd;
    const int N = qd + 2 * kd;
    // sum the split-K partial tiles of this row into LDS first
    extern __shared__ float row[];
    for (int i = threadIdx.x; 4 * i < N; i += 1024) {
        float4 v = *reinterpret_cast<const float4 *>(qkv + (size_t)r * N + 4 * i);
        if (nsplit > 1) v = add_partials(v, qkv + (size_t)R * N, nsplit - 1, R, r, N, i);
        *reinterpret_cast<float4 *>(row + 4 * i) = v;
    }
    __syncthreads();
    const float *cs = rcos + (size_t)ri.pos * half;
    const float *sn = rsin + (size_t)ri.pos * half;
    T *cache = (T *)dc.cache;
    const size_t head_stride = (size_t)dc.n_cap * hd;
    T *kbase = cache + ((size_t)layer * 2 + 0) * Hkv * head_stride + (size_t)ri.pos * hd;
    T *vbase = cache + ((size_t)layer * 2 + 1) * Hkv * head_stride + (size_t)ri.pos * hd;
    for (int idx = threadIdx.x; idx < (Hq + Hkv) * half; idx += 1024) {
        const int j = idx / half, i = idx - j * half;
        float a, b;
        if (j < Hq) {
            a = row[j * hd + i];
            b = row[j * hd + i + half];
            if (bq) { a += to_f32(bq[j * hd + i]); b += to_f32(bq[j * hd + i + half]); }
        } else {
            const int g = j - Hq;
            a = row[qd + g * hd + i];
            b = row[qd + g * hd + i + half];
            if (bk) { a += to_f32(bk[g * hd + i]); b += to_f32(bk[g * hd + i + half]); }
        }
        const float c = cs[i], s = sn[i];
        const float o1 = a * c - b * s, o2 = b * c + a * s;
        if (j < Hq) {
            store_operand(Q, Q_lo, (size_t)r * qd + j * hd + i, o1);
            store_operand(Q, Q_lo, (size_t)r * qd + j * hd + i + half, o2);
        } else {
            const int g = j - Hq;
            kbase[g * head_stride + i] = from_f32<T>(o1);
            kbase[g * head_stride + i + half] = from_f32<T>(o2);
        }
    }
    for (int idx = threadIdx.x; idx < kd; idx += 1024) {
        const int g = idx / hd, i = idx - g * hd;
        float v = row[qd + kd + idx];
        if (bv) v += to_f32(bv[idx]);
        vbase[g * head_stride + i] = from_f32<T>(v);
    }
}

// Residual update for a pass whose projections apply the RMS scale to their
// outputs (the skinny path): H[r] += the `nsplit` partial tiles (in order),
// X = H * gain as a compensated operand in operand order, and ssq[b][r] = the
// sum of H[r][c]^2 over the 1024 columns of column block b (fixed reduction
// order).  RMSNorm's scale is one factor per row and the projection is
// linear, so the projection that reads X multiplies its output row r by
// rsqrt((ssq[0][r] + ... ) / d + eps) instead; the work then spreads over
// (row, column block) blocks rather than one block per row.
template <typename G>
__global__ __launch_bounds__(256) void resid_gain_kernel(float *H, const float *part, int nsplit, int R, const G *gain,
                                                         int d, bf16_t *X, bf16_t *X_lo, float *ssq) {
    __shared__ float red[4];
    const int r = blockIdx.x, b = blockIdx.y;
    const int i = b * 256 + threadIdx.x;  // float4 index within the row
    float ss = 0.f;
    if (4 * i < d) {
        float *hp = H + (size_t)r * d + 4 * i;
        float4 h = *reinterpret_cast<const float4 *>(hp);
        if (nsplit) {
            h = add_partials(h, part, nsplit, R, r, d, i);
            *reinterpret_cast<float4 *>(hp) = h;
        }
        ss = h.x * h.x + h.y * h.y + h.z * h.z + h.w * h.w;
        const float4 x = {h.x * to_f32(gain[4 * i]), h.y * to_f32(gain[4 * i + 1]), h.z * to_f32(gain[4 * i + 2]),
                          h.w * to_f32(gain[4 * i + 3])};
        const bf16_t hi[4] = {f32_to_bf16(x.x), f32_to_bf16(x.y), f32_to_bf16(x.z), f32_to_bf16(x.w)};
        const bf16_t lo[4] = {f32_to_bf16(x.x - bf16_to_f32(hi[0])), f32_to_bf16(x.y - bf16_to_f32(hi[1])),
                              f32_to_bf16(x.z - bf16_to_f32(hi[2])), f32_to_bf16(x.w - bf16_to_f32(hi[3]))};
        const size_t o = perm_offset(r, 4 * i, d);  // four consecutive columns are adjacent in operand order
        *reinterpret_cast<uint2 *>(X + o) =
            make_uint2((uint32_t)hi[0] | ((uint32_t)hi[1] << 16), (uint32_t)hi[2] | ((uint32_t)hi[3] << 16));
        *reinterpret_cast<uint2 *>(X_lo + o) =
            make_uint2((uint32_t)lo[0] | ((uint32_t)lo[1] << 16), (uint32_t)lo[2] | ((uint32_t)lo[3] << 16));
    }
    ss = warp_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    if (threadIdx.x == 0) ssq[(size_t)b * R + r] = ((red[0] + red[1]) + red[2]) + red[3];
}

// Four values of row-major type T at p (8-byte or 16-byte store).
template <typename T>
__device__ __forceinline__ void store4(T *p, float4 v) {
    if constexpr (sizeof(T) == 4) {
        *reinterpret_cast<float4 *>(p) = v;
    } else {
        const uint32_t a = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
        const uint32_t b = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
        *reinterpret_cast<uint2 *>(p) = make_uint2(a, b);
    }
}
// Four consecutive operand values (store_operand for each, vectorised).
template <typename T>
__device__ __forceinline__ void store4_operand(T *hi, T *lo, size_t i, float4 v) {
    if constexpr (sizeof(T) == 4) {
        store4(hi + i, v);
    } else {
        const bf16_t h[4] = {f32_to_bf16(v.x), f32_to_bf16(v.y), f32_to_bf16(v.z), f32_to_bf16(v.w)};
        *reinterpret_cast<uint2 *>(hi + i) =
            make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
        if (lo) {
            const float4 d = {v.x - bf16_to_f32(h[0]), v.y - bf16_to_f32(h[1]), v.z - bf16_to_f32(h[2]),
                              v.w - bf16_to_f32(h[3])};
            store4(lo + i, d);
        }
    }
}
template <typename T>
__device__ __forceinline__ float4 load4_f32(const T *p) {
    if constexpr (sizeof(T) == 4) return *reinterpret_cast<const float4 *>(p);
    else return float4{to_f32(p[0]), to_f32(p[1]), to_f32(p[2]), to_f32(p[3])};
}

// The same as rope_scatter_kernel with one thread per (row, head, four
// rotary pairs) and per (row, four value dimensions): nothing in it is
// reduced over a row, so the work spreads over all compute units instead of
// one block per row (head_dim a multiple of 8).
template <typename T>
__global__ __launch_bounds__(256) void rope_scatter_vec_kernel(const float *qkv, int nsplit, int R, const T *bq,
                                                               const T *bk, const T *bv, const RowInfo *rows,
                                                               const DocInfo *docs, int layer, int Hq, int Hkv, int hd,
                                                               const float *rcos, const float *rsin, T *Q, T *Q_lo) {
    const int r = blockIdx.x;
    const int idx = blockIdx.y * 256 + threadIdx.x;
    const int half = hd >> 1, hq4 = half >> 2;
    const int qd = Hq * hd, kd = Hkv * hd;
    const int N = qd + 2 * kd;
    const int nrot = (Hq + Hkv) * hq4;
    if (idx >= nrot + (kd >> 2)) return;
    const RowInfo ri = rows[r];
    const DocInfo dc = docs[ri.doc];
    // columns c..c+3 of this row, the split-K partial tiles summed in order
    auto load4 = [&](int c) {
        float4 v = *reinterpret_cast<const float4 *>(qkv + (size_t)r * N + c);
        for (int q = 1; q < nsplit; ++q) {
            const float4 p = *reinterpret_cast<const float4 *>(qkv + ((size_t)q * R + r) * N + c);
            v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
        }
        return v;
    };
    T *cache = (T *)dc.cache;
    const size_t head_stride = (size_t)dc.n_cap * hd;
    if (idx < nrot) {
        const int j = idx / hq4, i = (idx - j * hq4) * 4;
        const bool isq = j < Hq;
        const int g = j - Hq;
        const int ca = isq ? j * hd + i : qd + g * hd + i;
        float4 a = load4(ca), b = load4(ca + half);
        const T *bias = isq ? bq : bk;
        if (bias) {
            const int bo = (isq ? j : g) * hd + i;
            const float4 ba = load4_f32(bias + bo), bb = load4_f32(bias + bo + half);
            a.x += ba.x; a.y += ba.y; a.z += ba.z; a.w += ba.w;
            b.x += bb.x; b.y += bb.y; b.z += bb.z; b.w += bb.w;
        }
        const float4 c = *reinterpret_cast<const float4 *>(rcos + (size_t)ri.pos * half + i);
        const float4 sn = *reinterpret_cast<const float4 *>(rsin + (size_t)ri.pos * half + i);
        const float4 o1 = {a.x * c.x - b.x * sn.x, a.y * c.y - b.y * sn.y, a.z * c.z - b.z * sn.z, a.w * c.w - b.w * sn.w};
        const float4 o2 = {b.x * c.x + a.x * sn.x, b.y * c.y + a.y * sn.y, b.z * c.z + a.z * sn.z, b.w * c.w + a.w * sn.w};
        if (isq) {
            store4_operand(Q, Q_lo, (size_t)r * qd + j * hd + i, o1);
            store4_operand(Q, Q_lo, (size_t)r * qd + j * hd + i + half, o2);
        } else {
            T *kb = cache + (((size_t)layer * 2 + 0) * Hkv + g) * head_stride + (size_t)ri.pos * hd;
            store4(kb + i, o1);
            store4(kb + i + half, o2);
        }
    } else {
        const int c4 = (idx - nrot) * 4;  // column of the value part [0, kd)
        float4 v = load4(qd + kd + c4);
        if (bv) {
            const float4 bb = load4_f32(bv + c4);
            v.x += bb.x; v.y += bb.y; v.z += bb.z; v.w += bb.w;
        }
        const int g = c4 / hd, i = c4 - g * hd;
        T *vb = cache + (((size_t)layer * 2 + 1) * Hkv + g) * head_stride + (size_t)ri.pos * hd;
        store4(vb + i, v);
    }
}

// One wavefront per (row, query head): online softmax over keys 0..pos.
// When `lse` is given, lse[r * Hq + j] = log2 of the softmax normaliser of the
// scores q.k * log2(e)/sqrt(hd) (the base-2 log-sum-exp).
template <typename T>
__global__ __launch_bounds__(64) void attention_simple_kernel(const T *Q, const T *Q_lo, const RowInfo *rows,
                                                              const DocInfo *docs, int layer, int Hq, int Hkv, int hd,
                                                              T *O, T *O_lo, int o_perm, float *lse) {
    const int r = blockIdx.x, j = blockIdx.y, lane = threadIdx.x;
    const RowInfo ri = rows[r];
    const DocInfo dc = docs[ri.doc];
    const int g = j / (Hq / Hkv);
    const size_t head_stride = (size_t)dc.n_cap * hd;
    const T *K = (const T *)dc.cache + (((size_t)layer * 2 + 0) * Hkv + g) * head_stride;
    const T *V = (const T *)dc.cache + (((size_t)layer * 2 + 1) * Hkv + g) * head_stride;
    const int qd = Hq * hd;
    const bool has0 = lane < hd, has1 = lane + 64 < hd;
    const float scale = 1.0f / sqrtf((float)hd);
    const float q0 = has0 ? load_operand(Q, Q_lo, (size_t)r * qd + j * hd + lane) * scale : 0.f;
    const float q1 = has1 ? load_operand(Q, Q_lo, (size_t)r * qd + j * hd + lane + 64) * scale : 0.f;
    float m = -INFINITY, l = 0.f, a0 = 0.f, a1 = 0.f;
    for (int t = 0; t <= ri.pos; ++t) {
        const T *kr = K + (size_t)t * hd;
        float p = (has0 ? q0 * to_f32(kr[lane]) : 0.f) + (has1 ? q1 * to_f32(kr[lane + 64]) : 0.f);
        p = warp_sum(p);
        const float mn = fmaxf(m, p);
        const float corr = expf(m - mn);
        const float e = expf(p - mn);
        const T *vr = V + (size_t)t * hd;
        l = l * corr + e;
        a0 = a0 * corr + (has0 ? e * to_f32(vr[lane]) : 0.f);
        a1 = a1 * corr + (has1 ? e * to_f32(vr[lane + 64]) : 0.f);
        m = mn;
    }
    const float inv = 1.0f / l;
    if (has0) store_operand(O, O_lo, o_perm ? perm_offset(r, j * hd + lane, qd) : (size_t)r * qd + j * hd + lane, a0 * inv);
    if (has1)
        store_operand(O, O_lo, o_perm ? perm_offset(r, j * hd + lane + 64, qd) : (size_t)r * qd + j * hd + lane + 64,
                      a1 * inv);
    if (lse && lane == 0) lse[(size_t)r * Hq + j] = (m + logf(l)) * 1.4426950408889634f;
}

__device__ __forceinline__ float silu_f(float z) { return z / (1.0f + expf(-z)); }

// Generic tiled linear layer: 64x64 output tile, 16-wide K steps, 4x4 outputs
// per thread.  Every index is bounds-checked, so any R, N, K works.
template <typename T, int EPI>
__global__ __launch_bounds__(256) void linear_simple_kernel(LinearArgs a) {
    __shared__ float xs[16][65];
    __shared__ float ws[16][65];
    __shared__ float tile[64][65];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int r0 = blockIdx.y * 64;
    const int c0 = blockIdx.x * 64;
    const T *X = (const T *)a.x;
    const T *Xl = (const T *)a.x_lo;
    // weight row pointer of the tile's column c (0..63); null if out of range
    auto wrow = [&](int c) -> const T * {
        if (EPI == EPI_SWIGLU) {
            const int f = blockIdx.x * 32 + (c & 31);
            if (f >= a.N) return nullptr;
            return (const T *)a.w[c >> 5] + (size_t)f * a.K;
        }
        const int n = c0 + c;
        if (n >= a.N) return nullptr;
        if (n < a.seg_end[0]) return (const T *)a.w[0] + (size_t)n * a.K;
        if (n < a.seg_end[1]) return (const T *)a.w[1] + (size_t)(n - a.seg_end[0]) * a.K;
        return (const T *)a.w[2] + (size_t)(n - a.seg_end[1]) * a.K;
    };
    float acc[4][4] = {};
    const int lr = threadIdx.x >> 2;        // 0..63: tile row / column loaded
    const int lk = (threadIdx.x & 3) * 4;   // 0,4,8,12
    const T *wr = wrow(lr);
    const int xr = r0 + lr;
    for (int k0 = 0; k0 < a.K; k0 += 16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int k = k0 + lk + e;
            xs[lk + e][lr] = (xr < a.R && k < a.K) ? load_operand(X, Xl, (size_t)xr * a.ldx + k) : 0.f;
            ws[lk + e][lr] = (wr && k < a.K) ? to_f32(wr[k]) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float xv[4], wv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) { xv[i] = xs[kk][ty * 4 + i]; wv[i] = ws[kk][tx * 4 + i]; }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) acc[i][jj] += xv[i] * wv[jj];
        }
        __syncthreads();
    }
    if (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) tile[ty * 4 + i][tx * 4 + jj] = acc[i][jj];
        __syncthreads();
        T *A = (T *)a.out;
        T *Al = (T *)a.out_lo;
        for (int idx = threadIdx.x; idx < 64 * 32; idx += 256) {
            const int rr = idx >> 5, f = idx & 31;
            const int row = r0 + rr, feat = blockIdx.x * 32 + f;
            if (row < a.R && feat < a.N)
                store_operand(A, Al, (size_t)row * a.ldo + feat, silu_f(tile[rr][f]) * tile[rr][32 + f]);
        }
        return;
    }
    float *out = (float *)a.out;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = r0 + ty * 4 + i;
        if (row >= a.R) continue;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int n = c0 + tx * 4 + jj;
            if (n >= a.N) continue;
            if (EPI == EPI_RESID) out[(size_t)row * a.ldo + n] += acc[i][jj];
            else out[(size_t)row * a.ldo + n] = acc[i][jj];
        }
    }
}

}  // namespace

hipError_t launch_embed(bool bf16, const RowInfo *rows, const DocInfo *docs, int R, const void *embed, int d,
                        int vocab, float *H, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (bf16)
        kvr_launch(embed_kernel<bf16_t>, dim3(R), dim3(256), 0, s, rows, docs, (const bf16_t *)embed, d, vocab,
                           H);
    else
        kvr_launch(embed_kernel<float>, dim3(R), dim3(256), 0, s, rows, docs, (const float *)embed, d, vocab,
                           H);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(bool bf16_out, bool bf16_gain, float *H, const float *part, int nsplit, const void *gain,
                          int R, int d, float eps, void *X, void *X_lo, int ldx, bool perm, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (d % 4 != 0 || d > 4 * 1024 * NORM_V || (!perm && ldx % 4 != 0)) return hipErrorInvalidValue;
    // many rows and at most two partial tiles: a wavefront per row (d <= 4096)
    if (bf16_out && bf16_gain && perm && R >= 512 && nsplit <= 2 && d <= 4096) {
        kvr_launch((rmsnorm_wave_kernel<bf16_t, bf16_t, true, 16>), dim3((R + 7) / 8), dim3(512), 0, s, H, part, nsplit,
                   R, (const bf16_t *)gain, d, eps, (bf16_t *)X, (bf16_t *)X_lo, ldx);
        return hipGetLastError();
    }
    if (bf16_out && bf16_gain) {
        if (perm)
            kvr_launch((rmsnorm_kernel<bf16_t, bf16_t, true>), dim3(R), dim3(1024), 0, s, H, part, nsplit, R,
                               (const bf16_t *)gain, d, eps, (bf16_t *)X, (bf16_t *)X_lo, ldx);
        else
            kvr_launch((rmsnorm_kernel<bf16_t, bf16_t, false>), dim3(R), dim3(1024), 0, s, H, part, nsplit, R,
                               (const bf16_t *)gain, d, eps, (bf16_t *)X, (bf16_t *)X_lo, ldx);
    } else if (!bf16_out && !bf16_gain && !perm) {
        kvr_launch((rmsnorm_kernel<float, float, false>), dim3(R), dim3(1024), 0, s, H, part, nsplit, R,
                           (const float *)gain, d, eps, (float *)X, (float *)nullptr, ldx);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int resid_gain_blocks(int d) { return (d + 1023) / 1024; }

hipError_t launch_resid_gain(bool bf16_gain, float *H, const float *part, int nsplit, const void *gain, int R, int d,
                             void *X, void *X_lo, float *ssq, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (d % 32 != 0 || !X || !X_lo || !ssq) return hipErrorInvalidValue;
    const dim3 grid(R, resid_gain_blocks(d));
    if (bf16_gain)
        kvr_launch(resid_gain_kernel<bf16_t>, grid, dim3(256), 0, s, H, part, nsplit, R, (const bf16_t *)gain, d,
                   (bf16_t *)X, (bf16_t *)X_lo, ssq);
    else
        kvr_launch(resid_gain_kernel<float>, grid, dim3(256), 0, s, H, part, nsplit, R, (const float *)gain, d,
                   (bf16_t *)X, (bf16_t *)X_lo, ssq);
    return hipGetLastError();
}

hipError_t launch_final_norm(bool bf16_gain, float *H, const float *part, int nsplit, const void *gain,
                             const RowInfo *rows, const DocInfo *docs, int R, int d, float eps, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (d % 4 != 0) return hipErrorInvalidValue;
    if (bf16_gain)
        kvr_launch(final_norm_kernel<bf16_t>, dim3(R), dim3(1024), 0, s, H, part, nsplit, R,
                           (const bf16_t *)gain, rows, docs, d, eps);
    else
        kvr_launch(final_norm_kernel<float>, dim3(R), dim3(1024), 0, s, H, part, nsplit, R,
                           (const float *)gain, rows, docs, d, eps);
    return hipGetLastError();
}

hipError_t launch_rope_scatter(bool bf16, const float *qkv, int nsplit, const void *bq, const void *bk,
                               const void *bv, const RowInfo *rows, const DocInfo *docs, int R, int layer, int Hq,
                               int Hkv, int hd, const float *rope_cos, const float *rope_sin, void *Q, void *Q_lo,
                               hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (hd % 8 == 0) {
        const int work = (Hq + Hkv) * (hd / 8) + Hkv * hd / 4;  // threads per row
        const dim3 grid(R, (work + 255) / 256);
        if (bf16)
            kvr_launch(rope_scatter_vec_kernel<bf16_t>, grid, dim3(256), 0, s, qkv, nsplit, R, (const bf16_t *)bq,
                       (const bf16_t *)bk, (const bf16_t *)bv, rows, docs, layer, Hq, Hkv, hd, rope_cos, rope_sin,
                       (bf16_t *)Q, (bf16_t *)Q_lo);
        else
            kvr_launch(rope_scatter_vec_kernel<float>, grid, dim3(256), 0, s, qkv, nsplit, R, (const float *)bq,
                       (const float *)bk, (const float *)bv, rows, docs, layer, Hq, Hkv, hd, rope_cos, rope_sin,
                       (float *)Q, (float *)nullptr);
        return hipGetLastError();
    }
    const size_t lds = (size_t)(Hq + 2 * Hkv) * hd * sizeof(float);
    if (lds > 160 * 1024 || ((Hq + 2 * Hkv) * hd) % 4 != 0) return hipErrorInvalidValue;
    if (bf16)
        kvr_launch(rope_scatter_kernel<bf16_t>, dim3(R), dim3(1024), lds, s, qkv, nsplit, R,
                           (const bf16_t *)bq, (const bf16_t *)bk, (const bf16_t *)bv, rows, docs, layer, Hq, Hkv, hd,
                           rope_cos, rope_sin, (bf16_t *)Q, (bf16_t *)Q_lo);
    else
        kvr_launch(rope_scatter_kernel<float>, dim3(R), dim3(1024), lds, s, qkv, nsplit, R,
                           (const float *)bq, (const float *)bk, (const float *)bv, rows, docs, layer, Hq, Hkv, hd,
                           rope_cos, rope_sin, (float *)Q, (float *)nullptr);
    return hipGetLastError();
}

hipError_t launch_attention_simple(bool bf16, const void *Q, const void *Q_lo, const RowInfo *rows,
                                   const DocInfo *docs, int R, int layer, int Hq, int Hkv, int hd, void *O, void *O_lo,
                                   bool o_perm, float *lse, hipStream_t s) {
    if (R <= 0) return hipSuccess;
    if (bf16)
        kvr_launch(attention_simple_kernel<bf16_t>, dim3(R, Hq), dim3(64), 0, s, (const bf16_t *)Q,
                           (const bf16_t *)Q_lo, rows, docs, layer, Hq, Hkv, hd, (bf16_t *)O, (bf16_t *)O_lo, (int)o_perm, lse);
    else if (!o_perm)
        kvr_launch(attention_simple_kernel<float>, dim3(R, Hq), dim3(64), 0, s, (const float *)Q,
                           (const float *)nullptr, rows, docs, layer, Hq, Hkv, hd, (float *)O, (float *)nullptr, 0, lse);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_linear_simple(bool bf16, int epi, const LinearArgs &a, hipStream_t s) {
    if (a.R <= 0) return hipSuccess;
    const int cols_per_block = epi == EPI_SWIGLU ? 32 : 64;
    dim3 grid((a.N + cols_per_block - 1) / cols_per_block, (a.R + 63) / 64);
#define KVR_LS(T, E) kvr_launch((linear_simple_kernel<T, E>), grid, dim3(256), 0, s, a)
    if (bf16) {
        if (epi == EPI_STORE) KVR_LS(bf16_t, EPI_STORE);
        else if (epi == EPI_RESID) KVR_LS(bf16_t, EPI_RESID);
        else KVR_LS(bf16_t, EPI_SWIGLU);
    } else {
        if (epi == EPI_STORE) KVR_LS(float, EPI_STORE);
        else if (epi == EPI_RESID) KVR_LS(float, EPI_RESID);
        else KVR_LS(float, EPI_SWIGLU);
    }
#undef KVR_LS
    return hipGetLastError();
}

}  // namespace kvr
