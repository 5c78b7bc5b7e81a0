// One-time repacking of a projection's weight matrices into MFMA operand order.
//
// The projections read every weight exactly once per pass, so the weight
// stream sets their speed.  In the caller's row-major [out][in] layout a
// wavefront's B-operand load (16 rows x 64 bytes) touches sixteen half cache
// lines in sixteen different DRAM rows.  Stored in operand order instead
// (perm_offset with the output feature as the row), the 16-row x 32-k tile a
// wavefront consumes per k-step is one contiguous 1 KB block and consecutive
// k-steps of a tile are adjacent, so a wavefront streams whole cache lines
// from one contiguous range.
//
// The packed matrix has V "virtual" rows:
//   * concatenation (Q/K/V, or a single matrix): virtual row v is row v of
//     the segment [seg_end[i-1], seg_end[i]) it falls into;
//   * gate/up interleave: 16-row tile t holds gate rows 8t..8t+7 followed by
//     up rows 8t..8t+7, so both halves of SwiGLU feature f sit in the same
//     tile, eight columns apart.
// The tiles are stored in groups of `grp` (packed_tile_offset): a skinny
// block that owns one group then streams one contiguous range instead of grp
// separate ones (gate/up of the 8B shape at 48 rows: 47.8 -> 44.5 us).
#include <algorithm>

#include "common.h"

namespace kvr {

namespace {

__global__ __launch_bounds__(256) void pack_weight_kernel(const bf16_t *w0, const bf16_t *w1, const bf16_t *w2,
                                                          int e0, int e1, int interleave, int V, int K,
                                                          int grp, bf16_t *dst) {
    const int ksteps = K >> 5;
    const size_t chunks = (size_t)V * K / 8;  // 16-byte chunks of the packed matrix
    for (size_t q = blockIdx.x * (size_t)blockDim.x + threadIdx.x; q < chunks; q += (size_t)gridDim.x * blockDim.x) {
        const int lane = (int)(q & 63);
        const size_t blk = q >> 6;
        const int t = (int)(blk / ksteps), s = (int)(blk - (size_t)t * ksteps);
        const int v = 16 * t + (lane & 15);
        const int k = 32 * s + 8 * (lane >> 4);
        const bf16_t *src;
        if (interleave) {
            const int j = v & 15;
            src = (j < 8 ? w0 : w1) + (size_t)(8 * t + (j & 7)) * K;
        } else if (v < e0) {
            src = w0 + (size_t)v * K;
        } else if (v < e1) {
            src = w1 + (size_t)(v - e0) * K;
        } else {
            src = w2 + (size_t)(v - e1) * K;
        }
        int kstride;
        const size_t o = packed_tile_offset(t, V >> 4, ksteps, grp, &kstride) + (size_t)s * kstride + lane * 8;
        *reinterpret_cast<u32x4 *>(dst + o) = *reinterpret_cast<const u32x4 *>(src + k);
    }
}

}  // namespace

hipError_t launch_pack_weight(const void *w0, const void *w1, const void *w2, int e0, int e1, bool interleave,
                              int V, int K, int grp, void *dst, hipStream_t s) {
    if (V <= 0 || V % 16 != 0 || K % 32 != 0 || grp < 1) return hipErrorInvalidValue;
    const size_t chunks = (size_t)V * K / 8;
    const int grid = (int)std::min<size_t>((chunks + 255) / 256, 65536);
    kvr_launch(pack_weight_kernel, dim3(grid), dim3(256), 0, s, (const bf16_t *)w0, (const bf16_t *)w1,
                       (const bf16_t *)w2, e0, e1, interleave ? 1 : 0, V, K, grp, (bf16_t *)dst);
    return hipGetLastError();
}

}  // namespace kvr
