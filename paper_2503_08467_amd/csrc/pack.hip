// loadShard: cut this device's inner slice out of every expert's weights (W_i by columns,
// W_o by the matching rows) and store it K-contiguous for the grouped GEMM:
//   W1^T[e][n][j] = W1[e][j][col0 + n]        n < f, zero for f <= n < fp
//   W2^T[e][c][n] = W2[e][col0 + n][c]        n < f, zero for f <= n < fp
// Both are batched 2-D transposes of a sub-matrix with zero padding, done through a
// 64 x 64 LDS tile so that reads and writes are both row-contiguous.
//
// bf16 weights are stored K-blocked: the K (reduction) index is split into blocks of 32, and
// block kb holds every row's 32 elements side by side -- element (row, k) of a [rows][K]
// matrix sits at ((k / 32) * rows + row) * 32 + k % 32.  A GEMM stage that takes 32 K values
// of consecutive rows then reads one contiguous run of memory.  W1^T / W3^T (K = h) use it
// when h is a multiple of 32; W2^T (K = fp, a multiple of 128) always does.  fp32 weights
// stay row-major.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kTile = 64;

// dst[e](c, r) = (r < nr && c < nc) ? src[e][(r0 + r) * src_ld + c0 + c] : 0
// for c < dst_rows, r < dst_cols, where dst(c, r) is dst[c * dst_cols + r] (row-major) or,
// with blocked, dst[((r / 32) * dst_rows + c) * 32 + r % 32] (dst_cols a multiple of 32).
template <typename Te>
__global__ __launch_bounds__(256) void transpose_pad(const Te* __restrict__ src, int64_t src_estride,
                                                     int64_t src_ld, int64_t r0, int64_t c0, int64_t nr,
                                                     int64_t nc, Te* __restrict__ dst, int64_t dst_estride,
                                                     int64_t dst_rows, int64_t dst_cols, int blocked) {
    __shared__ Te tile[kTile][kTile + 1];
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int64_t rt = static_cast<int64_t>(blockIdx.x) * kTile;  // source rows = dst cols
    const int64_t ct = static_cast<int64_t>(blockIdx.y) * kTile;  // source cols = dst rows
    const Te* s = src + blockIdx.z * src_estride;
    Te* d = dst + blockIdx.z * dst_estride;
    for (int i = ty; i < kTile; i += 4) {
        const int64_t r = rt + i, c = ct + tx;
        tile[i][tx] = (r < nr && c < nc) ? s[(r0 + r) * src_ld + c0 + c] : Te(0);
    }
    __syncthreads();
    for (int i = ty; i < kTile; i += 4) {
        const int64_t c = ct + i, r = rt + tx;
        if (c < dst_rows && r < dst_cols)
            d[blocked ? ((r >> 5) * dst_rows + c) * 32 + (r & 31) : c * dst_cols + r] = tile[tx][i];
    }
}

template <typename Te>
hipError_t pack_t(const void* w1, const void* w3, const void* w2, int E, int64_t h, int64_t F,
                  int64_t col0, int64_t f, int64_t fp, void* w1t, void* w3t, void* w2t, hipStream_t s) {
    const int blk1 = (sizeof(Te) == 2 && h % 32 == 0) ? 1 : 0;
    const int blk2 = sizeof(Te) == 2 ? 1 : 0;
    // W1 (and W3): source [h rows][F cols] -> dst [fp rows][h cols]
    const dim3 g1(static_cast<unsigned>(ceil_div(h, kTile)), static_cast<unsigned>(ceil_div(fp, kTile)), E);
    hipLaunchKernelGGL(transpose_pad<Te>, g1, dim3(256), 0, s, static_cast<const Te*>(w1), h * F, F,
                       int64_t(0), col0, h, f, static_cast<Te*>(w1t), fp * h, fp, h, blk1);
    if (w3)
        hipLaunchKernelGGL(transpose_pad<Te>, g1, dim3(256), 0, s, static_cast<const Te*>(w3), h * F, F,
                           int64_t(0), col0, h, f, static_cast<Te*>(w3t), fp * h, fp, h, blk1);
    // W2: source [F rows][h cols], rows col0.. -> dst [h rows][fp cols]
    const dim3 g2(static_cast<unsigned>(ceil_div(fp, kTile)), static_cast<unsigned>(ceil_div(h, kTile)), E);
    hipLaunchKernelGGL(transpose_pad<Te>, g2, dim3(256), 0, s, static_cast<const Te*>(w2), F * h, h, col0,
                       int64_t(0), f, h, static_cast<Te*>(w2t), h * fp, h, fp, blk2);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_pack(const void* w1, const void* w3, const void* w2, int E, int64_t h, int64_t F,
                       int64_t col0, int64_t f, int64_t fp, int elem_bytes, void* w1t, void* w3t,
                       void* w2t, hipStream_t s) {
    if (elem_bytes == 2) return pack_t<uint16_t>(w1, w3, w2, E, h, F, col0, f, fp, w1t, w3t, w2t, s);
    return pack_t<uint32_t>(w1, w3, w2, E, h, F, col0, f, fp, w1t, w3t, w2t, s);
}

}  // namespace moe
