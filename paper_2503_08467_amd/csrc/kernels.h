// Internal launchers of the MoE layer kernels (called by the C ABI after validation).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

// Tile constants shared by the packer and the grouped GEMM.
constexpr int kInnerAlign = 128;  // packed inner width is a multiple of this
constexpr int kDispatchChunk = 1024;  // assignments per dispatch workgroup

// K parts of the down-projection.  A call with few rows has few row tiles, each with a long
// K loop, and leaves most CUs idle; splitting K spreads the weight reads over more workgroups
// (fp32 partial tiles, summed in a fixed order afterwards).  A function of the call's sizes
// only (the row bound, not the routing), so every launch path of one call shape rounds the
// same way.  fp is the packed inner width (a multiple of kInnerAlign).
//   bf16: up to 8 parts for at most 512 rows (measured: no gain from 1024 rows up);
//   fp32: 4 parts for at most 1024 rows (its K loop is four times as slow as bf16's).
inline int down_ksplit(int64_t A_max, int64_t fp, bool bf16) {
    const int64_t nk = fp / 32;  // K steps of 32
    if (!bf16) return (A_max <= 1024 && nk % 4 == 0 && nk / 4 >= 8) ? 4 : 1;
    if (A_max > 512) return 1;
    int s = A_max <= 256 ? 8 : 4;
    while (s > 1 && (nk % s != 0 || nk / s < 8)) s >>= 1;
    return s;
}

// Bytes of fp32 partial tiles to reserve past the H buffer for a call bound of A_max rows:
// the most that any call with at most A_max rows needs (down_ksplit * rows * h * 4), so
// that a workspace sized for a bound also serves every smaller call.  The product is
// largest at the ends of the split ranges (256, 512 and 1024 rows).
inline size_t down_partial_bytes(int64_t A_max, int64_t h, int64_t fp, bool bf16) {
    int64_t most = 0;
    for (int64_t end : {int64_t(256), int64_t(512), int64_t(1024)}) {
        const int64_t a = A_max < end ? A_max : end;
        const int64_t s = down_ksplit(a, fp, bf16);
        if (s > 1 && s * a > most) most = s * a;
    }
    return static_cast<size_t>(most) * static_cast<size_t>(h) * 4u;
}

hipError_t launch_route(const void* x, bool bf16, int64_t T, int h, const void* wg, int E, int k,
                        const float* bias, int64_t bias_stride, int renorm, int32_t* idx, float* w,
                        hipStream_t s);

// Step 2's outputs written by the routing launch itself (moe_dispatch's counts, offsets,
// row_src, pos_of; no x_perm).
struct RouteDispatchOut {
    int32_t* counts;
    int32_t* offsets;
    int32_t* row_src;
    int32_t* pos_of;
};

// Whether one routing workgroup covers the whole batch, so that it can also group the
// assignments: bf16, h % 64 == 0, 32 < E <= 256, 1 <= T <= 64, k <= 8.
bool route_dispatch_fusable(bool bf16, int64_t T, int h, int E, int k);

// Steps 1 and 2 in one launch (only when route_dispatch_fusable).
hipError_t launch_route_dispatch(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                                 int64_t bias_stride, int renorm, int32_t* idx, float* w, RouteDispatchOut out,
                                 hipStream_t s);

hipError_t launch_dispatch(const int32_t* idx, int64_t T, int k, int E, const void* x, int elem_bytes,
                           int h, int32_t* counts, int32_t* offsets, int32_t* row_src,
                           int32_t* pos_of, void* x_perm, int32_t* ws, hipStream_t s);

hipError_t launch_pack(const void* w1, const void* w3, const void* w2, int E, int64_t h, int64_t F,
                       int64_t col0, int64_t f, int64_t fp, int elem_bytes, void* w1t, void* w3t,
                       void* w2t, hipStream_t s);

hipError_t launch_ffn(const void* x_perm, const int32_t* offsets, int64_t A_max, int E, int h,
                      int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                      const void* w2t, void* y_perm, bool y_bf16, void* hbuf, hipStream_t s);

hipError_t launch_ffn_gather(const void* x, int64_t T, const int32_t* row_src, const int32_t* offsets, int64_t A_max,
                             int E, int h, int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                             const void* w2t, void* y_perm, bool y_bf16, void* hbuf, hipStream_t s);

// launch_ffn_gather followed by launch_combine; when the second product's K is split, its
// parts' sum and the combine run as one kernel and y_perm is not written (*y_perm_written).
hipError_t launch_ffn_gather_combine(const void* x, int64_t T, const int32_t* row_src, const int32_t* offsets, int k,
                                     int E, int h, int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                                     const void* w2t, void* y_perm, bool y_bf16, const int32_t* pos_of,
                                     const float* topk_w, void* y, bool out_bf16, void* hbuf, hipStream_t s,
                                     bool* y_perm_written);

hipError_t launch_ffn_top1(const void* x, int64_t T, const int32_t* row_src, const float* topk_w,
                           const int32_t* offsets, int64_t A_max, int E, int h, int64_t fp, int act, bool bf16,
                           const void* w1t, const void* w3t, const void* w2t, void* y, bool y_bf16, void* hbuf,
                           hipStream_t s);

hipError_t launch_ffn_per_expert(const void* x_perm, const int32_t* offsets, const int32_t* offsets_host,
                                 int64_t A_max, int E, int h, int64_t fp, int act, bool bf16, const void* w1t,
                                 const void* w3t, const void* w2t, void* y_perm, bool y_bf16, void* hbuf,
                                 hipStream_t s);

// moe_expert_ffn_shard with its workspace in the library's static per-device array.
hipError_t launch_ffn_noalloc(const void* x_perm, const int32_t* offsets, int64_t A_max, int E, int h, int64_t fp,
                              int act, bool bf16, const void* w1t, const void* w3t, const void* w2t, void* y_perm,
                              bool y_bf16, hipStream_t s);

hipError_t launch_combine(const void* y_perm, bool y_bf16, const int32_t* pos_of, const float* w,
                          int64_t T, int k, int h, void* y, bool out_bf16, hipStream_t s);

}  // namespace moe
