// C ABI of the MoE layer: argument validation, workspace sizing and kernel launches.
// Nothing is launched unless every argument checks out.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "../../include/moeshard.h"
#include "kernels.h"

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool valid_dtype(moe_dtype d) { return d == MOE_F32 || d == MOE_BF16; }

bool valid_act(moe_act a) { return a == MOE_ACT_GELU || a == MOE_ACT_GELU_TANH || a == MOE_ACT_SWIGLU; }

int elem_bytes(moe_dtype d) { return d == MOE_BF16 ? 2 : 4; }

bool valid_h(int64_t h) { return h >= 8 && h % 8 == 0 && h <= (1 << 20); }

bool valid_ek(int32_t E, int32_t k) { return E >= 1 && k >= 1 && k <= E; }

moe_status from_hip(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_ERR_HIP; }

// A tensor pointer must be present and 16-byte aligned whenever it holds data.
bool ok_ptr(const void* p, bool needed) { return !needed || (p != nullptr && aligned16(p)); }

int64_t dispatch_chunks(int64_t A) { return (A + moe::kDispatchChunk - 1) / moe::kDispatchChunk; }

}  // namespace

extern "C" {

const char* moe_status_string(moe_status status) {
    switch (status) {
        case MOE_OK: return "MOE_OK";
        case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG: invalid size, pointer, alignment or enum";
        case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED: request not implemented in this build";
        case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE: workspace or packed buffer too small";
        case MOE_ERR_HIP: return "MOE_ERR_HIP: HIP runtime error at launch";
        case MOE_ERR_TOO_LARGE: return "MOE_ERR_TOO_LARGE: the call needs more than the static scratch array holds";
    }
    return "unknown moe_status";
}

moe_status moe_route(const void* x, moe_dtype xdt, int64_t T, int64_t h, const void* w_gate,
                     int32_t E, int32_t k, const float* sel_bias, int64_t bias_row_stride,
                     int32_t renorm, int32_t* topk_idx, float* topk_w, hipStream_t stream) {
    if (!valid_dtype(xdt) || T < 0 || !valid_h(h) || !valid_ek(E, k)) return MOE_ERR_INVALID_ARG;
    if (E > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
    if (T * k >= INT32_MAX) return MOE_ERR_INVALID_ARG;
    if (renorm != 0 && renorm != 1) return MOE_ERR_INVALID_ARG;
    if (bias_row_stride != 0 && bias_row_stride != E) return MOE_ERR_INVALID_ARG;
    const bool any = T > 0;
    if (!ok_ptr(x, any) || !ok_ptr(w_gate, true) || !ok_ptr(topk_idx, any) || !ok_ptr(topk_w, any))
        return MOE_ERR_INVALID_ARG;
    if (sel_bias && (reinterpret_cast<uintptr_t>(sel_bias) & 3u)) return MOE_ERR_INVALID_ARG;
    if (!any) return MOE_OK;
    return from_hip(moe::launch_route(x, xdt == MOE_BF16, T, static_cast<int>(h), w_gate, E, k, sel_bias,
                                      bias_row_stride, renorm, topk_idx, topk_w, stream));
}

size_t moe_dispatch_workspace_size(int64_t T, int32_t k, int32_t E) {
    if (T < 0 || k < 1 || E < 1) return 0;
    const int64_t L = static_cast<int64_t>(E) * dispatch_chunks(T * k);
    return align_up(sizeof(int32_t) * static_cast<size_t>(2 * L + 1));
}

moe_status moe_dispatch(const int32_t* topk_idx, int64_t T, int32_t k, int32_t E, const void* x,
                        moe_dtype xdt, int64_t h, int32_t* counts, int32_t* offsets, int32_t* row_src,
                        int32_t* pos_of, void* x_perm, void* ws, size_t ws_bytes, hipStream_t stream) {
    if (!valid_dtype(xdt) || T < 0 || !valid_h(h) || !valid_ek(E, k)) return MOE_ERR_INVALID_ARG;
    if (E > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
    if (T * k >= INT32_MAX) return MOE_ERR_INVALID_ARG;
    const bool any = T > 0;
    // x_perm may be NULL: the grouped rows are then not written (moe_expert_ffn_shard_gather
    // reads them through row_src); x is only read when x_perm is given
    const bool gather = x_perm != nullptr;
    if (!ok_ptr(topk_idx, any) || !ok_ptr(x, any && gather) || !ok_ptr(counts, true) || !ok_ptr(offsets, true) ||
        !ok_ptr(row_src, any) || !ok_ptr(pos_of, any) || (x_perm && !aligned16(x_perm)) || !ok_ptr(ws, true))
        return MOE_ERR_INVALID_ARG;
    if (ws_bytes < moe_dispatch_workspace_size(T, k, E)) return MOE_ERR_WORKSPACE;
    return from_hip(moe::launch_dispatch(topk_idx, T, k, E, x, elem_bytes(xdt), static_cast<int>(h), counts,
                                         offsets, row_src, pos_of, x_perm, static_cast<int32_t*>(ws), stream));
}

moe_status moe_route_dispatch(const void* x, moe_dtype xdt, int64_t T, int64_t h, const void* w_gate, int32_t E,
                              int32_t k, const float* sel_bias, int64_t bias_row_stride, int32_t renorm,
                              int32_t* topk_idx, float* topk_w, int32_t* counts, int32_t* offsets,
                              int32_t* row_src, int32_t* pos_of, void* ws, size_t ws_bytes, hipStream_t stream) {
    // every check of both calls, before any launch
    if (!valid_dtype(xdt) || T < 0 || !valid_h(h) || !valid_ek(E, k)) return MOE_ERR_INVALID_ARG;
    if (E > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
    if (T * k >= INT32_MAX) return MOE_ERR_INVALID_ARG;
    if (renorm != 0 && renorm != 1) return MOE_ERR_INVALID_ARG;
    if (bias_row_stride != 0 && bias_row_stride != E) return MOE_ERR_INVALID_ARG;
    const bool any = T > 0;
    if (!ok_ptr(x, any) || !ok_ptr(w_gate, true) || !ok_ptr(topk_idx, any) || !ok_ptr(topk_w, any) ||
        !ok_ptr(counts, true) || !ok_ptr(offsets, true) || !ok_ptr(row_src, any) || !ok_ptr(pos_of, any) ||
        !ok_ptr(ws, true))
        return MOE_ERR_INVALID_ARG;
    if (sel_bias && (reinterpret_cast<uintptr_t>(sel_bias) & 3u)) return MOE_ERR_INVALID_ARG;
    if (ws_bytes < moe_dispatch_workspace_size(T, k, E)) return MOE_ERR_WORKSPACE;
    const bool bf16 = xdt == MOE_BF16;
    if (moe::route_dispatch_fusable(bf16, T, static_cast<int>(h), E, k))
        return from_hip(moe::launch_route_dispatch(x, T, static_cast<int>(h), w_gate, E, k, sel_bias, bias_row_stride,
                                                   renorm, topk_idx, topk_w,
                                                   moe::RouteDispatchOut{counts, offsets, row_src, pos_of}, stream));
    if (any) {
        const hipError_t err = moe::launch_route(x, bf16, T, static_cast<int>(h), w_gate, E, k, sel_bias,
                                                 bias_row_stride, renorm, topk_idx, topk_w, stream);
        if (err != hipSuccess) return from_hip(err);
    }
    return from_hip(moe::launch_dispatch(topk_idx, T, k, E, x, elem_bytes(xdt), static_cast<int>(h), counts, offsets,
                                         row_src, pos_of, nullptr, static_cast<int32_t*>(ws), stream));
}

int64_t moe_padded_inner_width(int64_t f) {
    if (f < 1) return 0;
    return (f + moe::kInnerAlign - 1) / moe::kInnerAlign * moe::kInnerAlign;
}

static size_t packed_matrix_bytes(int32_t E, int64_t h, int64_t f, moe_dtype wdt) {
    return align_up(static_cast<size_t>(E) * static_cast<size_t>(moe_padded_inner_width(f)) *
                    static_cast<size_t>(h) * static_cast<size_t>(elem_bytes(wdt)));
}

size_t moe_packed_weights_size(int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype wdt) {
    if (E < 1 || h < 1 || f < 1 || !valid_act(act) || !valid_dtype(wdt)) return 0;
    return packed_matrix_bytes(E, h, f, wdt) * (act == MOE_ACT_SWIGLU ? 3 : 2);
}

moe_status moe_pack_weights(const void* w1, const void* w3, const void* w2, int32_t E, int64_t h, int64_t F,
                            int64_t col0, int64_t f, moe_act act, moe_dtype wdt, void* packed,
                            size_t packed_bytes, hipStream_t stream) {
    if (!valid_dtype(wdt) || !valid_act(act) || !valid_h(h) || E < 1 || f < 1 || col0 < 0 || col0 + f > F)
        return MOE_ERR_INVALID_ARG;
    if (E > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
    const bool swiglu = act == MOE_ACT_SWIGLU;
    if (!ok_ptr(w1, true) || !ok_ptr(w2, true) || !ok_ptr(packed, true) || (swiglu && !ok_ptr(w3, true)))
        return MOE_ERR_INVALID_ARG;
    if (packed_bytes < moe_packed_weights_size(E, h, f, act, wdt)) return MOE_ERR_WORKSPACE;
    const size_t mb = packed_matrix_bytes(E, h, f, wdt);
    unsigned char* base = static_cast<unsigned char*>(packed);
    void* w1t = base;
    void* w3t = swiglu ? base + mb : nullptr;
    void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_pack(w1, swiglu ? w3 : nullptr, w2, E, h, F, col0, f, moe_padded_inner_width(f),
                                     elem_bytes(wdt), w1t, w3t, w2t, stream));
}

size_t moe_ffn_workspace_size(int64_t A_max, int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt) {
    (void)E;
    (void)act;
    if (A_max < 0 || f < 1 || h < 0 || !valid_dtype(dt)) return 0;
    const int64_t fp = moe_padded_inner_width(f);
    // H (A_max x fp), then the down-projection's fp32 partial tiles when its K is split
    return align_up(static_cast<size_t>(A_max) * static_cast<size_t>(fp) * static_cast<size_t>(elem_bytes(dt))) +
           align_up(moe::down_partial_bytes(A_max, h, fp, dt == MOE_BF16)) + kAlign;
}

// Checks shared by the expert-step calls, all but the workspace.
static moe_status ffn_args_check(const void* x_perm, const int32_t* offsets, int64_t A_max, int32_t E, int64_t h,
                                 int64_t f, moe_act act, moe_dtype dt, const void* packed, const void* y_perm,
                                 moe_dtype ydt) {
    if (!valid_dtype(dt) || !valid_dtype(ydt) || !valid_act(act) || !valid_h(h) || E < 1 || f < 1 || A_max < 0)
        return MOE_ERR_INVALID_ARG;
    if (E > MOE_MAX_EXPERTS) return MOE_ERR_UNSUPPORTED;
    if (A_max >= INT32_MAX) return MOE_ERR_INVALID_ARG;
    if (moe_padded_inner_width(f) >= INT32_MAX / 2) return MOE_ERR_UNSUPPORTED;
    const bool any = A_max > 0;
    if (!ok_ptr(x_perm, any) || !ok_ptr(offsets, true) || !ok_ptr(packed, true) || !ok_ptr(y_perm, any))
        return MOE_ERR_INVALID_ARG;
    return MOE_OK;
}

static moe_status ffn_check(const void* x_perm, const int32_t* offsets, int64_t A_max, int32_t E, int64_t h,
                            int64_t f, moe_act act, moe_dtype dt, const void* packed, const void* y_perm,
                            moe_dtype ydt, const void* ws, size_t ws_bytes) {
    const moe_status st = ffn_args_check(x_perm, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt);
    if (st != MOE_OK) return st;
    if (!ok_ptr(ws, A_max > 0)) return MOE_ERR_INVALID_ARG;
    if (ws_bytes < moe_ffn_workspace_size(A_max, E, h, f, act, dt)) return MOE_ERR_WORKSPACE;
    return MOE_OK;
}

moe_status moe_expert_ffn_shard(const void* x_perm, const int32_t* offsets, int64_t A_max, int32_t E, int64_t h,
                                int64_t f, moe_act act, moe_dtype dt, const void* packed, void* y_perm,
                                moe_dtype ydt, void* ws, size_t ws_bytes, hipStream_t stream) {
    const moe_status st = ffn_check(x_perm, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt, ws, ws_bytes);
    if (st != MOE_OK) return st;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_ffn(x_perm, offsets, A_max, E, static_cast<int>(h), moe_padded_inner_width(f),
                                    static_cast<int>(act), dt == MOE_BF16, w1t, w3t, w2t, y_perm, ydt == MOE_BF16,
                                    ws, stream));
}

moe_status moe_expert_ffn_shard_gather(const void* x, int64_t T, const int32_t* row_src, const int32_t* offsets,
                                       int64_t A_max, int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                       const void* packed, void* y_perm, moe_dtype ydt, void* ws, size_t ws_bytes,
                                       hipStream_t stream) {
    const moe_status st = ffn_check(x, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt, ws, ws_bytes);
    if (st != MOE_OK) return st;
    if (T < 0 || (A_max > 0 && (T < 1 || !ok_ptr(row_src, true)))) return MOE_ERR_INVALID_ARG;
    // a source row's byte offset must fit the kernels' 32-bit per-lane offsets
    if (T * h * elem_bytes(dt) >= (int64_t(1) << 32)) return MOE_ERR_UNSUPPORTED;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_ffn_gather(x, T, row_src, offsets, A_max, E, static_cast<int>(h),
                                           moe_padded_inner_width(f), static_cast<int>(act), dt == MOE_BF16, w1t, w3t,
                                           w2t, y_perm, ydt == MOE_BF16, ws, stream));
}

moe_status moe_expert_ffn_shard_gather_combine(const void* x, int64_t T, const int32_t* row_src,
                                               const int32_t* offsets, const int32_t* pos_of, const float* topk_w,
                                               int32_t k, int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                               const void* packed, void* y_perm, moe_dtype ydt, void* y,
                                               moe_dtype out_dt, int32_t* y_perm_written, void* ws, size_t ws_bytes,
                                               hipStream_t stream) {
    if (k < 1 || T < 0 || T * static_cast<int64_t>(k) >= INT32_MAX || !valid_dtype(out_dt)) return MOE_ERR_INVALID_ARG;
    const int64_t A_max = T * k;
    const moe_status st = ffn_check(x, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt, ws, ws_bytes);
    if (st != MOE_OK) return st;
    const bool any = T > 0;
    if (!ok_ptr(row_src, any) || !ok_ptr(pos_of, any) || !ok_ptr(y, any) ||
        (any && (!topk_w || (reinterpret_cast<uintptr_t>(topk_w) & 3u))))
        return MOE_ERR_INVALID_ARG;
    if (T * h * elem_bytes(dt) >= (int64_t(1) << 32)) return MOE_ERR_UNSUPPORTED;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    bool written = true;
    moe_status out = MOE_OK;
    if (any)
        out = from_hip(moe::launch_ffn_gather_combine(x, T, row_src, offsets, k, E, static_cast<int>(h),
                                                      moe_padded_inner_width(f), static_cast<int>(act), dt == MOE_BF16,
                                                      w1t, w3t, w2t, y_perm, ydt == MOE_BF16, pos_of, topk_w, y,
                                                      out_dt == MOE_BF16, ws, stream, &written));
    if (y_perm_written) *y_perm_written = written ? 1 : 0;
    return out;
}

moe_status moe_expert_ffn_shard_top1(const void* x, int64_t T, const int32_t* row_src, const float* topk_w,
                                     const int32_t* offsets, int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                     const void* packed, void* y, moe_dtype out_dt, void* ws, size_t ws_bytes,
                                     hipStream_t stream) {
    const moe_status st = ffn_check(x, offsets, T, E, h, f, act, dt, packed, y, out_dt, ws, ws_bytes);
    if (st != MOE_OK) return st;
    if (T > 0 && (!ok_ptr(row_src, true) || !topk_w || (reinterpret_cast<uintptr_t>(topk_w) & 3u)))
        return MOE_ERR_INVALID_ARG;
    if (T * h * elem_bytes(dt) >= (int64_t(1) << 32)) return MOE_ERR_UNSUPPORTED;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_ffn_top1(x, T, row_src, topk_w, offsets, T, E, static_cast<int>(h),
                                         moe_padded_inner_width(f), static_cast<int>(act), dt == MOE_BF16, w1t, w3t,
                                         w2t, y, out_dt == MOE_BF16, ws, stream));
}

moe_status moe_expert_ffn_shard_per_expert(const void* x_perm, const int32_t* offsets, const int32_t* offsets_host,
                                           int64_t A_max, int32_t E, int64_t h, int64_t f, moe_act act,
                                           moe_dtype dt, const void* packed, void* y_perm, moe_dtype ydt, void* ws,
                                           size_t ws_bytes, hipStream_t stream) {
    const moe_status st = ffn_check(x_perm, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt, ws, ws_bytes);
    if (st != MOE_OK) return st;
    if (!offsets_host || offsets_host[0] < 0 || offsets_host[E] > A_max) return MOE_ERR_INVALID_ARG;
    for (int32_t e = 0; e < E; ++e)
        if (offsets_host[e + 1] < offsets_host[e]) return MOE_ERR_INVALID_ARG;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_ffn_per_expert(x_perm, offsets, offsets_host, A_max, E, static_cast<int>(h),
                                               moe_padded_inner_width(f), static_cast<int>(act), dt == MOE_BF16, w1t,
                                               w3t, w2t, y_perm, ydt == MOE_BF16, ws, stream));
}

moe_status moe_expert_ffn_shard_noalloc(const void* x_perm, const int32_t* offsets, int64_t A_max, int32_t E,
                                        int64_t h, int64_t f, moe_act act, moe_dtype dt, const void* packed,
                                        void* y_perm, moe_dtype ydt, hipStream_t stream) {
    // the argument checks of moe_expert_ffn_shard; the static array is the workspace
    const moe_status st = ffn_args_check(x_perm, offsets, A_max, E, h, f, act, dt, packed, y_perm, ydt);
    if (st != MOE_OK) return st;
    if (moe_ffn_workspace_size(A_max, E, h, f, act, dt) > MOE_NOALLOC_SCRATCH_BYTES) return MOE_ERR_TOO_LARGE;
    const size_t mb = packed_matrix_bytes(E, h, f, dt);
    const unsigned char* base = static_cast<const unsigned char*>(packed);
    const bool swiglu = act == MOE_ACT_SWIGLU;
    const void* w1t = base;
    const void* w3t = swiglu ? base + mb : nullptr;
    const void* w2t = base + (swiglu ? 2 : 1) * mb;
    return from_hip(moe::launch_ffn_noalloc(x_perm, offsets, A_max, E, static_cast<int>(h),
                                            moe_padded_inner_width(f), static_cast<int>(act), dt == MOE_BF16, w1t,
                                            w3t, w2t, y_perm, ydt == MOE_BF16, stream));
}

moe_status moe_combine(const void* y_perm, moe_dtype ydt, const int32_t* pos_of, const float* topk_w, int64_t T,
                       int32_t k, int64_t h, void* y, moe_dtype out_dt, hipStream_t stream) {
    if (!valid_dtype(ydt) || !valid_dtype(out_dt) || T < 0 || k < 1 || !valid_h(h)) return MOE_ERR_INVALID_ARG;
    if (T * k >= INT32_MAX) return MOE_ERR_INVALID_ARG;
    const bool any = T > 0;
    if (!ok_ptr(y_perm, any) || !ok_ptr(pos_of, any) || !ok_ptr(topk_w, any) || !ok_ptr(y, any))
        return MOE_ERR_INVALID_ARG;
    if (!any) return MOE_OK;
    return from_hip(moe::launch_combine(y_perm, ydt == MOE_BF16, pos_of, topk_w, T, k, static_cast<int>(h), y,
                                        out_dt == MOE_BF16, stream));
}

}  // extern "C"
