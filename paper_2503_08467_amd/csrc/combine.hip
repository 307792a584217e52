// Step 5 of the layer: y[t] = sum_j w[t, j] * y_perm[pos_of[t, j]], accumulated in fp32 in
// pick order and rounded once.  One thread produces 8 consecutive outputs of one token.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

template <bool YB>
struct Row8;

template <>
struct Row8<true> {
    static __device__ __forceinline__ void load(const void* base, int64_t off, float v[8]) {
        const uint4 q = *reinterpret_cast<const uint4*>(static_cast<const bf16_t*>(base) + off);
        const uint32_t u[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(u[i] << 16);
            v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
        }
    }
    static __device__ __forceinline__ void store(void* base, int64_t off, const float v[8]) {
        uint4 q;
        q.x = pack_bf16x2(v[0], v[1]);
        q.y = pack_bf16x2(v[2], v[3]);
        q.z = pack_bf16x2(v[4], v[5]);
        q.w = pack_bf16x2(v[6], v[7]);
        *reinterpret_cast<uint4*>(static_cast<bf16_t*>(base) + off) = q;
    }
};

template <>
struct Row8<false> {
    static __device__ __forceinline__ void load(const void* base, int64_t off, float v[8]) {
        const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(base) + off);
        const float4 a = p[0], b = p[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
    static __device__ __forceinline__ void store(void* base, int64_t off, const float v[8]) {
        float4* p = reinterpret_cast<float4*>(static_cast<float*>(base) + off);
        p[0] = make_float4(v[0], v[1], v[2], v[3]);
        p[1] = make_float4(v[4], v[5], v[6], v[7]);
    }
};

constexpr int kCombineUnroll = 4;  // picks whose rows are loaded together

template <bool YB, bool OB>
__global__ __launch_bounds__(256) void combine_kernel(const void* __restrict__ y_perm,
                                                      const int32_t* __restrict__ pos_of,
                                                      const float* __restrict__ w, int64_t T, int k,
                                                      int h, void* __restrict__ y) {
    const int nv = h / 8;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= T * nv) return;
    const int64_t t = i / nv;
    const int c = static_cast<int>(i - t * nv) * 8;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (k <= kCombineUnroll) {
        // every position and weight first, then every row from a clamped position (a load
        // behind a per-lane condition would wait for each row in turn); rows of positions out
        // of range are loaded but not added
        int32_t pos[kCombineUnroll];
        float wt[kCombineUnroll];
#pragma unroll
        for (int j = 0; j < kCombineUnroll; ++j)
            if (j < k) {
                pos[j] = pos_of[t * k + j];
                wt[j] = w[t * k + j];
            }
        float v[kCombineUnroll][8];
#pragma unroll
        for (int j = 0; j < kCombineUnroll; ++j)
            if (j < k) {
                const bool ok = pos[j] >= 0 && pos[j] < T * k;
                Row8<YB>::load(y_perm, static_cast<int64_t>(ok ? pos[j] : 0) * h + c, v[j]);
            }
#pragma unroll
        for (int j = 0; j < kCombineUnroll; ++j)
            if (j < k) {
                const bool ok = pos[j] >= 0 && pos[j] < T * k;
#pragma unroll
                for (int q = 0; q < 8; ++q) acc[q] = ok ? acc[q] + wt[j] * v[j][q] : acc[q];
            }
    } else {
        for (int j = 0; j < k; ++j) {
            const int32_t p = pos_of[t * k + j];
            if (p < 0 || p >= T * k) continue;
            const float wt = w[t * k + j];
            float v[8];
            Row8<YB>::load(y_perm, static_cast<int64_t>(p) * h + c, v);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[q] += wt * v[q];
        }
    }
    Row8<OB>::store(y, t * h + c, acc);
}

}  // namespace

hipError_t launch_combine(const void* y_perm, bool y_bf16, const int32_t* pos_of, const float* w,
                          int64_t T, int k, int h, void* y, bool out_bf16, hipStream_t s) {
    if (T == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(ceil_div(T * (h / 8), 256)));
    if (y_bf16 && out_bf16)
        hipLaunchKernelGGL((combine_kernel<true, true>), grid, dim3(256), 0, s, y_perm, pos_of, w, T, k, h, y);
    else if (y_bf16)
        hipLaunchKernelGGL((combine_kernel<true, false>), grid, dim3(256), 0, s, y_perm, pos_of, w, T, k, h, y);
    else if (out_bf16)
        hipLaunchKernelGGL((combine_kernel<false, true>), grid, dim3(256), 0, s, y_perm, pos_of, w, T, k, h, y);
    else
        hipLaunchKernelGGL((combine_kernel<false, false>), grid, dim3(256), 0, s, y_perm, pos_of, w, T, k, h, y);
    return hipGetLastError();
}

}  // namespace moe
