// Step 1 of the layer: gate logits, top-k selection and softmax weights.
//
// The gate product logits[t, e] = x[t] . w_gate[e] runs on MFMA (16x16 output blocks,
// fp32 accumulation).  Each wave owns 16 tokens and all (padded) experts: its
// accumulators hold the 16 x E_pad logit block, which it parks in LDS and then reduces
// per token across the wave (max, sum of exponentials, k rounds of arg-max with the
// lower expert id winning ties).  The four waves of a workgroup are independent.
#include "common.h"
#include "kernels.h"

namespace moe {
namespace {

constexpr int kRouteTokensPerWave = 16;
constexpr int kRouteWaves = 4;

// One K chunk of the gate product for one 16 x 16 block.
template <typename Tin>
struct GateChunk;

template <>
struct GateChunk<bf16_t> {
    static constexpr int kStep = 32;  // K covered by one v_mfma_f32_16x16x32_bf16
    typedef uint4 frag_t;
    static __device__ __forceinline__ frag_t load(const bf16_t* base, int64_t row, int64_t nrows,
                                                  int h, int k) {
        if (row < nrows && k < h) return *reinterpret_cast<const uint4*>(base + row * h + k);
        return make_uint4(0, 0, 0, 0);
    }
    static __device__ __forceinline__ int lane_k(int k0, int g) { return k0 + g * 8; }
    static __device__ __forceinline__ f32x4_t mma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
    }
};

template <>
struct GateChunk<float> {
    static constexpr int kStep = 16;  // four v_mfma_f32_16x16x4_f32 on one float4 per lane
    typedef float4 frag_t;
    static __device__ __forceinline__ frag_t load(const float* base, int64_t row, int64_t nrows,
                                                  int h, int k) {
        if (row < nrows && k < h) return *reinterpret_cast<const float4*>(base + row * h + k);
        return make_float4(0.f, 0.f, 0.f, 0.f);
    }
    static __device__ __forceinline__ int lane_k(int k0, int g) { return k0 + g * 4; }
    static __device__ __forceinline__ f32x4_t mma(frag_t a, frag_t b, f32x4_t c) {
        // lane (r, g) supplies element c of its float4 as K index g of MFMA number c; A and B
        // use the same mapping, so the four products sum over all 16 K values of the chunk.
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, c, 0, 0, 0);
        return c;
    }
};

template <typename Tin, int NB>
__global__ __launch_bounds__(kRouteWaves * kWave) void route_kernel(
    const Tin* __restrict__ x, const Tin* __restrict__ wg, int64_t T, int h, int E, int k,
    const float* __restrict__ bias, int64_t bias_stride, int renorm, int32_t* __restrict__ idx,
    float* __restrict__ w) {
    constexpr int EP = NB * 16;             // padded expert count
    constexpr int LDW = (NB == 16) ? EP : EP + 1;  // LDS row stride (floats); <= 64 KiB per block
    constexpr int NV = (EP + kWave - 1) / kWave;  // experts per lane in the reductions
    extern __shared__ float lds[];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    float* lg = lds + wave * kRouteTokensPerWave * LDW;
    const int64_t tok0 = (static_cast<int64_t>(blockIdx.x) * kRouteWaves + wave) * kRouteTokensPerWave;
    const int r = lane & 15, g = lane >> 4;

    typedef GateChunk<Tin> C;
    f32x4_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int k0 = 0; k0 < h; k0 += C::kStep) {
        const int kk = C::lane_k(k0, g);
        typename C::frag_t a = C::load(x, tok0 + r, T, h, kk);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            typename C::frag_t b = C::load(wg, nb * 16 + r, E, h, kk);
            acc[nb] = C::mma(a, b, acc[nb]);
        }
    }
    // D[token][expert]: lane holds expert column r of each block, tokens 4g .. 4g+3.
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i) lg[(4 * g + i) * LDW + nb * 16 + r] = acc[nb][i];
    __syncthreads();

    for (int rr = 0; rr < kRouteTokensPerWave; ++rr) {
        const int64_t t = tok0 + rr;
        if (t >= T) break;  // uniform across the wave
        float v[NV], s[NV];
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int e = lane + i * kWave;
            v[i] = (e < E) ? lg[rr * LDW + e] : -INFINITY;
            s[i] = (e < E) ? v[i] + (bias ? bias[t * bias_stride + e] : 0.f) : -INFINITY;
            mx = fmaxf(mx, v[i]);
        }
        mx = wave_max(mx);
        float den = 0.f;
#pragma unroll
        for (int i = 0; i < NV; ++i) den += (lane + i * kWave < E) ? expf(v[i] - mx) : 0.f;
        den = wave_sum(den);

        uint32_t taken = 0;
        float wsum = 0.f;
        for (int j = 0; j < k; ++j) {
            float bs = -INFINITY;
            int be = 0x7fffffff;
#pragma unroll
            for (int i = 0; i < NV; ++i) {
                const int e = lane + i * kWave;
                if (e < E && !((taken >> i) & 1u) && (s[i] > bs || be == 0x7fffffff)) {
                    bs = s[i];
                    be = e;
                }
            }
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) {
                const float os = __shfl_xor(bs, o, kWave);
                const int oe = __shfl_xor(be, o, kWave);
                if (os > bs || (os == bs && oe < be)) {
                    bs = os;
                    be = oe;
                }
            }
            if (be != 0x7fffffff && (be & (kWave - 1)) == lane) taken |= 1u << (be / kWave);
            const float p = (be != 0x7fffffff) ? expf(lg[rr * LDW + be] - mx) / den : 0.f;
            wsum += p;
            if (lane == 0) {
                idx[t * k + j] = be;
                w[t * k + j] = p;
            }
        }
        if (renorm && lane == 0)
            for (int j = 0; j < k; ++j) w[t * k + j] = w[t * k + j] / wsum;
    }
}

template <typename Tin, int NB>
hipError_t launch_route_nb(const void* x, int64_t T, int h, const void* wg, int E, int k,
                           const float* bias, int64_t bias_stride, int renorm, int32_t* idx,
                           float* w, hipStream_t s) {
    const int64_t per_block = kRouteWaves * kRouteTokensPerWave;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, per_block)));
    const size_t lds = sizeof(float) * kRouteWaves * kRouteTokensPerWave * (NB == 16 ? NB * 16 : NB * 16 + 1);
    hipLaunchKernelGGL((route_kernel<Tin, NB>), grid, dim3(kRouteWaves * kWave), lds, s,
                       static_cast<const Tin*>(x), static_cast<const Tin*>(wg), T, h, E, k, bias,
                       bias_stride, renorm, idx, w);
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_route_t(const void* x, int64_t T, int h, const void* wg, int E, int k,
                          const float* bias, int64_t bias_stride, int renorm, int32_t* idx,
                          float* w, hipStream_t s) {
    if (E <= 16) return launch_route_nb<Tin, 1>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    if (E <= 32) return launch_route_nb<Tin, 2>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    if (E <= 64) return launch_route_nb<Tin, 4>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    if (E <= 128) return launch_route_nb<Tin, 8>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    return launch_route_nb<Tin, 16>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
}

}  // namespace

hipError_t launch_route(const void* x, bool bf16, int64_t T, int h, const void* wg, int E, int k,
                        const float* bias, int64_t bias_stride, int renorm, int32_t* idx, float* w,
                        hipStream_t s) {
    if (T == 0) return hipSuccess;
    return bf16 ? launch_route_t<bf16_t>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s)
                : launch_route_t<float>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
}

}  // namespace moe
