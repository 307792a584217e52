// Step 1 of the layer: gate logits, top-k selection and softmax weights.
//
// A workgroup of four waves routes 32 tokens.  The gate product
// logits[t, e] = x[t] . w_gate[e] runs on MFMA 32x32 blocks with fp32 accumulation; the
// K dimension is split across the four waves (wave w takes K chunks w, w + 4, ...), each
// wave keeping its 32 x E_pad partial block in accumulators with several chunks' loads in
// flight.  The partials meet in LDS and are summed in a fixed order.  Each token is then
// reduced by eight lanes: max and sum of exponentials for the softmax, then k rounds of
// arg-max over logit + bias in which the lower expert id wins ties.
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace moe {
namespace {

constexpr int kTok = 32;  // tokens per workgroup

template <typename Tin>
struct GateFrag;

// bf16: v_mfma_f32_32x32x16_bf16; lane (r = l % 32, g = l / 32) holds K values 8g .. 8g+7
template <>
struct GateFrag<bf16_t> {
    static constexpr int kStep = 16;
    typedef uint4 frag_t;
    static __device__ __forceinline__ frag_t load(const bf16_t* base, int64_t row, int64_t nrows, int h, int k) {
        if (row < nrows && k < h) return *reinterpret_cast<const uint4*>(base + row * h + k);
        return make_uint4(0, 0, 0, 0);
    }
    static __device__ __forceinline__ int lane_k(int k0, int g) { return k0 + g * 8; }
    static __device__ __forceinline__ f32x16_t mma(frag_t a, frag_t b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(b), c, 0, 0, 0);
    }
};

// fp32: four v_mfma_f32_32x32x2_f32 per float4; lane (r, g) supplies element c of its
// float4 (K index 4g + c of the chunk) to MFMA number c.  A and B use the same mapping,
// so the four products sum over all 8 K values of the chunk.
template <>
struct GateFrag<float> {
    static constexpr int kStep = 8;
    typedef float4 frag_t;
    static __device__ __forceinline__ frag_t load(const float* base, int64_t row, int64_t nrows, int h, int k) {
        if (row < nrows && k < h) return *reinterpret_cast<const float4*>(base + row * h + k);
        return make_float4(0.f, 0.f, 0.f, 0.f);
    }
    static __device__ __forceinline__ int lane_k(int k0, int g) { return k0 + g * 4; }
    static __device__ __forceinline__ f32x16_t mma(frag_t a, frag_t b, f32x16_t c) {
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, b.x, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, b.y, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, b.z, c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, b.w, c, 0, 0, 0);
        return c;
    }
};

constexpr int kWaves = 4;

template <int NB>
constexpr int route_ldw() { return NB * 32 + 8; }  // padded row: 8 token rows hit 8 bank groups

template <typename Tin, int NB>
__global__ __launch_bounds__(kWaves * kWave) void route_kernel(const Tin* __restrict__ x,
                                                               const Tin* __restrict__ wg, int64_t T, int h,
                                                               int E, int k, const float* __restrict__ bias,
                                                               int64_t bias_stride, int renorm,
                                                               int32_t* __restrict__ idx, float* __restrict__ w) {
    constexpr int EP = NB * 32;
    constexpr int LDW = route_ldw<NB>();
    constexpr int U = (NB == 1) ? 8 : (NB == 2) ? 4 : 2;  // K chunks in flight per wave
    constexpr int NV = EP / 8;                             // experts per lane in the epilogue
    extern __shared__ float part[];                        // [kWaves][kTok][LDW] partial logits
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kTok;
    const int r = lane & 31, g = lane >> 5;

    typedef GateFrag<Tin> F;
    f32x16_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[nb][i] = 0.f;

    for (int k0 = wave * F::kStep; k0 < h; k0 += kWaves * U * F::kStep) {
        typename F::frag_t a[U], b[U][NB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = F::lane_k(k0 + u * kWaves * F::kStep, g);
            a[u] = F::load(x, tok0 + r, T, h, kk);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) b[u][nb] = F::load(wg, nb * 32 + r, E, h, kk);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = F::mma(a[u], b[u][nb], acc[nb]);
    }

    // 32x32 accumulator layout: lane holds expert column r of each block; register i holds
    // token row 8 * (i / 4) + 4 * g + i % 4.
    float* mine = part + wave * kTok * LDW;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 16; ++i) mine[(8 * (i >> 2) + 4 * g + (i & 3)) * LDW + nb * 32 + r] = acc[nb][i];
    __syncthreads();

    // eight lanes per token: lane q = lane & 7 holds experts q, q + 8, q + 16, ...
    const int tt = wave * 8 + (lane >> 3), q = lane & 7;
    const int64_t t = tok0 + tt;
    float lv[NV], sv[NV];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int e = q + 8 * j;
        const int o = tt * LDW + e;
        const float v = ((part[o] + part[kTok * LDW + o]) + part[2 * kTok * LDW + o]) + part[3 * kTok * LDW + o];
        const bool ok = e < E;
        lv[j] = ok ? v : -INFINITY;
        sv[j] = ok ? ((bias && t < T) ? v + bias[t * bias_stride + e] : v) : -INFINITY;
        mx = fmaxf(mx, lv[j]);
    }
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    float den = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) den += (q + 8 * j < E) ? expf(lv[j] - mx) : 0.f;
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) den += __shfl_xor(den, o, kWave);

    uint32_t taken = 0;
    float wsum = 0.f;
    for (int j = 0; j < k; ++j) {
        float bs = -INFINITY, bl = -INFINITY;
        int be = 0x7fffffff;
#pragma unroll
        for (int jj = 0; jj < NV; ++jj) {
            const int e = q + 8 * jj;
            if (e < E && !((taken >> jj) & 1u) && (sv[jj] > bs || be == 0x7fffffff)) {
                bs = sv[jj];
                bl = lv[jj];
                be = e;
            }
        }
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) {
            const float os = __shfl_xor(bs, o, kWave);
            const float ol = __shfl_xor(bl, o, kWave);
            const int oe = __shfl_xor(be, o, kWave);
            if (oe != 0x7fffffff && (be == 0x7fffffff || os > bs || (os == bs && oe < be))) {
                bs = os;
                bl = ol;
                be = oe;
            }
        }
        const bool found = be != 0x7fffffff;
        if (found && (be & 7) == q) taken |= 1u << (be >> 3);
        const float p = found ? expf(bl - mx) / den : 0.f;
        wsum += p;
        if (q == 0 && t < T) {
            idx[t * k + j] = found ? be : -1;
            w[t * k + j] = p;
        }
    }
    if (renorm && q == 0 && t < T)
        for (int j = 0; j < k; ++j) w[t * k + j] = w[t * k + j] / wsum;
}

// ---------------------------------------------------------------- bf16, h % 64 == 0, E > 32
//
// A workgroup of four waves routes 64 tokens against all experts (padded to EP = 64 NBW).
// K advances in chunks of 64 (128 bytes of every row): each chunk of the 64 token rows and
// the EP gate rows goes straight to LDS with 1 KiB direct loads (8 rows x 128 bytes each),
// several chunks in flight.  Wave (wt, we) multiplies tokens 32 wt .. 32 wt + 31 by experts
// we EP/2 .. (we + 1) EP/2 - 1 on 32x32x16 MFMAs, gate rows as the first operand, so a lane
// ends up holding one token's logits.  The logits then go through LDS to the same per-token
// epilogue as above (eight lanes per token).  Token rows past T and gate rows past E are
// clamped to the last valid row; their results are never used.

constexpr int kRTok = 64;      // tokens per workgroup
constexpr int kRK = 64;        // K elements per chunk (128-byte rows)

template <int NBW>
struct RouteLds {
    static constexpr int EP = 64 * NBW;                  // padded experts
    static constexpr int kRows = kRTok + EP;             // LDS rows per chunk
    static constexpr int kChunkBytes = kRows * kRK * 2;
    // chunks in flight, sized so that two workgroups share a CU (one's epilogue then
    // overlaps the other's loads)
    static constexpr int kStages = NBW == 1 ? 4 : NBW == 2 ? 3 : 2;
    static constexpr int kLPW = kRows / 8 / 4;           // 1 KiB loads per wave per chunk
    static constexpr int kLDW = EP + 4;                  // logits row stride (floats)
    static constexpr size_t kStageBytes = (size_t)kStages * kChunkBytes;
    static constexpr size_t kLogitBytes = (size_t)kRTok * kLDW * 4;
    static constexpr size_t kBytes = kStageBytes > kLogitBytes ? kStageBytes : kLogitBytes;
};

template <int NBW>
__global__ __launch_bounds__(kWaves * kWave) void route_lds_kernel(const bf16_t* __restrict__ x,
                                                                   const bf16_t* __restrict__ wg, int64_t T,
                                                                   int h, int E, int k,
                                                                   const float* __restrict__ bias,
                                                                   int64_t bias_stride, int renorm,
                                                                   int32_t* __restrict__ idx,
                                                                   float* __restrict__ w) {
    typedef RouteLds<NBW> S;
    constexpr int EP = S::EP, LPW = S::kLPW, LDW = S::kLDW, NS = S::kStages;
    constexpr int kXJ = kRTok / 8 / 4;  // loads per wave per chunk that carry token rows
    extern __shared__ __align__(1024) unsigned char smem[];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kRTok;
    const uint32_t lds0 = lds_address(smem);
    const int nk = h / kRK;

    // per-lane offsets of this wave's loads: load j fills LDS rows 8 (4 j + wave) + lane / 8
    // of a chunk, 16-byte slot lane % 8, with global chunk slot ^ swz(row)
    uint32_t voff[LPW];
    {
        const int t_lim = static_cast<int>(T - tok0 < kRTok ? T - tok0 : kRTok) - 1;
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
            const int R = 8 * (4 * j + wave) + (lane >> 3);
            const int kc = (lane & 7) ^ ((R >> 1) & 7);
            const int r = j < kXJ ? min(R, t_lim) : min(R - kRTok, E - 1);
            voff[j] = static_cast<uint32_t>(r) * static_cast<uint32_t>(2 * h) + static_cast<uint32_t>(kc * 16);
        }
    }
    const unsigned char* xb = uniform_ptr(reinterpret_cast<const unsigned char*>(x + tok0 * h));
    const unsigned char* gb = uniform_ptr(reinterpret_cast<const unsigned char*>(wg));
    // every workgroup walks K in the same order, so a token's logits are summed in the same
    // order wherever it sits in the batch (its picks do not depend on T or its position)
    int issued = 0;
    auto issue = [&]() {
        const uint32_t dst = lds0 + (issued % NS) * S::kChunkBytes;
        const int kb = issued * kRK * 2;
#pragma unroll
        for (int j = 0; j < LPW; ++j)
            load_lds16((j < kXJ ? xb : gb) + kb, voff[j], dst + (4 * j + wave) * 1024);
        ++issued;
    };
#pragma unroll
    for (int st = 0; st < NS - 1; ++st)
        if (issued < nk) issue();

    // Each epilogue lane owns NV consecutive experts of one token (two passes of 32 tokens).
    // The selection bias of those tokens is fetched now, in contiguous runs per lane, so
    // that its latency hides behind the K loop.
    constexpr int NV = EP / 8;
    const int q = lane & 7;
    float bv[2][NV];
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int64_t t = tok0 + pass * 32 + wave * 8 + (lane >> 3);
        const int e0 = NV * q;
        const float* bp = bias ? bias + t * bias_stride + e0 : nullptr;
        if (bias && t < T && e0 + NV <= E && (reinterpret_cast<uintptr_t>(bp) & 15u) == 0) {
#pragma unroll
            for (int j = 0; j < NV; j += 4) {
                const float4 v = *reinterpret_cast<const float4*>(bp + j);
                bv[pass][j] = v.x;
                bv[pass][j + 1] = v.y;
                bv[pass][j + 2] = v.z;
                bv[pass][j + 3] = v.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < NV; ++j) bv[pass][j] = (bias && t < T && e0 + j < E) ? bp[j] : 0.f;
        }
    }

    const int wt = wave & 1, we = wave >> 1;
    const int l32 = lane & 31, lhi = lane >> 5;
    f32x16_t acc[NBW];
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[b][i] = 0.f;

    for (int kc = 0; kc < nk; ++kc) {
        wait_stages<LPW, NS>(issued - kc - 1);
        stage_barrier();
        if (issued < nk) issue();
        const unsigned char* st = smem + (kc % NS) * S::kChunkBytes;
#pragma unroll
        for (int ks = 0; ks < kRK / 16; ++ks) {
            const int ch = 2 * ks + lhi;
            const int Rt = 32 * wt + l32;
            const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(st + Rt * 128 + ((ch ^ ((Rt >> 1) & 7)) << 4));
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const int Re = kRTok + we * (EP / 2) + 32 * b + l32;
                const bf16x8_t gf =
                    *reinterpret_cast<const bf16x8_t*>(st + Re * 128 + ((ch ^ ((Re >> 1) & 7)) << 4));
                acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(gf, xf, acc[b], 0, 0, 0);
            }
        }
    }

    // logits to LDS: D[expert][token] layout, lane = token 32 wt + l32, register i = expert
    // we EP/2 + 32 b + 8 (i / 4) + 4 lhi + i % 4
    stage_barrier();  // every wave is done reading the last chunk
    float* part = reinterpret_cast<float*>(smem);
#pragma unroll
    for (int b = 0; b < NBW; ++b)
#pragma unroll
        for (int i = 0; i < 16; ++i)
            part[(32 * wt + l32) * LDW + we * (EP / 2) + 32 * b + 8 * (i >> 2) + 4 * lhi + (i & 3)] = acc[b][i];
    __syncthreads();

    // eight lanes per token, 32 tokens per pass; lane q holds experts NV q .. NV q + NV - 1
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
        const int tt = pass * 32 + wave * 8 + (lane >> 3);
        const int64_t t = tok0 + tt;
        float lv[NV], sv[NV];
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < NV; ++j) {
            const int e = NV * q + j;
            const float v = part[tt * LDW + e];
            const bool ok = e < E;
            lv[j] = ok ? v : -INFINITY;
            sv[j] = ok ? v + bv[pass][j] : -INFINITY;
            mx = fmaxf(mx, lv[j]);
        }
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
        float den = 0.f;
#pragma unroll
        for (int j = 0; j < NV; ++j) den += (NV * q + j < E) ? expf(lv[j] - mx) : 0.f;
#pragma unroll
        for (int o = 1; o < 8; o <<= 1) den += __shfl_xor(den, o, kWave);

        // k rounds of arg-max over the selection score; equal scores -> lower expert id
        // (each lane scans its experts upward with a strict comparison, and the lane
        // reduction prefers the lower id on ties)
        uint32_t taken = 0;
        float wsum = 0.f;
        for (int j = 0; j < k; ++j) {
            float bs = -INFINITY, bl = -INFINITY;
            int be = 0x7fffffff;
#pragma unroll
            for (int jj = 0; jj < NV; ++jj) {
                const int e = NV * q + jj;
                if (e < E && !((taken >> jj) & 1u) && (sv[jj] > bs || be == 0x7fffffff)) {
                    bs = sv[jj];
                    bl = lv[jj];
                    be = e;
                }
            }
#pragma unroll
            for (int o = 1; o < 8; o <<= 1) {
                const float os = __shfl_xor(bs, o, kWave);
                const float ol = __shfl_xor(bl, o, kWave);
                const int oe = __shfl_xor(be, o, kWave);
                if (oe != 0x7fffffff && (be == 0x7fffffff || os > bs || (os == bs && oe < be))) {
                    bs = os;
                    bl = ol;
                    be = oe;
                }
            }
            const bool found = be != 0x7fffffff;
            if (found && be / NV == q) taken |= 1u << (be - NV * q);
            const float p = found ? expf(bl - mx) / den : 0.f;
            wsum += p;
            if (q == 0 && t < T) {
                idx[t * k + j] = found ? be : -1;
                w[t * k + j] = p;
            }
        }
        if (renorm && q == 0 && t < T)
            for (int j = 0; j < k; ++j) w[t * k + j] = w[t * k + j] / wsum;
    }
}

template <int NBW>
hipError_t launch_route_lds(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                            int64_t bias_stride, int renorm, int32_t* idx, float* w, hipStream_t s) {
    constexpr size_t lds = RouteLds<NBW>::kBytes;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&route_lds_kernel<NBW>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                                       static_cast<int>(lds));
    if (attr != hipSuccess) return attr;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kRTok)));
    hipLaunchKernelGGL((route_lds_kernel<NBW>), grid, dim3(kWaves * kWave), lds, s, static_cast<const bf16_t*>(x),
                       static_cast<const bf16_t*>(wg), T, h, E, k, bias, bias_stride, renorm, idx, w);
    return hipGetLastError();
}

template <typename Tin, int NB>
hipError_t launch_route_nb(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                           int64_t bias_stride, int renorm, int32_t* idx, float* w, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kTok)));
    const size_t lds = sizeof(float) * kWaves * kTok * route_ldw<NB>();
    if (lds > 64 * 1024) {
        static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&route_kernel<Tin, NB>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     static_cast<int>(lds));
        if (attr != hipSuccess) return attr;
    }
    hipLaunchKernelGGL((route_kernel<Tin, NB>), grid, dim3(kWaves * kWave), lds, s, static_cast<const Tin*>(x),
                       static_cast<const Tin*>(wg), T, h, E, k, bias, bias_stride, renorm, idx, w);
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_route_t(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                          int64_t bias_stride, int renorm, int32_t* idx, float* w, hipStream_t s) {
    if (E <= 32) return launch_route_nb<Tin, 1>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    if (E <= 64) return launch_route_nb<Tin, 2>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    if (E <= 128) return launch_route_nb<Tin, 4>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    return launch_route_nb<Tin, 8>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
}

}  // namespace

hipError_t launch_route(const void* x, bool bf16, int64_t T, int h, const void* wg, int E, int k,
                        const float* bias, int64_t bias_stride, int renorm, int32_t* idx, float* w,
                        hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (bf16 && h % kRK == 0 && E > 32) {
        if (E <= 64) return launch_route_lds<1>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
        if (E <= 128) return launch_route_lds<2>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
        return launch_route_lds<4>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
    }
    return bf16 ? launch_route_t<bf16_t>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s)
                : launch_route_t<float>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
}

}  // namespace moe
