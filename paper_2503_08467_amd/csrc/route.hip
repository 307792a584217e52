// Step 1 of the layer: gate logits, top-k selection and softmax weights.
//
// route_kernel: a workgroup of RW waves (8 for at most 64 experts, else 4) routes 32
// tokens.  The gate product logits[t, e] = x[t] . w_gate[e] runs on MFMA 32x32 blocks with
// fp32 accumulation; the K dimension is split across the waves (wave w takes K chunks w,
// w + RW, ...), each wave keeping its 32 x E_pad partial block in accumulators with several
// chunks' loads in flight.  The partials meet in LDS and are summed in wave order.  Each
// token is then reduced by eight lanes of the first four waves: max and sum of exponentials
// for the softmax, then k rounds of arg-max over logit + bias in which the lower expert id
// wins ties.  route_lds_kernel (bf16, h % 64 == 0, more than 32 experts) is described below.
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

#include "../../include/moeshard.h"

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
constexpr int kNoExpert = 0x7fffffff;
constexpr int kRegPicks = 8;  // picks kept in registers (one per lane of a token's group)

// A token's picks as held by one lane of its group: pick q of the token (lane q), and the
// sum of the k pick weights.
struct Picks {
    int e;
    float p, wsum;
};

// Step 1's selection for one token, eight lanes per token: lane q of the group holds NV
// logits lv[] (-inf for padding) and selection scores sv[] = logit + bias for experts
// M::ex(q, j).  Softmax over the logits, then k rounds of arg-max over the scores in which
// the lower expert id wins ties (each lane scans its experts upward with a strict
// comparison, and the lane reduction prefers the lower id on ties); the weight of a pick is
// the softmax of its logit.  With k <= kRegPicks lane q keeps pick q and the caller stores
// it (store_pick) once every token of the workgroup is done, so no store waits on another;
// a larger k writes each pick as it is found and renormalises through memory afterwards.
template <int NV, typename M>
__device__ __forceinline__ Picks select_token(const float (&lv)[NV], const float (&sv)[NV], int q, int E, int k,
                                              int renorm, bool live, int64_t t, int32_t* __restrict__ idx,
                                              float* __restrict__ w) {
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < NV; ++j) mx = fmaxf(mx, lv[j]);
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    float den = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) den += (M::ex(q, j) < E) ? expf(lv[j] - mx) : 0.f;
#pragma unroll
    for (int o = 1; o < 8; o <<= 1) den += __shfl_xor(den, o, kWave);

    Picks r{-1, 0.f, 0.f};
    uint32_t taken = 0;
    float wsum = 0.f;
    for (int j = 0; j < k; ++j) {
        float bs = -INFINITY, bl = -INFINITY;
        int be = kNoExpert;
#pragma unroll
        for (int jj = 0; jj < NV; ++jj) {
            const int e = M::ex(q, jj);
            if (e < E && !((taken >> jj) & 1u) && (sv[jj] > bs || be == kNoExpert)) {
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
            if (oe != kNoExpert && (be == kNoExpert || os > bs || (os == bs && oe < be))) {
                bs = os;
                bl = ol;
                be = oe;
            }
        }
        const bool found = be != kNoExpert;
        if (found && M::owner(be) == q) taken |= 1u << M::slot(be);
        const float p = found ? expf(bl - mx) / den : 0.f;
        wsum += p;
        if (j == q) {
            r.e = found ? be : -1;
            r.p = p;
        }
        if (k > kRegPicks && q == 0 && live) {
            idx[t * k + j] = found ? be : -1;
            w[t * k + j] = p;
        }
    }
    r.wsum = wsum;
    if (k > kRegPicks && renorm && q == 0 && live)
        for (int j = 0; j < k; ++j) w[t * k + j] = w[t * k + j] / wsum;
    return r;
}

// Lane q's pick of its token (k <= kRegPicks): idx[t k + q], w[t k + q], renormalised over
// the k picks on request.
__device__ __forceinline__ void store_pick(const Picks& r, int q, int k, int renorm, bool live, int64_t t,
                                           int32_t* __restrict__ idx, float* __restrict__ w) {
    if (k <= kRegPicks && live && q < k) {
        idx[t * k + q] = r.e;
        w[t * k + q] = renorm ? r.p / r.wsum : r.p;
    }
}

// Lane exchanges inside a quad (four consecutive lanes) as DPP operand moves: a VALU
// instruction each, no LDS round trip.
constexpr int kDppXor1 = 0xB1;  // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;  // quad_perm [2, 3, 0, 1]

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}

// Arg-max step between quad partners: the higher score, the lower expert id on ties, a
// lane without a candidate (kNoExpert) losing to any other.  Symmetric, so both partners
// end with the same winner.
template <int CTRL>
__device__ __forceinline__ void quad_best(float& bs, float& bl, int& be) {
    const float os = dpp_f<CTRL>(bs);
    const float ol = dpp_f<CTRL>(bl);
    const int oe = dpp_i<CTRL>(be);
    const bool other = oe != kNoExpert && (be == kNoExpert || os > bs || (os == bs && oe < be));
    bs = other ? os : bs;
    bl = other ? ol : bl;
    be = other ? oe : be;
}

constexpr int kQuadPicks = 8;  // picks kept in registers with four lanes per token (two each)

struct QuadPicks {
    int e0, e1;  // picks q and q + 4 of the token
    float p0, p1, wsum;
};

// Step 1's selection with four lanes per token (a quad): lane q holds the logits lv[] and
// selection scores sv[] = logit + bias of experts NV q .. NV q + NV - 1 (sv = -inf for
// padding, whose lv is never used).  Every choice below is a select, not a branch: a
// branch around each element would serialise the LDS reads and exponentials.  Softmax
// over the logits (exponentials in base 2: e^(l - m) = 2^((l - m) log2 e)), then k rounds of
// arg-max over the scores in which the lower expert id wins ties; a pick's weight is the
// softmax of its logit.  Lane q keeps picks q and q + 4; with k > kQuadPicks every pick is
// written as it is found and renormalised through memory afterwards.
template <int NV>
__device__ __forceinline__ QuadPicks select_quad(const float (&lv)[NV], const float (&sv)[NV], int q, int E, int k,
                                                 int renorm, bool live, int64_t t, int32_t* __restrict__ idx,
                                                 float* __restrict__ w) {
    constexpr float kLog2e = 1.4426950408889634f;
    const int e0 = NV * q;
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < NV; ++j) mx = fmaxf(mx, lv[j]);
    mx = fmaxf(mx, dpp_f<kDppXor1>(mx));
    mx = fmaxf(mx, dpp_f<kDppXor2>(mx));
    float den = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const float x = __builtin_amdgcn_exp2f((lv[j] - mx) * kLog2e);
        den += e0 + j < E ? x : 0.f;
    }
    den += dpp_f<kDppXor1>(den);
    den += dpp_f<kDppXor2>(den);

    QuadPicks r{-1, -1, 0.f, 0.f, 0.f};
    uint64_t taken = 0;
    float wsum = 0.f;
    for (int j = 0; j < k; ++j) {
        float bs = -INFINITY, bl = -INFINITY;
        int be = kNoExpert;
#pragma unroll
        for (int jj = 0; jj < NV; ++jj) {
            const bool take = e0 + jj < E && !((taken >> jj) & 1u) && (sv[jj] > bs || be == kNoExpert);
            bs = take ? sv[jj] : bs;
            bl = take ? lv[jj] : bl;
            be = take ? e0 + jj : be;
        }
        quad_best<kDppXor1>(bs, bl, be);
        quad_best<kDppXor2>(bs, bl, be);
        const bool found = be != kNoExpert;
        const int rel = be - e0;
        taken |= (found && rel >= 0 && rel < NV) ? (1ull << rel) : 0ull;
        const float p = found ? __builtin_amdgcn_exp2f((bl - mx) * kLog2e) / den : 0.f;
        wsum += p;
        const int pe = found ? be : -1;
        r.e0 = j == q ? pe : r.e0;
        r.p0 = j == q ? p : r.p0;
        r.e1 = j == q + 4 ? pe : r.e1;
        r.p1 = j == q + 4 ? p : r.p1;
        if (k > kQuadPicks && q == 0 && live) {
            idx[t * k + j] = pe;
            w[t * k + j] = p;
        }
    }
    r.wsum = wsum;
    if (k > kQuadPicks && renorm && q == 0 && live)
        for (int j = 0; j < k; ++j) w[t * k + j] = w[t * k + j] / wsum;
    return r;
}

// Expert of lane q's j-th logit: experts q, q + 8, q + 16, ...; owner and slot invert it.
template <int NV>
struct StridedExperts {
    static __device__ __forceinline__ int ex(int q, int j) { return q + 8 * j; }
    static __device__ __forceinline__ int owner(int e) { return e & 7; }
    static __device__ __forceinline__ int slot(int e) { return e >> 3; }
};

template <int NB>
constexpr int route_ldw() { return NB * 32 + 8; }  // padded row: 8 token rows hit 8 bank groups

// Waves of route_kernel: 8 (each a K eighth) when its partial logits fit LDS comfortably,
// else 4.  The first four waves run the epilogue.
template <int NB>
constexpr int route_waves() { return NB <= 2 ? 8 : kWaves; }

template <typename Tin, int NB>
__global__ __launch_bounds__(route_waves<NB>() * kWave) void route_kernel(const Tin* __restrict__ x,
                                                               const Tin* __restrict__ wg, int64_t T, int h,
                                                               int E, int k, const float* __restrict__ bias,
                                                               int64_t bias_stride, int renorm,
                                                               int32_t* __restrict__ idx, float* __restrict__ w) {
    constexpr int EP = NB * 32;
    constexpr int LDW = route_ldw<NB>();
    constexpr int U = (NB == 1) ? 8 : (NB == 2) ? 4 : 2;  // K chunks in flight per wave
    constexpr int NV = EP / 8;                             // experts per lane in the epilogue
    constexpr int RW = route_waves<NB>();
    extern __shared__ float part[];                        // [RW][kTok][LDW] partial logits
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int64_t tok0 = static_cast<int64_t>(blockIdx.x) * kTok;
    const int r = lane & 31, g = lane >> 5;

    typedef GateFrag<Tin> F;
    // The epilogue's token and experts of this lane (waves 0..3): token tt, experts q, q + 8,
    // ...  Their selection bias is loaded now, from clamped addresses (entries past T or E
    // are loaded but never used), so that its latency hides behind the K loop instead of
    // costing a round trip per expert at the end.
    const int tt = wave * 8 + (lane >> 3), q = lane & 7;
    const int64_t t = tok0 + tt;
    float bv[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) bv[j] = 0.f;
    if (bias && wave < kTok / 8) {
        const float* bp = bias + (t < T ? t : T - 1) * bias_stride;
#pragma unroll
        for (int j = 0; j < NV; ++j) bv[j] = bp[min(q + 8 * j, E - 1)];
    }

    f32x16_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[nb][i] = 0.f;

    for (int k0 = wave * F::kStep; k0 < h; k0 += RW * U * F::kStep) {
        typename F::frag_t a[U], b[U][NB];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kk = F::lane_k(k0 + u * RW * F::kStep, g);
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

    if (wave >= kTok / 8) return;
    // eight lanes per token: lane q = lane & 7 holds experts q, q + 8, q + 16, ...
    float lv[NV], sv[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        const int e = q + 8 * j;
        const int o = tt * LDW + e;
        float v = part[o];  // the waves' partial sums in wave order
#pragma unroll
        for (int p = 1; p < RW; ++p) v += part[p * kTok * LDW + o];
        const bool ok = e < E;
        lv[j] = ok ? v : -INFINITY;
        sv[j] = ok ? v + bv[j] : -INFINITY;  // bv = 0 without a bias
    }
    const Picks pk = select_token<NV, StridedExperts<NV>>(lv, sv, q, E, k, renorm, t < T, t, idx, w);
    store_pick(pk, q, k, renorm, t < T, t, idx, w);
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

typedef RouteDispatchOut FusedDispatch;  // counts == nullptr: routing only
constexpr int kFusedGroups = kRTok * kQuadPicks / 64;  // groups of 64 assignments, at most
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

template <int NBW, int BIAS>
__global__ __launch_bounds__(kWaves * kWave) void route_lds_kernel(const bf16_t* __restrict__ x,
                                                                   const bf16_t* __restrict__ wg, int64_t T,
                                                                   int h, int E, int k,
                                                                   const float* __restrict__ bias,
                                                                   int64_t bias_stride, int renorm,
                                                                   int32_t* __restrict__ idx,
                                                                   float* __restrict__ w, FusedDispatch fd) {
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

    // Each epilogue lane owns NV consecutive experts of one token (four lanes per token, the
    // workgroup's 64 tokens in one pass).  The selection bias of those experts is fetched
    // now, behind the first stages, so that its latency hides behind the K loop: plain loads
    // from clamped addresses (entries past T or E are loaded but never used) and nothing that
    // reads the registers before the epilogue -- a select or a conditional copy here would
    // make the wave wait for every load in flight, the stages included.  BIAS: 0 none, 1
    // scalar loads, 2 16-byte loads (bias 16-byte aligned, E and the row stride multiples
    // of 4: a group starting below E then lies inside the row).
    constexpr int NV = EP / 4;
    const int q = lane & 3;
    const int tt = wave * 16 + (lane >> 2);
    const int64_t t = tok0 + tt;
    float bv[NV];
    if constexpr (BIAS == 0) {
#pragma unroll
        for (int j = 0; j < NV; ++j) bv[j] = 0.f;
    } else {
        const float* bp = bias + (t < T ? t : T - 1) * bias_stride;
        if constexpr (BIAS == 2) {
#pragma unroll
            for (int j = 0; j < NV; j += 4) {
                const float4 v = *reinterpret_cast<const float4*>(bp + min(NV * q + j, E - 4));
                bv[j] = v.x;
                bv[j + 1] = v.y;
                bv[j + 2] = v.z;
                bv[j + 3] = v.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < NV; ++j) bv[j] = bp[min(NV * q + j, E - 1)];
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
        // every fragment of the chunk is read before its MFMAs (one LDS latency per chunk)
        const unsigned char* st = smem + (kc % NS) * S::kChunkBytes;
        bf16x8_t xf[kRK / 16], gf[kRK / 16][NBW];
#pragma unroll
        for (int ks = 0; ks < kRK / 16; ++ks) {
            const int ch = 2 * ks + lhi;
            const int Rt = 32 * wt + l32;
            xf[ks] = *reinterpret_cast<const bf16x8_t*>(st + Rt * 128 + ((ch ^ ((Rt >> 1) & 7)) << 4));
#pragma unroll
            for (int b = 0; b < NBW; ++b) {
                const int Re = kRTok + we * (EP / 2) + 32 * b + l32;
                gf[ks][b] = *reinterpret_cast<const bf16x8_t*>(st + Re * 128 + ((ch ^ ((Re >> 1) & 7)) << 4));
            }
        }
        __builtin_amdgcn_sched_barrier(0);  // keep the reads ahead of the MFMAs
#pragma unroll
        for (int ks = 0; ks < kRK / 16; ++ks)
#pragma unroll
            for (int b = 0; b < NBW; ++b) acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(gf[ks][b], xf[ks], acc[b], 0, 0, 0);
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

    // four lanes per token; lane q holds experts NV q .. NV q + NV - 1 of token tt (read
    // whole, padding included: the row has EP + 4 entries)
    const float* lrow = part + tt * LDW + NV * q;
    float lv[NV], sv[NV];
#pragma unroll
    for (int j = 0; j < NV; j += 4) {
        const float4 v = *reinterpret_cast<const float4*>(lrow + j);
        lv[j] = v.x;
        lv[j + 1] = v.y;
        lv[j + 2] = v.z;
        lv[j + 3] = v.w;
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
        sv[j] = NV * q + j < E ? lv[j] + bv[j] : -INFINITY;
        lv[j] = NV * q + j < E ? lv[j] : -INFINITY;
    }
    const QuadPicks r = select_quad<NV>(lv, sv, q, E, k, renorm, t < T, t, idx, w);
    if (k <= kQuadPicks && t < T) {
        if (q < k) {
            idx[t * k + q] = r.e0;
            w[t * k + q] = renorm ? r.p0 / r.wsum : r.p0;
        }
        if (q + 4 < k) {
            idx[t * k + q + 4] = r.e1;
            w[t * k + q + 4] = renorm ? r.p1 / r.wsum : r.p1;
        }
    }
    if (fd.counts == nullptr) return;

    // ---- Step 2 in the same launch (this workgroup routed the whole batch): group the A = T k
    // assignments per expert, stable in (t, j) order -- the same counts, offsets, row_src and
    // pos_of as moe_dispatch -- from the picks still in registers.  The LDS of the logit
    // table is reused once every wave is done with it.
    __syncthreads();
    int* const sp = reinterpret_cast<int*>(smem);     // [T k] the picks, assignment a = t k + j
    int* const hist = sp + kRTok * kQuadPicks;         // [E] assignments per expert
    int* const off = hist + MOE_MAX_EXPERTS;           // [E + 1] exclusive prefix
    int* const gcnt = off + MOE_MAX_EXPERTS + 1;       // [group][E] count within each group of 64
    const int A = static_cast<int>(T) * k;
    if (t < T) {
        if (q < k) sp[tt * k + q] = r.e0;
        if (q + 4 < k) sp[tt * k + q + 4] = r.e1;
    }
    for (int e = threadIdx.x; e < MOE_MAX_EXPERTS; e += kWaves * kWave) hist[e] = 0;
    for (int i = threadIdx.x; i < kFusedGroups * MOE_MAX_EXPERTS; i += kWaves * kWave) gcnt[i] = 0;
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    __syncthreads();
    const int ngroups = (A + 63) / 64;
    for (int gi = wave; gi < ngroups; gi += kWaves) {  // wave-uniform
        const int a = gi * 64 + lane;
        const int e = a < A ? sp[a] : -1;
        const bool valid = static_cast<unsigned>(e) < static_cast<unsigned>(E);
        const uint64_t peers = same_expert_lanes(e, valid, nbits);
        if (valid && __popcll(peers & lt) == 0) {
            gcnt[gi * MOE_MAX_EXPERTS + e] = __popcll(peers);
            atomicAdd(&hist[e], __popcll(peers));
        }
    }
    __syncthreads();
    static_assert(MOE_MAX_EXPERTS == 4 * kWave, "four experts per lane of one wave");
    if (wave == 0) {
        int ex[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            ex[i] = sum;
            sum += (e < E) ? hist[e] : 0;
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int v = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += v;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            if (e < E) off[e] = incl - sum + ex[i];
        }
        if (lane == kWave - 1) off[E] = incl;
    }
    __syncthreads();
    for (int e = threadIdx.x; e <= E; e += kWaves * kWave) {
        fd.offsets[e] = off[e];
        if (e < E) fd.counts[e] = hist[e];
    }
    for (int gi = wave; gi < ngroups; gi += kWaves) {
        const int a = gi * 64 + lane;
        const int e = a < A ? sp[a] : -1;
        const bool valid = static_cast<unsigned>(e) < static_cast<unsigned>(E);
        const uint64_t peers = same_expert_lanes(e, valid, nbits);
        if (valid) {
            int pos = off[e] + __popcll(peers & lt);
            for (int g2 = 0; g2 < gi; ++g2) pos += gcnt[g2 * MOE_MAX_EXPERTS + e];
            fd.pos_of[a] = pos;
            fd.row_src[pos] = a / k;
        } else if (a < A) {
            fd.pos_of[a] = -1;
        }
    }
}

template <int NBW, int BIAS>
hipError_t launch_route_lds_b(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                              int64_t bias_stride, int renorm, int32_t* idx, float* w, FusedDispatch fd,
                              hipStream_t s) {
    constexpr size_t lds = RouteLds<NBW>::kBytes;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&route_lds_kernel<NBW, BIAS>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                                       static_cast<int>(lds));
    if (attr != hipSuccess) return attr;
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kRTok)));
    hipLaunchKernelGGL((route_lds_kernel<NBW, BIAS>), grid, dim3(kWaves * kWave), lds, s,
                       static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(wg), T, h, E, k, bias, bias_stride,
                       renorm, idx, w, fd);
    return hipGetLastError();
}

template <int NBW>
hipError_t launch_route_lds(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                            int64_t bias_stride, int renorm, int32_t* idx, float* w, FusedDispatch fd, hipStream_t s) {
    if (!bias) return launch_route_lds_b<NBW, 0>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
    if ((reinterpret_cast<uintptr_t>(bias) & 15u) == 0 && E % 4 == 0 && bias_stride % 4 == 0)
        return launch_route_lds_b<NBW, 2>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
    return launch_route_lds_b<NBW, 1>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
}

template <typename Tin, int NB>
hipError_t launch_route_nb(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                           int64_t bias_stride, int renorm, int32_t* idx, float* w, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(ceil_div(T, kTok)));
    const size_t lds = sizeof(float) * route_waves<NB>() * kTok * route_ldw<NB>();
    if (lds > 64 * 1024) {
        static hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&route_kernel<Tin, NB>),
                                                     hipFuncAttributeMaxDynamicSharedMemorySize,
                                                     static_cast<int>(lds));
        if (attr != hipSuccess) return attr;
    }
    hipLaunchKernelGGL((route_kernel<Tin, NB>), grid, dim3(route_waves<NB>() * kWave), lds, s, static_cast<const Tin*>(x),
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

static hipError_t route_any(const void* x, bool bf16, int64_t T, int h, const void* wg, int E, int k,
                            const float* bias, int64_t bias_stride, int renorm, int32_t* idx, float* w,
                            FusedDispatch fd, hipStream_t s) {
    if (T == 0) return hipSuccess;
    if (bf16 && h % kRK == 0 && E > 32) {
        if (E <= 64) return launch_route_lds<1>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
        if (E <= 128) return launch_route_lds<2>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
        return launch_route_lds<4>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, fd, s);
    }
    return bf16 ? launch_route_t<bf16_t>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s)
                : launch_route_t<float>(x, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, s);
}

hipError_t launch_route(const void* x, bool bf16, int64_t T, int h, const void* wg, int E, int k,
                        const float* bias, int64_t bias_stride, int renorm, int32_t* idx, float* w,
                        hipStream_t s) {
    return route_any(x, bf16, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, FusedDispatch{}, s);
}

bool route_dispatch_fusable(bool bf16, int64_t T, int h, int E, int k) {
    return bf16 && h % kRK == 0 && E > 32 && E <= MOE_MAX_EXPERTS && T >= 1 && T <= kRTok && k <= kQuadPicks;
}

hipError_t launch_route_dispatch(const void* x, int64_t T, int h, const void* wg, int E, int k, const float* bias,
                                 int64_t bias_stride, int renorm, int32_t* idx, float* w, RouteDispatchOut out,
                                 hipStream_t s) {
    return route_any(x, true, T, h, wg, E, k, bias, bias_stride, renorm, idx, w, out, s);
}

}  // namespace moe
