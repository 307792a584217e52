// Step 4 of the layer: this device's shard of every expert on the rows routed to it, as a
// grouped GEMM over variable-length expert segments -- one launch per matmul, whatever
// the number of experts.
//
//   GEMM1   H[p, n] = act(x_perm[p] . W1^T[e][n])       (SwiGLU: silu(.W1) * (.W3))
//   GEMM2   y_perm[p, c] = H[p] . W2^T[e][c]
//
// Each workgroup first turns offsets[] into a per-expert prefix of row tiles (in LDS),
// then maps its linear tile id to (expert, row tile, column tile).  Tiles past the last
// real one exit at once, so the grid can be sized from the host-known bound A_max
// without reading the counts back.
//
// bf16 path: 128-row tiles, 4 waves in a 2 x 2 arrangement, v_mfma_f32_32x32x16_bf16
// with fp32 accumulation, K staged through double-buffered LDS in steps of 64 with the
// next step's global loads in flight during the current step's MFMAs.  The epilogue
// applies the activation in fp32, rounds once, and goes through LDS so that every global
// store is a full 16-byte row segment.
// fp32 path: the same scheduling over a plain LDS-tiled fp32 FMA kernel (64 x 64 tiles).
#include "common.h"
#include "kernels.h"

#include "../../include/moeshard.h"

#include <mutex>

namespace moe {
namespace {

enum Epi { kEpiGelu = 0, kEpiGeluTanh = 1, kEpiSwiglu = 2, kEpiNone = 3 };

struct GroupedGemm {
    const void* a;           // [rows][K]
    const void* b;           // [E][N rows][K]  (K-contiguous weights)
    const void* b2;          // SwiGLU up projection, same layout as b
    void* c;                 // [rows][ldc]
    const int32_t* offsets;  // [E + 1] row segment of every expert
    int E, K, N, ldc, n_tiles;
    int64_t b_estride;  // elements from one expert's weights to the next
    int64_t rows_max;   // rows of a and c; no row at or past it is touched
};

constexpr int kThreads = 256;

// Exclusive prefix over experts of ceil(count / BM) into tstart[0..E]; returns the total.
template <int BM>
__device__ __forceinline__ int tile_prefix(const int32_t* __restrict__ offsets, int E, int* tstart) {
    const int tid = threadIdx.x;
    int v = 0;
    if (tid < E) v = (offsets[tid + 1] - offsets[tid] + BM - 1) / BM;
    tstart[tid + 1] = v;
    if (tid == 0) tstart[0] = 0;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
        const int add = (tid >= o) ? tstart[tid + 1 - o] : 0;
        __syncthreads();
        tstart[tid + 1] += add;
        __syncthreads();
    }
    return tstart[E];
}

// Largest expert e with tstart[e] <= mt (an expert that owns row tile mt).
__device__ __forceinline__ int find_expert(const int* tstart, int E, int mt) {
    int lo = 0, hi = E - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (tstart[mid] <= mt) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

template <int EPI>
__device__ __forceinline__ float epilogue(float u, float g) {
    if (EPI == kEpiGelu) return act_gelu(u);
    if (EPI == kEpiGeluTanh) return act_gelu_tanh(u);
    if (EPI == kEpiSwiglu) return silu(u) * g;
    return u;
}

// ------------------------------------------------------------------ bf16 MFMA kernel

constexpr int kBM = 128;
constexpr int kBK = 64;
constexpr int kLDK = kBK + 8;  // LDS row stride (elements): 144 B keeps ds_read_b128 conflict-free

template <int EPI>
struct BfShape {
    static constexpr bool kDual = (EPI == kEpiSwiglu);
    static constexpr int kNB = kDual ? 2 : 1;     // weight matrices per tile
    static constexpr int kJN = kDual ? 1 : 2;     // 32-column MFMA blocks per wave per matrix
    static constexpr int kBN = 2 * 32 * kJN;      // output columns per tile
    static constexpr int kAVec = kBM * kBK / 8 / kThreads;   // 16-B vectors per thread (A)
    static constexpr int kBVec = kBN * kBK / 8 / kThreads;   // per matrix (B)
    static constexpr size_t kStageBytes = 2 * (size_t)(kBM + kNB * kBN) * kLDK * sizeof(bf16_t);
};

template <bool OB>
constexpr size_t bf_cstage_bytes(int bn) {
    return OB ? (size_t)kBM * (bn + 8) * 2 : (size_t)kBM * (bn + 4) * 4;
}

template <int EPI, bool OB>
constexpr size_t bf_lds_bytes() {
    return BfShape<EPI>::kStageBytes > bf_cstage_bytes<OB>(BfShape<EPI>::kBN)
               ? BfShape<EPI>::kStageBytes
               : bf_cstage_bytes<OB>(BfShape<EPI>::kBN);
}

template <int EPI, bool OB>
__global__ __launch_bounds__(kThreads, 2) void gemm_bf16(GroupedGemm g) {
    typedef BfShape<EPI> S;
    constexpr int NB = S::kNB, JN = S::kJN, BN = S::kBN;
    __shared__ int tstart[kThreads + 1];
    extern __shared__ __align__(16) unsigned char smem_raw[];
    bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);

    const int total = tile_prefix<kBM>(g.offsets, g.E, tstart);
    const int mt = blockIdx.x / g.n_tiles;
    const int nt = blockIdx.x - mt * g.n_tiles;
    if (mt >= total) return;
    const int e = find_expert(tstart, g.E, mt);
    const int64_t row0 = g.offsets[e] + static_cast<int64_t>(mt - tstart[e]) * kBM;
    const int64_t row_end = g.offsets[e + 1] < g.rows_max ? g.offsets[e + 1] : g.rows_max;
    if (row0 < 0 || row0 >= row_end) return;
    const int n0 = nt * BN;

    const bf16_t* __restrict__ A = static_cast<const bf16_t*>(g.a);
    const bf16_t* __restrict__ Bm[NB];
    Bm[0] = static_cast<const bf16_t*>(g.b) + e * g.b_estride;
    if (NB > 1) Bm[NB - 1] = static_cast<const bf16_t*>(g.b2) + e * g.b_estride;

    bf16_t* As = smem;                    // [2][kBM][kLDK]
    bf16_t* Bs = smem + 2 * kBM * kLDK;   // [2][NB][BN][kLDK]
    const int tid = threadIdx.x;

    uint4 ra[S::kAVec], rb[NB][S::kBVec];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < S::kAVec; ++i) {
            const int v = tid + i * kThreads;
            const int row = v >> 3, kc = (v & 7) * 8;
            const int64_t ar = row0 + row;
            ra[i] = (ar < row_end && k0 + kc < g.K)
                        ? *reinterpret_cast<const uint4*>(A + ar * g.K + k0 + kc)
                        : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < S::kBVec; ++i) {
                const int v = tid + i * kThreads;
                const int row = v >> 3, kc = (v & 7) * 8;
                const int n = n0 + row;
                rb[nb][i] = (n < g.N && k0 + kc < g.K)
                                ? *reinterpret_cast<const uint4*>(Bm[nb] + static_cast<int64_t>(n) * g.K + k0 + kc)
                                : make_uint4(0, 0, 0, 0);
            }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < S::kAVec; ++i) {
            const int v = tid + i * kThreads;
            const int row = v >> 3, kc = (v & 7) * 8;
            *reinterpret_cast<uint4*>(As + (buf * kBM + row) * kLDK + kc) = ra[i];
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < S::kBVec; ++i) {
                const int v = tid + i * kThreads;
                const int row = v >> 3, kc = (v & 7) * 8;
                *reinterpret_cast<uint4*>(Bs + ((buf * NB + nb) * BN + row) * kLDK + kc) = rb[nb][i];
            }
    };

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lhi = lane >> 5;

    f32x16_t acc[NB][2][JN];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < JN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[nb][i][j][r] = 0.f;

    const int nk = (g.K + kBK - 1) / kBK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kBK);
        const bf16_t* as = As + buf * kBM * kLDK;
#pragma unroll
        for (int ks = 0; ks < kBK / 16; ++ks) {
            bf16x8_t af[2], bfr[NB][JN];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                af[i] = *reinterpret_cast<const bf16x8_t*>(as + (wm * 64 + i * 32 + l32) * kLDK + ks * 16 + lhi * 8);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int j = 0; j < JN; ++j)
                    bfr[nb][j] = *reinterpret_cast<const bf16x8_t*>(
                        Bs + ((buf * NB + nb) * BN + wn * 32 * JN + j * 32 + l32) * kLDK + ks * 16 + lhi * 8);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < JN; ++j)
                        acc[nb][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[nb][j], acc[nb][i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) sstore(buf ^ 1);
        __syncthreads();
    }

    // Epilogue.  32x32 accumulator layout: lane holds column l32; register r holds row
    // 8 * (r / 4) + 4 * lhi + r % 4 of the block.
    if (OB) {
        constexpr int LDC = BN + 8;
        bf16_t* cs = smem;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < JN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = wm * 64 + i * 32 + (r >> 2) * 8 + lhi * 4 + (r & 3);
                    const int n = wn * 32 * JN + j * 32 + l32;
                    const float v = epilogue<EPI>(acc[0][i][j][r], acc[NB - 1][i][j][r]);
                    cs[m * LDC + n] = f32_to_bf16(v);
                }
        __syncthreads();
        constexpr int VPR = BN / 8;  // 16-B vectors per row
        bf16_t* C = static_cast<bf16_t*>(g.c);
#pragma unroll
        for (int q = 0; q < kBM * VPR / kThreads; ++q) {
            const int v = tid + q * kThreads;
            const int row = v / VPR, c8 = (v % VPR) * 8;
            if (row0 + row < row_end && n0 + c8 < g.N)
                *reinterpret_cast<uint4*>(C + (row0 + row) * g.ldc + n0 + c8) =
                    *reinterpret_cast<const uint4*>(cs + row * LDC + c8);
        }
    } else {
        constexpr int LDC = BN + 4;
        float* cs = reinterpret_cast<float*>(smem_raw);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < JN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = wm * 64 + i * 32 + (r >> 2) * 8 + lhi * 4 + (r & 3);
                    const int n = wn * 32 * JN + j * 32 + l32;
                    cs[m * LDC + n] = epilogue<EPI>(acc[0][i][j][r], acc[NB - 1][i][j][r]);
                }
        __syncthreads();
        constexpr int VPR = BN / 4;
        float* C = static_cast<float*>(g.c);
#pragma unroll
        for (int q = 0; q < kBM * VPR / kThreads; ++q) {
            const int v = tid + q * kThreads;
            const int row = v / VPR, c4 = (v % VPR) * 4;
            if (row0 + row < row_end && n0 + c4 < g.N)
                *reinterpret_cast<float4*>(C + (row0 + row) * g.ldc + n0 + c4) =
                    *reinterpret_cast<const float4*>(cs + row * LDC + c4);
        }
    }
}

// ------------------------------------------------------------------ fp32 kernel

constexpr int kFBM = 64, kFBN = 64, kFBK = 16;

template <int EPI, bool OB>
__global__ __launch_bounds__(kThreads) void gemm_f32(GroupedGemm g) {
    constexpr int NB = (EPI == kEpiSwiglu) ? 2 : 1;
    __shared__ int tstart[kThreads + 1];
    __shared__ __align__(16) float As[kFBK][kFBM + 4];
    __shared__ __align__(16) float Bs[NB][kFBK][kFBN + 4];

    const int total = tile_prefix<kFBM>(g.offsets, g.E, tstart);
    const int mt = blockIdx.x / g.n_tiles;
    const int nt = blockIdx.x - mt * g.n_tiles;
    if (mt >= total) return;
    const int e = find_expert(tstart, g.E, mt);
    const int64_t row0 = g.offsets[e] + static_cast<int64_t>(mt - tstart[e]) * kFBM;
    const int64_t row_end = g.offsets[e + 1] < g.rows_max ? g.offsets[e + 1] : g.rows_max;
    if (row0 < 0 || row0 >= row_end) return;
    const int n0 = nt * kFBN;
    const float* __restrict__ A = static_cast<const float*>(g.a);
    const float* __restrict__ Bm[NB];
    Bm[0] = static_cast<const float*>(g.b) + e * g.b_estride;
    if (NB > 1) Bm[NB - 1] = static_cast<const float*>(g.b2) + e * g.b_estride;

    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int lrow = tid >> 2, lk = (tid & 3) * 4;
    float acc[NB][4][4] = {};
    for (int k0 = 0; k0 < g.K; k0 += kFBK) {
        const bool kv = k0 + lk < g.K;
        const int64_t ar = row0 + lrow;
        const float4 a = (ar < row_end && kv) ? *reinterpret_cast<const float4*>(A + ar * g.K + k0 + lk)
                                              : make_float4(0.f, 0.f, 0.f, 0.f);
        As[lk + 0][lrow] = a.x;
        As[lk + 1][lrow] = a.y;
        As[lk + 2][lrow] = a.z;
        As[lk + 3][lrow] = a.w;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int n = n0 + lrow;
            const float4 b = (n < g.N && kv)
                                 ? *reinterpret_cast<const float4*>(Bm[nb] + static_cast<int64_t>(n) * g.K + k0 + lk)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
            Bs[nb][lk + 0][lrow] = b.x;
            Bs[nb][lk + 1][lrow] = b.y;
            Bs[nb][lk + 2][lrow] = b.z;
            Bs[nb][lk + 3][lrow] = b.w;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < kFBK; ++kk) {
            const float4 av = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
            const float ar4[4] = {av.x, av.y, av.z, av.w};
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const float4 bv = *reinterpret_cast<const float4*>(&Bs[nb][kk][tx * 4]);
                const float br4[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[nb][i][j] = fmaf(ar4[i], br4[j], acc[nb][i][j]);
            }
        }
        __syncthreads();
    }
    const int n = n0 + tx * 4;
    if (n >= g.N) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t row = row0 + ty * 4 + i;
        if (row >= row_end) break;
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = epilogue<EPI>(acc[0][i][j], acc[NB - 1][i][j]);
        if (OB) {
            uint2 q;
            q.x = pack_bf16x2(v[0], v[1]);
            q.y = pack_bf16x2(v[2], v[3]);
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.c) + row * g.ldc + n) = q;
        } else {
            *reinterpret_cast<float4*>(static_cast<float*>(g.c) + row * g.ldc + n) = make_float4(v[0], v[1], v[2], v[3]);
        }
    }
}

// ------------------------------------------------------------------ launch

int64_t row_tile_bound(int64_t A_max, int E, int bm) {
    const int64_t b = ceil_div(A_max, bm) + E;
    return b < A_max ? b : A_max;
}

template <int EPI, bool OB>
hipError_t run_bf16(GroupedGemm g, int64_t A_max, hipStream_t s) {
    typedef BfShape<EPI> S;
    constexpr size_t lds = bf_lds_bytes<EPI, OB>();
    static std::once_flag once;
    static hipError_t attr_err = hipSuccess;
    std::call_once(once, [] {
        attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16<EPI, OB>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    });
    if (attr_err != hipSuccess) return attr_err;
    g.n_tiles = static_cast<int>(ceil_div(g.N, S::kBN));
    const int64_t blocks = row_tile_bound(A_max, g.E, kBM) * g.n_tiles;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_bf16<EPI, OB>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, s, g);
    return hipGetLastError();
}

template <int EPI, bool OB>
hipError_t run_f32(GroupedGemm g, int64_t A_max, hipStream_t s) {
    g.n_tiles = static_cast<int>(ceil_div(g.N, kFBN));
    const int64_t blocks = row_tile_bound(A_max, g.E, kFBM) * g.n_tiles;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_f32<EPI, OB>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s, g);
    return hipGetLastError();
}

template <int EPI>
hipError_t gemm1(bool bf16, GroupedGemm g, int64_t A_max, hipStream_t s) {
    return bf16 ? run_bf16<EPI, true>(g, A_max, s) : run_f32<EPI, false>(g, A_max, s);
}

}  // namespace

hipError_t launch_ffn(const void* x_perm, const int32_t* offsets, int64_t A_max, int E, int h,
                      int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                      const void* w2t, void* y_perm, bool y_bf16, void* hbuf, hipStream_t s) {
    if (A_max == 0) return hipSuccess;
    GroupedGemm g1{};
    g1.a = x_perm;
    g1.b = w1t;
    g1.b2 = w3t;
    g1.c = hbuf;
    g1.offsets = offsets;
    g1.E = E;
    g1.K = h;
    g1.N = static_cast<int>(fp);
    g1.ldc = static_cast<int>(fp);
    g1.b_estride = fp * h;
    g1.rows_max = A_max;
    hipError_t err;
    if (act == MOE_ACT_SWIGLU) err = gemm1<kEpiSwiglu>(bf16, g1, A_max, s);
    else if (act == MOE_ACT_GELU_TANH) err = gemm1<kEpiGeluTanh>(bf16, g1, A_max, s);
    else err = gemm1<kEpiGelu>(bf16, g1, A_max, s);
    if (err != hipSuccess) return err;

    GroupedGemm g2{};
    g2.a = hbuf;
    g2.b = w2t;
    g2.b2 = nullptr;
    g2.c = y_perm;
    g2.offsets = offsets;
    g2.E = E;
    g2.K = static_cast<int>(fp);
    g2.N = h;
    g2.ldc = h;
    g2.b_estride = static_cast<int64_t>(h) * fp;
    g2.rows_max = A_max;
    if (bf16) return y_bf16 ? run_bf16<kEpiNone, true>(g2, A_max, s) : run_bf16<kEpiNone, false>(g2, A_max, s);
    return y_bf16 ? run_f32<kEpiNone, true>(g2, A_max, s) : run_f32<kEpiNone, false>(g2, A_max, s);
}

}  // namespace moe
