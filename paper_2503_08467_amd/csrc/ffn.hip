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

#include <algorithm>
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
// One wave scans (four experts per lane, then a shuffle scan); one barrier publishes it.
template <int BM>
__device__ __forceinline__ int tile_prefix(const int32_t* __restrict__ offsets, int E, int* tstart) {
    static_assert(MOE_MAX_EXPERTS == 4 * 64, "four experts per lane of one wave");
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        int ex[4], run = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            const int cnt = (e < E) ? offsets[e + 1] - offsets[e] : 0;
            ex[i] = run;
            run += cnt > 0 ? (cnt + BM - 1) / BM : 0;
        }
        int incl = run;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(incl, o, 64);
            if (lane >= o) incl += t;
        }
        const int base = incl - run;
#pragma unroll
        for (int i = 0; i < 4; ++i) tstart[lane * 4 + i] = base + ex[i];
        if (lane == 63) tstart[4 * 64] = incl;
    }
    __syncthreads();
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

// The same activations through the fast forms (bf16 outputs: error far below rounding).
template <int EPI>
__device__ __forceinline__ float epilogue_fast(float u, float g) {
    if (EPI == kEpiGelu) return act_gelu_fast(u);
    if (EPI == kEpiGeluTanh) return act_gelu_tanh(u);
    if (EPI == kEpiSwiglu) return silu_fast(u) * g;
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

// ------------------------------------------------------------------ bf16 MFMA kernel, direct-to-LDS pipeline
//
// Tile: BM activation rows x BW weight rows (SwiGLU: BW/2 rows of W1 + the same rows of
// W3), K in steps of BK (32 or 64).  A row's BK-element slice is one LDS row of 2*BK bytes
// holding CPR = BK/8 chunks of 16 bytes; chunk c of row r is stored at position
// c ^ swz(r), which keeps the 32-row MFMA fragment reads free of bank conflicts.  Global
// data goes straight to LDS with global_load_lds_dwordx4 (lane l of a wave instruction
// fills bytes [16 l, 16 l + 16) of a 1 KiB span), NS stages deep, so NS - 1 K steps are in
// flight while one is multiplied.  The weight fragment is the MFMA's first operand, so each
// lane ends up holding 4 consecutive output columns of one row (one 8- or 16-byte store per
// group).  Rows past the segment end and weight rows past N are clamped to a valid row
// (their results are never stored); K must be a multiple of BK.

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt field is 6 bits");
    // gfx9 s_waitcnt: vmcnt[3:0] | expcnt[6:4]=7 | lgkmcnt[11:8]=15 | vmcnt[5:4] at [15:14]
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Wait until at most `newer` stages of LPW loads each are still in flight.
template <int LPW, int NS>
__device__ __forceinline__ void wait_stages(int newer) {
    static_assert(NS >= 2 && NS <= 6, "pipeline depth");
    if (NS > 5 && newer >= 4) { wait_vmcnt<(NS > 5 ? 4 * LPW : 0)>(); return; }
    if (NS > 4 && newer >= 3) { wait_vmcnt<(NS > 4 ? 3 * LPW : 0)>(); return; }
    if (NS > 3 && newer >= 2) { wait_vmcnt<(NS > 3 ? 2 * LPW : 0)>(); return; }
    if (NS > 2 && newer >= 1) { wait_vmcnt<(NS > 2 ? LPW : 0)>(); return; }
    wait_vmcnt<0>();
}

template <int BM, int BW, int BK, int NS, int EPI>
struct LdsShape {
    static constexpr bool kDual = (EPI == kEpiSwiglu);
    static constexpr int kNB = kDual ? 2 : 1;
    static constexpr int kBN = BW / kNB;          // output columns per tile
    static constexpr int kMI = BM / 64;           // 32-row blocks per wave (2 x 2 waves)
    static constexpr int kNI = kBN / 64;          // 32-column blocks per wave per matrix
    static constexpr int kCPR = BK / 8;           // 16-byte chunks per LDS row
    static constexpr int kRPI = 64 / kCPR;        // LDS rows per 1 KiB wave load
    static constexpr int kRows = BM + BW;         // LDS rows per stage
    static constexpr int kLPW = kRows / kRPI / 4;  // 1 KiB loads per wave per stage
    static constexpr int kSwzShift = (kCPR == 8) ? 1 : 2;  // rows sharing a 256-byte bank line
    static constexpr size_t kBytes = (size_t)NS * kRows * BK * 2;
    static_assert(kMI >= 1 && kNI >= 1, "tile too small for 2 x 2 waves of 32 x 32 blocks");
    static_assert(kRows % (kRPI * 4) == 0, "stage rows must split evenly over the waves");
    static_assert(BK == 32 || BK == 64, "BK");
};

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land at
// lds + 16 l (the LDS address is wave-uniform and goes through M0).  Issued as inline
// assembly on purpose: the compiler tracks the builtin form as an LDS write and then waits
// for it (vmcnt(0)) before every later LDS read it cannot prove disjoint -- which would make
// the prefetched stages synchronous.  The kernel orders these loads itself: wait_stages
// before the stage barrier, and a stage buffer is only refilled after every wave has read
// it.  The "memory" clobber keeps the compiler from moving LDS accesses across the issue.
__device__ __forceinline__ void load_lds16(const void* gptr, void* lds) {
    const uint32_t m0 = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) void*)lds)));
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(gptr) : "memory", "m0");
}

// Where a tile's loads come from: wave-uniform scalars, set once per tile.
struct TileSrc {
    const bf16_t* a;   // activation rows (x_perm or H)
    const bf16_t* b0;  // this expert's weights (W1^T or W2^T)
    const bf16_t* b1;  // SwiGLU: this expert's W3^T
    int64_t row0, last;  // first row of the tile, last valid row to read
    int n0;              // first weight row (output column) of the tile
};

// One stage of a wave's loads: 1 KiB per load, lane l landing at byte 16 l of it.  Load j
// of wave w fills LDS rows (4 j + w) * RPI ..., so whether a load carries activation rows
// or weight rows (and which weight matrix) is fixed by j at compile time.  LDS row R of the
// stage holds activation row R (R < BM) or weight row R - BM; rows past the segment or past
// N are clamped to a valid row, whose results are never stored.  Addresses are computed
// here from the tile scalars rather than cached, to keep registers for the accumulators.
template <int BM, int BN, int LPW, int RPI, int CPR, int SH>
__device__ __forceinline__ void issue_stage(const TileSrc& ts, int K, int N, int wave, int lane, bf16_t* stage,
                                            int k0) {
    const int r_lane = lane / CPR, c_lane = lane % CPR;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
        constexpr int kRowsPerJ = 4 * RPI;
        const int R = (j * 4 + wave) * RPI + r_lane;
        const int kc = c_lane ^ ((R >> SH) & (CPR - 1));
        const bf16_t* src;
        if (j * kRowsPerJ < BM) {
            src = ts.a + min(ts.row0 + R, ts.last) * K;
        } else {
            constexpr int kAJ = BM / kRowsPerJ;  // loads per wave that carry activation rows
            const int nb = ((j - kAJ) * kRowsPerJ) / BN;  // compile-time after unrolling
            const int n = min(ts.n0 + (R - BM - nb * BN), N - 1);
            src = (nb ? ts.b1 : ts.b0) + static_cast<int64_t>(n) * K;
        }
        load_lds16(src + k0 + kc * 8, stage + (j * 4 + wave) * RPI * (CPR * 8));
    }
}

// Bare workgroup barrier.  A fenced barrier (__syncthreads, or even an LDS-only fence)
// makes the compiler wait for every direct-to-LDS load in flight, which would drain the
// prefetched stages this pipeline keeps in flight across the barrier.  Ordering is kept
// by hand instead: each wave waits (wait_stages) for its own loads of the stage it is about
// to read before arriving, so after the barrier that stage is complete for all waves; and
// a wave only overwrites a stage buffer after the barrier that follows every wave's reads
// of it (its ds_reads have returned: their data fed the MFMAs before the wave arrived).
__device__ __forceinline__ void stage_barrier() { __builtin_amdgcn_s_barrier(); }

// Row tile mt's expert and row range, and the column offset of column tile nt.
struct TileRows {
    int64_t row0, row_end;
    int e;
};

template <int BM>
__device__ __forceinline__ TileRows tile_rows(const GroupedGemm& g, const int* tstart, int mt) {
    TileRows t;
    t.e = find_expert(tstart, g.E, mt);
    t.row0 = g.offsets[t.e] + static_cast<int64_t>(mt - tstart[t.e]) * BM;
    t.row_end = g.offsets[t.e + 1] < g.rows_max ? g.offsets[t.e + 1] : g.rows_max;
    return t;
}

// Logical tile L -> (row tile, column tile): groups of GM row tiles, column-major inside a
// group, so that neighbouring tiles share either rows or weights.
__device__ __forceinline__ void tile_coords(int L, int total_m, int n_tiles, int& mt, int& nt) {
    constexpr int GM = 8;
    const int grp = L / (GM * n_tiles);
    const int rem = L - grp * GM * n_tiles;
    const int gsz = min(GM, total_m - grp * GM);
    nt = rem / gsz;
    mt = grp * GM + (rem - nt * gsz);
}

// Persistent grouped GEMM.  The grid is a fixed number of workgroups (one or two per CU);
// the tiles are dealt to the 8 XCDs in contiguous runs (the hardware deals workgroups
// round-robin, so workgroup b sits on XCD b % 8) and, inside a run, round-robin to that
// XCD's workgroups, so concurrently running tiles share rows or weights in its L2.  The
// load pipeline runs across tile boundaries: while one tile's last K steps are multiplied
// and its epilogue runs, the next tile's first stages are already in flight.
template <int BM, int BW, int BK, int NS, int EPI, bool OB>
__global__ __launch_bounds__(kThreads, (LdsShape<BM, BW, BK, NS, EPI>::kBytes <= 80 * 1024) ? 2 : 1)
void gemm_bf16_lds(GroupedGemm g) {
    typedef LdsShape<BM, BW, BK, NS, EPI> S;
    constexpr int NB = S::kNB, BN = S::kBN, MI = S::kMI, NI = S::kNI, ROWS = S::kRows, LPW = S::kLPW;
    constexpr int CPR = S::kCPR, RPI = S::kRPI, SH = S::kSwzShift;
    __shared__ int tstart[kThreads + 1];
    extern __shared__ __align__(1024) unsigned char smem_raw[];
    bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);

    const int total_m = tile_prefix<BM>(g.offsets, g.E, tstart);
    const int total = total_m * g.n_tiles;
    const int per = (total + 7) >> 3;
    const int xcd = blockIdx.x & 7, nslot = gridDim.x >> 3;
    const int t_end = min(total, (xcd + 1) * per);
    const int t_first = xcd * per + static_cast<int>(blockIdx.x >> 3);
    if (t_first >= t_end) return;
    const int nk = g.K / BK;

    const int tid = threadIdx.x, lane = tid & 63;
    // the wave index is uniform across a wave; say so, so that per-wave choices stay scalar
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bf16_t* __restrict__ A = static_cast<const bf16_t*>(g.a);

    // ---- load cursor: tile lt, K step lk
    int lt = t_first, lk = 0;
    TileSrc ts;
    auto set_tile = [&](int L) {
        int mt, nt;
        tile_coords(L, total_m, g.n_tiles, mt, nt);
        const TileRows tr = tile_rows<BM>(g, tstart, mt);
        ts.a = A;
        ts.b0 = static_cast<const bf16_t*>(g.b) + tr.e * g.b_estride;
        ts.b1 = NB > 1 ? static_cast<const bf16_t*>(g.b2) + tr.e * g.b_estride : ts.b0;
        ts.row0 = max<int64_t>(0, tr.row0);
        // rows past the segment are clamped to its last row; inconsistent offsets (a segment
        // outside [0, rows_max)) still only ever read rows inside the buffer
        int64_t last = tr.row_end > tr.row0 ? tr.row_end - 1 : tr.row0;
        ts.last = max<int64_t>(0, min<int64_t>(last, g.rows_max - 1));
        ts.n0 = nt * BN;
    };
    set_tile(lt);
    int issued = 0;  // stages issued by this wave so far
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) {
        if (lt < t_end) {
            issue_stage<BM, BN, LPW, RPI, CPR, SH>(ts, g.K, g.N, wave, lane, smem + (issued % NS) * ROWS * BK, lk * BK);
            ++issued;
            if (++lk == nk) {
                lk = 0;
                lt += nslot;
                if (lt < t_end) set_tile(lt);
            }
        }
    }

    // ---- compute: one tile after another; the load cursor above runs NS - 1 stages ahead
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lhi = lane >> 5;
    int consumed = 0;
    for (int ct = t_first; ct < t_end; ct += nslot) {
        f32x16_t acc[NB][MI][NI];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[nb][i][j][r] = 0.f;

        for (int ck = 0; ck < nk; ++ck) {
            // the first step after an epilogue also waits for its stores (they share the counter)
            if (ck == 0 && ct != t_first) wait_vmcnt<0>();
            else wait_stages<LPW, NS>(issued - consumed - 1);
            stage_barrier();
            if (lt < t_end) {
                issue_stage<BM, BN, LPW, RPI, CPR, SH>(ts, g.K, g.N, wave, lane, smem + (issued % NS) * ROWS * BK,
                                                       lk * BK);
                ++issued;
                if (++lk == nk) {
                    lk = 0;
                    lt += nslot;
                    if (lt < t_end) set_tile(lt);
                }
            }
            const bf16_t* st = smem + (consumed % NS) * ROWS * BK;
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                const int ch = 2 * ks + lhi;
                bf16x8_t af[MI], wf[NB][NI];
#pragma unroll
                for (int i = 0; i < MI; ++i) {
                    const int R = wm * (BM / 2) + i * 32 + l32;
                    af[i] = *reinterpret_cast<const bf16x8_t*>(st + R * BK + ((ch ^ ((R >> SH) & (CPR - 1))) << 3));
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int j = 0; j < NI; ++j) {
                        const int R = BM + nb * BN + wn * (BN / 2) + j * 32 + l32;
                        wf[nb][j] = *reinterpret_cast<const bf16x8_t*>(st + R * BK + ((ch ^ ((R >> SH) & (CPR - 1))) << 3));
                    }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int i = 0; i < MI; ++i)
#pragma unroll
                        for (int j = 0; j < NI; ++j)
                            acc[nb][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[nb][j], af[i], acc[nb][i][j], 0, 0, 0);
            }
            ++consumed;
        }

        // ---- epilogue of tile ct.  D[n][m] layout: lane holds activation row l32 of the
        // block; register r holds weight row 8 * (r / 4) + 4 * lhi + r % 4, i.e. 4
        // consecutive output columns per group r / 4.
        int mt, nt;
        tile_coords(ct, total_m, g.n_tiles, mt, nt);
        const TileRows tr = tile_rows<BM>(g, tstart, mt);
        const int n0 = nt * BN;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            const int64_t row = tr.row0 + wm * (BM / 2) + i * 32 + l32;
            const bool row_ok = row >= 0 && row < tr.row_end;
#pragma unroll
            for (int j = 0; j < NI; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = n0 + wn * (BN / 2) + j * 32 + 8 * q + 4 * lhi;
                    float v[4];
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        v[c] = epilogue_fast<EPI>(acc[0][i][j][4 * q + c], acc[NB - 1][i][j][4 * q + c]);
                    if (row_ok && col < g.N) {
                        if (OB) {
                            uint2 pk;
                            pk.x = pack_bf16x2(v[0], v[1]);
                            pk.y = pack_bf16x2(v[2], v[3]);
                            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.c) + row * g.ldc + col) = pk;
                        } else {
                            *reinterpret_cast<float4*>(static_cast<float*>(g.c) + row * g.ldc + col) =
                                make_float4(v[0], v[1], v[2], v[3]);
                        }
                    }
                    // one block at a time: keeps the scheduler from pulling every accumulator
                    // into VGPRs at once
                    __builtin_amdgcn_sched_barrier(0);
                }
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

int device_cus() {
    static const int cus = [] {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = 256;
        return n;
    }();
    return cus;
}

template <int BM, int BW, int BK, int NS, int EPI, bool OB>
hipError_t run_bf16_lds(GroupedGemm g, int64_t A_max, hipStream_t s) {
    typedef LdsShape<BM, BW, BK, NS, EPI> S;
    constexpr size_t lds = S::kBytes;
    constexpr int per_cu = (lds <= 80 * 1024) ? 2 : 1;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&gemm_bf16_lds<BM, BW, BK, NS, EPI, OB>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (attr != hipSuccess) return attr;
    g.n_tiles = static_cast<int>(ceil_div(g.N, S::kBN));
    const int64_t tiles = row_tile_bound(A_max, g.E, BM) * g.n_tiles;
    if (tiles == 0) return hipSuccess;
    // persistent grid: at most per_cu workgroups per CU, a multiple of the 8 XCDs
    const int64_t blocks = round_up(std::min<int64_t>(tiles, static_cast<int64_t>(per_cu) * device_cus()), 8);
    hipLaunchKernelGGL((gemm_bf16_lds<BM, BW, BK, NS, EPI, OB>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads),
                       lds, s, g);
    return hipGetLastError();
}

// Tile shape: 128 activation rows x 256 weight rows, 32-wide K steps, three stages (two in
// flight) in 72 KiB of LDS, so that two workgroups share a CU and one's epilogue and
// pipeline fill overlap the other's MFMAs.
template <int EPI, bool OB>
hipError_t run_bf16_best(GroupedGemm g, int64_t A_max, hipStream_t s) {
    if (g.K % 32 == 0) return run_bf16_lds<128, 256, 32, 3, EPI, OB>(g, A_max, s);
    return run_bf16<EPI, OB>(g, A_max, s);
}

template <int EPI>
hipError_t gemm1(bool bf16, GroupedGemm g, int64_t A_max, hipStream_t s) {
    return bf16 ? run_bf16_best<EPI, true>(g, A_max, s) : run_f32<EPI, false>(g, A_max, s);
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
    if (bf16) return y_bf16 ? run_bf16_best<kEpiNone, true>(g2, A_max, s) : run_bf16_best<kEpiNone, false>(g2, A_max, s);
    return y_bf16 ? run_f32<kEpiNone, true>(g2, A_max, s) : run_f32<kEpiNone, false>(g2, A_max, s);
}

}  // namespace moe
