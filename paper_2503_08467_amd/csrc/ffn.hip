// Step 4 of the layer: this device's shard of every expert on the rows routed to it, as a
// grouped GEMM over variable-length expert segments -- one launch per matmul, whatever
// the number of experts.
//
//   GEMM1   H[p, n] = act(x_perm[p] . W1^T[e][n])       (SwiGLU: silu(.W1) * (.W3))
//   GEMM2   y_perm[p, c] = H[p] . W2^T[e][c]
//
// Each workgroup first turns offsets[] into a per-expert prefix of row tiles, then maps
// linear tile ids to (expert, row tile, column tile).  The grid is persistent (sized from
// the host-known bound A_max, at most as many workgroups per CU as LDS allows, a multiple
// of the 8 XCDs), so the counts are never read back to the host.
//
// bf16 path (gemm_bf16_lds, gemm_up_pairs): 128-row tiles, 256 (or 384 / 128) weight rows
// per tile, v_mfma_f32_32x32x16_bf16 with fp32 accumulation.  Weights and H are stored
// K-blocked (blocks of 32 K values, all rows side by side), so every stage of 32 K values
// of a run of rows is one contiguous stretch that 1 KiB direct-to-LDS loads fetch; three
// LDS stages, two in flight across K steps and tiles.  The epilogue applies the activation
// in fp32, rounds once, and stores 16-byte runs straight from the accumulators (into
// K-blocked H for GEMM1).  Calls of at most 512 rows split GEMM2's K into parts summed by
// split_reduce (or, with the combine folded in, split_combine) in a fixed order.
// fp32 path (gemm_f32_lds): 32 x 128 tiles on v_mfma_f32_32x32x2_f32, row-major operands in
// 128-byte row pieces through two direct-to-LDS stages, three workgroups per CU; gemm_f32
// (register-staged 64 x 64 tiles) only for an up-projection whose h is not a multiple of 32.
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

#include "../../include/moeshard.h"

#include <algorithm>
#include <mutex>
#include <type_traits>

namespace moe {
namespace {

enum Epi { kEpiGelu = 0, kEpiGeluTanh = 1, kEpiSwiglu = 2, kEpiNone = 3 };

struct GroupedGemm {
    const void* a;           // [rows][K], or with `gather` [a_rows][K] read through it
    const void* b;           // [E][N rows][K]  (K-contiguous weights)
    const void* b2;          // SwiGLU up projection, same layout as b
    void* c;                 // [rows][ldc]
    const int32_t* offsets;  // [E + 1] row segment of every expert
    int E, K, N, ldc, n_tiles;
    int64_t b_estride;  // elements from one expert's weights to the next
    int64_t rows_max;   // rows of a and c; no row at or past it is touched
    // Up-projection only: grouped row p reads row gather[p] of a (clamped to
    // [0, a_rows)) instead of row p -- the dispatch gather folded into the loads.
    const int32_t* gather;
    int64_t a_rows;
    // Down-projection, top-1 only: grouped row p is stored as w[t] * row into row
    // t = scatter[p] (clamped to [0, c_rows)) of c instead of row p -- Step 5 folded in.
    const int32_t* scatter;
    const float* scatter_w;
    int64_t c_rows;
    // Down-projection only: with ksplit > 1 every tile is computed as ksplit parts of K/ksplit
    // each, part s written in fp32 to partial[s][row][N] (no scale, no scatter); a reduce
    // kernel sums the parts in order afterwards.
    int ksplit;
    float* partial;
};

// Source row of grouped row p: p itself, or gather[p] clamped into a (entries past the
// assigned rows are never written by the dispatch, so their value is arbitrary).
__device__ __forceinline__ int64_t source_row(const GroupedGemm& g, int64_t p) {
    if (!g.gather) return p;
    const int64_t r = g.gather[p];
    return r < 0 ? 0 : (r >= g.a_rows ? g.a_rows - 1 : r);
}

constexpr int kThreads = 256;

// Exclusive prefix over experts of ceil(count / BM) into tstart[0..E]; returns the total.
// One wave scans (four experts per lane, then a shuffle scan); one barrier publishes it.
template <int BM>
__device__ __forceinline__ int tile_prefix(const int32_t* __restrict__ offsets, int E, int* tstart) {
    static_assert(MOE_MAX_EXPERTS == 4 * 64, "four experts per lane of one wave");
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        // offsets of the lane's four experts and the next, all loaded before any is used
        // (from clamped indices: a load behind a per-lane condition waits for itself)
        int o[5];
#pragma unroll
        for (int i = 0; i < 5; ++i) o[i] = offsets[min(lane * 4 + i, E)];
        int ex[4], run = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int cnt = (lane * 4 + i < E) ? o[i + 1] - o[i] : 0;
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

// CB: C is stored K-blocked for the next GEMM (element (row, n) at
// ((n / 32) * rows_max + row) * 32 + n % 32), else row-major with stride ldc.
template <int EPI, bool OB, bool CB>
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
                        ? *reinterpret_cast<const uint4*>(A + source_row(g, ar) * g.K + k0 + kc)
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
            const int64_t n = n0 + c8;
            const int64_t ci = CB ? ((n >> 5) * g.rows_max + row0 + row) * 32 + (n & 31) : (row0 + row) * g.ldc + n;
            if (row0 + row < row_end && n < g.N)
                *reinterpret_cast<uint4*>(C + ci) = *reinterpret_cast<const uint4*>(cs + row * LDC + c8);
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
            const int64_t n = n0 + c4;
            const int64_t ci = CB ? ((n >> 5) * g.rows_max + row0 + row) * 32 + (n & 31) : (row0 + row) * g.ldc + n;
            if (row0 + row < row_end && n < g.N)
                *reinterpret_cast<float4*>(C + ci) = *reinterpret_cast<const float4*>(cs + row * LDC + c4);
        }
    }
}

// ------------------------------------------------------------------ bf16 MFMA kernel, direct-to-LDS pipeline
//
// Tile: BM activation rows x BW weight rows (SwiGLU: BW/2 rows of W1 + the same rows of
// W3), K in steps of BK = 32.  A row's 32-element slice is one LDS row of 64 bytes holding
// 4 chunks of 16 bytes; chunk c of row r is stored at position c ^ swz(r), which keeps the
// 32-row MFMA fragment reads free of bank conflicts.  Global data goes straight to LDS with
// global_load_lds_dwordx4 (lane l of a wave instruction fills bytes [16 l, 16 l + 16) of a
// 1 KiB span: 16 LDS rows), NS stages deep.  The weights are K-blocked (see the pack step:
// a stage's rows are one contiguous run), and so is the intermediate H, which the
// up-projection writes and the down-projection reads: every 1 KiB load of those operands
// is 1 KiB of contiguous memory, eight full 128-byte lines.  The up-projection's
// activations (x_perm) are row-major: 64-byte pieces of 16 rows.  The weight fragment is
// the MFMA's first operand, so each lane ends up holding 4 consecutive output columns of
// one row (one 8- or 16-byte store per group).  K must be a multiple of 32.

// WN: waves along the tile's columns (the waves are 2 x WN; 4 or 8 per workgroup).
template <int BM, int BW, int BK, int NS, int EPI, int WN = 2>
struct LdsShape {
    static constexpr bool kDual = (EPI == kEpiSwiglu);
    static constexpr int kNB = kDual ? 2 : 1;
    static constexpr int kBN = BW / kNB;          // output columns per tile
    static constexpr int kWaves = 2 * WN;
    static constexpr int kThreadsWG = 64 * kWaves;
    static constexpr int kMI = BM / 64;           // 32-row blocks per wave (BM / 2 rows)
    static constexpr int kNI = kBN / (32 * WN);   // 32-column blocks per wave per matrix
    static constexpr int kCPR = BK / 8;           // 16-byte chunks per LDS row
    static constexpr int kRPI = 64 / kCPR;        // LDS rows per 1 KiB wave load
    static constexpr int kRows = BM + BW;         // LDS rows per stage
    static constexpr int kLPW = kRows / kRPI / kWaves;  // 1 KiB loads per wave per stage
    static constexpr int kKS = BK / 16;           // MFMA K steps per stage
    static constexpr int kSwzShift = (kCPR == 8) ? 1 : 2;  // rows sharing a 256-byte bank line
    static constexpr size_t kBytes = (size_t)NS * kRows * BK * 2;
    static constexpr int kPerCU = (kBytes <= 80 * 1024) ? 2 : 1;  // workgroups per CU
    static_assert(kMI >= 1 && kNI >= 1 && kBN % (32 * WN) == 0, "tile too small for the waves' 32 x 32 blocks");
    static_assert(kRows % (kRPI * kWaves) == 0, "stage rows must split evenly over the waves");
    static_assert(BM % (kWaves * kRPI) == 0 && kBN % (kWaves * kRPI) == 0, "a wave load carries one kind of row");
    static_assert(BK == 32, "the K-blocked operands come in blocks of 32");
};

// Stores one lane's share of a 32 x 32 bf16 output block.  The MFMA layout leaves lane
// (row, half) with columns 8 q + 4 half .. 8 q + 4 half + 3 of its row, q = 0..3, packed
// as pk[q].  Lanes l and l + 32 hold the same row; v_permlane32_swap trades lane l's pk[1]
// for lane l + 32's pk[0] (and pk[3] for pk[2]), after which lane l holds columns 0..7 and
// 16..23 of the row and lane l + 32 columns 8..15 and 24..31, each run stored as one
// 16-byte vector: half the store instructions of 8-byte groups, and 32 contiguous bytes of
// every row per instruction.  dst = the lane's row at column 8 half of the block (the
// second run is dst + 16); ok0 / ok1 say whether each run is stored.  Every lane of the
// wave must call it (the swap).
__device__ __forceinline__ void store_block_bf16(bf16_t* dst, const uint2 (&pk)[4], bool ok0, bool ok1) {
    // swap(vdst, src): lanes 32..63 of vdst <-> lanes 0..31 of src; returns {vdst, src}
    const auto a0 = __builtin_amdgcn_permlane32_swap(pk[0].x, pk[1].x, false, false);
    const auto a1 = __builtin_amdgcn_permlane32_swap(pk[0].y, pk[1].y, false, false);
    const auto b0 = __builtin_amdgcn_permlane32_swap(pk[2].x, pk[3].x, false, false);
    const auto b1 = __builtin_amdgcn_permlane32_swap(pk[2].y, pk[3].y, false, false);
    if (ok0) *reinterpret_cast<uint4*>(dst) = make_uint4(a0[0], a1[0], a0[1], a1[1]);
    if (ok1) *reinterpret_cast<uint4*>(dst + 16) = make_uint4(b0[0], b1[0], b0[1], b1[1]);
}

// One accumulator value for the epilogue.  With 256 accumulator registers per lane they
// live in AGPRs, and VALU work needs them in VGPRs; left to itself the compiler copies all of
// them at once when the K loop ends, which needs every VGPR and spills the loop's live
// values.  Reading them one at a time keeps the epilogue's VGPR use small.
template <bool IN_AGPR>
__device__ __forceinline__ float acc_read(float a) {
    if (!IN_AGPR) return a;
    float v;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(v) : "a"(a));
    return v;
}

// Row tile mt's expert and row range.
struct TileRows {
    int64_t row0, row_end;
    int e;
};

// The row-tile table (first row tile of every expert): in LDS, written by tile_prefix ...
struct LdsTiles {
    const int* tstart;
    int E;
    __device__ __forceinline__ int find(int mt) const { return find_expert(tstart, E, mt); }
    __device__ __forceinline__ int start(int e) const { return tstart[e]; }
};

// ... or in registers, one copy per wave (for kernels whose LDS is all stage buffers): lane l
// holds the first row tile of experts 4 l .. 4 l + 3.  Every lane of the wave must call.
template <int BM>
struct RegTiles {
    int ex[4];
    int E, total;
    __device__ __forceinline__ void build(const int32_t* __restrict__ offsets, int num_experts) {
        static_assert(MOE_MAX_EXPERTS == 4 * 64, "four experts per lane of one wave");
        E = num_experts;
        const int lane = threadIdx.x & 63;
        int o[5];  // loaded together from clamped indices, as in tile_prefix
#pragma unroll
        for (int i = 0; i < 5; ++i) o[i] = offsets[min(lane * 4 + i, num_experts)];
        int run = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int cnt = (lane * 4 + i < E) ? o[i + 1] - o[i] : 0;
            ex[i] = run;
            run += cnt > 0 ? (cnt + BM - 1) / BM : 0;
        }
        int incl = run;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(incl, o, 64);
            if (lane >= o) incl += t;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) ex[i] += incl - run;
        total = __builtin_amdgcn_readfirstlane(__shfl(incl, 63, 64));
    }
    // largest expert whose first row tile is <= mt (the table is non-decreasing): a count
    // over the wave by ballots, no cross-lane data movement
    __device__ __forceinline__ int find(int mt) const {
        const int lane = threadIdx.x & 63;
        int c = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) c += __popcll(__ballot(lane * 4 + i < E && ex[i] <= mt));
        return c - 1;
    }
    // e is wave-uniform: read it from lane e / 4
    __device__ __forceinline__ int start(int e) const {
        const int q = e & 3;
        const int v = q == 0 ? ex[0] : q == 1 ? ex[1] : q == 2 ? ex[2] : ex[3];
        return __builtin_amdgcn_readlane(v, e >> 2);
    }
};

template <int BM, typename Tiles>
__device__ __forceinline__ TileRows tile_rows(const GroupedGemm& g, const Tiles& tiles, int mt) {
    TileRows t;
    t.e = __builtin_amdgcn_readfirstlane(tiles.find(mt));
    const int first = __builtin_amdgcn_readfirstlane(tiles.start(t.e));
    const int64_t seg0 = g.offsets[t.e], seg1 = g.offsets[t.e + 1];
    t.row0 = seg0 + static_cast<int64_t>(mt - first) * BM;
    t.row_end = seg1 < g.rows_max ? seg1 : g.rows_max;
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

// Where a tile's rows are read from.  The tile reads BM activation rows starting at
// row_base and BN weight rows starting at n_base, both shifted back from the tile's own
// first row / column when the tile would run past the end of the buffer (so every load
// stays inside it without a per-row check); the epilogue stores only the tile's own rows
// [row0, row_end) and columns [n0, N).
struct TileGeom {
    int64_t row0, row_end, row_base;
    int n0, n_base, e;
};

template <int BM, int BN, typename Tiles>
__device__ __forceinline__ TileGeom tile_geom(const GroupedGemm& g, const Tiles& tiles, int total_m, int L) {
    int mt, nt;
    tile_coords(L, total_m, g.n_tiles, mt, nt);
    const TileRows tr = tile_rows<BM>(g, tiles, mt);
    TileGeom t;
    t.e = tr.e;
    t.row0 = tr.row0;
    t.row_end = tr.row_end;
    const int64_t top = g.rows_max > BM ? g.rows_max - BM : 0;
    t.row_base = tr.row0 < 0 ? 0 : (tr.row0 > top ? top : tr.row0);
    t.n0 = nt * BN;
    const int ntop = g.N > BN ? g.N - BN : 0;
    t.n_base = t.n0 > ntop ? ntop : t.n0;
    return t;
}

// Last activation row of a tile worth loading: rows past the tile's valid ones then load that
// row again (their results are never stored), so that a mostly empty tile's loads touch one
// line each.  A tile shifted back at the end of the buffer keeps the buffer's limit.
template <int BM>
__device__ __forceinline__ int tile_row_limit(const GroupedGemm& g, const TileGeom& t) {
    const int lim = static_cast<int>(g.rows_max < BM ? g.rows_max : BM) - 1;
    if (t.row_base != t.row0) return lim;
    const int64_t valid = t.row_end - t.row0;
    return valid >= 1 && valid - 1 < lim ? static_cast<int>(valid - 1) : lim;
}

// Persistent grouped GEMM.  The grid is a fixed number of workgroups (one or two per CU);
// the tiles are dealt to the 8 XCDs in contiguous runs (the hardware deals workgroups
// round-robin, so workgroup b sits on XCD b % 8) and, inside a run, round-robin to that
// XCD's workgroups, so concurrently running tiles share rows or weights in its L2.
//
// Pipeline (per wave; stage b = the b-th K step this workgroup multiplies, counted across
// tiles).  Loads run NS - 1 stages ahead, across tile boundaries.  Stage b is published by
// one barrier: before it each wave waits for its own loads of stage b (vmcnt) and for its
// own LDS reads of stage b - 1 (lgkmcnt); after it, stage b is complete for every wave and
// nobody reads stage b - 1 any more, so its buffer is refilled with stage b + NS - 1 right
// away.  Inside a tile, that barrier sits in front of the last MFMA step of stage b - 1:
// the first fragments of stage b are read from LDS while those MFMAs run, and every other
// MFMA step's fragments are read during the step before it (two fragment sets in
// registers).  Every 1 KiB load has a fixed per-lane offset (computed once) from a scalar
// base that moves by 2*BK bytes per stage.
//
// The activation epilogues belong to the up-projection (A = x_perm row-major, C = H
// K-blocked); the plain one to the down-projection (A = H K-blocked, C = y_perm row-major).
template <int BM, int BW, int BK, int NS, int EPI, bool OB, int WN = 2>
__global__ __launch_bounds__((LdsShape<BM, BW, BK, NS, EPI, WN>::kThreadsWG),
                             (LdsShape<BM, BW, BK, NS, EPI, WN>::kPerCU))
void gemm_bf16_lds(GroupedGemm g) {
    typedef LdsShape<BM, BW, BK, NS, EPI, WN> S;
    constexpr bool kUp = EPI != kEpiNone;
    constexpr int NB = S::kNB, BN = S::kBN, MI = S::kMI, NI = S::kNI, ROWS = S::kRows, LPW = S::kLPW;
    constexpr int CPR = S::kCPR, RPI = S::kRPI, SH = S::kSwzShift, KS = S::kKS, NW = S::kWaves;
    constexpr int kStageBytes = ROWS * BK * 2;
    constexpr int kAJ = BM / (NW * RPI);  // loads per wave per stage that carry activation rows
    __shared__ int tstart[kThreads + 1];
    extern __shared__ __align__(1024) unsigned char smem_raw[];

    const int total_m = tile_prefix<BM>(g.offsets, g.E, tstart);
    const LdsTiles tiles{tstart, g.E};
    // work item L = tile L / ks, K part L % ks (ks = 1 unless the down-projection is split)
    const int ks = (!kUp && g.ksplit > 1) ? g.ksplit : 1;
    const int total = total_m * g.n_tiles * ks;
    const int per = (total + 7) >> 3;
    const int xcd = blockIdx.x & 7, nslot = gridDim.x >> 3;
    const int t_end = min(total, (xcd + 1) * per);
    const int t_first = xcd * per + static_cast<int>(blockIdx.x >> 3);
    if (t_first >= t_end) return;
    const int nk = g.K / BK / ks;  // K steps per work item

    const int tid = threadIdx.x, lane = tid & 63;
    // the wave index is uniform across a wave; say so, so that per-wave choices stay scalar
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane(
        static_cast<uint32_t>(reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) void*)smem_raw)));

    // Per-lane byte offsets of this wave's loads: load j fills LDS rows (NW j + wave) * RPI
    // + lane / CPR of a stage, slot lane % CPR, with global chunk slot ^ swz(row).  Rows past
    // a buffer smaller than one tile repeat its last row.
    uint32_t voff[LPW];
    {
        const int r_lane = lane / CPR, c_lane = lane % CPR;
        const int a_lim = static_cast<int>(g.rows_max < BM ? g.rows_max : BM) - 1;
        const int b_lim = (g.N < BN ? g.N : BN) - 1;
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
            const int R = (j * NW + wave) * RPI + r_lane;
            const int kc = c_lane ^ ((R >> SH) & (CPR - 1));
            int r;
            if (j < kAJ) r = min(R, a_lim);
            else r = min((R - BM) % BN, b_lim);
            const uint32_t row_bytes = (j < kAJ && kUp) ? static_cast<uint32_t>(2 * g.K) : 64u;
            voff[j] = static_cast<uint32_t>(r) * row_bytes + static_cast<uint32_t>(kc * 16);
        }
    }

    // ---- load cursor: tile lt, K step lk, scalar bases of the tile's rows at K = 0
    int lt = t_first, lk = 0;
    const unsigned char *src_a = nullptr, *src_b0 = nullptr, *src_b1 = nullptr;
    auto set_tile = [&](int L) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, L / ks);
        const int64_t k0 = static_cast<int64_t>(L % ks) * nk;  // first K block of the work item
        const int64_t rb = kUp ? 2 * static_cast<int64_t>(g.K) : 64;
        if (kUp && g.gather) {
            // this lane's activation rows come from the gathered source rows (the index
            // load makes the compiler wait for the loads in flight: once per tile)
            const int r_lane = lane / CPR, c_lane = lane % CPR;
            const int a_lim = tile_row_limit<BM>(g, t);
#pragma unroll
            for (int j = 0; j < kAJ; ++j) {
                const int R = (j * NW + wave) * RPI + r_lane;
                const int kc = c_lane ^ ((R >> SH) & (CPR - 1));
                const int64_t src = source_row(g, t.row_base + min(R, a_lim));
                voff[j] = static_cast<uint32_t>(src) * static_cast<uint32_t>(2 * g.K) + static_cast<uint32_t>(kc * 16);
            }
            src_a = uniform_ptr(g.a);
        } else {
            const int r_lane = lane / CPR, c_lane = lane % CPR;
            const int a_lim = tile_row_limit<BM>(g, t);
#pragma unroll
            for (int j = 0; j < kAJ; ++j) {
                const int R = (j * NW + wave) * RPI + r_lane;
                const int kc = c_lane ^ ((R >> SH) & (CPR - 1));
                voff[j] = static_cast<uint32_t>(min(R, a_lim)) * static_cast<uint32_t>(rb) + static_cast<uint32_t>(kc * 16);
            }
            src_a = uniform_ptr(static_cast<const unsigned char*>(g.a) + t.row_base * rb +
                                (kUp ? 0 : k0 * g.rows_max * 64));
        }
        const int64_t boff = (t.e * g.b_estride) * 2 + static_cast<int64_t>(t.n_base) * 64 + k0 * g.N * 64;
        src_b0 = uniform_ptr(static_cast<const unsigned char*>(g.b) + boff);
        src_b1 = NB > 1 ? uniform_ptr(static_cast<const unsigned char*>(g.b2) + boff) : src_b0;
    };
    int issued = 0;  // stages issued by this wave so far
    auto issue_next = [&]() {
        if (lt >= t_end) return;
        const uint32_t dst = lds0 + (issued % NS) * kStageBytes;
        // K block lk of each operand: the next 64 bytes of every row (row-major x_perm), or
        // the next block of all rows (K-blocked)
        const int64_t ka = kUp ? static_cast<int64_t>(lk) * 64 : static_cast<int64_t>(lk) * g.rows_max * 64;
        const int64_t kb = static_cast<int64_t>(lk) * g.N * 64;
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
            const unsigned char* base = j < kAJ ? src_a + ka : ((NB > 1 && (j - kAJ) * NW * RPI >= BN) ? src_b1 : src_b0) + kb;
            load_lds16(base, voff[j], dst + (j * NW + wave) * RPI * CPR * 16);
        }
        ++issued;
        if (++lk == nk) {
            lk = 0;
            lt += nslot;
            if (lt < t_end) set_tile(lt);
        }
    };
    set_tile(lt);
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue_next();

    // ---- fragments: A block i = activation rows wm*BM/2 + 32 i + l32, B block (nb, j) =
    // weight rows BM + nb*BN + wn*BN/2 + 32 j + l32; K chunk 2 ks + lhi of the stage.  Only
    // the first NV row blocks of the wave are read (the rest hold no valid row).
    const int wm = wave / WN, wn = wave % WN;
    const int l32 = lane & 31, lhi = lane >> 5;
    typedef bf16x8_t Frags[MI + NB * NI];
    auto read_frags = [&](auto nv_tag, int stage_slot, int ks, Frags& f) {
        constexpr int NV = decltype(nv_tag)::value;
        const unsigned char* st = smem_raw + stage_slot * kStageBytes;
        const int ch = 2 * ks + lhi;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int R = wm * (BM / 2) + i * 32 + l32;
            f[i] = *reinterpret_cast<const bf16x8_t*>(st + R * (2 * BK) + ((ch ^ ((R >> SH) & (CPR - 1))) << 4));
        }
        if (NV == 0) return;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int R = BM + nb * BN + wn * (BN / WN) + j * 32 + l32;
                f[MI + nb * NI + j] =
                    *reinterpret_cast<const bf16x8_t*>(st + R * (2 * BK) + ((ch ^ ((R >> SH) & (CPR - 1))) << 4));
            }
    };

    // one workgroup per CU: the accumulators fill the AGPRs (see acc_read)
    constexpr bool kAccInAgpr = S::kPerCU == 1;
    int consumed = 0;
    for (int ct = t_first; ct < t_end; ct += nslot) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, ct / ks);
        // Row blocks of this wave that hold valid rows.  Valid rows start at the tile's first
        // row unless the tile was shifted back at the end of the buffer; then all count.  The
        // count is rounded up to MI / 2 or MI so that three loop bodies cover every case.
        int nv = MI;
        if (t.row_base == t.row0) {
            const int64_t left = t.row_end - (t.row0 + wm * (BM / 2));
            nv = left <= 0 ? 0 : (left > (MI / 2) * 32 ? MI : MI / 2);
        }
        nv = __builtin_amdgcn_readfirstlane(nv);

        f32x16_t acc[NB][MI][NI];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[nb][i][j][r] = 0.f;

        // publish the tile's first stage; after an epilogue its stores share the counter
        if (ct != t_first) wait_vmcnt<0>();
        else wait_stages<LPW, NS>(issued - consumed - 1);
        stage_barrier();
        issue_next();

        // the K loop with the MFMAs of the first NV row blocks; every wave takes part in the
        // loads, waits and barriers whatever its NV
        auto k_loop = [&](auto nv_tag) {
            constexpr int NV = decltype(nv_tag)::value;
            // weight block outer, row block inner: consecutive MFMAs share their first operand
            auto mma = [&](const Frags& f) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int j = 0; j < NI; ++j)
#pragma unroll
                        for (int i = 0; i < NV; ++i)
                            acc[nb][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[MI + nb * NI + j], f[i],
                                                                                    acc[nb][i][j], 0, 0, 0);
            };
            Frags f0, f1;
            read_frags(nv_tag, consumed % NS, 0, f0);
            for (int ck = 0; ck < nk; ++ck) {
                const int slot = consumed % NS;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    Frags& cur = (ks & 1) ? f1 : f0;
                    Frags& nxt = (ks & 1) ? f0 : f1;
                    if (ks + 1 < KS) {
                        read_frags(nv_tag, slot, ks + 1, nxt);
                    } else if (ck + 1 < nk) {
                        // publish stage consumed + 1 (see above), refill, start its fragments
                        wait_lgkm0();
                        wait_stages<LPW, NS>(issued - consumed - 2);
                        stage_barrier();
                        issue_next();
                        read_frags(nv_tag, (consumed + 1) % NS, 0, nxt);
                    }
                    if (NV > 0) {
                        mma(cur);
                        interleave_reads<NB * NV * NI, NV + NB * NI>();
                    }
                }
                // KS is even for BK 32 / 64, so the next step's first fragments are in f0
                ++consumed;
            }
        };
        if (nv == MI) k_loop(std::integral_constant<int, MI>());
        else if (nv > 0) k_loop(std::integral_constant<int, MI / 2>());
        else k_loop(std::integral_constant<int, 0>());

        // ---- epilogue of tile ct.  D[n][m] layout: lane holds activation row l32 of the
        // block; register r holds weight row 8 * (r / 4) + 4 * lhi + r % 4, i.e. 4
        // consecutive output columns per group r / 4.  bf16 output: two 16-byte runs per
        // lane and block (store_block_bf16); fp32 output: the four groups as 16-byte vectors,
        // 8 elements apart from the lane's address (immediate store offsets).
        const int64_t row_lo = t.row0 > 0 ? t.row0 : 0;
        if (ks > 1) {
            // a K part: its fp32 sums go to partial[part][row][N], the reduce kernel finishes
            float* const part = g.partial + static_cast<int64_t>(ct % ks) * g.rows_max * g.N;
#pragma unroll
            for (int i = 0; i < MI; ++i) {
                if (i >= nv) break;
                const int64_t row = t.row_base + wm * (BM / 2) + i * 32 + l32;
                const bool row_ok = row >= row_lo && row < t.row_end;
#pragma unroll
                for (int j = 0; j < NI; ++j) {
                    const int col0 = t.n_base + wn * (BN / WN) + j * 32 + 4 * lhi;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int col = col0 + 8 * q;
                        if (row_ok && col >= t.n0 && col < g.N)
                            *reinterpret_cast<float4*>(part + row * g.N + col) =
                                make_float4(acc_read<kAccInAgpr>(acc[0][i][j][4 * q]),
                                            acc_read<kAccInAgpr>(acc[0][i][j][4 * q + 1]),
                                            acc_read<kAccInAgpr>(acc[0][i][j][4 * q + 2]),
                                            acc_read<kAccInAgpr>(acc[0][i][j][4 * q + 3]));
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
            }
            continue;
        }
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            if (i >= nv) break;  // no valid row in this block or any later one
            int64_t row = t.row_base + wm * (BM / 2) + i * 32 + l32;
            const bool row_ok = row >= row_lo && row < t.row_end;
            float scale = 1.f;
            if (!kUp && g.scatter) {
                // the grouped row's token and gate weight (one index load per tile and row)
                const int64_t src = row_ok ? g.scatter[row] : 0;
                row = src < 0 ? 0 : (src >= g.c_rows ? g.c_rows - 1 : src);
                scale = row_ok ? g.scatter_w[row] : 0.f;
            }
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int cb = t.n_base + wn * (BN / WN) + j * 32;  // the block's first column
                if constexpr (OB) {
                    uint2 pk[4];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        float v[4];
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            v[c] = scale * epilogue_fast<EPI>(acc_read<kAccInAgpr>(acc[0][i][j][4 * q + c]),
                                                              acc_read<kAccInAgpr>(acc[NB - 1][i][j][4 * q + c]));
                        pk[q].x = pack_bf16x2(v[0], v[1]);
                        pk[q].y = pack_bf16x2(v[2], v[3]);
                    }
                    // runs of 8 columns from c0 and c0 + 16: inside one 32-column block of
                    // K-blocked H (N, n0 and cb are multiples of 32 there), or inside a row of
                    // y (N, n0 and cb are multiples of 8), wholly before n0 or wholly after it
                    const int c0 = cb + 8 * lhi;
                    bf16_t* const dst = static_cast<bf16_t*>(g.c) +
                                        (kUp ? ((static_cast<int64_t>(cb) >> 5) * g.rows_max + row) * 32 + 8 * lhi
                                             : row * g.ldc + c0);
                    store_block_bf16(dst, pk, row_ok && c0 >= t.n0 && c0 < g.N,
                                     row_ok && c0 + 16 >= t.n0 && c0 + 16 < g.N);
                } else {
                    // fp32 y_perm (down-projection): groups of 4 columns, N % 4 == 0
                    const int col0 = cb + 4 * lhi;
                    float* const dst = static_cast<float*>(g.c) + row * g.ldc + col0;
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int col = col0 + 8 * q;
                        float v[4];
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            v[c] = scale * epilogue_fast<EPI>(acc_read<kAccInAgpr>(acc[0][i][j][4 * q + c]),
                                                              acc_read<kAccInAgpr>(acc[NB - 1][i][j][4 * q + c]));
                        if (row_ok && col >= t.n0 && col < g.N)
                            *reinterpret_cast<float4*>(dst + 8 * q) = make_float4(v[0], v[1], v[2], v[3]);
                        __builtin_amdgcn_sched_barrier(0);
                    }
                }
                // one block at a time: keeps the scheduler from pulling every accumulator
                // into VGPRs at once
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}
// ------------------------------------------------------------------ bf16 up-projection, paired A stages
//
// The up-projection's activations are rows of x (gathered through row_src) or of x_perm,
// row-major, so the kernel above reads them as 64-byte pieces: half a 128-byte line per
// stage, the other half a stage later.  This variant (K % 64 == 0) loads 128 bytes of an
// activation row for two stages at once.  The A side has two 16 KiB slots of 128 rows x
// 128 bytes (one in use, one filling; chunk c of row r sits at c ^ (r % 8), so the 8 rows
// that 8 lanes of a fragment read touch fall on 8 different bank groups); the weights keep
// the three-stage ring of K-blocked 256-row stages.  That is 80 KiB, two workgroups per CU
// with nothing left over, so the row-tile table is kept in registers.  Even stages issue 4
// A and 4 B loads per wave, odd stages 4 B loads; the vmcnt waits count them that way.
// Fragments, MFMA order and epilogue are those of gemm_bf16_lds<128, 256, 32, 3, EPI,
// true>, and so is every output bit.
constexpr int kUpASlot = 128 * 128;                       // bytes of one A slot
constexpr int kUpBSlot = 256 * 64;                        // bytes of one B stage
constexpr size_t kUpPairBytes = 2 * kUpASlot + 3 * kUpBSlot;  // 80 KiB

template <int EPI>
__global__ __launch_bounds__(kThreads, 2) void gemm_up_pairs(GroupedGemm g) {
    constexpr int BM = 128, BW = 256, NS = 3;
    typedef LdsShape<BM, BW, 32, NS, EPI> S;
    constexpr int NB = S::kNB, BN = S::kBN, MI = S::kMI, NI = S::kNI, KS = S::kKS;
    constexpr int kBBase = 2 * kUpASlot;
    constexpr int LPA = BM / 8 / 4;   // 1 KiB loads per wave of an A pair (8 rows x 128 bytes)
    constexpr int LPB = BW / 16 / 4;  // 1 KiB loads per wave of a B stage (16 rows x 64 bytes)
    static_assert(kUpPairBytes <= 80 * 1024, "two workgroups per CU");
    extern __shared__ __align__(1024) unsigned char smem_raw[];

    RegTiles<BM> tiles;
    tiles.build(g.offsets, g.E);
    const int total_m = tiles.total;
    const int total = total_m * g.n_tiles;
    const int per = (total + 7) >> 3;
    const int xcd = blockIdx.x & 7, nslot = gridDim.x >> 3;
    const int t_end = min(total, (xcd + 1) * per);
    const int t_first = xcd * per + static_cast<int>(blockIdx.x >> 3);
    if (t_first >= t_end) return;
    const int nk = g.K / 32;  // even: the host runs this kernel only for K % 64 == 0

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds0 = lds_address(smem_raw);
    const int a_lim = static_cast<int>(g.rows_max < BM ? g.rows_max : BM) - 1;
    const int b_lim = (g.N < BN ? g.N : BN) - 1;

    // B: load j fills B rows (4 j + wave) 16 + lane / 4 of a stage, slot lane % 4, with global
    // chunk slot ^ ((row / 4) % 4); the same for every tile
    uint32_t voffB[LPB];
#pragma unroll
    for (int j = 0; j < LPB; ++j) {
        const int R = (j * 4 + wave) * 16 + (lane >> 2);
        const int kc = (lane & 3) ^ ((R >> 2) & 3);
        voffB[j] = static_cast<uint32_t>(min(R % BN, b_lim)) * 64u + static_cast<uint32_t>(kc * 16);
    }
    // A: load j fills A rows (4 j + wave) 8 + lane / 8 of a slot, slot lane % 8, with global
    // chunk slot ^ (row % 8); set per tile
    uint32_t voffA[LPA];

    int lt = t_first, lk = 0;
    const unsigned char *src_a = nullptr, *src_b0 = nullptr, *src_b1 = nullptr;
    auto set_tile = [&](int L) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, L);
#pragma unroll
        for (int j = 0; j < LPA; ++j) {
            const int R = (j * 4 + wave) * 8 + (lane >> 3);
            const int c = (lane & 7) ^ (R & 7);
            // gathered: absolute source row (T h s < 4 GiB is checked by the host); else the
            // tile's base carries the row offset
            const int a_lim_t = tile_row_limit<BM>(g, t);
            const int64_t r = g.gather ? source_row(g, t.row_base + min(R, a_lim_t)) : min(R, a_lim_t);
            voffA[j] = static_cast<uint32_t>(r) * static_cast<uint32_t>(2 * g.K) + static_cast<uint32_t>(c * 16);
        }
        src_a = uniform_ptr(static_cast<const unsigned char*>(g.a) + (g.gather ? 0 : t.row_base * 2 * g.K));
        const int64_t boff = (t.e * g.b_estride) * 2 + static_cast<int64_t>(t.n_base) * 64;
        src_b0 = uniform_ptr(static_cast<const unsigned char*>(g.b) + boff);
        src_b1 = NB > 1 ? uniform_ptr(static_cast<const unsigned char*>(g.b2) + boff) : src_b0;
    };
    int issued = 0;  // stages issued by this wave so far (even at every tile start: nk is even)
    auto issue_next = [&]() {
        if (lt >= t_end) return;
        if ((lk & 1) == 0) {
            // the next 128 bytes of every activation row: K blocks lk and lk + 1
            const uint32_t da = lds0 + ((issued >> 1) & 1) * kUpASlot;
#pragma unroll
            for (int j = 0; j < LPA; ++j)
                load_lds16(src_a + static_cast<int64_t>(lk) * 64, voffA[j], da + (j * 4 + wave) * 1024);
        }
        const uint32_t db = lds0 + kBBase + (issued % NS) * kUpBSlot;
        const int64_t kb = static_cast<int64_t>(lk) * g.N * 64;
#pragma unroll
        for (int j = 0; j < LPB; ++j)
            load_lds16(((NB > 1 && j * 4 * 16 >= BN) ? src_b1 : src_b0) + kb, voffB[j], db + (j * 4 + wave) * 1024);
        ++issued;
        if (++lk == nk) {
            lk = 0;
            lt += nslot;
            if (lt < t_end) set_tile(lt);
        }
    };
    // wait until stage `st` is in LDS while `newer` later stages stay in flight
    auto wait_stage = [&](int st, int newer) {
        if (newer >= 2) wait_vmcnt<LPA + 2 * LPB>();
        else if (newer == 1 && ((st + 1) & 1) == 0) wait_vmcnt<LPA + LPB>();
        else if (newer == 1) wait_vmcnt<LPB>();
        else wait_vmcnt<0>();
    };
    set_tile(lt);
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue_next();

    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lhi = lane >> 5;
    typedef bf16x8_t Frags[MI + NB * NI];
    // fragments of stage st (its A slot and half of the slot's rows, its B ring slot)
    auto read_frags = [&](auto nv_tag, int st, int ks, Frags& f) {
        constexpr int NV = decltype(nv_tag)::value;
        const unsigned char* sa = smem_raw + ((st >> 1) & 1) * kUpASlot;
        const int ca = (st & 1) * 4 + 2 * ks + lhi;
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int R = wm * (BM / 2) + i * 32 + l32;
            f[i] = *reinterpret_cast<const bf16x8_t*>(sa + R * 128 + ((ca ^ (R & 7)) << 4));
        }
        if (NV == 0) return;
        const unsigned char* sb = smem_raw + kBBase + (st % NS) * kUpBSlot;
        const int cb = 2 * ks + lhi;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int R = nb * BN + wn * (BN / 2) + j * 32 + l32;
                f[MI + nb * NI + j] = *reinterpret_cast<const bf16x8_t*>(sb + R * 64 + ((cb ^ ((R >> 2) & 3)) << 4));
            }
    };

    int consumed = 0;
    for (int ct = t_first; ct < t_end; ct += nslot) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, ct);
        int nv = MI;
        if (t.row_base == t.row0) {
            const int64_t left = t.row_end - (t.row0 + wm * (BM / 2));
            nv = left <= 0 ? 0 : (left > (MI / 2) * 32 ? MI : MI / 2);
        }
        nv = __builtin_amdgcn_readfirstlane(nv);

        f32x16_t acc[NB][MI][NI];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NI; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[nb][i][j][r] = 0.f;

        // publish the tile's first stage; after an epilogue its stores share the counter
        if (ct != t_first) wait_vmcnt<0>();
        else wait_stage(consumed, issued - consumed - 1);
        stage_barrier();
        issue_next();

        auto k_loop = [&](auto nv_tag) {
            constexpr int NV = decltype(nv_tag)::value;
            auto mma = [&](const Frags& f) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int j = 0; j < NI; ++j)
#pragma unroll
                        for (int i = 0; i < NV; ++i)
                            acc[nb][i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[MI + nb * NI + j], f[i],
                                                                                    acc[nb][i][j], 0, 0, 0);
            };
            Frags f0, f1;
            read_frags(nv_tag, consumed, 0, f0);
            for (int ck = 0; ck < nk; ++ck) {
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    Frags& cur = (ks & 1) ? f1 : f0;
                    Frags& nxt = (ks & 1) ? f0 : f1;
                    if (ks + 1 < KS) {
                        read_frags(nv_tag, consumed, ks + 1, nxt);
                    } else if (ck + 1 < nk) {
                        wait_lgkm0();
                        wait_stage(consumed + 1, issued - consumed - 2);
                        stage_barrier();
                        issue_next();
                        read_frags(nv_tag, consumed + 1, 0, nxt);
                    }
                    if (NV > 0) {
                        mma(cur);
                        interleave_reads<NB * NV * NI, NV + NB * NI>();
                    }
                }
                ++consumed;
            }
        };
        if (nv == MI) k_loop(std::integral_constant<int, MI>());
        else if (nv > 0) k_loop(std::integral_constant<int, MI / 2>());
        else k_loop(std::integral_constant<int, 0>());

        // epilogue: as in gemm_bf16_lds (bf16 H, K-blocked)
        const int64_t row_lo = t.row0 > 0 ? t.row0 : 0;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
            if (i >= nv) break;
            const int64_t row = t.row_base + wm * (BM / 2) + i * 32 + l32;
            const bool row_ok = row >= row_lo && row < t.row_end;
#pragma unroll
            for (int j = 0; j < NI; ++j) {
                const int cb = t.n_base + wn * (BN / 2) + j * 32;  // the block's first column
                uint2 pk[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float v[4];
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        v[c] = epilogue_fast<EPI>(acc[0][i][j][4 * q + c], acc[NB - 1][i][j][4 * q + c]);
                    pk[q].x = pack_bf16x2(v[0], v[1]);
                    pk[q].y = pack_bf16x2(v[2], v[3]);
                }
                bf16_t* const dst = static_cast<bf16_t*>(g.c) +
                                    ((static_cast<int64_t>(cb) >> 5) * g.rows_max + row) * 32 + 8 * lhi;
                const bool ok = row_ok && cb >= t.n0 && cb < g.N;  // N, n0, cb: multiples of 32
                store_block_bf16(dst, pk, ok, ok);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// ------------------------------------------------------------------ fp32 kernel
//
// 64 x 64 tiles on the fp32 matrix cores: four waves, each one 32 x 32 block of
// v_mfma_f32_32x32x2_f32 (lane l supplies A[row l % 32][k l / 32] and B[k l / 32][column
// l % 32] of a two-wide K step, and ends holding column l % 32 of the block).  K advances
// 32 at a time through two LDS buffers stored K-major ([k][row], 4 floats of padding),
// each filled from registers loaded two steps earlier (two register sets take turns), so
// a step's MFMAs overlap the loads of the next two.  Gathered rows are looked up once.

constexpr int kFBM = 64, kFBN = 64, kFBK = 32, kFLD = kFBM + 4;

template <int EPI, bool OB>
__global__ __launch_bounds__(kThreads) void gemm_f32(GroupedGemm g) {
    constexpr int NB = (EPI == kEpiSwiglu) ? 2 : 1;
    __shared__ int tstart[kThreads + 1];
    __shared__ __align__(16) float As[2][kFBK][kFLD];
    __shared__ __align__(16) float Bs[2][NB][kFBK][kFLD];

    const int total = tile_prefix<kFBM>(g.offsets, g.E, tstart);
    // work item = tile blockIdx / ks, K part blockIdx % ks (ks = 1 unless the down-projection
    // is split: then part p covers K steps [p nk, (p + 1) nk) and writes fp32 partial sums)
    const int ks = (EPI == kEpiNone && g.ksplit > 1) ? g.ksplit : 1;
    const int tile = blockIdx.x / ks, part = blockIdx.x - tile * ks;
    const int mt = tile / g.n_tiles;
    const int nt = tile - mt * g.n_tiles;
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

    // loader: thread t brings rows t / 8 and t / 8 + 32, K values 4 (t % 8) .. + 3 of the step
    // (K % 4 == 0, so a float4 never straddles the end of K)
    const int tid = threadIdx.x;
    const int lrow = tid >> 3, lk = (tid & 7) * 4;
    const float* arow[2];  // this thread's two activation rows (null: past the segment)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int64_t ar = row0 + lrow + 32 * h;
        arow[h] = ar < row_end ? A + source_row(g, ar) * g.K : nullptr;
    }
    struct Regs {
        float4 a[2], b[NB][2];
    };
    const int nk = (g.K + kFBK - 1) / kFBK / ks;  // K steps of this work item (exact when ks > 1)
    const int kt0 = part * nk;
    auto gload = [&](Regs& R, int kt) {
        const int k = (kt0 + kt) * kFBK + lk;
        const bool kv = k < g.K;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            R.a[h] = (arow[h] && kv) ? *reinterpret_cast<const float4*>(arow[h] + k) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int n = n0 + lrow + 32 * h;
                R.b[nb][h] = (n < g.N && kv)
                                 ? *reinterpret_cast<const float4*>(Bm[nb] + static_cast<int64_t>(n) * g.K + k)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    };
    auto sstore = [&](const Regs& R, int buf) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = lrow + 32 * h;
            As[buf][lk + 0][r] = R.a[h].x;
            As[buf][lk + 1][r] = R.a[h].y;
            As[buf][lk + 2][r] = R.a[h].z;
            As[buf][lk + 3][r] = R.a[h].w;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                Bs[buf][nb][lk + 0][r] = R.b[nb][h].x;
                Bs[buf][nb][lk + 1][r] = R.b[nb][h].y;
                Bs[buf][nb][lk + 2][r] = R.b[nb][h].z;
                Bs[buf][nb][lk + 3][r] = R.b[nb][h].w;
            }
        }
    };

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31, lhi = lane >> 5;
    f32x16_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;

    // step kt: MFMAs on LDS buffer kt % 2; register set `next` holds step kt + 1 and goes to
    // the other buffer after them (that buffer was last read before the previous step's
    // barrier), then takes the loads of step kt + 3
    // a wave whose 32 rows all lie past the segment skips its MFMAs (it still loads and
    // takes part in the barriers); its block is never stored
    const bool live = row0 + wm * 32 < row_end;
    auto step = [&](int kt, Regs& next) {
        const int buf = kt & 1;
        if (live) {
#pragma unroll
            for (int ks = 0; ks < kFBK / 2; ++ks) {
                const float a = As[buf][2 * ks + lhi][wm * 32 + l32];
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, Bs[buf][nb][2 * ks + lhi][wn * 32 + l32],
                                                                   acc[nb], 0, 0, 0);
            }
        }
        if (kt + 1 < nk) sstore(next, buf ^ 1);
        __syncthreads();
        if (kt + 3 < nk) gload(next, kt + 3);
    };
    Regs r0, r1;
    gload(r0, 0);
    sstore(r0, 0);
    if (nk > 1) gload(r1, 1);
    if (nk > 2) gload(r0, 2);
    __syncthreads();
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        step(kt, r1);      // r1 holds step kt + 1, then loads kt + 3
        step(kt + 1, r0);  // r0 holds step kt + 2, then loads kt + 4
    }
    if (kt < nk) step(kt, r1);

    // epilogue: register r holds row 8 (r / 4) + 4 lhi + r % 4 of the wave's block; for a
    // fixed r the 32 lanes of a half-wave store 32 consecutive columns
    const int n = n0 + wn * 32 + l32;
    if (n >= g.N) return;
    if (ks > 1) {
        // a K part: its fp32 sums go to partial[part][row][N], the reduce kernel finishes
        float* const dst = g.partial + static_cast<int64_t>(part) * g.rows_max * g.N;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = row0 + wm * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
            if (row < row_end) dst[row * g.N + n] = acc[0][r];
        }
        return;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        int64_t row = row0 + wm * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3);
        if (row >= row_end) continue;
        float scale = 1.f;
        if (g.scatter) {
            const int64_t src = g.scatter[row];
            row = src < 0 ? 0 : (src >= g.c_rows ? g.c_rows - 1 : src);
            scale = g.scatter_w[row];
        }
        const float v = scale * epilogue<EPI>(acc[0][r], acc[NB - 1][r]);
        if (OB) static_cast<bf16_t*>(g.c)[row * g.ldc + n] = f32_to_bf16(v);
        else static_cast<float*>(g.c)[row * g.ldc + n] = v;
    }
}

// ------------------------------------------------------------------ fp32 pipelined kernel
//
// fp32 operands whose K is a multiple of 32 (every down-projection; the up-projection when
// h % 32 == 0).  Tiles of 32 activation rows x 128 weight rows of each matrix; four waves,
// wave w owning output columns 32 w .. 32 w + 31 of the tile in every matrix.
// v_mfma_f32_32x32x2_f32 takes the weights as its first operand, so a lane ends up holding
// one activation row and, in each group of four registers, four consecutive output columns.
// K advances 32 values (128 bytes of every row) per stage; a stage goes straight to LDS as
// 1 KiB direct loads of 8 rows x 128 bytes, NS stages with NS - 1 in flight across K steps
// and work items (the bf16 kernel's pipeline).  Inside a stage a lane reads, for each group
// of 8 K values, 4 consecutive K values of its row as one 16-byte fragment and feeds element
// c to the c-th of four MFMAs; the other half-wave supplies the group's other 4 K values, so
// the four MFMAs together sum over the whole group.  32-row tiles hold at least one valid
// row each, and an expert's rows waste at most 31 padded rows.  Persistent grid: work items
// (tile, K part) are dealt to the XCDs in contiguous runs and round-robin to each XCD's
// workgroups.  Two stages (one in flight): with one matrix a workgroup needs 40 KiB and
// three share a CU (three waves per SIMD hide each other's waits; measured 3 % faster on a
// 512-token top-1 step than three stages at two per CU), with two matrices 72 KiB and two.
constexpr int kF2BM = 32, kF2BN = 128, kF2BK = 32;  // kF2BK counts floats: 128-byte row pieces

template <int NB>
struct F32Shape {
    static constexpr int kRows = kF2BM + NB * kF2BN;  // LDS rows per stage
    static constexpr int kStageBytes = kRows * kF2BK * 4;
    static constexpr int kLPW = kRows / 8 / 4;         // 1 KiB loads per wave per stage
    static constexpr int kStages = 2;
    static constexpr size_t kBytes = static_cast<size_t>(kStages) * kStageBytes;
    static constexpr int kPerCU = NB == 1 ? 3 : 2;      // workgroups per CU (160 KiB of LDS)
    static_assert(kPerCU * kBytes <= 160 * 1024, "LDS per CU");
};

template <int EPI, bool OB>
__global__ __launch_bounds__(kThreads, (F32Shape<(EPI == kEpiSwiglu) ? 2 : 1>::kPerCU)) void gemm_f32_lds(GroupedGemm g) {
    constexpr int NB = (EPI == kEpiSwiglu) ? 2 : 1;
    typedef F32Shape<NB> S;
    constexpr int BM = kF2BM, BN = kF2BN, LPW = S::kLPW, NS = S::kStages;
    constexpr int kStageBytes = S::kStageBytes;
    constexpr bool kUp = EPI != kEpiNone;
    static_assert(LPW == 1 + 4 * NB, "load 0 carries the 32 activation rows, loads 4 nb + 1 .. 4 nb + 4 matrix nb");
    __shared__ int tstart[kThreads + 1];
    extern __shared__ __align__(1024) unsigned char smem_raw[];

    const int total_m = tile_prefix<BM>(g.offsets, g.E, tstart);
    const LdsTiles tiles{tstart, g.E};
    // work item L: tile L / ks, K part L % ks (ks = 1 unless the down-projection is split)
    const int ks = (!kUp && g.ksplit > 1) ? g.ksplit : 1;
    const int total = total_m * g.n_tiles * ks;
    const int per = (total + 7) >> 3;
    const int xcd = blockIdx.x & 7, nslot = gridDim.x >> 3;
    const int t_first = xcd * per + static_cast<int>(blockIdx.x >> 3);
    const int t_end = min(total, xcd * per + per);
    if (t_first >= t_end) return;
    const int nk = g.K / kF2BK / ks;  // stages per work item

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t lds0 = lds_address(smem_raw);

    // Per-lane byte offsets of this wave's loads: load j fills LDS rows 8 (4 j + wave) + lane
    // / 8 of a stage, 16-byte slot lane % 8, from global slot (lane % 8) ^ swz(row).  Rows past
    // a buffer smaller than one tile repeat its last row.
    const int r_lane = lane >> 3;
    const int a_lim = static_cast<int>(g.rows_max < BM ? g.rows_max : BM) - 1;
    const int b_lim = (g.N < BN ? g.N : BN) - 1;
    uint32_t voff[LPW];
#pragma unroll
    for (int j = 1; j < LPW; ++j) {
        const int R = 8 * (4 * j + wave) + r_lane;
        const int kc = (lane & 7) ^ ((R >> 1) & 7);
        const int r = min((R - BM) % BN, b_lim);
        voff[j] = static_cast<uint32_t>(r) * static_cast<uint32_t>(4 * g.K) + static_cast<uint32_t>(kc * 16);
    }
    const int ra = min(8 * wave + r_lane, a_lim);  // this lane's activation row in load 0
    const uint32_t kca = static_cast<uint32_t>(((lane & 7) ^ (((8 * wave + r_lane) >> 1) & 7)) * 16);

    // ---- load cursor: work item li, K step lk, scalar bases of the item's rows
    int li = t_first, lk = 0;
    const unsigned char *src_a = nullptr, *src_b0 = nullptr, *src_b1 = nullptr;
    auto set_item = [&](int L) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, L / ks);
        const int64_t k0 = static_cast<int64_t>(L % ks) * nk * kF2BK;  // first K value of the item
        if (g.gather) {
            // absolute source row (T h 4 < 4 GiB is checked by the host)
            const int64_t src = source_row(g, t.row_base + ra);
            voff[0] = static_cast<uint32_t>(src) * static_cast<uint32_t>(4 * g.K) + kca;
            src_a = uniform_ptr(static_cast<const float*>(g.a) + k0);
        } else {
            voff[0] = static_cast<uint32_t>(ra) * static_cast<uint32_t>(4 * g.K) + kca;
            src_a = uniform_ptr(static_cast<const float*>(g.a) + t.row_base * g.K + k0);
        }
        const int64_t boff = t.e * g.b_estride + static_cast<int64_t>(t.n_base) * g.K + k0;
        src_b0 = uniform_ptr(static_cast<const float*>(g.b) + boff);
        src_b1 = NB > 1 ? uniform_ptr(static_cast<const float*>(g.b2) + boff) : src_b0;
    };
    int issued = 0;  // stages issued by this wave so far
    auto issue_next = [&]() {
        if (li >= t_end) return;
        const uint32_t dst = lds0 + (issued % NS) * kStageBytes;
        const int kb = lk * kF2BK * 4;  // bytes into every row
#pragma unroll
        for (int j = 0; j < LPW; ++j) {
            const unsigned char* base = j == 0 ? src_a : ((j - 1) / 4 == 0 ? src_b0 : src_b1);
            load_lds16(base + kb, voff[j], dst + (4 * j + wave) * 1024);
        }
        ++issued;
        if (++lk == nk) {
            lk = 0;
            li += nslot;
            if (li < t_end) set_item(li);
        }
    };
    set_item(li);
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue_next();

    const int l32 = lane & 31, lhi = lane >> 5;
    int consumed = 0;
    for (int L = t_first; L < t_end; L += nslot) {
        const TileGeom t = tile_geom<BM, BN>(g, tiles, total_m, L / ks);
        f32x16_t acc[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;

        // publish the item's first stage (after an epilogue its stores share the counter)
        wait_lgkm0();
        if (L != t_first) wait_vmcnt<0>();
        else wait_stages<LPW, NS>(issued - consumed - 1);
        stage_barrier();
        issue_next();
        for (int ck = 0; ck < nk; ++ck) {
            const unsigned char* st = smem_raw + (consumed % NS) * kStageBytes;
#pragma unroll
            for (int q = 0; q < kF2BK / 8; ++q) {
                const int slot = 2 * q + lhi;
                const float4 xf = *reinterpret_cast<const float4*>(st + l32 * 128 + ((slot ^ ((l32 >> 1) & 7)) << 4));
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const int Rw = BM + nb * BN + 32 * wave + l32;
                    const float4 wf =
                        *reinterpret_cast<const float4*>(st + Rw * 128 + ((slot ^ ((Rw >> 1) & 7)) << 4));
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wf.x, xf.x, acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wf.y, xf.y, acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wf.z, xf.z, acc[nb], 0, 0, 0);
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(wf.w, xf.w, acc[nb], 0, 0, 0);
                }
            }
            ++consumed;
            if (ck + 1 < nk) {
                // publish the next stage: own reads of this one done, own loads of the next
                // landed; then refill this stage's buffer
                wait_lgkm0();
                wait_stages<LPW, NS>(issued - consumed - 1);
                stage_barrier();
                issue_next();
            }
        }

        // ---- epilogue.  Lane: activation row row_base + l32; register 4 q + c: output column
        // n_base + 32 wave + 8 q + 4 lhi + c.
        const int64_t row = t.row_base + l32;
        const int64_t row_lo = t.row0 > 0 ? t.row0 : 0;
        const bool row_ok = row >= row_lo && row < t.row_end;
        const int cb = t.n_base + 32 * wave + 4 * lhi;
        if (ks > 1) {
            // a K part: its fp32 sums go to partial[part][row][N], the reduce kernel finishes
            float* const dst = g.partial + static_cast<int64_t>(L % ks) * g.rows_max * g.N;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = cb + 8 * q;
                if (row_ok && col >= t.n0 && col < g.N)
                    *reinterpret_cast<float4*>(dst + row * g.N + col) =
                        make_float4(acc[0][4 * q], acc[0][4 * q + 1], acc[0][4 * q + 2], acc[0][4 * q + 3]);
            }
            continue;
        }
        int64_t orow = row;
        float scale = 1.f;
        if (!kUp && g.scatter) {
            // the grouped row's token and gate weight
            const int64_t src = row_ok ? g.scatter[row] : 0;
            orow = src < 0 ? 0 : (src >= g.c_rows ? g.c_rows - 1 : src);
            scale = row_ok ? g.scatter_w[orow] : 0.f;
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int col = cb + 8 * q;
            if (!row_ok || col < t.n0 || col >= g.N) continue;
            float v[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) v[c] = scale * epilogue<EPI>(acc[0][4 * q + c], acc[NB - 1][4 * q + c]);
            if constexpr (OB) {
                uint2 pk;
                pk.x = pack_bf16x2(v[0], v[1]);
                pk.y = pack_bf16x2(v[2], v[3]);
                *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.c) + orow * g.ldc + col) = pk;
            } else {
                *reinterpret_cast<float4*>(static_cast<float*>(g.c) + orow * g.ldc + col) =
                    make_float4(v[0], v[1], v[2], v[3]);
            }
        }
    }
}

// ------------------------------------------------------------------ split-K reduce
//
// out[p] = sum over s of partial[s][p] (s ascending) for the grouped rows p of the call,
// [offsets[0], offsets[E]); with scatter (top-1), out[t] = w[t] * that sum for
// t = scatter[p] instead (the down-projection's own epilogue, applied after the parts
// meet).  N % 4 == 0.  S (2, 4 or 8 parts) is a template argument so that a thread's S
// loads are issued together (one memory round trip) before the sum.

template <bool OB, int S>
__global__ __launch_bounds__(256) void split_reduce(const float* __restrict__ partial, int64_t rows_max,
                                                     int N, const int32_t* __restrict__ offsets, int E,
                                                     void* __restrict__ out, int ldo,
                                                     const int32_t* __restrict__ scatter,
                                                     const float* __restrict__ scatter_w, int64_t c_rows) {
    const int64_t p0 = offsets[0];
    const int64_t p1 = offsets[E] < rows_max ? offsets[E] : rows_max;
    const int nv = N / 4;
    const int64_t n = (p1 - p0) * nv;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * 256) {
        const int64_t p = p0 + i / nv;
        const int c = static_cast<int>(i % nv) * 4;
        float4 u[S];
#pragma unroll
        for (int s = 0; s < S; ++s)
            u[s] = *reinterpret_cast<const float4*>(partial + (static_cast<int64_t>(s) * rows_max + p) * N + c);
        float4 v = u[0];
#pragma unroll
        for (int s = 1; s < S; ++s) {
            v.x += u[s].x;
            v.y += u[s].y;
            v.z += u[s].z;
            v.w += u[s].w;
        }
        int64_t row = p;
        if (scatter) {
            const int64_t t = scatter[p];
            row = t < 0 ? 0 : (t >= c_rows ? c_rows - 1 : t);
            const float w = scatter_w[row];
            v.x *= w;
            v.y *= w;
            v.z *= w;
            v.w *= w;
        }
        if (OB) {
            uint2 pk;
            pk.x = pack_bf16x2(v.x, v.y);
            pk.y = pack_bf16x2(v.z, v.w);
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(out) + row * ldo + c) = pk;
        } else {
            *reinterpret_cast<float4*>(static_cast<float*>(out) + row * ldo + c) = v;
        }
    }
}


// Steps 4 and 5 together when the second product's K is split: for token t and 8 columns,
//     y[t] = sum over picks j of w[t, j] * round_ydt(sum over s of partial[s][pos_of[t, j]])
// -- exactly split_reduce's sum (parts in order), rounded to y_perm's type as split_reduce
// stores it, then combine's weighted sum (fp32, pick order, invalid picks skipped) rounded
// once: the same bits as the two launches, without writing or reading y_perm.
template <bool YB, bool OB, int S>
__global__ __launch_bounds__(256) void split_combine(const float* __restrict__ partial, int64_t rows_max,
                                                     int h, const int32_t* __restrict__ pos_of,
                                                     const float* __restrict__ w, int64_t T, int k,
                                                     void* __restrict__ y) {
    const int nv = h / 8;
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= T * nv) return;
    const int64_t t = i / nv;
    const int c = static_cast<int>(i - t * nv) * 8;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
        const int32_t p = pos_of[t * k + j];
        if (p < 0 || p >= T * k) continue;
        const float wt = w[t * k + j];
        const float* src = partial + static_cast<int64_t>(p) * h + c;
        float4 u[S], v[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const float* q = src + static_cast<int64_t>(s) * rows_max * h;
            u[s] = *reinterpret_cast<const float4*>(q);
            v[s] = *reinterpret_cast<const float4*>(q + 4);
        }
        float4 a = u[0], b = v[0];
#pragma unroll
        for (int s = 1; s < S; ++s) {
            a.x += u[s].x;
            a.y += u[s].y;
            a.z += u[s].z;
            a.w += u[s].w;
            b.x += v[s].x;
            b.y += v[s].y;
            b.z += v[s].z;
            b.w += v[s].w;
        }
        float r[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        if (YB) {
            // y_perm's bf16 rounding, as split_reduce stores it and combine reads it back
#pragma unroll
            for (int q = 0; q < 8; q += 2) {
                const uint32_t pk = pack_bf16x2(r[q], r[q + 1]);
                r[q] = __uint_as_float(pk << 16);
                r[q + 1] = __uint_as_float(pk & 0xffff0000u);
            }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += wt * r[q];
    }
    if (OB) {
        uint4 q;
        q.x = pack_bf16x2(acc[0], acc[1]);
        q.y = pack_bf16x2(acc[2], acc[3]);
        q.z = pack_bf16x2(acc[4], acc[5]);
        q.w = pack_bf16x2(acc[6], acc[7]);
        *reinterpret_cast<uint4*>(static_cast<bf16_t*>(y) + t * h + c) = q;
    } else {
        float4* o = reinterpret_cast<float4*>(static_cast<float*>(y) + t * h + c);
        o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
        o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
    }
}

// ------------------------------------------------------------------ launch

int64_t row_tile_bound(int64_t A_max, int E, int bm) {
    const int64_t b = ceil_div(A_max, bm) + E;
    return b < A_max ? b : A_max;
}

template <int EPI, bool OB, bool CB>
hipError_t run_bf16(GroupedGemm g, int64_t A_max, hipStream_t s) {
    typedef BfShape<EPI> S;
    constexpr size_t lds = bf_lds_bytes<EPI, OB>();
    static std::once_flag once;
    static hipError_t attr_err = hipSuccess;
    std::call_once(once, [] {
        attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16<EPI, OB, CB>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    });
    if (attr_err != hipSuccess) return attr_err;
    g.n_tiles = static_cast<int>(ceil_div(g.N, S::kBN));
    const int64_t blocks = row_tile_bound(A_max, g.E, kBM) * g.n_tiles;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((gemm_bf16<EPI, OB, CB>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, s, g);
    return hipGetLastError();
}

int device_cus();

template <int EPI, bool OB>
hipError_t run_f32_lds(GroupedGemm g, int64_t A_max, hipStream_t s) {
    typedef F32Shape<(EPI == kEpiSwiglu) ? 2 : 1> S;
    constexpr size_t lds = S::kBytes;
    static const hipError_t attr = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_f32_lds<EPI, OB>),
                                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                                       static_cast<int>(lds));
    if (attr != hipSuccess) return attr;
    g.n_tiles = static_cast<int>(ceil_div(g.N, kF2BN));
    const int64_t items = row_tile_bound(A_max, g.E, kF2BM) * g.n_tiles * (g.ksplit > 1 ? g.ksplit : 1);
    if (items == 0) return hipSuccess;
    // persistent grid: at most kPerCU workgroups per CU, a multiple of the 8 XCDs
    const int64_t blocks = round_up(std::min<int64_t>(items, S::kPerCU * static_cast<int64_t>(device_cus())), 8);
    hipLaunchKernelGGL((gemm_f32_lds<EPI, OB>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), lds, s, g);
    return hipGetLastError();
}

template <int EPI, bool OB>
hipError_t run_f32(GroupedGemm g, int64_t A_max, hipStream_t s) {
    if (g.K % kF2BK == 0) return run_f32_lds<EPI, OB>(g, A_max, s);
    g.n_tiles = static_cast<int>(ceil_div(g.N, kFBN));
    const int64_t blocks = row_tile_bound(A_max, g.E, kFBM) * g.n_tiles * (g.ksplit > 1 ? g.ksplit : 1);
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

template <int BM, int BW, int BK, int NS, int EPI, bool OB, int WN = 2>
hipError_t run_bf16_lds(GroupedGemm g, int64_t A_max, hipStream_t s) {
    typedef LdsShape<BM, BW, BK, NS, EPI, WN> S;
    constexpr size_t lds = S::kBytes;
    constexpr int per_cu = S::kPerCU;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&gemm_bf16_lds<BM, BW, BK, NS, EPI, OB, WN>),
        hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (attr != hipSuccess) return attr;
    g.n_tiles = static_cast<int>(ceil_div(g.N, S::kBN));
    const int64_t tiles = row_tile_bound(A_max, g.E, BM) * g.n_tiles * (g.ksplit > 1 ? g.ksplit : 1);
    if (tiles == 0) return hipSuccess;
    // persistent grid: at most per_cu workgroups per CU, a multiple of the 8 XCDs
    const int64_t blocks = round_up(std::min<int64_t>(tiles, static_cast<int64_t>(per_cu) * device_cus()), 8);
    hipLaunchKernelGGL((gemm_bf16_lds<BM, BW, BK, NS, EPI, OB, WN>), dim3(static_cast<unsigned>(blocks)),
                       dim3(S::kThreadsWG), lds, s, g);
    return hipGetLastError();
}

// Tile shape: 128 activation rows x 256 weight rows, 32-wide K steps, three stages (two in
// flight) in 72 KiB of LDS, so that two workgroups share a CU and one's epilogue and
// pipeline fill overlap the other's MFMAs.
//
// The up-projection needs h % 32 == 0 for the pipelined kernel (the packed W1 is K-blocked
// exactly then); otherwise the register-staged kernel runs it on row-major weights and still
// writes H K-blocked.  The down-projection's K is fp, always a multiple of 128.
//
// When the down-projection's tiles fit on the CUs in one round even 384 columns wide (few
// rows, e.g. a top-1 layer of a few thousand tokens or a decode batch), it runs 128 x 384
// tiles, one workgroup per CU with 96 KiB of stages: every tile then streams its weights
// with more bytes in flight instead of a third of the CUs taking a second tile.  That
// workgroup has 8 waves (2 x 4, each 64 x 96), two per SIMD, so that one wave's LDS reads,
// loads and barrier waits overlap the other's MFMAs.  Each output element's K sum is the
// same in any of these shapes.
template <int EPI>
hipError_t run_up_pairs(GroupedGemm g, int64_t A_max, hipStream_t s) {
    static const hipError_t attr =
        hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_up_pairs<EPI>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kUpPairBytes));
    if (attr != hipSuccess) return attr;
    g.n_tiles = static_cast<int>(ceil_div(g.N, LdsShape<128, 256, 32, 3, EPI>::kBN));
    const int64_t tiles = row_tile_bound(A_max, g.E, 128) * g.n_tiles;
    if (tiles == 0) return hipSuccess;
    const int64_t blocks = round_up(std::min<int64_t>(tiles, 2 * static_cast<int64_t>(device_cus())), 8);
    hipLaunchKernelGGL((gemm_up_pairs<EPI>), dim3(static_cast<unsigned>(blocks)), dim3(kThreads), kUpPairBytes, s,
                       g);
    return hipGetLastError();
}

template <int EPI, bool OB>
hipError_t run_bf16_best(GroupedGemm g, int64_t A_max, hipStream_t s) {
    constexpr bool kUp = EPI != kEpiNone;
    if constexpr (kUp) {
        // Decode-sized calls (at most 128 rows: a few row tiles) take 64 x 128 tiles: twice
        // the workgroups of 256-column tiles streaming the weights, and half the activation
        // rows per stage of 128-row tiles, most of which are empty at this size (measured on
        // a 64-token top-2 step: about 10 us less than 128 x 256, 1.6 us less than 128 x 128;
        // no gain from 256 rows up, where the tiles already cover the CUs).
        if (A_max <= 128 && g.K % 32 == 0) return run_bf16_lds<64, 128, 32, 3, EPI, OB>(g, A_max, s);
        // activation rows in 128-byte pieces when K allows it (see gemm_up_pairs)
        if constexpr (OB) {
            if (g.K % 64 == 0) return run_up_pairs<EPI>(g, A_max, s);
        }
        if (g.K % 32 == 0) return run_bf16_lds<128, 256, 32, 3, EPI, OB>(g, A_max, s);
        return run_bf16<EPI, OB, true>(g, A_max, s);
    } else {
        if (g.K % 32 != 0) return hipErrorInvalidValue;  // not reachable through the C ABI (fp % 128 == 0)
        if (g.ksplit > 1 && A_max <= 128) return run_bf16_lds<64, 256, 32, 3, EPI, OB>(g, A_max, s);
        if (g.ksplit > 1) return run_bf16_lds<128, 256, 32, 3, EPI, OB>(g, A_max, s);
        if (g.N >= 384 && row_tile_bound(A_max, g.E, 128) * ceil_div(g.N, 384) <= device_cus())
            return run_bf16_lds<128, 384, 32, 3, EPI, OB, 4>(g, A_max, s);
        return run_bf16_lds<128, 256, 32, 3, EPI, OB>(g, A_max, s);
    }
}

template <int EPI>
hipError_t gemm1(bool bf16, GroupedGemm g, int64_t A_max, hipStream_t s) {
    return bf16 ? run_bf16_best<EPI, true>(g, A_max, s) : run_f32<EPI, false>(g, A_max, s);
}

// Both matmuls of the expert step.  grid_rows sizes the launches (an upper bound of the
// rows the offsets describe); rows_max is the row count of x_perm, H and y_perm.
// Step 5 folded into the expert step (CombineArgs given and the second product split): the
// parts' sum goes straight into y through split_combine instead of into y_perm.
struct CombineArgs {
    const int32_t* pos_of;
    const float* w;
    int64_t T;
    int k;
    void* y;
    bool y_bf16;
};


template <bool OB, int S>
hipError_t launch_split_reduce_t(const float* partial, int64_t rows_max, int h, int64_t grid_rows,
                                 const int32_t* offsets, int E, void* out, const int32_t* scatter,
                                 const float* scatter_w, int64_t c_rows, hipStream_t s) {
    const int64_t n4 = grid_rows * (h / 4);
    const int blocks = static_cast<int>(std::min<int64_t>(ceil_div(n4, 256), 8LL * device_cus()));
    hipLaunchKernelGGL((split_reduce<OB, S>), dim3(blocks), dim3(256), 0, s, partial, rows_max, h, offsets, E, out, h,
                       scatter, scatter_w, c_rows);
    return hipGetLastError();
}

// S = the down-projection's K parts: 2, 4 or 8 (down_ksplit)
hipError_t launch_split_reduce(bool ob, int S, const float* partial, int64_t rows_max, int h, int64_t grid_rows,
                               const int32_t* offsets, int E, void* out, const int32_t* scatter,
                               const float* scatter_w, int64_t c_rows, hipStream_t s) {
#define MOE_SPLIT_REDUCE(OBV, SV) \
    return launch_split_reduce_t<OBV, SV>(partial, rows_max, h, grid_rows, offsets, E, out, scatter, scatter_w, c_rows, s)
    if (ob) {
        if (S == 2) MOE_SPLIT_REDUCE(true, 2);
        if (S == 4) MOE_SPLIT_REDUCE(true, 4);
        if (S == 8) MOE_SPLIT_REDUCE(true, 8);
    } else {
        if (S == 2) MOE_SPLIT_REDUCE(false, 2);
        if (S == 4) MOE_SPLIT_REDUCE(false, 4);
        if (S == 8) MOE_SPLIT_REDUCE(false, 8);
    }
#undef MOE_SPLIT_REDUCE
    return hipErrorInvalidValue;
}

template <bool YB, bool OB, int S>
hipError_t launch_split_combine_t(const float* partial, int64_t rows_max, int h, const CombineArgs& c, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(ceil_div(c.T * (h / 8), 256)));
    hipLaunchKernelGGL((split_combine<YB, OB, S>), grid, dim3(256), 0, s, partial, rows_max, h, c.pos_of, c.w, c.T,
                       c.k, c.y);
    return hipGetLastError();
}

hipError_t launch_split_combine(bool yb, int S, const float* partial, int64_t rows_max, int h, const CombineArgs& c,
                                hipStream_t s) {
#define MOE_SPLIT_COMBINE(YBV, OBV)                                                              \
    do {                                                                                       \
        if (S == 2) return launch_split_combine_t<YBV, OBV, 2>(partial, rows_max, h, c, s);   \
        if (S == 4) return launch_split_combine_t<YBV, OBV, 4>(partial, rows_max, h, c, s);   \
        if (S == 8) return launch_split_combine_t<YBV, OBV, 8>(partial, rows_max, h, c, s);   \
    } while (0)
    if (yb && c.y_bf16) MOE_SPLIT_COMBINE(true, true);
    else if (yb) MOE_SPLIT_COMBINE(true, false);
    else if (c.y_bf16) MOE_SPLIT_COMBINE(false, true);
    else MOE_SPLIT_COMBINE(false, false);
#undef MOE_SPLIT_COMBINE
    return hipErrorInvalidValue;
}

hipError_t ffn_pair(const void* x_perm, const int32_t* offsets, int64_t grid_rows, int64_t rows_max, int E,
                    int h, int64_t fp, int act, bool bf16, const void* w1t, const void* w3t, const void* w2t,
                    void* y_perm, bool y_bf16, void* hbuf, hipStream_t s, const int32_t* gather = nullptr,
                    int64_t a_rows = 0, const float* scatter_w = nullptr, const CombineArgs* comb = nullptr) {
    if (grid_rows == 0) return hipSuccess;
    GroupedGemm g1{};
    g1.a = x_perm;
    g1.gather = gather;
    g1.a_rows = a_rows;
    g1.b = w1t;
    g1.b2 = w3t;
    g1.c = hbuf;
    g1.offsets = offsets;
    g1.E = E;
    g1.K = h;
    g1.N = static_cast<int>(fp);
    g1.ldc = static_cast<int>(fp);
    g1.b_estride = fp * h;
    g1.rows_max = rows_max;
    hipError_t err;
    if (act == MOE_ACT_SWIGLU) err = gemm1<kEpiSwiglu>(bf16, g1, grid_rows, s);
    else if (act == MOE_ACT_GELU_TANH) err = gemm1<kEpiGeluTanh>(bf16, g1, grid_rows, s);
    else err = gemm1<kEpiGelu>(bf16, g1, grid_rows, s);
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
    g2.rows_max = rows_max;
    if (scatter_w) {
        g2.scatter = gather;
        g2.scatter_w = scatter_w;
        g2.c_rows = a_rows;
    }
    // the split is chosen from rows_max (the call's row bound), so a per-expert launch of
    // this call splits like the grouped one
    g2.ksplit = down_ksplit(rows_max, fp, bf16);
    if (g2.ksplit <= 1) {
        if (!bf16) return y_bf16 ? run_f32<kEpiNone, true>(g2, grid_rows, s) : run_f32<kEpiNone, false>(g2, grid_rows, s);
        return y_bf16 ? run_bf16_best<kEpiNone, true>(g2, grid_rows, s) : run_bf16_best<kEpiNone, false>(g2, grid_rows, s);
    }
    // partial tiles after H in the workspace: ksplit x rows_max x h fp32
    g2.partial = reinterpret_cast<float*>(static_cast<unsigned char*>(hbuf) +
                                          round_up(rows_max * fp * (bf16 ? 2 : 4), 256));
    if (bf16)
        err = y_bf16 ? run_bf16_best<kEpiNone, true>(g2, grid_rows, s) : run_bf16_best<kEpiNone, false>(g2, grid_rows, s);
    else
        err = run_f32<kEpiNone, false>(g2, grid_rows, s);  // partial tiles only
    if (err != hipSuccess) return err;
    if (comb) {
        if (comb->T == 0) return hipSuccess;
        return launch_split_combine(y_bf16, g2.ksplit, g2.partial, rows_max, h, *comb, s);
    }
    return launch_split_reduce(y_bf16, g2.ksplit, g2.partial, rows_max, h, grid_rows, offsets, E, y_perm,
                               g2.scatter, g2.scatter_w, g2.c_rows, s);
}

}  // namespace

hipError_t launch_ffn(const void* x_perm, const int32_t* offsets, int64_t A_max, int E, int h,
                      int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                      const void* w2t, void* y_perm, bool y_bf16, void* hbuf, hipStream_t s) {
    return ffn_pair(x_perm, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y_perm, y_bf16, hbuf, s);
}

hipError_t launch_ffn_gather(const void* x, int64_t T, const int32_t* row_src, const int32_t* offsets, int64_t A_max,
                             int E, int h, int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                             const void* w2t, void* y_perm, bool y_bf16, void* hbuf, hipStream_t s) {
    return ffn_pair(x, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y_perm, y_bf16, hbuf, s, row_src, T);
}

hipError_t launch_ffn_gather_combine(const void* x, int64_t T, const int32_t* row_src, const int32_t* offsets, int k,
                                     int E, int h, int64_t fp, int act, bool bf16, const void* w1t, const void* w3t,
                                     const void* w2t, void* y_perm, bool y_bf16, const int32_t* pos_of,
                                     const float* topk_w, void* y, bool out_bf16, void* hbuf, hipStream_t s,
                                     bool* y_perm_written) {
    const int64_t A_max = T * k;
    const bool split = down_ksplit(A_max, fp, bf16) > 1;
    *y_perm_written = !split;
    if (split) {
        const CombineArgs comb{pos_of, topk_w, T, k, y, out_bf16};
        return ffn_pair(x, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y_perm, y_bf16, hbuf, s,
                        row_src, T, nullptr, &comb);
    }
    const hipError_t err =
        ffn_pair(x, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y_perm, y_bf16, hbuf, s, row_src, T);
    if (err != hipSuccess) return err;
    return launch_combine(y_perm, y_bf16, pos_of, topk_w, T, k, h, y, out_bf16, s);
}

// One expert at a time: expert e's segment is the one-expert grouping (offsets + e), its
// weights start e matrices into each packed block, and the launches are sized by its own
// row count, read from the host copy of the offsets.
// Top-1 layer output in one call: gathered rows in, y[t] = w[t] * FFN(x[t]) out.
hipError_t launch_ffn_top1(const void* x, int64_t T, const int32_t* row_src, const float* topk_w,
                           const int32_t* offsets, int64_t A_max, int E, int h, int64_t fp, int act, bool bf16,
                           const void* w1t, const void* w3t, const void* w2t, void* y, bool y_bf16, void* hbuf,
                           hipStream_t s) {
    return ffn_pair(x, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y, y_bf16, hbuf, s, row_src, T,
                    topk_w);
}

// ------------------------------------------------------------------ no-allocation variant
//
// The workspace of one call (H, then the split second product's partial tiles) lives in a
// static device array instead of caller memory.  Each GPU the library runs on holds its own
// copy of the array for the life of the process.  In host code the array's name only stands
// in for it: the device address comes from hipGetSymbolAddress, taken once per device with
// that device current, and only that address is ever handed to a kernel.  Nothing in the
// array needs to start at zero (every H row and partial tile a kernel reads is written
// earlier in the same call; rows of a tile past its segment only feed outputs that are not
// stored).  Calls that overlap on one GPU share the array and race.
namespace {

__device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of `scratch` on the current device (resolved on the first call there).
hipError_t static_scratch(void** out) {
    int dev = -1;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

hipError_t launch_ffn_noalloc(const void* x_perm, const int32_t* offsets, int64_t A_max, int E, int h, int64_t fp,
                              int act, bool bf16, const void* w1t, const void* w3t, const void* w2t, void* y_perm,
                              bool y_bf16, hipStream_t s) {
    if (s) {  // the stream must belong to the current device, whose copy of the array is used
        int sdev = -1, dev = -1;
        hipError_t err = hipStreamGetDevice(s, &sdev);
        if (err != hipSuccess) return err;
        err = hipGetDevice(&dev);
        if (err != hipSuccess) return err;
        if (sdev != dev) return hipErrorInvalidDevice;
    }
    void* ws = nullptr;
    const hipError_t err = static_scratch(&ws);
    if (err != hipSuccess) return err;
    return ffn_pair(x_perm, offsets, A_max, A_max, E, h, fp, act, bf16, w1t, w3t, w2t, y_perm, y_bf16, ws, s);
}

hipError_t launch_ffn_per_expert(const void* x_perm, const int32_t* offsets, const int32_t* offsets_host,
                                 int64_t A_max, int E, int h, int64_t fp, int act, bool bf16, const void* w1t,
                                 const void* w3t, const void* w2t, void* y_perm, bool y_bf16, void* hbuf,
                                 hipStream_t s) {
    const int64_t es = bf16 ? 2 : 4;
    const int64_t mat = fp * h * es;  // bytes of one expert's matrix in each packed block
    for (int e = 0; e < E; ++e) {
        const int64_t count = static_cast<int64_t>(offsets_host[e + 1]) - offsets_host[e];
        if (count <= 0) continue;
        const unsigned char* b1 = static_cast<const unsigned char*>(w1t) + e * mat;
        const unsigned char* b3 = w3t ? static_cast<const unsigned char*>(w3t) + e * mat : nullptr;
        const unsigned char* b2 = static_cast<const unsigned char*>(w2t) + e * mat;
        const hipError_t err = ffn_pair(x_perm, offsets + e, count, A_max, 1, h, fp, act, bf16, b1, b3, b2, y_perm,
                                        y_bf16, hbuf, s);
        if (err != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace moe
