// Step 2 of the layer: count the assignments per expert, scan, and group them stably.
//
//   count   one workgroup per chunk of kDispatchChunk assignments builds an LDS histogram
//           and writes it expert-major: cc[e * nchunks + c]
//   scan    one workgroup scans cc in that order; the exclusive prefix at (e, c) is the
//           first grouped position of chunk c's expert-e assignments, and at (e, 0) it is
//           offsets[e]
//   rank    per chunk, each wave walks its 256 assignments in 4 rounds of 64; lanes with
//           the same expert find each other with ballots over the id bits, so an
//           assignment's position is   chunk base + earlier waves' count + running count
//           + number of lower lanes with the same expert   -- stable in (t, j) order
//   gather  x_perm[p] = x[row_src[p]] with 16-byte vector copies
// When the count table (experts x chunks) is small, the scan runs inside every rank
// workgroup instead (dispatch_rank_scan: two launches).  Up to kFusedMaxA assignments,
// count, scan and rank run as one kernel (same output): every chunk's workgroup, 16 waves,
// counts all assignments itself into per-wave LDS histograms, keeping the counts of the
// chunks before its own apart, scans the totals, and ranks its chunk in one round (one
// group of 64 per wave).
// Integer atomics are used only for the LDS histograms, whose result does not depend on
// their order.
#include "common.h"
#include "kernels.h"

#include "../../include/moeshard.h"

namespace moe {
namespace {

constexpr int kDispThreads = 256;
constexpr int kDispWaves = kDispThreads / kWave;
constexpr int kPerWave = kDispatchChunk / kDispWaves;  // 256
constexpr int kRounds = kPerWave / kWave;              // 4

// The ids of this wave's kRounds groups of 64 assignments from a0 on (-1 past A): every load
// is issued before any is used, from a clamped index, so that they make one memory round
// trip (a load guarded by its own condition becomes a branch that waits for it).
__device__ __forceinline__ void load_wave_ids(const int32_t* __restrict__ idx, int64_t A, int64_t a0, int lane,
                                              int (&ev)[kRounds]) {
#pragma unroll
    for (int s = 0; s < kRounds; ++s) {
        const int64_t a = a0 + s * kWave + lane;
        ev[s] = idx[a < A ? a : A - 1];
    }
#pragma unroll
    for (int s = 0; s < kRounds; ++s) ev[s] = a0 + s * kWave + lane < A ? ev[s] : -1;
}

__global__ __launch_bounds__(kDispThreads) void dispatch_count(const int32_t* __restrict__ idx, int64_t A,
                                                               int E, int nchunks, int32_t* __restrict__ cc) {
    __shared__ int hist[MOE_MAX_EXPERTS];
    for (int e = threadIdx.x; e < E; e += kDispThreads) hist[e] = 0;
    __syncthreads();
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    int ev[kRounds];
    load_wave_ids(idx, A, static_cast<int64_t>(blockIdx.x) * kDispatchChunk + wave * kPerWave, lane, ev);
#pragma unroll
    for (int s = 0; s < kRounds; ++s)
        if (static_cast<unsigned>(ev[s]) < static_cast<unsigned>(E)) atomicAdd(&hist[ev[s]], 1);
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kDispThreads)
        cc[static_cast<int64_t>(e) * nchunks + blockIdx.x] = hist[e];
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void dispatch_scan(const int32_t* __restrict__ cc, int E,
                                                              int nchunks, int32_t* __restrict__ base,
                                                              int32_t* __restrict__ counts,
                                                              int32_t* __restrict__ offsets) {
    __shared__ int part[kScanThreads];
    __shared__ int off[MOE_MAX_EXPERTS + 1];
    const int tid = threadIdx.x;
    const int64_t L = static_cast<int64_t>(E) * nchunks;
    for (int e = tid; e <= E; e += kScanThreads) off[e] = 0;
    const int64_t per = ceil_div(L, kScanThreads);
    const int64_t lo = tid * per;
    const int64_t hi = (lo + per < L) ? lo + per : L;
    int sum = 0;
    for (int64_t i = lo; i < hi; ++i) sum += cc[i];
    part[tid] = sum;
    __syncthreads();
    for (int o = 1; o < kScanThreads; o <<= 1) {
        const int v = (tid >= o) ? part[tid - o] : 0;
        __syncthreads();
        part[tid] += v;
        __syncthreads();
    }
    int run = part[tid] - sum;
    for (int64_t i = lo; i < hi; ++i) {
        if (i % nchunks == 0) off[i / nchunks] = run;
        base[i] = run;
        run += cc[i];
    }
    if (tid == 0) off[E] = part[kScanThreads - 1];
    __syncthreads();
    for (int e = tid; e <= E; e += kScanThreads) {
        offsets[e] = off[e];
        if (e < E) counts[e] = off[e + 1] - off[e];
    }
}

__global__ __launch_bounds__(kDispThreads) void dispatch_rank(const int32_t* __restrict__ idx, int64_t A,
                                                              int k, int E, int nbits, int nchunks,
                                                              const int32_t* __restrict__ base,
                                                              int32_t* __restrict__ row_src,
                                                              int32_t* __restrict__ pos_of) {
    __shared__ int wcnt[kDispWaves][MOE_MAX_EXPERTS];
    __shared__ int run[kDispWaves][MOE_MAX_EXPERTS];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int c = blockIdx.x;
    for (int e = lane; e < E; e += kWave) wcnt[wave][e] = 0;
    __syncthreads();
    const int64_t a0 = static_cast<int64_t>(c) * kDispatchChunk + wave * kPerWave;
    int ev[kRounds];
    load_wave_ids(idx, A, a0, lane, ev);
#pragma unroll
    for (int s = 0; s < kRounds; ++s)
        if (static_cast<unsigned>(ev[s]) < static_cast<unsigned>(E)) atomicAdd(&wcnt[wave][ev[s]], 1);
    __syncthreads();
    for (int e = lane; e < E; e += kWave) {
        int b = base[static_cast<int64_t>(e) * nchunks + c];
        for (int w = 0; w < wave; ++w) b += wcnt[w][e];
        run[wave][e] = b;
    }
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int s = 0; s < kRounds; ++s) {
        const int64_t a = a0 + s * kWave + lane;
        const int e = ev[s];
        const bool valid = static_cast<unsigned>(e) < static_cast<unsigned>(E);
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < nbits; ++b) {
            const bool bit = valid && ((e >> b) & 1);
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const int rank = __popcll(peers & lt);
        if (valid) {
            const int pos = run[wave][e] + rank;
            pos_of[a] = pos;
            if (pos >= 0 && pos < A) row_src[pos] = static_cast<int32_t>(a / k);
        } else if (a < A) {
            pos_of[a] = -1;
        }
        __syncthreads();  // every lane has read run[] before the group leaders advance it
        if (valid && rank == 0) run[wave][e] += __popcll(peers);
        __syncthreads();
    }
}

// Rank with the scan folded in (two launches instead of three, for count tables that fit
// kRankScanMaxTable entries of LDS): every chunk's workgroup reads the whole table cc, sums each
// expert's row (the totals, and separately the chunks before its own), scans the totals, and
// ranks its chunk from base = offsets[e] + (earlier chunks' count of e).  Workgroup 0 writes
// counts and offsets.
constexpr int64_t kRankScanMaxTable = 8192;

__global__ __launch_bounds__(kDispThreads) void dispatch_rank_scan(const int32_t* __restrict__ idx, int64_t A,
                                                                   int k, int E, int nbits, int nchunks,
                                                                   const int32_t* __restrict__ cc,
                                                                   int32_t* __restrict__ counts,
                                                                   int32_t* __restrict__ offsets,
                                                                   int32_t* __restrict__ row_src,
                                                                   int32_t* __restrict__ pos_of) {
    __shared__ int table[kRankScanMaxTable];
    __shared__ int tot[MOE_MAX_EXPERTS];
    __shared__ int before[MOE_MAX_EXPERTS];
    __shared__ int off[MOE_MAX_EXPERTS + 1];
    __shared__ int wcnt[kDispWaves][MOE_MAX_EXPERTS];
    __shared__ int run[kDispWaves][MOE_MAX_EXPERTS];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int c = blockIdx.x;
    const int64_t a0 = static_cast<int64_t>(c) * kDispatchChunk + wave * kPerWave;
    // this chunk's ids and the whole count table, loaded together (one memory round trip):
    // every load from a clamped index, issued before any is stored
    int ev[kRounds];
    load_wave_ids(idx, A, a0, lane, ev);
    constexpr int kTablePer = kRankScanMaxTable / kDispThreads;
    const int L = E * nchunks;
    int tv[kTablePer];
#pragma unroll
    for (int u = 0; u < kTablePer; ++u)
        if (u * kDispThreads < L) tv[u] = cc[min(static_cast<int>(threadIdx.x) + u * kDispThreads, L - 1)];
    // stored chunk-major with a padded row (E + 1 counters), so that both the copy and the
    // per-expert sums below touch distinct banks
#pragma unroll
    for (int u = 0; u < kTablePer; ++u) {
        const int i = threadIdx.x + u * kDispThreads;
        const int e = i / nchunks, ch = i - e * nchunks;
        if (i < L) table[ch * (E + 1) + e] = tv[u];
    }
    __syncthreads();
    // each expert's total and its count in the chunks before this one: G = 256 / E threads
    // per expert (G = 1 .. 256) sum every G-th chunk, then one thread per expert adds the G
    // partial sums (integers: the order does not matter)
    static_assert(MOE_MAX_EXPERTS <= kDispThreads, "one expert per thread");
    {
        const int G = kDispThreads / E;
        const int e = threadIdx.x % E, g = threadIdx.x / E;
        int t = 0, b = 0;
        if (g < G)
            for (int i = g; i < nchunks; i += G) {
                const int v = table[i * (E + 1) + e];
                t += v;
                b += i < c ? v : 0;
            }
        if (g < G) {
            wcnt[0][threadIdx.x] = t;  // scratch for the partial sums (wcnt is cleared again below)
            run[0][threadIdx.x] = b;
        }
    }
    __syncthreads();
    if (threadIdx.x < E) {
        const int G = kDispThreads / E;
        int t = 0, b = 0;
        for (int g = 0; g < G; ++g) {
            t += wcnt[0][g * E + threadIdx.x];
            b += run[0][g * E + threadIdx.x];
        }
        tot[threadIdx.x] = t;
        before[threadIdx.x] = b;
    }
    __syncthreads();
    for (int e = lane; e < E; e += kWave) wcnt[wave][e] = 0;
    __syncthreads();
#pragma unroll
    for (int s = 0; s < kRounds; ++s)
        if (static_cast<unsigned>(ev[s]) < static_cast<unsigned>(E)) atomicAdd(&wcnt[wave][ev[s]], 1);
    // exclusive scan of the totals: one wave, four experts per lane
    static_assert(MOE_MAX_EXPERTS == 4 * kWave, "four experts per lane of one wave");
    if (wave == 0) {
        int ex[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            ex[i] = sum;
            sum += (e < E) ? tot[e] : 0;
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int t = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += t;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            if (e < E) off[e] = incl - sum + ex[i];
        }
        if (lane == kWave - 1) off[E] = incl;
    }
    __syncthreads();
    if (c == 0) {
        for (int e = threadIdx.x; e <= E; e += kDispThreads) {
            offsets[e] = off[e];
            if (e < E) counts[e] = tot[e];
        }
    }
    for (int e = lane; e < E; e += kWave) {
        int b = off[e] + before[e];
        for (int w = 0; w < wave; ++w) b += wcnt[w][e];
        run[wave][e] = b;
    }
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int s = 0; s < kRounds; ++s) {
        const int64_t a = a0 + s * kWave + lane;
        const int e = ev[s];
        const bool valid = static_cast<unsigned>(e) < static_cast<unsigned>(E);
        uint64_t peers = __ballot(valid);
        for (int b = 0; b < nbits; ++b) {
            const bool bit = valid && ((e >> b) & 1);
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const int rank = __popcll(peers & lt);
        if (valid) {
            const int pos = run[wave][e] + rank;
            pos_of[a] = pos;
            if (pos >= 0 && pos < A) row_src[pos] = static_cast<int32_t>(a / k);
        } else if (a < A) {
            pos_of[a] = -1;
        }
        __syncthreads();  // every lane has read run[] before the group leaders advance it
        if (valid && rank == 0) run[wave][e] += __popcll(peers);
        __syncthreads();
    }
}

constexpr int64_t kFusedMaxA = 16384;

// One workgroup of 16 waves per chunk of 1024 assignments (one group of 64 per wave), so
// that counting every assignment is spread over 1024 threads and the chunk is ranked in a
// single round.
constexpr int kFusedThreads = 1024;
constexpr int kFusedWaves = kFusedThreads / kWave;
static_assert(kFusedWaves * kWave == kDispatchChunk, "one wave per 64 assignments of a chunk");
constexpr int kFusedLoads = 8;  // groups of 64 assignments per wave whose loads go out together

__global__ __launch_bounds__(kFusedThreads) void dispatch_fused(const int32_t* __restrict__ idx, int64_t A, int k,
                                                                 int E, int nbits, int32_t* __restrict__ counts,
                                                                 int32_t* __restrict__ offsets,
                                                                 int32_t* __restrict__ row_src,
                                                                 int32_t* __restrict__ pos_of) {
    // per-wave histograms: all assignments (h_all) and those before this chunk (h_bef);
    // h_all then holds each wave's counts within this chunk
    __shared__ int h_all[kFusedWaves][MOE_MAX_EXPERTS];
    __shared__ int h_bef[kFusedWaves][MOE_MAX_EXPERTS];
    __shared__ int tot[MOE_MAX_EXPERTS];
    __shared__ int before[MOE_MAX_EXPERTS];
    __shared__ int off[MOE_MAX_EXPERTS + 1];
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int c = blockIdx.x;
    const int64_t cbeg = static_cast<int64_t>(c) * kDispatchChunk;
    // this lane's assignment of the chunk, loaded first (its latency hides behind the count)
    const int64_t my_a = cbeg + wave * kWave + lane;
    int my_e = idx[my_a < A ? my_a : A - 1];
    for (int e = lane; e < E; e += kWave) h_all[wave][e] = h_bef[wave][e] = 0;
    __syncthreads();

    // every assignment into this wave's histograms, kFusedLoads groups of 64 per round with
    // their loads issued together (clamped indices; a group lies wholly before the chunk or
    // wholly in or after it, as chunks are multiples of 64)
    for (int64_t b0 = static_cast<int64_t>(wave) * kWave; b0 < A; b0 += kFusedThreads * kFusedLoads) {
        int eb[kFusedLoads];
#pragma unroll
        for (int u = 0; u < kFusedLoads; ++u) {
            const int64_t a = b0 + static_cast<int64_t>(u) * kFusedThreads + lane;
            eb[u] = idx[a < A ? a : A - 1];
        }
#pragma unroll
        for (int u = 0; u < kFusedLoads; ++u) {
            const int64_t g0 = b0 + static_cast<int64_t>(u) * kFusedThreads;
            const int e = g0 + lane < A ? eb[u] : -1;
            if (static_cast<unsigned>(e) < static_cast<unsigned>(E)) {
                atomicAdd(&h_all[wave][e], 1);
                if (g0 < cbeg) atomicAdd(&h_bef[wave][e], 1);
            }
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += kFusedThreads) {
        int t = 0, b = 0;
#pragma unroll
        for (int w = 0; w < kFusedWaves; ++w) {
            t += h_all[w][e];
            b += h_bef[w][e];
        }
        tot[e] = t;
        before[e] = b;
    }
    __syncthreads();

    // exclusive scan of the totals: one wave, four experts per lane
    if (wave == 0) {
        int ex[4], sum = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            ex[i] = sum;
            sum += (e < E) ? tot[e] : 0;
        }
        int incl = sum;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int t = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += t;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane * 4 + i;
            if (e < E) off[e] = incl - sum + ex[i];
        }
        if (lane == kWave - 1) off[E] = incl;
    }
    // each wave's counts within the chunk (h_all is free again after the sums above)
    my_e = my_a < A ? my_e : -1;
    const bool valid = static_cast<unsigned>(my_e) < static_cast<unsigned>(E);
    const uint64_t peers = same_expert_lanes(my_e, valid, nbits);
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int rank = __popcll(peers & lt);
    for (int e = lane; e < E; e += kWave) h_all[wave][e] = 0;
    __syncthreads();
    if (valid && rank == 0) h_all[wave][my_e] = __popcll(peers);
    if (c == 0) {
        for (int e = threadIdx.x; e <= E; e += kFusedThreads) {
            offsets[e] = off[e];
            if (e < E) counts[e] = tot[e];
        }
    }
    __syncthreads();

    // position = expert start + earlier chunks + earlier waves of this chunk + earlier lanes
    if (valid) {
        int pos = off[my_e] + before[my_e] + rank;
        for (int w = 0; w < wave; ++w) pos += h_all[w][my_e];
        pos_of[my_a] = pos;
        if (pos >= 0 && pos < A) row_src[pos] = static_cast<int32_t>(my_a / k);
    } else if (my_a < A) {
        pos_of[my_a] = -1;
    }
}

// x_perm[p] = x[row_src[p]] for p < offsets[E]: each wave copies kGatherRows rows, its lanes
// striding over the 16-byte vectors of a row, with the loads of all its rows issued before
// their stores.
constexpr int kGatherRows = 8;

__global__ __launch_bounds__(256) void dispatch_gather(const uint4* __restrict__ x,
                                                       const int32_t* __restrict__ row_src,
                                                       const int32_t* __restrict__ offsets, int E,
                                                       uint32_t A_cap, uint32_t T, uint32_t nvec,
                                                       uint4* __restrict__ x_perm) {
    const uint32_t A = min(static_cast<uint32_t>(offsets[E]), A_cap);
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t p0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kGatherRows;
    if (p0 >= A) return;
    uint32_t src[kGatherRows];
#pragma unroll
    for (int r = 0; r < kGatherRows; ++r) {
        const uint32_t p = p0 + r;
        const uint32_t s = (p < A) ? static_cast<uint32_t>(row_src[p]) : 0u;
        src[r] = (s < T) ? s : 0u;
    }
    for (uint32_t c = lane; c < nvec; c += 64) {
        uint4 v[kGatherRows];
#pragma unroll
        for (int r = 0; r < kGatherRows; ++r) v[r] = x[static_cast<uint64_t>(src[r]) * nvec + c];
#pragma unroll
        for (int r = 0; r < kGatherRows; ++r)
            if (p0 + r < A) x_perm[static_cast<uint64_t>(p0 + r) * nvec + c] = v[r];
    }
}

}  // namespace

hipError_t launch_dispatch(const int32_t* idx, int64_t T, int k, int E, const void* x, int elem_bytes,
                           int h, int32_t* counts, int32_t* offsets, int32_t* row_src,
                           int32_t* pos_of, void* x_perm, int32_t* ws, hipStream_t s) {
    const int64_t A = T * k;
    const int nchunks = static_cast<int>(ceil_div(A, kDispatchChunk));
    int32_t* cc = ws;
    int32_t* base = ws + static_cast<int64_t>(E) * nchunks;
    int nbits = 0;
    while ((1 << nbits) < E) ++nbits;
    if (nchunks > 0 && A <= kFusedMaxA) {
        hipLaunchKernelGGL(dispatch_fused, dim3(nchunks), dim3(kFusedThreads), 0, s, idx, A, k, E, nbits, counts,
                           offsets, row_src, pos_of);
    } else {
        if (nchunks > 0) {
            hipLaunchKernelGGL(dispatch_count, dim3(nchunks), dim3(kDispThreads), 0, s, idx, A, E, nchunks, cc);
        }
        if (nchunks > 0 && static_cast<int64_t>(E + 1) * nchunks <= kRankScanMaxTable) {
            hipLaunchKernelGGL(dispatch_rank_scan, dim3(nchunks), dim3(kDispThreads), 0, s, idx, A, k, E, nbits,
                               nchunks, cc, counts, offsets, row_src, pos_of);
        } else {
            hipLaunchKernelGGL(dispatch_scan, dim3(1), dim3(kScanThreads), 0, s, cc, E, nchunks, base, counts,
                               offsets);
            if (nchunks > 0) {
                hipLaunchKernelGGL(dispatch_rank, dim3(nchunks), dim3(kDispThreads), 0, s, idx, A, k, E, nbits,
                                   nchunks, base, row_src, pos_of);
            }
        }
    }
    if (nchunks > 0) {
        if (x_perm) {  // without x_perm the expert step gathers the rows itself
            const uint32_t nvec = static_cast<uint32_t>(static_cast<int64_t>(h) * elem_bytes / 16);
            const int64_t blocks = ceil_div(A, 4 * kGatherRows);
            hipLaunchKernelGGL(dispatch_gather, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                               static_cast<const uint4*>(x), row_src, offsets, E, static_cast<uint32_t>(A),
                               static_cast<uint32_t>(T), nvec, static_cast<uint4*>(x_perm));
        }
    }
    return hipGetLastError();
}

}  // namespace moe
