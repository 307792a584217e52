/*
 * moeshard.h -- C ABI of the sharded expert-FFN MoE layer for AMD Instinct MI355X (gfx950).
 *
 * The layer is the one the MoEShard paper ("Accelerating MoE Model Inference with Expert
 * Sharding", EuroMLSys '25) speeds up: every device holds a contiguous slice of the FFN
 * inner width of *every* expert -- columns of W_i and the matching rows of W_o (Section
 * 3.2) -- so it runs every expert on every token routed to it, and the devices' partial
 * outputs sum to the unsharded result.  On one device the forward pass of Algorithm 1
 * reduces to four calls made in order on one stream:
 *
 *   moe_route            Step 1, token routing (Section 3.1)
 *   moe_dispatch         Step 2, group tokens per expert and count them (Section 3.1)
 *   moe_expert_ffn_shard Step 4, this device's shard of every expert on its tokens, as
 *                        one grouped computation over all experts (Sections 3.2 and 3.3)
 *   moe_combine          Step 5, point-wise gate-weighted sum of each token's results
 *
 * plus moe_pack_weights, the one-time loadShard of Step 4.
 *
 * Conventions shared by every call
 *  - Every data pointer is caller-owned DEVICE memory (e.g. allocated by torch); the
 *    library never allocates, frees or keeps per-call state.  Scratch memory comes from
 *    the caller, sized by the *_workspace_size queries.
 *  - Every call is asynchronous on `stream` (0 = the null stream) and never synchronises
 *    the host.  Per-expert counts stay on the device.
 *  - Arguments are validated before anything is launched.  On an error nothing is
 *    launched and no output is written.  Status codes: see moe_status.
 *  - Matrices are row-major.  bf16 tensors hold raw bfloat16 bit patterns (uint16).
 *  - Alignment: every tensor pointer must be 16-byte aligned.
 *  - Limits: 1 <= k <= E <= MOE_MAX_EXPERTS; h >= 8 and h % 8 == 0; T * k < 2^31.
 *  - Outputs are bitwise deterministic: no floating-point atomics, fixed reduction order.
 *  - Calls on different streams that share no output buffers may run concurrently.
 */
#ifndef MOESHARD_H
#define MOESHARD_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_MAX_EXPERTS 256

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1, /* a size, pointer, alignment or enum value is invalid */
    MOE_ERR_UNSUPPORTED = 2, /* valid request this build does not implement */
    MOE_ERR_WORKSPACE = 3,   /* the workspace or packed buffer is too small */
    MOE_ERR_HIP = 4,         /* the HIP runtime reported a launch error */
    MOE_ERR_TOO_LARGE = 5    /* the call needs more than MOE_NOALLOC_SCRATCH_BYTES of scratch
                                (moe_expert_ffn_shard_noalloc only) */
} moe_status;

/* Bytes of the static per-device scratch array behind moe_expert_ffn_shard_noalloc. */
#define MOE_NOALLOC_SCRATCH_BYTES (64u * 1024u * 1024u)

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

/* Activation between the two expert matrices.  The paper writes the expert as two
 * matmuls (Section 3.2) and never names the activation; any element-wise activation
 * keeps the shard-sum property, because it acts on each inner column independently.
 *   MOE_ACT_GELU       u * Phi(u)                          (erf form)
 *   MOE_ACT_GELU_TANH  0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))
 *   MOE_ACT_SWIGLU     silu(x W1) * (x W3), W1 and W3 sliced on the same inner columns */
typedef enum { MOE_ACT_GELU = 0, MOE_ACT_GELU_TANH = 1, MOE_ACT_SWIGLU = 2 } moe_act;

/* Human-readable name of a status code (static storage, never NULL). */
const char *moe_status_string(moe_status status);

/* Step 1 (Algorithm 1, token routing; Section 3.1: the router maps each token to its
 * expert(s)).
 *   x         [T, h]  activations, dtype xdt (MOE_BF16 or MOE_F32)
 *   w_gate    [E, h]  gate projection, dtype xdt; row e is expert e's gate vector
 *   sel_bias  nullable fp32 selection bias: bias_row_stride == 0 -> [E] shared by all
 *             tokens, bias_row_stride == E -> [T, E] per token
 *   renorm    0: weights are the softmax probabilities; 1: divided by their sum over k
 *   topk_idx  [T, k] int32 out: expert ids in decreasing order of logit + bias; equal
 *             scores go to the lower expert id
 *   topk_w    [T, k] fp32 out: softmax of the UNBIASED logits (fp32 accumulation) at the
 *             picked experts; the bias only changes which experts are picked
 * T == 0 is a valid no-op. */
moe_status moe_route(const void *x, moe_dtype xdt, int64_t T, int64_t h, const void *w_gate,
                     int32_t E, int32_t k, const float *sel_bias, int64_t bias_row_stride,
                     int32_t renorm, int32_t *topk_idx, float *topk_w, hipStream_t stream);

/* Bytes of workspace moe_dispatch needs for T tokens, k picks and E experts. */
size_t moe_dispatch_workspace_size(int64_t T, int32_t k, int32_t E);

/* Step 2 (Algorithm 1, groupPerExpert and countPerExpert; Section 3.1).  The A = T*k
 * assignments (t, j) are grouped by expert; inside a group they keep (t, j) order.
 *   topk_idx  [T, k] int32 expert ids; an id outside [0, E) is dropped: it is not
 *             counted, gets pos_of = -1 and contributes nothing in moe_combine
 *   x         [T, h] rows to permute, dtype xdt
 *   counts    [E]   out: assignments per expert (m_sizes of the paper)
 *   offsets   [E+1] out: exclusive prefix sum of counts; offsets[E] = A when every id
 *             is valid
 *   row_src   [A]   out: token of the assignment at grouped position p
 *   pos_of    [T,k] out: grouped position of assignment (t, j)
 *   x_perm    [A, h] out: x_perm[p] = x[row_src[p]], bit copies; may be NULL, and then
 *             only the indices are written (x is not read; moe_expert_ffn_shard_gather
 *             reads the rows through row_src instead)
 *   ws        moe_dispatch_workspace_size(T, k, E) bytes, 16-byte aligned
 * T == 0 writes zero counts and offsets. */
moe_status moe_dispatch(const int32_t *topk_idx, int64_t T, int32_t k, int32_t E,
                        const void *x, moe_dtype xdt, int64_t h, int32_t *counts,
                        int32_t *offsets, int32_t *row_src, int32_t *pos_of, void *x_perm,
                        void *ws, size_t ws_bytes, hipStream_t stream);

/* Steps 1 and 2 in one call: moe_route followed by moe_dispatch without x_perm (the grouped
 * rows are read through row_src by moe_expert_ffn_shard_gather / _top1 / _gather_combine),
 * with the same outputs bit for bit.  When one routing workgroup covers the whole batch
 * (bf16, h % 64 == 0, 32 < E <= 256, 1 <= T <= 64, k <= 8: decode-sized batches) that
 * workgroup also groups the assignments from its picks, in the same launch; otherwise the
 * two steps run as the two calls would.
 *   arguments as moe_route and moe_dispatch (ws: moe_dispatch_workspace_size(T, k, E)
 *   bytes, 16-byte aligned); every argument of both is checked before any launch. */
moe_status moe_route_dispatch(const void *x, moe_dtype xdt, int64_t T, int64_t h, const void *w_gate,
                              int32_t E, int32_t k, const float *sel_bias, int64_t bias_row_stride,
                              int32_t renorm, int32_t *topk_idx, float *topk_w, int32_t *counts,
                              int32_t *offsets, int32_t *row_src, int32_t *pos_of, void *ws,
                              size_t ws_bytes, hipStream_t stream);

/* Inner width after padding to the grouped GEMM's tile multiple (the packed layout). */
int64_t moe_padded_inner_width(int64_t f);

/* Bytes of the packed shard for E experts, hidden h, shard inner width f. */
size_t moe_packed_weights_size(int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype wdt);

/* loadShard of Step 4: cut this device's shard out of full expert weights and lay it out
 * for the grouped GEMM (Section 3.2: W_i split by columns, W_o by the matching rows; the
 * shard is the contiguous inner slice [col0, col0 + f)).
 *   w1  [E, h, F]  W_i of every expert, dtype wdt (SwiGLU: the gate projection)
 *   w3  [E, h, F]  SwiGLU up projection (same columns), NULL otherwise
 *   w2  [E, F, h]  W_o of every expert
 *   0 <= col0, f >= 1, col0 + f <= F
 *   packed  moe_packed_weights_size(...) bytes.  Layout (internal, may change):
 *           W1^T [E][fp][h], (W3^T [E][fp][h]), W2^T [E][h][fp], fp = padded f;
 *           padded inner columns are zero, which is exact: every activation maps 0 to 0.
 *           bf16 matrices are stored K-blocked (K = the second index: element (r, k) of
 *           an [R][K] matrix at ((k / 32) * R + r) * 32 + k % 32), W1^T / W3^T only when
 *           h % 32 == 0; fp32 matrices are row-major.
 * Run once per shard; the result is read-only for moe_expert_ffn_shard. */
moe_status moe_pack_weights(const void *w1, const void *w3, const void *w2, int32_t E,
                            int64_t h, int64_t F, int64_t col0, int64_t f, moe_act act,
                            moe_dtype wdt, void *packed, size_t packed_bytes,
                            hipStream_t stream);

/* Bytes of workspace moe_expert_ffn_shard needs: the activated inner rows (A_max x fp) and,
 * for bf16, room for fp32 partial sums of the second product (at most 2048 x h floats):
 * calls with A_max <= 512 split its K into up to 8 parts so that few rows still occupy
 * the whole GPU.  Non-decreasing in A_max, so a workspace sized for a bound serves every
 * call with a smaller A_max. */
size_t moe_ffn_workspace_size(int64_t A_max, int32_t E, int64_t h, int64_t f, moe_act act,
                              moe_dtype dt);

/* Step 4 (Algorithm 1, expert computation; Section 3.3's single grouped operation over
 * all experts): for every expert e and every grouped row p in [offsets[e], offsets[e+1]):
 *     y_perm[p] = act(x_perm[p] . W1_e^g) . W2_e^g        (shard g = the packed slice)
 * computed with bf16 MFMA and fp32 accumulation (dt = MOE_BF16) or fp32 arithmetic
 * (dt = MOE_F32).  The activated row is rounded to dt before the second product.  One
 * launch per matmul regardless of E; the per-expert counts are read on the device.  A small
 * bf16 call (A_max <= 512) sums the second product's K in parts, each part in fp32, the
 * parts added in a fixed order by one more launch; the split depends only on A_max and f,
 * so results are deterministic and every entry point agrees bit for bit on one call.
 *   x_perm  [A, h] dtype dt, grouped rows from moe_dispatch
 *   offsets [E+1] int32, device; offsets[E] must not exceed A_max
 *   A_max   host-known upper bound of offsets[E] (normally T*k); sizes the launch
 *   packed  from moe_pack_weights with the same E, h, f, act and dt
 *   y_perm  [A, h] out, dtype ydt (MOE_F32 keeps an unrounded shard partial)
 *   ws      moe_ffn_workspace_size(A_max, E, h, f, act, dt) bytes */
moe_status moe_expert_ffn_shard(const void *x_perm, const int32_t *offsets, int64_t A_max,
                                int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                const void *packed, void *y_perm, moe_dtype ydt, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/* Step 4 with Step 2's row gather folded into it (Section 3.3's concatenation of an
 * expert's tokens done by the loads of the first matmul): the same result as
 * moe_expert_ffn_shard on x_perm[p] = x[row_src[p]], bit for bit, without x_perm.
 *   x        [T, h] dtype dt, the unpermuted rows; T * h * sizeof(dt) < 4 GiB
 *            (else MOE_ERR_UNSUPPORTED)
 *   row_src  [A_max] int32 from moe_dispatch (entries past offsets[E] are never used as
 *            more than a clamped row index)
 *   other arguments as moe_expert_ffn_shard. */
moe_status moe_expert_ffn_shard_gather(const void *x, int64_t T, const int32_t *row_src,
                                       const int32_t *offsets, int64_t A_max, int32_t E,
                                       int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                       const void *packed, void *y_perm, moe_dtype ydt, void *ws,
                                       size_t ws_bytes, hipStream_t stream);

/* Steps 4 and 5 together for any k (Algorithm 1's expert computation and weighted
 * combination): moe_expert_ffn_shard_gather on rows_max = T * k followed by moe_combine,
 * with the same y bit for bit.  When the second product's K is split (calls of at most 512
 * bf16 or 1024 fp32 rows, the decode-sized ones), the parts' sum and the combine run as one
 * launch: each token's rows are summed over the parts, rounded to ydt exactly as y_perm
 * would hold them, weighted and accumulated in pick order, and y_perm is not written;
 * otherwise y_perm is written as by moe_expert_ffn_shard_gather and then combined.
 *   x, row_src, offsets, E, h, f, act, dt, packed, ydt, ws: as moe_expert_ffn_shard_gather
 *            with A_max = T * k (T * k < 2^31)
 *   pos_of   [T, k] int32 from moe_dispatch;  topk_w [T, k] fp32 from moe_route
 *   y_perm   [T * k, h] dtype ydt scratch (written only when K is not split)
 *   y        [T, h] out, dtype out_dt
 *   y_perm_written  optional host int: set to 1 if y_perm was written, else 0 (may be NULL) */
moe_status moe_expert_ffn_shard_gather_combine(const void *x, int64_t T, const int32_t *row_src,
                                               const int32_t *offsets, const int32_t *pos_of,
                                               const float *topk_w, int32_t k, int32_t E, int64_t h,
                                               int64_t f, moe_act act, moe_dtype dt, const void *packed,
                                               void *y_perm, moe_dtype ydt, void *y, moe_dtype out_dt,
                                               int32_t *y_perm_written, void *ws, size_t ws_bytes,
                                               hipStream_t stream);

/* Steps 4 and 5 together for top-1 routing (k = 1): the expert step reads its rows through
 * row_src and its down-projection epilogue writes each token's gate-weighted result
 * straight into y, so neither x_perm nor y_perm nor moe_combine is needed:
 *     y[t] = topk_w[t] * (act(x[t] . W1_e^g) . W2_e^g),   e = the token's expert
 * computed in fp32 and rounded once to out_dt.  A token whose pick was dropped (an id
 * outside [0, E) in moe_dispatch) is not written.
 *   x        [T, h] dtype dt; T * h * sizeof(dt) < 4 GiB (else MOE_ERR_UNSUPPORTED)
 *   row_src  [T] int32 and offsets [E+1] from moe_dispatch with k = 1
 *   topk_w   [T] fp32 gate weights from moe_route
 *   y        [T, h] out, dtype out_dt
 *   ws       moe_ffn_workspace_size(T, E, h, f, act, dt) bytes
 *   other arguments as moe_expert_ffn_shard (A_max = T). */
moe_status moe_expert_ffn_shard_top1(const void *x, int64_t T, const int32_t *row_src,
                                     const float *topk_w, const int32_t *offsets, int32_t E,
                                     int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                     const void *packed, void *y, moe_dtype out_dt, void *ws,
                                     size_t ws_bytes, hipStream_t stream);

/* Ablation of the single grouped operation (Section 3.3's second optimization, the one the
 * paper's ablation study removes): the same result as moe_expert_ffn_shard, bit for bit,
 * computed with one launch of each matmul per expert that has rows -- Step 4's per-expert
 * loop without the grouped formulation.  The launches are sized from a host copy of the
 * offsets, so the caller reads them back first (the synchronization such a loop needs).
 * Arguments as moe_expert_ffn_shard, plus
 *   offsets_host [E+1] int32 in host memory, equal to the device offsets: nondecreasing,
 *                offsets_host[0] >= 0 and offsets_host[E] <= A_max, else
 *                MOE_ERR_INVALID_ARG (nothing is launched). */
moe_status moe_expert_ffn_shard_per_expert(const void *x_perm, const int32_t *offsets,
                                           const int32_t *offsets_host, int64_t A_max, int32_t E,
                                           int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                           const void *packed, void *y_perm, moe_dtype ydt,
                                           void *ws, size_t ws_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory -- code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc: moe_expert_ffn_shard with the same
 * arguments, result and bits, but with no caller workspace.  The scratch it needs (the
 * activated inner rows and, for A_max <= 512 in bf16, the partial sums of the second
 * product) lives in a static device array of MOE_NOALLOC_SCRATCH_BYTES that the library
 * holds on every GPU it runs on until the process ends.  The call itself allocates and
 * frees nothing; its first call on a device looks up that device's copy of the array
 * (hipGetSymbolAddress) once.
 *   Limit: moe_ffn_workspace_size(A_max, E, h, f, act, dt) must not exceed
 *          MOE_NOALLOC_SCRATCH_BYTES, else MOE_ERR_TOO_LARGE and nothing is launched
 *          (e.g. bf16 with f = 4096 takes A_max up to about 8000 rows).
 *   stream must belong to the current device (else MOE_ERR_HIP, nothing launched).
 *   Every call on one GPU uses the same array: calls that may overlap on one GPU (other
 *   streams, other threads) race and give wrong results; order them on one stream.  The
 *   array keeps the last call's contents; no call depends on them. */
moe_status moe_expert_ffn_shard_noalloc(const void *x_perm, const int32_t *offsets, int64_t A_max,
                                        int32_t E, int64_t h, int64_t f, moe_act act, moe_dtype dt,
                                        const void *packed, void *y_perm, moe_dtype ydt,
                                        hipStream_t stream);

/* Step 5 (Algorithm 1, aggregateTokens): point-wise weighted sum of each token's expert
 * results, accumulated in fp32 in pick order j = 0..k-1 and rounded once:
 *     y[t] = sum_j topk_w[t, j] * y_perm[pos_of[t, j]]
 *   y_perm [A, h] dtype ydt; pos_of [T, k] (negative entries are skipped); topk_w [T, k]
 *   fp32; y [T, h] out, dtype out_dt */
moe_status moe_combine(const void *y_perm, moe_dtype ydt, const int32_t *pos_of,
                       const float *topk_w, int64_t T, int32_t k, int64_t h, void *y,
                       moe_dtype out_dt, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* MOESHARD_H */
