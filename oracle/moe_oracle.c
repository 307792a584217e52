/*
 * moe_oracle.c -- fp64 reference of the sharded expert-FFN MoE layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link or call this code;
 * only the tests, the smoke check and the benchmark's CPU-baseline leg use it.  It shares
 * no source with the HIP library.
 *
 * It follows the paper's forward pass (Algorithm 1): Step 1 routing (Section 3.1, the
 * token -> expert map), Step 2 grouping tokens per expert and counting them, Step 4
 * running every expert on its tokens with this device's shard of W_i (column slice) and
 * W_o (row slice) (Section 3.2), and Step 5 summing the per-token results.  The cross-
 * device exchanges (Steps 2b, 3, 5's transfers) do not exist on one device.
 *
 * Every input arrives as float32 holding values that are exact in the workload's dtype
 * (bf16 or fp32); every operation below is carried out in double, in the plain order of
 * the definition, with no blocking or reordering.  OpenMP only splits independent tokens
 * or rows across threads; each value is still computed by one sequential loop.
 *
 * Readings of points the paper leaves open (each is listed in the design notes):
 *  - activation between the two expert matmuls: GELU (erf form, default), GELU with the
 *    tanh approximation, or SwiGLU (silu(x W1) * (x W3), W1/W3 sliced on the same columns);
 *  - gate weighting (Switch convention): each expert output is scaled by the softmax
 *    probability of the unbiased logits; with renorm the k picked weights are divided by
 *    their sum;
 *  - top-k order: decreasing selection score, equal scores -> lower expert id first; the
 *    optional selection bias changes only which experts are picked, not the weights;
 *  - order inside an expert's group: by token, then by pick slot (stable).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_ACT_GELU = 0, ORACLE_ACT_GELU_TANH = 1, ORACLE_ACT_SWIGLU = 2 };

/* ---- Step 1: routing -------------------------------------------------------------
 * logits[t,e] = sum_j x[t,j] * wg[e,j]         (wg holds one gate vector per expert)
 * score[t,e]  = logits[t,e] + bias[t*bias_stride + e]   (bias may be NULL)
 * idx[t,:]    = first k entries of a stable sort of e = 0..E-1 by decreasing score
 * p[t,:]      = softmax(logits[t,:]);  w[t,j] = p[t, idx[t,j]]  (renorm: / sum_j w)
 * Returns 0, or -1 on invalid sizes. */
int oracle_route(const float *x, const float *wg, int64_t T, int64_t h, int32_t E, int32_t k,
                 const float *bias, int64_t bias_stride, int32_t renorm,
                 int32_t *idx, double *w, double *logits)
{
    if (T < 0 || h < 1 || E < 1 || k < 1 || k > E) return -1;
#pragma omp parallel
    {
        double *score = (double *)malloc(sizeof(double) * (size_t)E);
        int32_t *order = (int32_t *)malloc(sizeof(int32_t) * (size_t)E);
#pragma omp for schedule(static)
        for (int64_t t = 0; t < T; ++t) {
            double *lg = logits + t * E;
            for (int32_t e = 0; e < E; ++e) {
                double acc = 0.0;
                for (int64_t j = 0; j < h; ++j)
                    acc += (double)x[t * h + j] * (double)wg[(int64_t)e * h + j];
                lg[e] = acc;
                score[e] = acc + (bias ? (double)bias[t * bias_stride + e] : 0.0);
            }
            /* stable insertion sort of expert ids by decreasing score */
            for (int32_t e = 0; e < E; ++e) {
                int32_t pos = e;
                while (pos > 0 && score[order[pos - 1]] < score[e]) {
                    order[pos] = order[pos - 1];
                    --pos;
                }
                order[pos] = e;
            }
            double mx = lg[0];
            for (int32_t e = 1; e < E; ++e) if (lg[e] > mx) mx = lg[e];
            double den = 0.0;
            for (int32_t e = 0; e < E; ++e) den += exp(lg[e] - mx);
            double wsum = 0.0;
            for (int32_t j = 0; j < k; ++j) {
                idx[t * k + j] = order[j];
                w[t * k + j] = exp(lg[order[j]] - mx) / den;
                wsum += w[t * k + j];
            }
            if (renorm)
                for (int32_t j = 0; j < k; ++j) w[t * k + j] /= wsum;
        }
        free(score);
        free(order);
    }
    return 0;
}

/* ---- Step 2: group per expert and count (counting sort) ---------------------------
 * counts[e]   = number of (t,j) with idx[t,j] == e
 * offsets[0]  = 0, offsets[e+1] = offsets[e] + counts[e]
 * walking t = 0..T-1, j = 0..k-1:  p = cursor[e]++  (cursor starts at offsets)
 *     row_src[p] = t,  pos_of[t*k+j] = p
 * Returns 0, or -1 if an id is out of range. */
int oracle_dispatch(const int32_t *idx, int64_t T, int32_t k, int32_t E, int32_t *counts,
                    int32_t *offsets, int32_t *row_src, int32_t *pos_of)
{
    for (int32_t e = 0; e < E; ++e) counts[e] = 0;
    for (int64_t i = 0; i < T * k; ++i) {
        if (idx[i] < 0 || idx[i] >= E) return -1;
        counts[idx[i]]++;
    }
    offsets[0] = 0;
    for (int32_t e = 0; e < E; ++e) offsets[e + 1] = offsets[e] + counts[e];
    int32_t *cursor = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
    for (int32_t e = 0; e < E; ++e) cursor[e] = offsets[e];
    for (int64_t t = 0; t < T; ++t)
        for (int32_t j = 0; j < k; ++j) {
            int32_t p = cursor[idx[t * k + j]]++;
            row_src[p] = (int32_t)t;
            pos_of[t * k + j] = p;
        }
    free(cursor);
    return 0;
}

static double act_gelu(double u) { return u * 0.5 * (1.0 + erf(u / sqrt(2.0))); }

static double act_gelu_tanh(double u)
{
    const double c = sqrt(2.0 / M_PI);
    return 0.5 * u * (1.0 + tanh(c * (u + 0.044715 * u * u * u)));
}

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* ---- Step 4: one expert-shard FFN on one row ----------------------------------------
 * Full weights are laid out as the paper writes them: w1[e] is h x F (W_i), w2[e] is
 * F x h (W_o); w3[e] (SwiGLU up projection) is h x F like w1.  This device's shard is
 * the contiguous inner slice [col0, col0+f): columns of W_i, rows of W_o (Section 3.2).
 *   u[n]  = sum_j xr[j] * w1[e][j][col0+n]            n < f
 *   a[n]  = act(u[n])   (SwiGLU: silu(u[n]) * sum_j xr[j] * w3[e][j][col0+n])
 *   out[c] = sum_n a[n] * w2[e][col0+n][c]           c < h                         */
static void ffn_row(const float *xr, int32_t e, const float *w1, const float *w3,
                    const float *w2, int64_t h, int64_t F, int64_t col0, int64_t f, int act,
                    double *u, double *g, double *out)
{
    const float *W1 = w1 + (int64_t)e * h * F;
    const float *W2 = w2 + (int64_t)e * F * h;
    for (int64_t n = 0; n < f; ++n) u[n] = 0.0;
    for (int64_t j = 0; j < h; ++j) {
        const double xv = (double)xr[j];
        const float *row = W1 + j * F + col0;
        for (int64_t n = 0; n < f; ++n) u[n] += xv * (double)row[n];
    }
    if (act == ORACLE_ACT_SWIGLU) {
        const float *W3 = w3 + (int64_t)e * h * F;
        for (int64_t n = 0; n < f; ++n) g[n] = 0.0;
        for (int64_t j = 0; j < h; ++j) {
            const double xv = (double)xr[j];
            const float *row = W3 + j * F + col0;
            for (int64_t n = 0; n < f; ++n) g[n] += xv * (double)row[n];
        }
        for (int64_t n = 0; n < f; ++n) u[n] = silu(u[n]) * g[n];
    } else if (act == ORACLE_ACT_GELU_TANH) {
        for (int64_t n = 0; n < f; ++n) u[n] = act_gelu_tanh(u[n]);
    } else {
        for (int64_t n = 0; n < f; ++n) u[n] = act_gelu(u[n]);
    }
    for (int64_t c = 0; c < h; ++c) out[c] = 0.0;
    for (int64_t n = 0; n < f; ++n) {
        const double a = u[n];
        const float *row = W2 + (col0 + n) * h;
        for (int64_t c = 0; c < h; ++c) out[c] += a * (double)row[c];
    }
}

/* FFN of `n` independent rows: rows[r] (h values) through expert expert[r]'s shard. */
int oracle_ffn_rows(int64_t n, const float *rows, const int32_t *expert, int32_t E,
                    const float *w1, const float *w3, const float *w2, int64_t h, int64_t F,
                    int64_t col0, int64_t f, int32_t act, double *out)
{
    if (n < 0 || h < 1 || f < 0 || col0 < 0 || col0 + f > F) return -1;
    if (act == ORACLE_ACT_SWIGLU && !w3) return -1;
    for (int64_t r = 0; r < n; ++r)
        if (expert[r] < 0 || expert[r] >= E) return -1;
#pragma omp parallel
    {
        double *u = (double *)malloc(sizeof(double) * (size_t)(f > 0 ? f : 1));
        double *g = (double *)malloc(sizeof(double) * (size_t)(f > 0 ? f : 1));
#pragma omp for schedule(dynamic, 4)
        for (int64_t r = 0; r < n; ++r)
            ffn_row(rows + r * h, expert[r], w1, w3, w2, h, F, col0, f, act, u, g, out + r * h);
        free(u);
        free(g);
    }
    return 0;
}

/* Step 4 over grouped rows: x_perm rows [offsets[e], offsets[e+1]) go through expert e. */
int oracle_expert_ffn(const float *x_perm, const int32_t *offsets, int32_t E,
                      const float *w1, const float *w3, const float *w2, int64_t h, int64_t F,
                      int64_t col0, int64_t f, int32_t act, double *y_perm)
{
    const int64_t A = offsets[E];
    int32_t *ex = (int32_t *)malloc(sizeof(int32_t) * (size_t)(A > 0 ? A : 1));
    for (int32_t e = 0; e < E; ++e)
        for (int64_t p = offsets[e]; p < offsets[e + 1]; ++p) ex[p] = e;
    int rc = oracle_ffn_rows(A, x_perm, ex, E, w1, w3, w2, h, F, col0, f, act, y_perm);
    free(ex);
    return rc;
}

/* ---- Step 5: combine ------------------------------------------------------------------
 * y[t,c] = sum_{j=0..k-1} w[t,j] * y_perm[pos_of[t,j], c]   (j ascending)              */
int oracle_combine(const double *y_perm, const int32_t *pos_of, const double *w, int64_t T,
                   int32_t k, int64_t h, double *y)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t)
        for (int64_t c = 0; c < h; ++c) {
            double acc = 0.0;
            for (int32_t j = 0; j < k; ++j)
                acc += w[t * k + j] * y_perm[(int64_t)pos_of[t * k + j] * h + c];
            y[t * h + c] = acc;
        }
    return 0;
}

/* The layer output of selected tokens straight from the definition, without grouping:
 *   y[i] = sum_j w[t,j] * FFN_{idx[t,j]}(x[t])   for t = toks[i]                        */
int oracle_layer_tokens(int64_t n, const int64_t *toks, const float *x, const int32_t *idx,
                        const double *w, int32_t k, int32_t E, const float *w1,
                        const float *w3, const float *w2, int64_t h, int64_t F, int64_t col0,
                        int64_t f, int32_t act, double *y)
{
    if (n < 0 || k < 1 || h < 1 || f < 0 || col0 < 0 || col0 + f > F) return -1;
    if (act == ORACLE_ACT_SWIGLU && !w3) return -1;
    int bad = 0;
    for (int64_t i = 0; i < n; ++i)
        for (int32_t j = 0; j < k; ++j)
            if (idx[toks[i] * k + j] < 0 || idx[toks[i] * k + j] >= E) bad = 1;
    if (bad) return -1;
#pragma omp parallel
    {
        double *u = (double *)malloc(sizeof(double) * (size_t)(f > 0 ? f : 1));
        double *g = (double *)malloc(sizeof(double) * (size_t)(f > 0 ? f : 1));
        double *o = (double *)malloc(sizeof(double) * (size_t)h);
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < n; ++i) {
            const int64_t t = toks[i];
            double *yr = y + i * h;
            for (int64_t c = 0; c < h; ++c) yr[c] = 0.0;
            for (int32_t j = 0; j < k; ++j) {
                ffn_row(x + t * h, idx[t * k + j], w1, w3, w2, h, F, col0, f, act, u, g, o);
                const double wt = w[t * k + j];
                for (int64_t c = 0; c < h; ++c) yr[c] += wt * o[c];
            }
        }
        free(u);
        free(g);
        free(o);
    }
    return 0;
}

int oracle_num_threads(void)
{
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
