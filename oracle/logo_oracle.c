/*
 * logo_oracle.c -- plain fp64 CPU oracle for the forward pass of one LoGo
 * attention layer (LoGo: Token-Level Dynamic Local-Global Attention).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the definition the GPU path is
 * checked against.  It shares no code with the HIP library: it is compiled by
 * gcc into its own shared object and is called only by the tests, by the
 * package smoke check and by the benchmark's CPU-baseline leg.  Nothing on
 * the product path may load it.
 *
 * Every function writes out a plain definition from the paper, in double
 * precision, without tiling, online rescaling or any reordering beyond what
 * the definition states:
 *
 *   - softmax attention over a context set C_t           (Sec. 3.1, Eq. attention)
 *   - global context {1..t}, local context {max(1,t-w+1)..t}
 *                                                         (Sec. 3.1, below Eq. attention)
 *   - hard routing z_t = [p_t > b_th], strict, shared by all heads
 *                                                         (Sec. 3.2, Eq. gate-routing;
 *                                                          Sec. 3.1, Eq. token-routing)
 *   - query-sparse global branch: global rows only for selected tokens,
 *     keys/values dense                                   (Sec. 3.2, Eq. query-sparse-global)
 *   - ContextNorm: head-wise RMSNorm of each branch       (Sec. 3.2, Eq. contextnorm)
 *   - output fusion (1-p) oL + p oG for selected tokens,
 *     oL otherwise                                        (Sec. 3.2, Eq. output-fusion)
 *   - realized ratio F = (selected tokens) / (valid tokens)
 *                                                         (Sec. 3.1, Eq. realized-ratio)
 *   - budget controller b_th <- b_th + gamma sign(F - rho) and the P-mask
 *     starting threshold                                  (Sec. 3.2, Eq. threshold-update
 *                                                          and the P-mask paragraph)
 *   - one autoregressive decoding step: the new token's local and (when
 *     selected) global attention over the KV cache, fused as above
 *                                                         (Sec. 3.3 and App. B,
 *                                                          Autoregressive Decoding)
 *   - the gate projection p = sigmoid(x . w_g)            (Sec. 3.2, Eq. gate-routing)
 *   - the backward pass: gradients of the layer's inputs given dL/d out,
 *     the selection held fixed                            (Sec. 3.3 and App. B, the
 *                                                          row-sparse backward)
 *   - the branch transforms LP (U A) and SO (U * s + b)   (Sec. 3.2, Eq. branch-transform)
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - positions are 0-based: key j is visible to query i iff j <= i (global)
 *     or i-w < j <= i (local); the local context holds exactly min(i+1, w)
 *     keys, the query itself included.
 *   - a target ratio rho becomes a per-sequence threshold: k = floor(rho*T)
 *     in IEEE double; thr = -inf if k == T, else the (k+1)-th largest gate
 *     value of the sequence (an input value, no interpolation).  A zero
 *     threshold is reported as +0.0.
 *   - GQA: query head h reads key/value head floor(h / (Hq/Hkv)).
 *   - ContextNorm: o / sqrt(mean_c o_c^2 + eps) * g per (token, head), with a
 *     per-branch gain g[Hq][d] (1 when absent).
 *   - the fusion weight is the fp32 gate value p, widened to double.
 *
 * Inputs: bf16 tensors are raw uint16 bit patterns, widened exactly.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_SEL_THRESHOLD 0
#define ORACLE_SEL_RATIO 1

static double bf16_to_double(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Sequence that owns packed token t: largest b with cu[b] <= t < cu[b+1]. */
static int owner_sequence(const int32_t *cu, int B, int64_t t)
{
    int lo = 0, hi = B - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) / 2;
        if ((int64_t)cu[mid] <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    /* skip empty sequences that start at the same offset */
    while (lo + 1 < B && (int64_t)cu[lo + 1] <= t)
        lo++;
    return lo;
}

static int cmp_float_ascending(const void *a, const void *b)
{
    float x = *(const float *)a, y = *(const float *)b;
    return (x < y) ? -1 : (x > y) ? 1 : 0;
}

/*
 * Realized global ratio of one routing pass (Sec. 3.1, Eq. realized-ratio):
 * the fraction of the n_valid token positions whose z is 1, in double.
 */
double oracle_realized_ratio(int64_t n_selected, int64_t n_valid)
{
    return n_valid > 0 ? (double)n_selected / (double)n_valid : 0.0;
}

/*
 * One budget-controller step (Sec. 3.2, Eq. threshold-update):
 *   b_th <- b_th + gamma * sign(F - rho)
 * with sign(0) = 0: the threshold rises when more tokens than the target
 * went global (fewer pass next time) and falls when fewer did.  F is the
 * realized ratio above and is compared with rho in double; the update itself
 * is one fp32 multiply-free add of +-gamma (or nothing).  No valid tokens:
 * no update.
 */
float oracle_budget_update(float b_th, int64_t n_selected, int64_t n_valid, double rho,
                           float gamma)
{
    if (n_valid <= 0)
        return b_th;
    double f = oracle_realized_ratio(n_selected, n_valid);
    if (f > rho)
        return b_th + gamma;
    if (f < rho)
        return b_th - gamma;
    return b_th;
}

/*
 * P-mask starting threshold (Sec. 3.2, progressive masking): chosen so that
 * pmask_steps controller steps of +gamma (every token is selected while the
 * threshold is below every gate, so F = 1 > rho) bring b_th to the initial
 * gate centre 0.5: b_th,0 = 0.5 - gamma * pmask_steps, evaluated in double
 * and rounded once to fp32.
 */
float oracle_pmask_initial_threshold(float gamma, int64_t pmask_steps)
{
    return (float)(0.5 - (double)gamma * (double)pmask_steps);
}

/*
 * Per-sequence threshold b_th (Sec. 3.2, Eq. gate-routing).
 * Threshold mode: every sequence uses `threshold`.
 * Ratio mode: the order statistic described in the header.
 */
void oracle_thresholds(const float *gate, const int32_t *cu, int B, int mode,
                       float threshold, double ratio, float *thr_out)
{
    for (int b = 0; b < B; b++) {
        if (mode == ORACLE_SEL_THRESHOLD) {
            thr_out[b] = threshold;
            continue;
        }
        int64_t T = (int64_t)cu[b + 1] - cu[b];
        int64_t k = (int64_t)floor(ratio * (double)T);
        if (k >= T) {
            thr_out[b] = -INFINITY;
            continue;
        }
        float *s = (float *)malloc((size_t)T * sizeof(float));
        memcpy(s, gate + cu[b], (size_t)T * sizeof(float));
        qsort(s, (size_t)T, sizeof(float), cmp_float_ascending);
        float thr = s[T - k - 1];
        if (thr == 0.0f)
            thr = 0.0f; /* -0.0 -> +0.0 */
        thr_out[b] = thr;
        free(s);
    }
}

/*
 * Hard routing (Sec. 3.2, Eq. gate-routing): z_t = [p_t > thr_b], compared in
 * fp32, selected tokens kept in ascending order.  Writes sel_idx (packed
 * token index), cu_sel[B+1] (selections before each sequence), tok2sel[N]
 * (rank or -1).  Returns the number of selected tokens.
 */
int64_t oracle_select(const float *gate, const int32_t *cu, int B, const float *thr,
                      int32_t *sel_idx, int32_t *cu_sel, int32_t *tok2sel)
{
    int64_t n = 0;
    for (int b = 0; b < B; b++) {
        cu_sel[b] = (int32_t)n;
        for (int64_t t = cu[b]; t < cu[b + 1]; t++) {
            if (gate[t] > thr[b]) {
                if (sel_idx)
                    sel_idx[n] = (int32_t)t;
                if (tok2sel)
                    tok2sel[t] = (int32_t)n;
                n++;
            } else if (tok2sel) {
                tok2sel[t] = -1;
            }
        }
    }
    cu_sel[B] = (int32_t)n;
    return n;
}

/*
 * Softmax attention for a list of query rows (Sec. 3.1, Eq. attention).
 * rows[r] is a packed token index; out is [n_rows][Hq][d].
 * window <= 0 : global context, keys 0..pos
 * window >= 1 : local context, keys max(0, pos-window+1)..pos
 * Two passes per (row, head): scores and their maximum, then the weighted
 * sum of values divided by the sum of weights.
 */
void oracle_attn_rows(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                      int Hq, int Hkv, int d, const int32_t *cu, int B,
                      const int32_t *rows, int64_t n_rows, int window, double scale,
                      double *out)
{
    const int G = Hq / Hkv;
    int64_t max_T = 0;
    for (int b = 0; b < B; b++)
        if ((int64_t)cu[b + 1] - cu[b] > max_T)
            max_T = (int64_t)cu[b + 1] - cu[b];

#pragma omp parallel
    {
        double *s = (double *)malloc((size_t)(max_T > 0 ? max_T : 1) * sizeof(double));
        double *qd = (double *)malloc((size_t)d * sizeof(double));
        double *acc = (double *)malloc((size_t)d * sizeof(double));
#pragma omp for schedule(dynamic, 4)
        for (int64_t job = 0; job < n_rows * Hq; job++) {
            int64_t r = job / Hq;
            int h = (int)(job % Hq);
            int hk = h / G;
            int64_t t = rows[r];
            int b = owner_sequence(cu, B, t);
            int64_t base = cu[b];
            int64_t pos = t - base;
            int64_t lo = (window >= 1) ? (pos - window + 1 > 0 ? pos - window + 1 : 0) : 0;
            int64_t nk = pos - lo + 1;

            for (int c = 0; c < d; c++)
                qd[c] = bf16_to_double(q[(t * Hq + h) * (int64_t)d + c]);

            double m = -INFINITY;
            for (int64_t j = 0; j < nk; j++) {
                const uint16_t *kr = k + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                double dot = 0.0;
                for (int c = 0; c < d; c++)
                    dot += qd[c] * bf16_to_double(kr[c]);
                s[j] = scale * dot;
                if (s[j] > m)
                    m = s[j];
            }

            double den = 0.0;
            for (int c = 0; c < d; c++)
                acc[c] = 0.0;
            for (int64_t j = 0; j < nk; j++) {
                double e = exp(s[j] - m);
                const uint16_t *vr = v + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                den += e;
                for (int c = 0; c < d; c++)
                    acc[c] += e * bf16_to_double(vr[c]);
            }
            double *o = out + (r * Hq + h) * (int64_t)d;
            for (int c = 0; c < d; c++)
                o[c] = acc[c] / den;
        }
        free(s);
        free(qd);
        free(acc);
    }
}

/*
 * ContextNorm (Sec. 3.2, Eq. contextnorm): head-wise RMSNorm, in place on
 * o[n_rows][Hq][d].  gain is [Hq][d] (NULL means 1).
 */
void oracle_contextnorm(double *o, int64_t n_rows, int Hq, int d, const float *gain,
                        double eps)
{
#pragma omp parallel for schedule(static)
    for (int64_t job = 0; job < n_rows * Hq; job++) {
        int h = (int)(job % Hq);
        double *row = o + job * (int64_t)d;
        double ss = 0.0;
        for (int c = 0; c < d; c++)
            ss += row[c] * row[c];
        double inv = 1.0 / sqrt(ss / (double)d + eps);
        for (int c = 0; c < d; c++) {
            double g = gain ? (double)gain[h * d + c] : 1.0;
            row[c] = row[c] * inv * g;
        }
    }
}

/*
 * Output fusion (Sec. 3.2, Eq. output-fusion).  ol is [N][Hq][d] (all
 * tokens), og is [n_sel][Hq][d] (compact, rank order); out is [N][Hq][d].
 */
void oracle_fuse(const double *ol, const double *og, const float *gate,
                 const int32_t *tok2sel, int64_t N, int Hq, int d, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N; t++) {
        const int64_t row = (int64_t)Hq * d;
        const double *l = ol + t * row;
        double *o = out + t * row;
        int32_t r = tok2sel[t];
        if (r < 0) {
            for (int64_t e = 0; e < row; e++)
                o[e] = l[e];
        } else {
            double p = (double)gate[t];
            const double *g = og + (int64_t)r * row;
            for (int64_t e = 0; e < row; e++)
                o[e] = (1.0 - p) * l[e] + p * g[e];
        }
    }
}

/*
 * The whole layer.  q_g/k_g/v_g may be NULL (identity branch transform:
 * the global branch reads the local tensors, Sec. 3.2, Eq. branch-transform
 * at initialisation).  apply_norm = 0 skips ContextNorm (raw fusion, a
 * diagnostic).  Outputs (all caller-allocated):
 *   thr_out[B], sel_idx[N], cu_sel[B+1], tok2sel[N],
 *   o_local[N][Hq][d]  (raw local branch),
 *   o_global[N][Hq][d] (raw global branch, compact: first n_sel rows used),
 *   out[N][Hq][d]      (fused output).
 * Returns n_sel.
 */
int64_t oracle_logo_fwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const uint16_t *q_g, const uint16_t *k_g, const uint16_t *v_g,
                        const float *gate, const int32_t *cu, int B, int Hq, int Hkv,
                        int d, int window, double scale, int mode, float threshold,
                        double ratio, const float *gain_local, const float *gain_global,
                        double eps, int apply_norm, float *thr_out, int32_t *sel_idx,
                        int32_t *cu_sel, int32_t *tok2sel, double *o_local,
                        double *o_global, double *out)
{
    const int64_t N = cu[B];
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    if (!q_g)
        q_g = q;
    if (!k_g)
        k_g = k;
    if (!v_g)
        v_g = v;

    oracle_thresholds(gate, cu, B, mode, threshold, ratio, thr_out);
    int64_t n_sel = oracle_select(gate, cu, B, thr_out, sel_idx, cu_sel, tok2sel);

    int32_t *all = (int32_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int32_t));
    for (int64_t t = 0; t < N; t++)
        all[t] = (int32_t)t;
    oracle_attn_rows(q, k, v, Hq, Hkv, d, cu, B, all, N, window, scale, o_local);
    free(all);
    oracle_attn_rows(q_g, k_g, v_g, Hq, Hkv, d, cu, B, sel_idx, n_sel, 0, scale, o_global);

    const int64_t row = (int64_t)Hq * d;
    double *nl = (double *)malloc((size_t)(N > 0 ? N : 1) * row * sizeof(double));
    double *ng = (double *)malloc((size_t)(n_sel > 0 ? n_sel : 1) * row * sizeof(double));
    memcpy(nl, o_local, (size_t)N * row * sizeof(double));
    memcpy(ng, o_global, (size_t)n_sel * row * sizeof(double));
    if (apply_norm) {
        oracle_contextnorm(nl, N, Hq, d, gain_local, eps);
        oracle_contextnorm(ng, n_sel, Hq, d, gain_global, eps);
    }
    oracle_fuse(nl, ng, gate, tok2sel, N, Hq, d, out);
    free(nl);
    free(ng);
    return n_sel;
}

/*
 * One autoregressive decoding step of the layer (Sec. 3.3, Autoregressive
 * Decoding; App. B, Autoregressive Decoding).
 *
 * Sequence b's cache holds L_b = cu[b+1] - cu[b] >= 1 tokens (rows cu[b] ..
 * cu[b+1]-1 of k/v and k_g/v_g); the last of them is the new token itself,
 * at position L_b - 1, its key and value already appended.  Its query
 * q_new[b] attends over the local context (the last min(L_b, w) cached keys,
 * itself included).  Its gate value gate_new[b] decides the global branch
 * (z = [p > threshold], strict, as in Eq. gate-routing); a selected token's
 * global query q_g_new[b] attends over all L_b cached global keys.  Both
 * outputs are ContextNorm-ed and fused as in Eqs. contextnorm and
 * output-fusion; an unselected token's output is Norm^L of its local output.
 *
 * Inputs as in oracle_logo_fwd; q_new, q_g_new are [B][Hq][d] (q_g_new,
 * k_g, v_g may be NULL: the local tensors).  Outputs: o_local[B][Hq][d] and
 * o_global[B][Hq][d] (raw branch outputs; rows of unselected tokens are
 * zero), out[B][Hq][d], z_out[B].  Returns the number of selected tokens.
 */
int64_t oracle_decode(const uint16_t *q_new, const uint16_t *q_g_new, const uint16_t *k,
                      const uint16_t *v, const uint16_t *k_g, const uint16_t *v_g,
                      const float *gate_new, const int32_t *cu, int B, int Hq, int Hkv, int d,
                      int window, double scale, float threshold, const float *gain_local,
                      const float *gain_global, double eps, double *o_local, double *o_global,
                      double *out, int32_t *z_out)
{
    const int G = Hq / Hkv;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    if (!q_g_new)
        q_g_new = q_new;
    if (!k_g)
        k_g = k;
    if (!v_g)
        v_g = v;
    int64_t max_L = 1;
    int64_t n_sel = 0;
    for (int b = 0; b < B; b++) {
        if ((int64_t)cu[b + 1] - cu[b] > max_L)
            max_L = (int64_t)cu[b + 1] - cu[b];
        z_out[b] = gate_new[b] > threshold ? 1 : 0;
        n_sel += z_out[b];
    }

#pragma omp parallel
    {
        double *score = (double *)malloc((size_t)max_L * sizeof(double));
        double *qd = (double *)malloc((size_t)d * sizeof(double));
        double *acc = (double *)malloc((size_t)d * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t job = 0; job < (int64_t)B * Hq * 2; job++) {
            const int branch = (int)(job % 2); /* 0 local, 1 global */
            const int h = (int)((job / 2) % Hq);
            const int b = (int)(job / 2 / Hq);
            const int kvh = h / G;
            const int64_t base = cu[b];
            const int64_t L = (int64_t)cu[b + 1] - base;
            double *o = (branch == 0 ? o_local : o_global) + ((int64_t)b * Hq + h) * d;
            if (branch == 1 && !z_out[b]) {
                for (int c = 0; c < d; c++)
                    o[c] = 0.0;
                continue;
            }
            const uint16_t *qq = (branch == 0 ? q_new : q_g_new) + ((int64_t)b * Hq + h) * d;
            const uint16_t *kk = branch == 0 ? k : k_g;
            const uint16_t *vv = branch == 0 ? v : v_g;
            /* context: keys lo .. L-1 of the cache */
            const int64_t lo = (branch == 0 && L > window) ? L - window : 0;
            const int64_t nk = L - lo;
            for (int c = 0; c < d; c++)
                qd[c] = bf16_to_double(qq[c]);
            double m = -INFINITY;
            for (int64_t j = 0; j < nk; j++) {
                const uint16_t *kr = kk + ((base + lo + j) * Hkv + kvh) * (int64_t)d;
                double dot = 0.0;
                for (int c = 0; c < d; c++)
                    dot += qd[c] * bf16_to_double(kr[c]);
                score[j] = scale * dot;
                if (score[j] > m)
                    m = score[j];
            }
            double wsum = 0.0;
            for (int c = 0; c < d; c++)
                acc[c] = 0.0;
            for (int64_t j = 0; j < nk; j++) {
                const double e = exp(score[j] - m);
                const uint16_t *vr = vv + ((base + lo + j) * Hkv + kvh) * (int64_t)d;
                wsum += e;
                for (int c = 0; c < d; c++)
                    acc[c] += e * bf16_to_double(vr[c]);
            }
            for (int c = 0; c < d; c++)
                o[c] = acc[c] / wsum;
        }
        free(score);
        free(qd);
        free(acc);
    }

    /* ContextNorm of both branches, then the fusion */
    const int64_t row = (int64_t)Hq * d;
    double *nl = (double *)malloc((size_t)B * row * sizeof(double));
    double *ng = (double *)malloc((size_t)B * row * sizeof(double));
    memcpy(nl, o_local, (size_t)B * row * sizeof(double));
    memcpy(ng, o_global, (size_t)B * row * sizeof(double));
    oracle_contextnorm(nl, B, Hq, d, gain_local, eps);
    oracle_contextnorm(ng, B, Hq, d, gain_global, eps);
    for (int b = 0; b < B; b++) {
        const double p = (double)gate_new[b];
        for (int64_t e = 0; e < row; e++) {
            const double l = nl[b * row + e];
            out[b * row + e] = z_out[b] ? (1.0 - p) * l + p * ng[b * row + e] : l;
        }
    }
    free(nl);
    free(ng);
    return n_sel;
}

/*
 * Gate projection (Sec. 3.2, Eq. gate-routing): p_t = sigmoid(x_t . w_g) for
 * every token, x [N][dm] and w_g [dm] bf16, the dot product and the sigmoid
 * in double, p rounded once to fp32.
 */
void oracle_gate_proj(const uint16_t *x, const uint16_t *w_g, int64_t N, int dm, float *p_out)
{
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < N; t++) {
        double dot = 0.0;
        for (int c = 0; c < dm; c++)
            dot += bf16_to_double(x[t * dm + c]) * bf16_to_double(w_g[c]);
        p_out[t] = (float)(1.0 / (1.0 + exp(-dot)));
    }
}

/*
 * Branch transform phi_{U,h} from local to global representations (Sec.
 * 3.2, Eq. branch-transform), per head h of u [N][H][d] (bf16):
 *   kind 0 (LP): out[t][h][j] = sum_c u[t][h][c] * A[h][c][j]   (A bf16 [H][d][d])
 *   kind 1 (SO): out[t][h][j] = u[t][h][j] * s[h][j] + b[h][j] (s, b fp32 [H][d])
 * for the token rows listed in rows[0..n_rows) (all N tokens when rows is
 * NULL, n_rows = N).  out is [n_rows][H][d] in double (not rounded).
 */
void oracle_branch_transform(const uint16_t *u, int H, int d, int kind, const uint16_t *A,
                             const float *s, const float *b, const int32_t *rows,
                             int64_t n_rows, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n_rows; r++) {
        const int64_t t = rows ? rows[r] : r;
        for (int h = 0; h < H; h++) {
            const uint16_t *ur = u + (t * H + h) * (int64_t)d;
            double *o = out + (r * H + h) * (int64_t)d;
            for (int j = 0; j < d; j++) {
                if (kind == 0) {
                    double acc = 0.0;
                    for (int c = 0; c < d; c++)
                        acc += bf16_to_double(ur[c]) *
                               bf16_to_double(A[((int64_t)h * d + c) * d + j]);
                    o[j] = acc;
                } else {
                    o[j] = bf16_to_double(ur[j]) * (double)s[h * d + j] + (double)b[h * d + j];
                }
            }
        }
    }
}

/*
 * Backward pass of the layer for training (Sec. 3.3 and App. B: the backward
 * keeps the forward's row-sparse structure; query gradients exist only for
 * the rows a branch computes).  The selection is the forward's (threshold /
 * ratio as in oracle_logo_fwd) and is held fixed: z is a hard decision with
 * no gradient.  Given dout = dL/d out [N][Hq][d] (double), the chain rule is
 * written out per (row, head), in double:
 *   fusion (Eq. output-fusion):  d~oL = (z ? 1-p : 1) dout,  d~oG = p dout,
 *                                dL/dp = z * sum_{h,c} dout (~oG - ~oL)
 *   ContextNorm (Eq. contextnorm), y = o g / r, r = sqrt(mean o^2 + eps):
 *                                dg_c += dy_c o_c / r,
 *                                do_c = g_c dy_c / r - o_c (sum_k g_k dy_k o_k) / (d r^3)
 *   attention (Eq. attention):   P = softmax(scale q.k_j) over the context,
 *                                dv_j += P_j do,  dP_j = do . v_j,
 *                                dS_j = P_j (dP_j - sum_k P_k dP_k),
 *                                dq += scale sum_j dS_j k_j,  dk_j += scale dS_j q
 * Outputs (caller-allocated, overwritten): dq, dk, dv for the local-branch
 * tensors and dq_g, dk_g, dv_g for the global-branch ones (with aliased
 * global tensors the caller adds each pair), dgate [N], dgain_l and dgain_g
 * [Hq][d].  Returns n_sel.
 */
int64_t oracle_logo_bwd(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                        const uint16_t *q_g, const uint16_t *k_g, const uint16_t *v_g,
                        const float *gate, const int32_t *cu, int B, int Hq, int Hkv, int d,
                        int window, double scale, int mode, float threshold, double ratio,
                        const float *gain_local, const float *gain_global, double eps,
                        const double *dout, double *dq, double *dk, double *dv, double *dq_g,
                        double *dk_g, double *dv_g, double *dgate, double *dgain_l,
                        double *dgain_g)
{
    const int64_t N = cu[B];
    const int G = Hq / Hkv;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    if (!q_g)
        q_g = q;
    if (!k_g)
        k_g = k;
    if (!v_g)
        v_g = v;
    float *thr = (float *)malloc((size_t)B * sizeof(float));
    int32_t *sel = (int32_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int32_t));
    int32_t *cu_sel = (int32_t *)malloc((size_t)(B + 1) * sizeof(int32_t));
    int32_t *t2s = (int32_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int32_t));
    oracle_thresholds(gate, cu, B, mode, threshold, ratio, thr);
    const int64_t n_sel = oracle_select(gate, cu, B, thr, sel, cu_sel, t2s);

    const int64_t row = (int64_t)Hq * d;
    memset(dq, 0, (size_t)N * row * sizeof(double));
    memset(dq_g, 0, (size_t)N * row * sizeof(double));
    memset(dk, 0, (size_t)N * Hkv * d * sizeof(double));
    memset(dv, 0, (size_t)N * Hkv * d * sizeof(double));
    memset(dk_g, 0, (size_t)N * Hkv * d * sizeof(double));
    memset(dv_g, 0, (size_t)N * Hkv * d * sizeof(double));
    memset(dgain_l, 0, (size_t)row * sizeof(double));
    memset(dgain_g, 0, (size_t)row * sizeof(double));
    /* normalised branch outputs ~oL (all rows) and ~oG (selected rows, by token) */
    double *yl = (double *)calloc((size_t)(N > 0 ? N : 1) * row, sizeof(double));
    double *yg = (double *)calloc((size_t)(N > 0 ? N : 1) * row, sizeof(double));
    int64_t max_T = 1;
    for (int b = 0; b < B; b++)
        if ((int64_t)cu[b + 1] - cu[b] > max_T)
            max_T = (int64_t)cu[b + 1] - cu[b];

    /* one job per (branch, KV head): the rows of its G query heads, so the
       dk / dv / gain accumulations of a job touch only its own heads */
#pragma omp parallel for schedule(dynamic, 1)
    for (int job = 0; job < 2 * Hkv; job++) {
        const int branch = job / Hkv; /* 0 local, 1 global */
        const int hk = job % Hkv;
        const uint16_t *Q = branch ? q_g : q, *K = branch ? k_g : k, *V = branch ? v_g : v;
        double *dQ = branch ? dq_g : dq, *dK = branch ? dk_g : dk, *dV = branch ? dv_g : dv;
        double *dG = branch ? dgain_g : dgain_l, *Y = branch ? yg : yl;
        const float *gain = branch ? gain_global : gain_local;
        double *P = (double *)malloc((size_t)max_T * sizeof(double));
        double *dP = (double *)malloc((size_t)max_T * sizeof(double));
        double *qd = (double *)malloc((size_t)d * sizeof(double));
        double *o = (double *)malloc((size_t)d * sizeof(double));
        double *dy = (double *)malloc((size_t)d * sizeof(double));
        double *dO = (double *)malloc((size_t)d * sizeof(double));
        for (int b = 0; b < B; b++) {
            const int64_t base = cu[b], T = (int64_t)cu[b + 1] - base;
            for (int64_t i = 0; i < T; i++) {
                const int64_t t = base + i;
                const int z = t2s[t] >= 0;
                if (branch == 1 && !z)
                    continue;
                const int64_t lo = (branch == 0 && i - window + 1 > 0) ? i - window + 1 : 0;
                const int64_t nk = i - lo + 1;
                const double p = (double)gate[t];
                for (int h = hk * G; h < (hk + 1) * G; h++) {
                    for (int c = 0; c < d; c++)
                        qd[c] = bf16_to_double(Q[(t * Hq + h) * (int64_t)d + c]);
                    /* forward recomputation: P, o, r, y */
                    double m = -INFINITY;
                    for (int64_t j = 0; j < nk; j++) {
                        const uint16_t *kr = K + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        double dot = 0.0;
                        for (int c = 0; c < d; c++)
                            dot += qd[c] * bf16_to_double(kr[c]);
                        P[j] = scale * dot;
                        if (P[j] > m)
                            m = P[j];
                    }
                    double den = 0.0;
                    for (int64_t j = 0; j < nk; j++) {
                        P[j] = exp(P[j] - m);
                        den += P[j];
                    }
                    for (int c = 0; c < d; c++)
                        o[c] = 0.0;
                    for (int64_t j = 0; j < nk; j++) {
                        P[j] /= den;
                        const uint16_t *vr = V + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        for (int c = 0; c < d; c++)
                            o[c] += P[j] * bf16_to_double(vr[c]);
                    }
                    double ms = 0.0;
                    for (int c = 0; c < d; c++)
                        ms += o[c] * o[c];
                    const double r = sqrt(ms / (double)d + eps);
                    double *yr = Y + (t * Hq + h) * (int64_t)d;
                    const double *dr = dout + (t * Hq + h) * (int64_t)d;
                    const double wgt = branch ? p : (z ? 1.0 - p : 1.0);
                    const float *gh = gain ? gain + (int64_t)h * d : NULL;
                    double gdo = 0.0;
                    for (int c = 0; c < d; c++) {
                        const double gc = gh ? (double)gh[c] : 1.0;
                        yr[c] = o[c] / r * gc;
                        dy[c] = wgt * dr[c];
                        dG[h * d + c] += dy[c] * o[c] / r;
                        gdo += gc * dy[c] * o[c];
                    }
                    /* ContextNorm backward */
                    for (int c = 0; c < d; c++) {
                        const double gc = gh ? (double)gh[c] : 1.0;
                        dO[c] = gc * dy[c] / r - o[c] * gdo / ((double)d * r * r * r);
                    }
                    /* softmax attention backward */
                    double delta = 0.0;
                    for (int64_t j = 0; j < nk; j++) {
                        const uint16_t *vr = V + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        double s = 0.0;
                        for (int c = 0; c < d; c++)
                            s += dO[c] * bf16_to_double(vr[c]);
                        dP[j] = s;
                        delta += P[j] * s;
                    }
                    double *dqr = dQ + (t * Hq + h) * (int64_t)d;
                    for (int64_t j = 0; j < nk; j++) {
                        const double ds = P[j] * (dP[j] - delta);
                        const uint16_t *kr = K + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        double *dkr = dK + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        double *dvr = dV + ((base + lo + j) * Hkv + hk) * (int64_t)d;
                        for (int c = 0; c < d; c++) {
                            dqr[c] += scale * ds * bf16_to_double(kr[c]);
                            dkr[c] += scale * ds * qd[c];
                            dvr[c] += P[j] * dO[c];
                        }
                    }
                }
            }
        }
        free(P);
        free(dP);
        free(qd);
        free(o);
        free(dy);
        free(dO);
    }
    /* gate gradient through the fusion weight */
    for (int64_t t = 0; t < N; t++) {
        double acc = 0.0;
        if (t2s[t] >= 0)
            for (int64_t e = 0; e < row; e++)
                acc += dout[t * row + e] * (yg[t * row + e] - yl[t * row + e]);
        dgate[t] = acc;
    }
    free(yl);
    free(yg);
    free(thr);
    free(sel);
    free(cu_sel);
    free(t2s);
    return n_sel;
}

/*
 * Backward of ContextNorm and the fusion alone (Eqs. contextnorm and
 * output-fusion), per (token, head), given the raw branch outputs:
 *   ol [N][Hq][d] (every token), og [N][Hq][d] (rows of selected tokens,
 *   indexed by token; others unused), gate p [N], z [N] (1 = selected),
 *   gains (NULL = 1), eps, dout [N][Hq][d].
 * Writes dol = dL/d oL, dog = dL/d oG (zero for unselected tokens), the
 * row sums delta_l[t][h] = sum_c dol * ol and delta_g[t][h] = sum_c dog * og,
 * dgate [N] and the gain gradients dgain_l, dgain_g [Hq][d].  The same chain
 * rule as in oracle_logo_bwd, in double.
 */
void oracle_fusion_bwd(const double *ol, const double *og, const float *gate, const int32_t *z,
                       int64_t N, int Hq, int d, const float *gain_local,
                       const float *gain_global, double eps, const double *dout, double *dol,
                       double *dog, double *delta_l, double *delta_g, double *dgate,
                       double *dgain_l, double *dgain_g)
{
    memset(dgain_l, 0, (size_t)Hq * d * sizeof(double));
    memset(dgain_g, 0, (size_t)Hq * d * sizeof(double));
    for (int64_t t = 0; t < N; t++) {
        const double p = (double)gate[t];
        double dp = 0.0;
        for (int h = 0; h < Hq; h++) {
            const int64_t off = (t * Hq + h) * (int64_t)d;
            const double *dr = dout + off;
            for (int branch = 0; branch < 2; branch++) {
                const double *o = (branch ? og : ol) + off;
                double *dO = (branch ? dog : dol) + off;
                double *delta = branch ? delta_g : delta_l;
                double *dgn = branch ? dgain_g : dgain_l;
                const float *gn = branch ? gain_global : gain_local;
                if (branch == 1 && !z[t]) {
                    for (int c = 0; c < d; c++)
                        dO[c] = 0.0;
                    delta[t * Hq + h] = 0.0;
                    continue;
                }
                const double wgt = branch ? p : (z[t] ? 1.0 - p : 1.0);
                double sq = 0.0;
                for (int c = 0; c < d; c++)
                    sq += o[c] * o[c];
                const double rr = sqrt(sq / (double)d + eps);
                double proj = 0.0, side = 0.0;
                for (int c = 0; c < d; c++) {
                    const double gc = gn ? (double)gn[(int64_t)h * d + c] : 1.0;
                    const double y = o[c] / rr * gc;
                    proj += gc * wgt * dr[c] * o[c];
                    dgn[(int64_t)h * d + c] += wgt * dr[c] * o[c] / rr;
                    side += (branch ? 1.0 : -1.0) * dr[c] * y;
                }
                if (z[t])
                    dp += side;
                double dl = 0.0;
                for (int c = 0; c < d; c++) {
                    const double gc = gn ? (double)gn[(int64_t)h * d + c] : 1.0;
                    dO[c] = gc * wgt * dr[c] / rr - o[c] * proj / ((double)d * rr * rr * rr);
                    dl += dO[c] * o[c];
                }
                delta[t * Hq + h] = dl;
            }
        }
        dgate[t] = dp;
    }
}

/*
 * Backward of plain causal softmax attention (Eq. attention; with window >= 1
 * the local context of Sec. 3.1, keys max(0, i-w+1)..i; window <= 0 = full
 * causal): the dense baseline's training step.  Given dout = dL/do
 * [N][Hq][d] (double) for o_i = sum_j P_ij v_j, P_i = softmax(scale q_i.k_j):
 *   dv_j += P_ij dout_i,   dP_ij = dout_i . v_j,
 *   dS_ij = P_ij (dP_ij - sum_k P_ik dP_ik),
 *   dq_i += scale sum_j dS_ij k_j,   dk_j += scale dS_ij q_i
 * Outputs dq [N][Hq][d], dk, dv [N][Hkv][d] (overwritten), in double.
 */
void oracle_attn_bwd(const uint16_t *q, const uint16_t *k, const uint16_t *v, const int32_t *cu,
                     int B, int Hq, int Hkv, int d, int window, double scale, const double *dout,
                     double *dq, double *dk, double *dv)
{
    const int64_t N = cu[B];
    const int G = Hq / Hkv;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    memset(dq, 0, (size_t)N * Hq * d * sizeof(double));
    memset(dk, 0, (size_t)N * Hkv * d * sizeof(double));
    memset(dv, 0, (size_t)N * Hkv * d * sizeof(double));
    int64_t max_T = 1;
    for (int b = 0; b < B; b++)
        if ((int64_t)cu[b + 1] - cu[b] > max_T)
            max_T = (int64_t)cu[b + 1] - cu[b];
    /* one job per KV head: the dk / dv rows it accumulates are its own */
#pragma omp parallel for schedule(dynamic, 1)
    for (int hk = 0; hk < Hkv; hk++) {
        double *w_p = (double *)malloc((size_t)max_T * sizeof(double));
        double *w_dp = (double *)malloc((size_t)max_T * sizeof(double));
        double *qrow = (double *)malloc((size_t)d * sizeof(double));
        for (int b = 0; b < B; b++) {
            const int64_t base = cu[b], T = (int64_t)cu[b + 1] - base;
            for (int64_t i = 0; i < T; i++) {
                const int64_t first = (window >= 1 && i - window + 1 > 0) ? i - window + 1 : 0;
                const int64_t cnt = i - first + 1;
                for (int h = hk * G; h < (hk + 1) * G; h++) {
                    const int64_t qo = ((base + i) * Hq + h) * (int64_t)d;
                    for (int c = 0; c < d; c++)
                        qrow[c] = bf16_to_double(q[qo + c]);
                    double mx = -INFINITY;
                    for (int64_t j = 0; j < cnt; j++) {
                        const int64_t ko = ((base + first + j) * Hkv + hk) * (int64_t)d;
                        double acc = 0.0;
                        for (int c = 0; c < d; c++)
                            acc += qrow[c] * bf16_to_double(k[ko + c]);
                        w_p[j] = scale * acc;
                        mx = w_p[j] > mx ? w_p[j] : mx;
                    }
                    double sum = 0.0;
                    for (int64_t j = 0; j < cnt; j++) {
                        w_p[j] = exp(w_p[j] - mx);
                        sum += w_p[j];
                    }
                    const double *go = dout + qo;
                    double rowdot = 0.0;
                    for (int64_t j = 0; j < cnt; j++) {
                        w_p[j] /= sum;
                        const int64_t vo = ((base + first + j) * Hkv + hk) * (int64_t)d;
                        double acc = 0.0;
                        for (int c = 0; c < d; c++)
                            acc += go[c] * bf16_to_double(v[vo + c]);
                        w_dp[j] = acc;
                        rowdot += w_p[j] * acc;
                    }
                    for (int64_t j = 0; j < cnt; j++) {
                        const int64_t ko = ((base + first + j) * Hkv + hk) * (int64_t)d;
                        const double g_s = w_p[j] * (w_dp[j] - rowdot);
                        for (int c = 0; c < d; c++) {
                            dq[qo + c] += scale * g_s * bf16_to_double(k[ko + c]);
                            dk[ko + c] += scale * g_s * qrow[c];
                            dv[ko + c] += w_p[j] * go[c];
                        }
                    }
                }
            }
        }
        free(w_p);
        free(w_dp);
        free(qrow);
    }
}

/*
 * The layer backward (as oracle_logo_bwd, same chain rule, fp64) evaluated
 * only where a test samples it: dq and dq_g of the query tokens qrows[], dgate
 * of those tokens, and dk, dv, dk_g, dv_g of the key tokens keys[].  The
 * selection is given (tok2sel [N], rank or -1).  A key's gradient sums over
 * every row that sees it: rows j..j+w-1 of its sequence for the local branch,
 * every selected row at or after it for the global branch; those rows are
 * recomputed in full (forward, ContextNorm backward, softmax backward).
 * Outputs: dq_s, dqg_s [n_q][Hq][d], dgate_s [n_q], dk_s, dv_s, dkg_s, dvg_s
 * [n_k][Hkv][d] (overwritten; the global ones are the global-branch tensors'
 * gradients; a caller with aliased tensors adds the pairs).
 */
void oracle_logo_bwd_sample(const uint16_t *q, const uint16_t *k, const uint16_t *v,
                            const uint16_t *q_g, const uint16_t *k_g, const uint16_t *v_g,
                            const float *gate, const int32_t *cu, int B, int Hq, int Hkv, int d,
                            int window, double scale, const int32_t *tok2sel,
                            const float *gain_local, const float *gain_global, double eps,
                            const double *dout, int64_t n_q, const int32_t *qrows, int64_t n_k,
                            const int32_t *keys, double *dq_s, double *dqg_s, double *dgate_s,
                            double *dk_s, double *dv_s, double *dkg_s, double *dvg_s)
{
    const int64_t N = cu[B];
    const int G = Hq / Hkv;
    if (scale <= 0.0)
        scale = 1.0 / sqrt((double)d);
    if (!q_g)
        q_g = q;
    if (!k_g)
        k_g = k;
    if (!v_g)
        v_g = v;
    const int64_t row = (int64_t)Hq * d;
    /* sample index of each token as a query / as a key, or -1 */
    int64_t *qpos = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    int64_t *kpos = (int64_t *)malloc((size_t)(N > 0 ? N : 1) * sizeof(int64_t));
    for (int64_t t = 0; t < N; t++)
        qpos[t] = kpos[t] = -1;
    for (int64_t a = 0; a < n_q; a++)
        qpos[qrows[a]] = a;
    for (int64_t a = 0; a < n_k; a++)
        kpos[keys[a]] = a;
    memset(dq_s, 0, (size_t)n_q * row * sizeof(double));
    memset(dqg_s, 0, (size_t)n_q * row * sizeof(double));
    memset(dgate_s, 0, (size_t)n_q * sizeof(double));
    memset(dk_s, 0, (size_t)n_k * Hkv * d * sizeof(double));
    memset(dv_s, 0, (size_t)n_k * Hkv * d * sizeof(double));
    memset(dkg_s, 0, (size_t)n_k * Hkv * d * sizeof(double));
    memset(dvg_s, 0, (size_t)n_k * Hkv * d * sizeof(double));
    /* rows to recompute, per branch: the sampled queries and every row that
       sees a sampled key */
    char *need = (char *)calloc((size_t)(N > 0 ? N : 1) * 2, 1);
    for (int b = 0; b < B; b++) {
        const int64_t base = cu[b], T = (int64_t)cu[b + 1] - base;
        for (int64_t i = 0; i < T; i++) {
            const int64_t t = base + i;
            if (qpos[t] >= 0) {
                need[2 * t] = 1;
                need[2 * t + 1] = tok2sel[t] >= 0;
            }
            if (kpos[t] >= 0) {
                const int64_t hi = (window >= 1 && i + window < T) ? i + window : T;
                for (int64_t r = i; r < hi; r++)
                    need[2 * (base + r)] = 1;
                for (int64_t r = i; r < T; r++)
                    if (tok2sel[base + r] >= 0)
                        need[2 * (base + r) + 1] = 1;
            }
        }
    }
    int64_t max_T = 1;
    for (int b = 0; b < B; b++)
        if ((int64_t)cu[b + 1] - cu[b] > max_T)
            max_T = (int64_t)cu[b + 1] - cu[b];
    /* one job per (branch, KV head): its keys' and its heads' outputs only */
#pragma omp parallel for schedule(dynamic, 1)
    for (int job = 0; job < 2 * Hkv; job++) {
        const int br = job / Hkv, hk = job % Hkv;
        const uint16_t *Qm = br ? q_g : q, *Km = br ? k_g : k, *Vm = br ? v_g : v;
        const float *gmat = br ? gain_global : gain_local;
        double *wts = (double *)malloc((size_t)max_T * sizeof(double));
        double *gsc = (double *)malloc((size_t)max_T * sizeof(double));
        double *qv = (double *)malloc((size_t)d * sizeof(double));
        double *ov = (double *)malloc((size_t)d * sizeof(double));
        double *go = (double *)malloc((size_t)d * sizeof(double));
        for (int b = 0; b < B; b++) {
            const int64_t base = cu[b], T = (int64_t)cu[b + 1] - base;
            for (int64_t i = 0; i < T; i++) {
                const int64_t t = base + i;
                if (!need[2 * t + br])
                    continue;
                const int64_t j0 = (br == 0 && window >= 1 && i - window + 1 > 0) ? i - window + 1 : 0;
                const int64_t cnt = i - j0 + 1;
                const double pg = (double)gate[t];
                const int sel = tok2sel[t] >= 0;
                const double wb = br ? pg : (sel ? 1.0 - pg : 1.0);
                for (int h = hk * G; h < (hk + 1) * G; h++) {
                    const int64_t qo = (t * Hq + h) * (int64_t)d;
                    for (int c = 0; c < d; c++)
                        qv[c] = bf16_to_double(Qm[qo + c]);
                    double mx = -INFINITY;
                    for (int64_t j = 0; j < cnt; j++) {
                        const int64_t ko = ((base + j0 + j) * Hkv + hk) * (int64_t)d;
                        double acc = 0.0;
                        for (int c = 0; c < d; c++)
                            acc += qv[c] * bf16_to_double(Km[ko + c]);
                        wts[j] = scale * acc;
                        mx = wts[j] > mx ? wts[j] : mx;
                    }
                    double z = 0.0;
                    for (int64_t j = 0; j < cnt; j++) {
                        wts[j] = exp(wts[j] - mx);
                        z += wts[j];
                    }
                    for (int c = 0; c < d; c++)
                        ov[c] = 0.0;
                    for (int64_t j = 0; j < cnt; j++) {
                        wts[j] /= z;
                        const int64_t vo = ((base + j0 + j) * Hkv + hk) * (int64_t)d;
                        for (int c = 0; c < d; c++)
                            ov[c] += wts[j] * bf16_to_double(Vm[vo + c]);
                    }
                    double msq = 0.0;
                    for (int c = 0; c < d; c++)
                        msq += ov[c] * ov[c];
                    const double rms = sqrt(msq / (double)d + eps);
                    const double *gr = dout + qo;
                    double gsum = 0.0, yside = 0.0;
                    for (int c = 0; c < d; c++) {
                        const double gc = gmat ? (double)gmat[(int64_t)h * d + c] : 1.0;
                        gsum += gc * wb * gr[c] * ov[c];
                        yside += gr[c] * ov[c] / rms * gc;
                    }
                    if (br == 0 && qpos[t] >= 0 && sel) {
#pragma omp atomic
                        dgate_s[qpos[t]] -= yside;
                    }
                    if (br == 1 && qpos[t] >= 0) {
#pragma omp atomic
                        dgate_s[qpos[t]] += yside;
                    }
                    for (int c = 0; c < d; c++) {
                        const double gc = gmat ? (double)gmat[(int64_t)h * d + c] : 1.0;
                        go[c] = gc * wb * gr[c] / rms - ov[c] * gsum / ((double)d * rms * rms * rms);
                    }
                    double rdot = 0.0;
                    for (int64_t j = 0; j < cnt; j++) {
                        const int64_t vo = ((base + j0 + j) * Hkv + hk) * (int64_t)d;
                        double acc = 0.0;
                        for (int c = 0; c < d; c++)
                            acc += go[c] * bf16_to_double(Vm[vo + c]);
                        gsc[j] = acc;
                        rdot += wts[j] * acc;
                    }
                    double *dqr = qpos[t] >= 0 ? (br ? dqg_s : dq_s) + (qpos[t] * Hq + h) * (int64_t)d
                                               : NULL;
                    for (int64_t j = 0; j < cnt; j++) {
                        const double g_s = wts[j] * (gsc[j] - rdot);
                        const int64_t kt = base + j0 + j;
                        const int64_t ko = (kt * Hkv + hk) * (int64_t)d;
                        if (dqr)
                            for (int c = 0; c < d; c++)
                                dqr[c] += scale * g_s * bf16_to_double(Km[ko + c]);
                        if (kpos[kt] >= 0) {
                            double *dkr = (br ? dkg_s : dk_s) + (kpos[kt] * Hkv + hk) * (int64_t)d;
                            double *dvr = (br ? dvg_s : dv_s) + (kpos[kt] * Hkv + hk) * (int64_t)d;
                            for (int c = 0; c < d; c++) {
                                dkr[c] += scale * g_s * qv[c];
                                dvr[c] += wts[j] * go[c];
                            }
                        }
                    }
                }
            }
        }
        free(wts);
        free(gsc);
        free(qv);
        free(ov);
        free(go);
    }
    free(qpos);
    free(kpos);
    free(need);
}
