/*
 * logo.h -- C ABI of liblogo: the forward pass of one LoGo attention layer
 * (LoGo: Token-Level Dynamic Local-Global Attention) on AMD MI355X (gfx950).
 *
 * The layer (Sec. 3.2):
 *   O^L = SoftmaxAttn_w(Q, K, V)             for every token   (Eq. branch-attention)
 *   z_t = [p_t > b_th]                        per token, all heads share it
 *                                             (Eq. gate-routing, Eq. token-routing)
 *   O^G_I = SoftmaxAttn_inf(Q^G_I, K^G, V^G)  for selected tokens only, K/V dense
 *                                             (Eq. query-sparse-global)
 *   out_t = (1-p_t) Norm^L(O^L_t) + p_t Norm^G(O^G_t)  if z_t = 1
 *         = Norm^L(O^L_t)                               otherwise
 *                                             (Eq. contextnorm, Eq. output-fusion)
 *
 * Conventions for every entry point
 *   - Tensors are DEVICE pointers, row-major and contiguous, in packed varlen
 *     layout: Q [N][Hq][d], K and V [N][Hkv][d], gate [N], with sequence b
 *     occupying tokens cu_seqlens[b] .. cu_seqlens[b+1]-1.
 *   - bf16 tensors are passed as raw 16-bit patterns (logo_bf16).
 *   - Positions are 0-based within a sequence.  Key j is visible to query i
 *     iff j <= i (global) or i-w < j <= i (local: exactly min(i+1, w) keys,
 *     the query included; the paper's 1-based context {max(1,t-w+1)..t}).
 *   - GQA: query head h reads key/value head h / (Hq/Hkv).
 *   - A per-token array ([N] or [N][...]) may be NULL when N = 0 (every
 *     sequence empty); per-sequence arrays ([B+1], [B]) are still required
 *     and are written (cu_sel all zeros).
 *   - The caller owns every buffer.  The library never allocates or frees
 *     device memory, keeps no pointer after a call returns, and never
 *     synchronises: every call only enqueues work on `stream` (NULL = the
 *     default stream) and returns.  Device-side faults surface at the
 *     caller's next synchronisation.
 *   - Arguments are validated on the host before anything is enqueued: on
 *     any error status nothing has been launched.  No C++ exception crosses
 *     this interface.
 *   - Calls are thread-safe.  Two calls that share output or workspace
 *     buffers must be ordered by the caller (same stream or events).
 */
#ifndef LOGO_H
#define LOGO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t logo_bf16;      /* raw bfloat16 bits                              */
typedef void *logo_stream;       /* a hipStream_t; NULL selects the default stream */

typedef enum {
    LOGO_OK = 0,
    LOGO_ERR_NULL = 1,        /* a required pointer is NULL                        */
    LOGO_ERR_SHAPE = 2,       /* inconsistent sizes (heads, tokens, capacity)      */
    LOGO_ERR_UNSUPPORTED = 3, /* a valid but unimplemented case (head_dim)         */
    LOGO_ERR_ARG = 4,         /* an argument out of its domain (ratio, window...)  */
    LOGO_ERR_WORKSPACE = 5,   /* workspace missing, misaligned or too small        */
    LOGO_ERR_HIP = 6,         /* the HIP runtime refused a launch                  */
    LOGO_ERR_SCRATCH_LIMIT = 7 /* logo_decode_noalloc: the step needs more scratch
                                  than LOGO_NOALLOC_SCRATCH_BYTES                  */
} logo_status;

typedef enum {
    LOGO_SEL_THRESHOLD = 0,   /* one scalar threshold b_th for every sequence      */
    LOGO_SEL_RATIO = 1,       /* per-sequence threshold from a target ratio rho    */
    LOGO_SEL_THRESHOLD_DEVICE = 2  /* b_th read on the device from thr_out[0]      */
} logo_sel_mode;

/* Which entry point logo_workspace_bytes() sizes. */
typedef enum {
    LOGO_ENTRY_SELECT = 0,
    LOGO_ENTRY_LOCAL = 1,
    LOGO_ENTRY_GLOBAL = 2,
    LOGO_ENTRY_COMBINE = 3,
    LOGO_ENTRY_FWD = 4,
    LOGO_ENTRY_DENSE = 5,
    LOGO_ENTRY_DECODE = 6,
    LOGO_ENTRY_FWD_TRAIN = 7,
    LOGO_ENTRY_BWD = 8,
    LOGO_ENTRY_DENSE_BWD = 9,
    LOGO_ENTRY_GLOBAL_BWD = 10,
    LOGO_ENTRY_FWD_QPHI = 11
} logo_entry;

/* Problem description (a host struct; only cu_seqlens is a device pointer). */
typedef struct {
    int32_t num_seqs;               /* B >= 1                                            */
    int32_t total_tokens;           /* N = cu_seqlens[B] >= 0                            */
    int32_t max_seqlen;             /* >= every T_b; bounds the launch grids             */
    const int32_t *cu_seqlens;      /* device [B+1]: 0 = cu[0] <= cu[1] <= ... = N       */
    const int32_t *cu_seqlens_host; /* optional host copy of cu_seqlens (NULL allowed);
                                       when given it is checked against N / max_seqlen
                                       and sizes the ratio-mode selection bound          */
    int32_t num_q_heads;            /* Hq >= 1                                           */
    int32_t num_kv_heads;           /* Hkv >= 1, Hq % Hkv == 0                            */
    int32_t head_dim;               /* d in {64, 128}                                    */
    int32_t window;                 /* w >= 1 (local span, Sec. 3.1); w >= max_seqlen
                                       makes the local branch full causal attention      */
    float softmax_scale;            /* <= 0 selects 1/sqrt(d) (Eq. attention)            */
} logo_problem;

/*
 * logo_select -- hard routing and stream compaction (Eq. gate-routing;
 * Sec. 3.3 and App. B: selected queries in ascending order with their
 * original positions and compacted cu_seqlens).
 *
 *   gate       device [N] fp32: the preference p_t (already through the
 *              sigmoid of Eq. gate-routing).  A NaN gate is never selected.
 *   mode       LOGO_SEL_THRESHOLD: thr_b = threshold for every b (NaN is
 *              rejected; -inf selects every non-NaN gate, +inf none).
 *              LOGO_SEL_RATIO: k_b = floor(ratio * T_b) in IEEE double,
 *              thr_b = -inf if k_b == T_b, else the (k_b+1)-th largest gate
 *              of sequence b (an input value, -0 reported as +0).  Gates
 *              must be finite in this mode.  0 <= ratio <= 1.
 *              LOGO_SEL_THRESHOLD_DEVICE: thr_b = b_th for every b, where
 *              b_th is read on the device from thr_out[0] when the
 *              selection runs (the threshold the budget controller keeps on
 *              the device, see logo_budget_update); thr_out must not be
 *              NULL and every thr_out[b] is set to b_th.  A NaN b_th
 *              selects nothing.
 *   Selection: z_t = gate[t] > thr_b, strict, compared in fp32.
 *   sel_idx    device [sel_capacity] int32: packed token indices of the
 *              selected tokens, strictly ascending (sequence-major).
 *   cu_sel     device [B+1] int32: cu_sel[b] = number of selected tokens in
 *              sequences 0..b-1; cu_sel[B] = n_sel (the realized ratio of
 *              Eq. realized-ratio is n_sel / N).
 *   tok2sel    device [N] int32 or NULL: rank of token t in sel_idx, or -1.
 *   thr_out    device [B] fp32 or NULL: the thresholds used.
 *   Capacity:  in ratio mode sel_capacity must be >= sum_b floor(ratio*T_b)
 *              (checked when cu_seqlens_host is given, else it must be >= N).
 *              In the threshold modes any sel_capacity >= 0 is accepted; if more
 *              tokens pass, sel_idx keeps the first sel_capacity of them,
 *              tok2sel marks the rest -1, and cu_sel still counts all of
 *              them, so cu_sel[B] > sel_capacity reports the overflow.
 *   ws         device workspace of >= logo_workspace_bytes(p, LOGO_ENTRY_SELECT, 0)
 *              bytes, 256-byte aligned.
 */
logo_status logo_select(const logo_problem *p, const float *gate, logo_sel_mode mode,
                        float threshold, double ratio, int32_t *sel_idx, int32_t sel_capacity,
                        int32_t *cu_sel, int32_t *tok2sel, float *thr_out, void *ws,
                        size_t ws_bytes, logo_stream stream);

/*
 * logo_local_attn -- the local branch O^L = SoftmaxAttn_w(Q, K, V) for every
 * token and query head (Eq. branch-attention; local context of Sec. 3.1).
 *   q [N][Hq][d], k/v [N][Hkv][d] bf16; o_local [N][Hq][d] fp32 (raw
 *   attention output, not normalised).  No workspace.
 */
logo_status logo_local_attn(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                            const logo_bf16 *v, float *o_local, logo_stream stream);

/*
 * logo_global_attn_sparse_q -- the query-sparse global branch
 * O^G_I = SoftmaxAttn_inf(Q_I, K, V) (Eq. query-sparse-global): full causal
 * attention for the selected rows only, keys and values dense.
 *   sel_idx/cu_sel as produced by logo_select (only the first
 *   min(cu_sel[B], sel_capacity) rows are computed).
 *   o_global [sel_capacity][Hq][d] fp32, compact in rank order (row r is
 *   token sel_idx[r]); rows at or past n_sel are left untouched.
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_GLOBAL, sel_capacity) bytes,
 *   256-byte aligned (tile table and work-queue counters).
 */
logo_status logo_global_attn_sparse_q(const logo_problem *p, const logo_bf16 *q,
                                      const logo_bf16 *k, const logo_bf16 *v,
                                      const int32_t *sel_idx, const int32_t *cu_sel,
                                      int32_t sel_capacity, float *o_global, void *ws,
                                      size_t ws_bytes, logo_stream stream);

/*
 * logo_combine -- ContextNorm and output fusion, scattered back to token
 * order (Eq. contextnorm, Eq. output-fusion).
 *   Norm(o) = o / sqrt(mean_c o_c^2 + eps) * g[h][c] per (token, head).
 *   out_t = (1-p_t) Norm^L(O^L_t) + p_t Norm^G(O^G_{tok2sel[t]}) if tok2sel[t] >= 0,
 *         = Norm^L(O^L_t) otherwise;  with apply_norm == 0 Norm is the identity.
 *   o_local [N][Hq][d] fp32, o_global [*][Hq][d] fp32 compact (may be NULL
 *   when no token is selected), gate [N] fp32, tok2sel [N] int32,
 *   gain_local / gain_global [Hq][d] fp32 or NULL (= 1), eps >= 0,
 *   out [N][Hq][d] bf16 (round to nearest even, once).  No workspace.
 */
logo_status logo_combine(const logo_problem *p, const float *o_local, const float *o_global,
                         const float *gate, const int32_t *tok2sel, const float *gain_local,
                         const float *gain_global, float eps, int apply_norm, logo_bf16 *out,
                         logo_stream stream);

/*
 * logo_attn_fwd -- the whole layer: select, local branch, query-sparse
 * global branch, ContextNorm and fusion, in one stream-ordered sequence with
 * no host synchronisation (Sec. 3.2-3.3).  ContextNorm and the fusion run in
 * the epilogues of the attention kernels: the local branch writes
 * Norm^L(O^L) (bf16) for unselected tokens and keeps (1-p) Norm^L(O^L) (fp32,
 * workspace) for selected ones.  When Hq / Hkv is a multiple of 4, or 1,
 * both branches run in one persistent launch (global work first, local work
 * filling in behind it) that keeps p Norm^G(O^G) (fp32, workspace) too, and a
 * short pass sums the two into the selected rows of `out`; otherwise the
 * global branch's kernel, launched after the local one, completes them.
 *   q_g/k_g/v_g: global-branch tensors of the same shapes as q/k/v, or NULL
 *   to use q/k/v (the identity branch transform of Eq. branch-transform).
 *   gain_local / gain_global [Hq][d] fp32 or NULL (= 1); eps >= 0.
 *   sel_idx [sel_capacity], cu_sel [B+1], tok2sel [N], thr_out [B]: outputs
 *   as for logo_select; each may be NULL, in which case it lives in the
 *   workspace.  sel_capacity bounds the selection as for logo_select; with
 *   sel_idx NULL, 0 selects the mode's bound (ratio mode: the ratio bound,
 *   threshold mode: N).  In threshold mode, tokens past the capacity are
 *   fused as unselected (cu_sel[B] > sel_capacity reports it).
 *   out [N][Hq][d] bf16.
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_FWD, sel_capacity) bytes,
 *   256-byte aligned (selection scratch, tile table, queue counters and the
 *   compact fp32 buffers of the selected rows).
 */
logo_status logo_attn_fwd(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                          const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                          const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                          float threshold, double ratio, const float *gain_local,
                          const float *gain_global, float eps, logo_bf16 *out,
                          int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                          int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                          logo_stream stream);

/*
 * logo_attn_fwd_profiled -- logo_attn_fwd that additionally records five
 * caller-created HIP events (hipEvent_t, passed as void*) on `stream`:
 *   events[0] before the selection kernel(s), events[1] after them,
 *   events[2] after the local branch (which also applies Norm^L and writes
 *   the unselected rows of `out`), events[3] after the tile plan of the
 *   global branch, events[4] after the query-sparse attention kernel (which
 *   applies Norm^G and the fusion for the selected rows).  Elapsed times
 *   between consecutive events are the stage times (select, local, plan,
 *   global).  With the one-launch layer (Hq / Hkv a multiple of 4, or 1) events[2]
 *   and events[3] both follow that launch and events[4] the selected rows'
 *   sum: the stages are (select, layer, -, sum).  `events` must not be NULL;
 *   everything else is as for logo_attn_fwd.
 */
logo_status logo_attn_fwd_profiled(const logo_problem *p, const logo_bf16 *q,
                                   const logo_bf16 *k, const logo_bf16 *v,
                                   const logo_bf16 *q_g, const logo_bf16 *k_g,
                                   const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                   float threshold, double ratio, const float *gain_local,
                                   const float *gain_global, float eps, logo_bf16 *out,
                                   int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                                   int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                                   logo_stream stream, void *const *events);

/*
 * logo_attn_fwd_train -- the layer forward for training: logo_attn_fwd (the
 * same launches and output) whose attention epilogues also keep what
 * logo_attn_bwd needs.  The selection outputs are required here (they are the saved
 * routing decision of Sec. 3.3, held fixed by the backward pass).
 *   sel_idx [sel_capacity], cu_sel [B+1], tok2sel [N]: as for logo_select
 *   (sel_idx may be NULL only when sel_capacity is 0); thr_out [B] or NULL.
 *   o_local  [N][Hq][d] fp32: raw O^L (Eq. branch-attention, local context).
 *   lse_local [Hq][N] fp32: per (head, token) the base-2 log-sum-exp of the
 *            scaled scores, log2 sum_j 2^(c s_j) with c = softmax_scale *
 *            log2(e) over the keys of the row's window.
 *   o_global [sel_capacity][Hq][d] fp32, lse_global [Hq][sel_capacity]:
 *            the same for the selected rows of the global branch (Eq.
 *            query-sparse-global), compact in rank order.
 *   Everything else as for logo_attn_fwd.
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_FWD_TRAIN, sel_capacity) bytes,
 *   256-byte aligned.
 */
logo_status logo_attn_fwd_train(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                                const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                                const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                float threshold, double ratio, const float *gain_local,
                                const float *gain_global, float eps, logo_bf16 *out,
                                int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                                int32_t *tok2sel, float *thr_out, float *o_local,
                                float *lse_local, float *o_global, float *lse_global, void *ws,
                                size_t ws_bytes, logo_stream stream);

/*
 * logo_attn_bwd -- gradients of the layer given dL/d out, with the routing
 * decision z held fixed (it is a hard threshold, Eq. gate-routing; the
 * gate receives its gradient through the fusion weight p_t of Eq.
 * output-fusion).  The chain rule runs through Eq. output-fusion, Eq.
 * contextnorm and the two attentions (Eq. branch-attention with the local
 * window; Eq. query-sparse-global, whose backward visits the selected rows
 * only: App. B, backward traversal).
 *   Inputs: the forward's tensors and gains, and the saved outputs of
 *   logo_attn_fwd_train (sel_idx, sel_capacity, cu_sel, tok2sel, o_local,
 *   lse_local, o_global, lse_global); dout [N][Hq][d] bf16 = dL/d out.
 *   Outputs (fp32, row-major like the inputs, overwritten):
 *     dq [N][Hq][d], dk, dv [N][Hkv][d]: gradients of the local-branch
 *       tensors.  Where a global-branch tensor is NULL (it aliases the local
 *       one), its gradient is added in here and its d*_g must be NULL.
 *     dq_g, dk_g, dv_g: gradients of q_g, k_g, v_g when those are given
 *       (each must be non-NULL exactly when its tensor is); rows of dq_g of
 *       unselected tokens are zero.
 *     dgate [N] or NULL: dL/dp_t (zero for unselected tokens).
 *     dgain_local, dgain_global [Hq][d] or NULL: gain gradients (the gains
 *       themselves may be NULL, meaning 1).
 *   Numerics: P and dS are recomputed from lse and rounded to bf16 for the
 *   matrix products (fp32 accumulation); dO of each branch is rounded to
 *   bf16 once.
 *   Limits: Hq * d / 8 must be <= 256 or 512 or 1024 (Hq * d <= 8192).
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_BWD, sel_capacity) bytes,
 *   256-byte aligned.
 */
logo_status logo_attn_bwd(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                          const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                          const logo_bf16 *v_g, const float *gate, const float *gain_local,
                          const float *gain_global, float eps, const int32_t *sel_idx,
                          int32_t sel_capacity, const int32_t *cu_sel, const int32_t *tok2sel,
                          const float *o_local, const float *lse_local, const float *o_global,
                          const float *lse_global, const logo_bf16 *dout, float *dq, float *dk,
                          float *dv, float *dq_g, float *dk_g, float *dv_g, float *dgate,
                          float *dgain_local, float *dgain_global, void *ws, size_t ws_bytes,
                          logo_stream stream);

/*
 * logo_dense_causal_attn -- dense causal softmax attention for every token
 * (Eq. attention with the global context), bf16 output [N][Hq][d].  This is
 * the dense baseline the query-sparse layer is measured against; it uses
 * the same kernel template as the global branch.  No workspace.
 */
logo_status logo_dense_causal_attn(const logo_problem *p, const logo_bf16 *q,
                                   const logo_bf16 *k, const logo_bf16 *v, logo_bf16 *out,
                                   logo_stream stream);

/*
 * logo_global_attn_sparse_q_fwd_train -- logo_global_attn_sparse_q that also
 * keeps lse_global [Hq][sel_capacity] fp32: per (head, selected rank) the
 * base-2 log-sum-exp of the scaled scores over keys 0..pos (Eq.
 * query-sparse-global).  Arguments and workspace otherwise as for
 * logo_global_attn_sparse_q (LOGO_ENTRY_GLOBAL).
 */
logo_status logo_global_attn_sparse_q_fwd_train(const logo_problem *p, const logo_bf16 *q,
                                                const logo_bf16 *k, const logo_bf16 *v,
                                                const int32_t *sel_idx, const int32_t *cu_sel,
                                                int32_t sel_capacity, float *o_global,
                                                float *lse_global, void *ws, size_t ws_bytes,
                                                logo_stream stream);

/*
 * logo_global_attn_sparse_q_bwd -- gradients of the query-sparse global
 * attention alone (Eq. query-sparse-global; App. B, backward traversal):
 * the loss depends on the selected rows' outputs only.
 *   sel_idx, cu_sel, sel_capacity: as for logo_global_attn_sparse_q;
 *   o_global [sel_capacity][Hq][d] fp32 and lse_global [Hq][sel_capacity]
 *   from logo_global_attn_sparse_q_fwd_train; dout [sel_capacity][Hq][d]
 *   bf16 = dL/d o_global (compact, rank order; rows at or past n_sel are
 *   not read).
 *   dq [N][Hq][d] fp32: rows of selected tokens, zero elsewhere; dk, dv
 *   [N][Hkv][d] fp32 (every key).  All overwritten.
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_GLOBAL_BWD, sel_capacity) bytes
 *   (compact Q rows and the row sums dout . o), 256-byte aligned.
 */
logo_status logo_global_attn_sparse_q_bwd(const logo_problem *p, const logo_bf16 *q,
                                          const logo_bf16 *k, const logo_bf16 *v,
                                          const int32_t *sel_idx, const int32_t *cu_sel,
                                          int32_t sel_capacity, const float *o_global,
                                          const float *lse_global, const logo_bf16 *dout,
                                          float *dq, float *dk, float *dv, void *ws,
                                          size_t ws_bytes, logo_stream stream);

/*
 * logo_dense_causal_attn_fwd_train -- logo_dense_causal_attn that also keeps
 * lse [Hq][N] fp32: per (head, token) the base-2 log-sum-exp of the scaled
 * scores over keys 0..i, log2 sum_j 2^(c s_j), c = softmax_scale * log2(e).
 * lse may be NULL (then this is logo_dense_causal_attn).  No workspace.
 */
logo_status logo_dense_causal_attn_fwd_train(const logo_problem *p, const logo_bf16 *q,
                                             const logo_bf16 *k, const logo_bf16 *v,
                                             logo_bf16 *out, float *lse, logo_stream stream);

/*
 * logo_dense_causal_attn_bwd -- gradients of dense causal softmax attention
 * (Eq. attention with the global context): the dense baseline's backward.
 *   out [N][Hq][d] bf16 and lse [Hq][N] from logo_dense_causal_attn_fwd_train,
 *   dout [N][Hq][d] bf16 = dL/d out; dq [N][Hq][d], dk, dv [N][Hkv][d] fp32
 *   (overwritten).  P and dS are recomputed from lse and rounded to bf16 for
 *   the matrix products (fp32 accumulation), as in logo_attn_bwd.
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_DENSE_BWD, 0) bytes (the row
 *   sums dout . out), 256-byte aligned.
 */
logo_status logo_dense_causal_attn_bwd(const logo_problem *p, const logo_bf16 *q,
                                       const logo_bf16 *k, const logo_bf16 *v,
                                       const logo_bf16 *out, const float *lse,
                                       const logo_bf16 *dout, float *dq, float *dk, float *dv,
                                       void *ws, size_t ws_bytes, logo_stream stream);

/*
 * logo_decode -- one autoregressive decoding step of the layer (Sec. 3.3 and
 * App. B, Autoregressive Decoding): each of the B sequences appends one
 * token.  Its query attends to the last min(L_b, w) cached keys (local
 * branch); when its gate passes the threshold (z = p > b_th, strict, fp32,
 * Eq. gate-routing) its global query also attends to all L_b cached global
 * keys; the outputs are ContextNorm-ed and fused as in logo_attn_fwd (Eqs.
 * contextnorm, output-fusion).  Only selected tokens get global work: the
 * selected sequences are compacted first, so an unselected token reads one
 * window of its cache.
 *   p          cu_seqlens = the caches: sequence b's cache is rows
 *              cu[b] .. cu[b+1]-1 of k / v, L_b = cu[b+1] - cu[b] >= 1, and
 *              its last row is the new token's own key and value (appended
 *              by the caller).  num_seqs = B; total_tokens = cu[B];
 *              max_seqlen >= every L_b; heads, head_dim, window, scale as in
 *              the layer.  With cu_seqlens_host given, L_b = 0 is rejected
 *              (LOGO_ERR_SHAPE); without it such a sequence outputs zeros.
 *   q          device [B][Hq][d] bf16: the new tokens' queries.
 *   k, v       device [N][Hkv][d] bf16: the caches (the prefill layout).
 *   q_g, k_g, v_g  the global branch's tensors, same shapes (NULL = the
 *              local ones, the identity branch transform).
 *   gate       device [B] fp32: p of the new tokens (NaN is never selected).
 *   mode       LOGO_SEL_THRESHOLD: b_th = threshold (NaN rejected);
 *              LOGO_SEL_THRESHOLD_DEVICE: b_th = thr_dev[0] read on the
 *              device (thr_dev must not be NULL); LOGO_SEL_RATIO is rejected
 *              (LOGO_ERR_ARG): decoding routes with the layer's threshold.
 *   gain_local, gain_global, eps   ContextNorm, as in logo_combine.
 *   out        device [B][Hq][d] bf16.
 *   active     device [B] int32 or NULL: the selected sequences, ascending,
 *              in its first n_active entries.
 *   n_active   device int32 or NULL: the number of selected sequences.
 *   ws         >= logo_workspace_bytes(p, LOGO_ENTRY_DECODE, 0) bytes,
 *              256-byte aligned (partial results of the key chunks).
 * Asynchronous on `stream`; nothing is enqueued on error.
 */
logo_status logo_decode(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                        const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                        const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                        float threshold, const float *thr_dev, const float *gain_local,
                        const float *gain_global, float eps, logo_bf16 *out, int32_t *active,
                        int32_t *n_active, void *ws, size_t ws_bytes, logo_stream stream);

/*
 * logo_decode_noalloc -- logo_decode for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same decoding step with the same arguments and
 * results, minus the workspace.  Its scratch memory (the partial results of
 * the key chunks, and the selected list and count when active / n_active
 * are NULL) is a fixed device array of LOGO_NOALLOC_SCRATCH_BYTES inside the
 * library, which every GPU the library runs on holds from the module's load
 * until the process ends.  The call allocates and frees nothing; the first
 * call on a device looks up the array's address there once.
 *   Errors: those of logo_decode, and LOGO_ERR_SCRATCH_LIMIT (nothing
 *   enqueued) when logo_workspace_bytes(p, LOGO_ENTRY_DECODE, 0) exceeds
 *   LOGO_NOALLOC_SCRATCH_BYTES (64 MiB; 32 caches of 32K tokens with 32
 *   query heads and 8 KV heads of d = 128 need 35 MB).
 *   Concurrency: every call on one GPU shares that GPU's array, which keeps
 *   the last call's contents (nothing in it must start at zero).  Calls that
 *   overlap on one GPU -- on different streams, or from different threads
 *   without ordering -- race on it; order them on one stream.
 */
#define LOGO_NOALLOC_SCRATCH_BYTES (64u << 20)
logo_status logo_decode_noalloc(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                                const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                                const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                float threshold, const float *thr_dev, const float *gain_local,
                                const float *gain_global, float eps, logo_bf16 *out,
                                int32_t *active, int32_t *n_active, logo_stream stream);

/*
 * logo_gate_proj -- the gate of Eq. gate-routing (Sec. 3.2):
 * gate_out[t] = sigmoid(x[t] . w_g) for t < n_tokens, in fp32 (bf16 products
 * accumulated in fp32).  The result is the `gate` input of logo_select /
 * logo_attn_fwd / logo_decode (both the routing preference and the fusion
 * weight).
 *   x          device [n_tokens][d_model] bf16, 16-byte aligned.
 *   w_g        device [d_model] bf16, 16-byte aligned.
 *   d_model    a multiple of 8 (LOGO_ERR_UNSUPPORTED otherwise), >= 8.
 *   gate_out   device [n_tokens] fp32.
 * Asynchronous on `stream`; nothing is enqueued on error.
 */
logo_status logo_gate_proj(int64_t n_tokens, int32_t d_model, const logo_bf16 *x,
                           const logo_bf16 *w_g, float *gate_out, logo_stream stream);

/* Branch transform kinds of Eq. branch-transform. */
typedef enum {
    LOGO_PHI_LP = 0,   /* linear projection U A_h, A_h a d x d matrix per head */
    LOGO_PHI_SO = 1    /* scale and offset U * s_h + b_h                       */
} logo_phi_kind;

/*
 * logo_branch_transform -- the global branch's representation from the local
 * one, per head (Sec. 3.2, Eq. branch-transform): u_g[t][h] = u[t][h] A[h]
 * (LP) or u[t][h] * s[h] + b[h] (SO), fp32 arithmetic, one bf16 rounding.
 * Identity parameters (A = I; s = 1, b = 0) reproduce u exactly.
 *   n_tokens, num_heads, head_dim   u and u_g are [n_tokens][H][d] bf16,
 *              d in {64, 128}, 16-byte aligned; u_g must not overlap u.
 *   kind       LOGO_PHI_LP (A: device [H][d][d] bf16, row c of A[h] maps
 *              channel c to the output channels) or LOGO_PHI_SO (s, b:
 *              device [H][d] fp32).
 *   rows       device [n_rows] int32 token indices (each < n_tokens) or NULL
 *              for every token (then n_rows must be n_tokens); only the
 *              listed rows of u_g are written -- e.g. the selected queries
 *              (sel_idx) of the query-sparse global branch.
 *   n_rows_dev device int32 or NULL: the number of valid entries of rows when
 *              it is known only on the device (e.g. &cu_sel[B]); at most
 *              n_rows are used.
 * Asynchronous on `stream`; nothing is enqueued on error.
 */
logo_status logo_branch_transform(int64_t n_tokens, int32_t num_heads, int32_t head_dim,
                                  logo_phi_kind kind, const logo_bf16 *u, const logo_bf16 *A,
                                  const float *s, const float *b, const int32_t *rows,
                                  int64_t n_rows, const int32_t *n_rows_dev, logo_bf16 *u_g,
                                  logo_stream stream);

/*
 * logo_attn_fwd_qphi -- logo_attn_fwd whose global-branch queries are the
 * lightweight branch transform of the local ones (Sec. 3.2, Eq.
 * branch-transform), applied by the query-sparse attention kernel to the
 * selected rows only, as it loads them: q^G = q A_h (LP: bf16 products
 * accumulated in fp32) or q * s_h + b_h (SO: fp32), one bf16 rounding -- the
 * values logo_branch_transform writes (up to the fp32 summation order of
 * LP).  No Q^G tensor is written or read.
 *   q_phi      LOGO_PHI_LP (A: device [Hq][d][d] bf16, row c of A[h] maps
 *              channel c to the output channels; s, b ignored) or
 *              LOGO_PHI_SO (s, b: device [Hq][d] fp32; A ignored); anything
 *              else is LOGO_ERR_ARG, a missing operand LOGO_ERR_NULL.
 *   k_g, v_g   the global branch's keys / values (e.g. from
 *              logo_branch_transform, which runs once per token for them), or
 *              NULL for k / v.
 *   Everything else as for logo_attn_fwd (there is no q_g argument).
 *   ws >= logo_workspace_bytes(p, LOGO_ENTRY_FWD_QPHI, sel_capacity) bytes,
 *   256-byte aligned: LOGO_ENTRY_FWD's workspace plus, for LP, a permuted
 *   copy of A (2 Hq d^2 bytes) that the local-branch launch writes for the
 *   global one.
 */
logo_status logo_attn_fwd_qphi(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                               const logo_bf16 *v, logo_phi_kind q_phi, const logo_bf16 *A,
                               const float *s, const float *b, const logo_bf16 *k_g,
                               const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                               float threshold, double ratio, const float *gain_local,
                               const float *gain_global, float eps, logo_bf16 *out,
                               int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                               int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                               logo_stream stream);

/*
 * logo_budget_update -- one step of the global-budget controller
 * (Sec. 3.2, Eq. threshold-update) on the device, without a host sync:
 *   F    = cu_sel[B] / N, the realized global ratio of the last selection
 *          (Sec. 3.1, Eq. realized-ratio; N = total_tokens, the valid tokens)
 *   b_th <- b_th + gamma * sign(F - rho), sign(0) = 0
 * F and rho are compared in double; the update is one fp32 add of +-gamma.
 * With N == 0 nothing changes.
 *   cu_sel    device [B+1] int32, as written by logo_select / logo_attn_fwd
 *   rho       target ratio, 0 <= rho <= 1
 *   gamma     update rate, finite and >= 0
 *   b_th      device fp32 scalar, updated in place (the value a
 *             LOGO_SEL_THRESHOLD_DEVICE selection reads from thr_out[0])
 *   realized  device fp32 scalar or NULL: receives F rounded to fp32
 * Errors: LOGO_ERR_NULL (problem, cu_sel or b_th NULL), LOGO_ERR_ARG (rho or
 * gamma out of range), LOGO_ERR_HIP.  One single-thread launch.
 */
logo_status logo_budget_update(const logo_problem *p, const int32_t *cu_sel, double rho,
                               float gamma, float *b_th, float *realized, logo_stream stream);

/*
 * Starting threshold of the progressive-masking (P-mask) schedule (Sec. 3.2):
 * b_th,0 = 0.5 - gamma * pmask_steps (double, rounded once to fp32), so that
 * pmask_steps controller steps of +gamma -- every token is selected while
 * b_th is below every gate p in (0,1), so F = 1 > rho -- bring b_th to the
 * initial gate centre 0.5.  Host function, no device work.
 */
float logo_pmask_initial_threshold(float gamma, int64_t pmask_steps);

/*
 * Workspace size in bytes for `entry` (a logo_entry value); sel_capacity is
 * used by LOGO_ENTRY_GLOBAL and LOGO_ENTRY_FWD (0 = worst case of the
 * problem: N).  Returns 0 for an invalid problem.
 */
size_t logo_workspace_bytes(const logo_problem *p, int entry, int32_t sel_capacity);

/*
 * logo_attn_fwd_launches -- how logo_attn_fwd (and logo_attn_fwd_qphi /
 * _profiled) runs the two attention branches of problem p when the
 * selection capacity is nonzero: 1 = one persistent launch for both
 * (Hq / Hkv a multiple of 4, or 1, and enough local work per workgroup to
 * cover building the global work table inside the launch), 2 = the local
 * launch, then the global one.  Host-only (no GPU work; queries the current
 * device's CU count once).  The environment variable LOGO_FWD_LAUNCHES=1 or 2
 * forces one or the other where both are possible.  Returns -1 for an
 * invalid problem or a HIP error.
 */
int logo_attn_fwd_launches(const logo_problem *p);

/* Selection bound used by the ratio-mode capacity check: sum_b floor(ratio*T_b)
 * computed from cu_seqlens_host, or N when that is NULL.  -1 on bad input. */
int64_t logo_ratio_capacity(const logo_problem *p, double ratio);

/* Static string naming a status. */
const char *logo_status_str(logo_status s);

/* Library version, "MAJOR.MINOR.PATCH". */
const char *logo_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LOGO_H */
