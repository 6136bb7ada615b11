// logo_internal.h -- launch plans and kernel launchers shared by the host
// entry points (logo_api.cpp) and the HIP kernel files.  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace logo {

// ---------------------------------------------------------------------------
// Attention tiling.  A workgroup has W waves of 64 lanes; each wave owns 32
// query rows of one query head, and all W waves read the same key/value head,
// so a K/V tile staged in LDS serves 32 W rows.  With GQA group size G the
// waves cover HPW = gcd(G, 4) heads x (W / HPW) blocks of 32 tokens: a tile
// is TPW = 32 W / HPW tokens x HPW heads.  The global and dense modes use
// W = 8 (one workgroup per CU: each staged tile serves 256 rows), the global
// mode W = 4 when G = 1 (see global_waves).  The local
// branch uses W = 8 when HPW = 4 (64 tokens: with 64-key tiles both 32-token
// blocks need the same KV tiles of a window that is a multiple of 64) and
// W = 4 otherwise (two workgroups per CU; a wider token span would leave
// waves idle at the window's ends); its workgroups are persistent and
// prefetch the next item while they finish the current one.
// ---------------------------------------------------------------------------
constexpr int kRowsPerWave = 32;
constexpr int kBlockN = 64;   // keys per K/V tile
constexpr int kQueues = 8;    // one work queue per XCD
constexpr int kWavesLocal = 4;
constexpr int kWavesGlobal = 8;

enum AttnMode { kModeLocal = 0, kModeGlobal = 1, kModeDense = 2 };

// Waves of a local-branch workgroup for Hq / Hkv query / KV heads.
inline int local_waves(int hq, int hkv) { return (hq / hkv) % 4 == 0 ? 8 : kWavesLocal; }
// Waves of a global-branch workgroup: 4 (two workgroups per CU, 128 rows
// of one head per tile) when every KV head has a single query head, else 8.
// A 256-row tile of selected rows spans ~256 / ratio positions, so its causal
// band is long, and with one head per group there are few such tiles.
inline int global_waves(int hq, int hkv) { return hq == hkv ? kWavesLocal : kWavesGlobal; }

struct TilePlan {
    int hpw;      // heads per workgroup (1, 2 or 4)
    int tpw;      // tokens per workgroup
    int n_hg;     // head groups = Hq / hpw
};

inline TilePlan make_tile_plan(int hq, int hkv, int waves) {
    const int g = hq / hkv;
    TilePlan t;
    t.hpw = (g % 4 == 0) ? 4 : (g % 2 == 0) ? 2 : 1;
    t.tpw = kRowsPerWave * (waves / t.hpw);
    t.n_hg = hq / t.hpw;
    return t;
}

// One work entry of the query-sparse global branch (written on the device):
// a tile of selected rows and the range of 64-key KV blocks it covers.  A
// long tile is split into nsplit entries over consecutive KV ranges; each
// writes a partial (O, m, l) and the one that finishes last merges them in
// split order (attention.hip).
struct alignas(16) SparseTile {
    int32_t first;     // index of the tile's first row in sel_idx
    int32_t nrows;     // rows in the tile (1..tpw)
    int32_t seq;       // sequence b
    int32_t pos_max;   // position of the tile's last row
    int32_t kb_begin;  // first KV block of this entry
    int32_t kb_end;    // last KV block of this entry (inclusive)
    int32_t split;     // 0 .. nsplit-1
    int32_t nsplit;    // 1 = whole tile
    int32_t sid;       // first partial slot of a split tile (also its counter), -1 if whole
    int32_t pad[3];
};
constexpr int kMaxSplit = 4;          // KV ranges per tile at most
constexpr int kSplitDiv = 1;          // split tiles longer than 1/kSplitDiv of a workgroup's mean load
constexpr int kMinSplitBlocks = 4;    // never split tiles of 4 KV blocks or fewer
constexpr int kSplitGridRef = 512;    // persistent workgroups the split slots are sized for

// Partial result of one split entry for one head group, lane-major: the
// lanes of the global mode's waves each hold d/2 fp32 outputs, then m (exp2
// domain) and l of every lane.
__host__ __device__ constexpr size_t partial_floats(int head_dim) {
    return (size_t)kWavesGlobal * 64 * (kRowsPerWave / 32) * (head_dim / 2 + 2);
}
// Partial slots (per head group) for a problem with max_tiles tiles: split
// tiles have more than W / (kSplitDiv grid n_hg) blocks for a total of W
// (blocks x head groups), so their ceil(blocks / target) add up to at most
// 2 kSplitDiv grid / n_hg.
inline int split_slots(int max_tiles, int n_hg) {
    const long long a = (long long)max_tiles * kMaxSplit;
    const long long b = 2LL * kSplitDiv * kSplitGridRef / n_hg + kMaxSplit;
    return (int)(a < b ? a : b);
}

// Epilogue of the local / global modes.
//   kEpiRaw   : write the branch output O (fp32) -- logo_local_attn and
//               logo_global_attn_sparse_q.
//   kEpiFused : ContextNorm + output fusion in place (logo_attn_fwd): the local
//               kernel writes bf16 Norm^L(O^L) to `out` for unselected tokens and
//               (1-p) Norm^L(O^L) (fp32) to the compact buffer `lc` for selected
//               ones; the global kernel then writes bf16 lc + p Norm^G(O^G).
//   kEpiFusedTrain : kEpiFused, and also the raw branch output O (fp32, to
//               `out`) and the base-2 LSE of each row (to `lse`) -- the
//               training forward, which keeps them for the backward pass.
//   kEpiLayer : the one-launch layer (layer_kernel): the local items as in
//               kEpiFused; the global items write p Norm^G(O^G) (fp32) to the
//               compact buffer `gc` instead of finishing the rows, and a
//               separate pass sums lc + gc into `out`.
enum AttnEpi { kEpiRaw = 0, kEpiFused = 1, kEpiFusedTrain = 2, kEpiLayer = 3 };

// Tile plan of the global branch (device-built work table).  tmp and out each
// hold max_tiles + split_slots entries; scratch holds 2 * stride ints with
// stride >= max(B, max_tiles) + 1; split_cnt holds split_slots * n_hg ints.
struct PlanArgs {
    const int32_t *cu_sel;     // [B+1] compacted sequence offsets
    const int32_t *sel_idx;    // [cap] selected token indices
    int32_t tpw, cap, max_seqlen, n_hg, grid_wgs, split_slots, stride;
    // other work of the same persistent grid, in KV-block units (the local
    // items of the one-launch layer), counted into the split threshold
    int64_t extra_blocks;
    SparseTile *tmp, *out;
    int32_t *scratch, *queue, *split_cnt;
};
struct AttnArgs {
    const uint16_t *q;
    const uint16_t *k;
    const uint16_t *v;
    void *out;                 // fp32 [rows][Hq][d] or bf16 for dense
    const int32_t *cu_seqlens;
    const int32_t *sel_idx;    // global mode
    const SparseTile *tiles;   // global mode: work entries, longest first
    int32_t *queue;            // global mode: [0] = n_entries, [1 + x] = queue x counter
    int32_t *split_cnt;        // global mode: [sid * n_hg + hg] entries of a split tile done
    float *partial;            // global mode: [(sid + split) * n_hg + hg] partial results
    int32_t num_seqs;
    int32_t hq, hkv, group;    // group = hq / hkv
    int32_t hpw, tpw, n_hg;
    int32_t window;
    int32_t ntile_max;         // local/dense: ceil(max_seqlen / tpw)
    float scale_log2;          // softmax_scale * log2(e)
    // fused epilogue only
    const int32_t *tok2sel;    // [N] rank or -1
    const float *gate;         // [N]
    const float *gain;         // [Hq][d] of this branch, or NULL (= 1)
    float eps;
    float *lc;                 // [capacity][Hq][d] fp32: (1-p) Norm^L of selected rows
    uint16_t *out_bf16;        // [N][Hq][d]
    // fused local launch only: plan_wg = 1 makes the workgroup after the
    // item_stride persistent ones build the global branch's work table
    // (`plan`)
    int32_t plan_wg;
    // local mode: the persistent workgroups w < item_stride take items w,
    // w + item_stride, ... below n_items (head group fastest, then the
    // sequences' token tiles back to back)
    int32_t n_items, item_stride;
    // fused local launch only: prep_wgs workgroups (after the plan workgroup,
    // at the end of the grid)
    // write the permuted copy aperm of the LP matrices A [Hq][d][d] that the
    // global launch reads (one head each)
    int32_t prep_wgs;
    const uint16_t *prep_a;
    uint16_t *aperm;
    // fused global mode only: the branch transform of the selected queries,
    // applied as they are loaded (0 none, 1 LP with aperm, 2 SO with qphi_s /
    // qphi_b [Hq][d])
    int32_t qphi;
    const float *qphi_s, *qphi_b;
    PlanArgs plan;
    // raw epilogue only: lse (or NULL) receives each row's base-2
    // log-sum-exp of the scaled scores at [head * lse_stride + row]
    float *lse;
    int64_t lse_stride;
    // one-launch layer only: the global branch's Q / K / V (q, k, v are the
    // local branch's), the compact buffer of p Norm^G, and the launch's
    // control words (zeroed before the launch): [0] = the work table is
    // built, [1 + x] = local queue x's counter
    const uint16_t *qg, *kg, *vg;
    const float *gain_g;       // the global branch's gain (gain: the local one's)
    float *gc;
    int32_t *ctl;
};
// Control words of the one-launch layer.
constexpr int kLayerCtlWords = 1 + kQueues;

// Launchers (return hipSuccess or the launch error).
// waves: the workgroup's waves (8 for the global and dense modes; local_waves
// for the local mode).
hipError_t launch_attention(int mode, int epi, int head_dim, int waves, const AttnArgs &a,
                            int grid, hipStream_t s);
int attention_blocks_per_cu(int mode, int head_dim, int waves);

hipError_t launch_sparse_plan(const int32_t *cu_seqlens, int num_seqs, const PlanArgs &plan,
                              hipStream_t s);

// The one-launch layer, for problems whose two branches use workgroups of
// the same waves (and so the same tiles): 8 when Hq / Hkv is a multiple of 4,
// 4 when Hq = Hkv (layer_waves; 0 = not eligible).  grid persistent
// workgroups; a.n_items local items, the global items of the work table that
// workgroup 0 builds (a.plan).
inline int layer_waves(int hq, int hkv) {
    return local_waves(hq, hkv) == global_waves(hq, hkv) ? local_waves(hq, hkv) : 0;
}
hipError_t launch_layer(int head_dim, int waves, const AttnArgs &a, int grid, hipStream_t s);
int layer_blocks_per_cu(int head_dim, int waves);
// out[sel_idx[r]] = bf16(lc[r] + gc[r]) for the selected ranks r below
// min(cu_sel[B], cap) (read on the device).
hipError_t launch_sel_sum(int32_t cap, int hq, int head_dim, const int32_t *cu_sel, int num_seqs,
                          const int32_t *sel_idx, const float *lc, const float *gc,
                          uint16_t *out, hipStream_t s);

// Selection: thresholds, ranks and compaction.  seq_counts holds num_seqs
// ints (per-sequence selected counts when num_seqs > 1).  max_seqlen sizes
// the parts of a sequence that separate workgroups compact.
// zero_words (or NULL): n_zero ints the selection kernel clears (the control
// words of the layer launch that follows it).
hipError_t launch_select(const int32_t *cu_seqlens, int num_seqs, int max_seqlen,
                         const float *gate, int mode, float threshold, double ratio,
                         int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                         int32_t *tok2sel, float *thr, int32_t *seq_counts, hipStream_t s,
                         int32_t *zero_words = nullptr, int n_zero = 0);

// One decoding step (decode.hip).  Work items: local (sequence, KV head,
// head group, chunk) then global (selected rank, KV head, head group,
// chunk); partials [item][gh][m, l, acc[d]].
struct DecodeArgs {
    const uint16_t *q, *k, *v;       // q: [B][Hq][d] new tokens; k, v: caches [N][Hkv][d]
    const uint16_t *q_g, *k_g, *v_g; // global-branch tensors (aliases when not given)
    const int32_t *cu;               // [B+1] cache boundaries
    const float *gate;               // [B] gate of the new tokens
    const float *gain_local, *gain_global;
    float eps, scale_log2;
    int32_t num_seqs, hq, hkv, group, head_dim, window;
    int32_t gh, nhg;                 // query heads per item, head groups per KV head
    int32_t kc;                      // keys per chunk
    int32_t chunks_local, chunks_global;
    int32_t n_local_items, n_global_items;
    int32_t *act, *rank_of, *n_act;  // selected sequences (compacted), rank or -1, count
    int32_t sel_mode;                // 0: threshold thr_host, 2: device threshold thr_dev[0]
    float thr_host;
    const float *thr_dev;
    float *part_local, *part_global;
    uint16_t *out;                   // [B][Hq][d] bf16
};
hipError_t launch_decode(const DecodeArgs &a, hipStream_t s);

// Gate projection and branch transforms (transform.hip).  kind 0 = LP
// (A [H][d][d] bf16), 1 = SO (s, b [H][d] fp32); rows = token list or NULL,
// n_rows_dev = device row count (NULL: n_rows).
hipError_t launch_gate_proj(int64_t n, int dm, const uint16_t *x, const uint16_t *w, float *p,
                            hipStream_t s);
hipError_t launch_branch_transform(int kind, int64_t n_rows, int H, int d, const uint16_t *u,
                                   const uint16_t *A, const float *sc, const float *bi,
                                   const int32_t *rows, const int32_t *n_rows_dev, uint16_t *out,
                                   hipStream_t s);

// Backward pass (bwd.hip).  Rows of a branch: local = tokens (row index =
// token), global = selected rows in rank order (row index = rank, token =
// sel_idx[rank]).  q / dout are the branch's row-major [rows][Hq][d] bf16
// tensors (the global branch uses the compact copy of Q^G), lse / delta are
// [Hq][row_stride] fp32.  acc_*: add into the output instead of overwriting.
struct BwdArgs {
    const uint16_t *q, *k, *v, *dout;
    const float *lse, *delta;
    const int32_t *cu_seqlens, *sel_idx, *cu_sel;
    float *dq, *dk, *dv;
    int32_t num_seqs, hq, hkv, group, hpw, tpw, n_hg, window, ntile_max, cap;
    int32_t acc_q, acc_k, acc_v;
    int64_t row_stride;
    float scale_log2, scale;
};
struct FusionBwdArgs {
    const float *ol, *og;              // raw O^L [N][Hq][d], O^G [cap][Hq][d] (compact)
    const uint16_t *dout, *q_g;        // [N][Hq][d]
    const float *gate;
    const int32_t *tok2sel;
    const float *gain_l, *gain_g;      // [Hq][d] or NULL
    float eps;
    int32_t n, hq, cap, tokens_per_block;
    uint16_t *dol, *dog, *qc;          // [N][Hq][d], [cap][Hq][d], [cap][Hq][d]
    float *delta_l, *delta_g;          // [Hq][N], [Hq][cap]
    float *side;                       // [N][Hq]: row terms of dL/dp
    float *part_l, *part_g;            // gain-gradient partials or NULL
};
int fusion_bwd_tokens_per_pass(int hq, int head_dim);
bool fusion_bwd_supported(int hq, int head_dim);
hipError_t launch_fusion_bwd(const FusionBwdArgs &a, int grid, int head_dim, hipStream_t s);
hipError_t launch_gate_grad(int n, int hq, const float *side, float *dgate, hipStream_t s);
// gain-gradient column sums: tmp holds gain_grad_chunks(rows) x cols floats
int gain_grad_chunks(int rows);
hipError_t launch_gain_grad(int rows, int cols, const float *part, float *tmp, float *out,
                            hipStream_t s);
hipError_t launch_fill_zero(int64_t n, float *x, hipStream_t s);
// Compact Q rows + Delta for the standalone query-sparse backward: ranks
// below min(n_sel_dev[0], cap) (the selected count, read on the device).
hipError_t launch_sparse_prep(int64_t cap, int hq, int head_dim, const int32_t *n_sel_dev,
                              const int32_t *sel_idx, const uint16_t *q, const float *o,
                              const uint16_t *dout, uint16_t *qc, float *delta, hipStream_t s);
hipError_t launch_attn_delta(int64_t n, int hq, int head_dim, const uint16_t *o,
                             const uint16_t *dout, float *delta, hipStream_t s);
hipError_t launch_bwd_dq(int mode, int head_dim, const BwdArgs &a, int grid, hipStream_t s);
hipError_t launch_bwd_dkv(int mode, int head_dim, const BwdArgs &a, int grid, hipStream_t s);
int bwd_keys_per_block();

// One budget-controller step on the device (b_th += gamma sign(F - rho)).
hipError_t launch_budget_update(const int32_t *cu_sel, int num_seqs, int n_tokens, double rho,
                                float gamma, float *b_th, float *realized, hipStream_t s);

hipError_t launch_combine(int n_tokens, int hq, int head_dim, const float *o_local,
                          const float *o_global, const float *gate,
                          const int32_t *tok2sel, const float *gain_local,
                          const float *gain_global, float eps, int apply_norm,
                          uint16_t *out, hipStream_t s);

}  // namespace logo
