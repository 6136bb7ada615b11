// attention.hip -- softmax attention kernels for gfx950 (bf16 MFMA, fp32
// online softmax).  One template serves the three row sets of the layer:
//
//   kModeLocal  : every token, keys max(0, i-w+1)..i       (local branch,
//                 Sec. 3.1 local context; Eq. branch-attention)
//   kModeGlobal : selected tokens only, keys 0..i          (query-sparse global
//                 branch, Eq. query-sparse-global; App. B forward traversal)
//   kModeDense  : every token, keys 0..i                   (dense causal
//                 baseline, Eq. attention with the global context)
//
// Work decomposition.  A workgroup has W waves: 8 (one workgroup per CU) in
// the local mode when G = Hq/Hkv is a multiple of 4, else 4 (two per CU); 8
// in the global mode, except 4 when G = 1; 8 in the dense mode (see
// local_waves / global_waves).  Each wave owns 32 query rows of one query
// head, and all W waves read the same key/value head, so a staged K/V tile in
// LDS serves 32 W rows.  With GQA group size G the waves take gcd(G,4) heads
// of one KV group, which keeps the tile's token span -- and so its
// causal-diagonal band -- short.  The local and global modes run persistent
// workgroups (static item striding with a prefetch of the next item, and
// per-XCD work queues, respectively).  layer_kernel runs the items of both
// branches in one persistent launch (global items longest first, local items
// filling in behind them), where the two use workgroups of the same waves.
//
// MFMA formulation (v_mfma_f32_32x32x16_bf16, lane l: column l%32, rows
// 8*(i/4) + 4*(l/32) + i%4 of the 32x32 accumulator).  The kernel computes
// S^T = K Q^T, so each lane's accumulator column is ONE query: row max and
// row sum need only the lane and its partner l^32.  The same registers,
// rounded to bf16, are directly the B operand of O^T = V^T P^T when the V^T
// operand is read from LDS in the matching key order (see read_vt_frag).  O^T
// again has one query per lane column, so the online-softmax rescale is a
// per-lane multiply.
//
// Causal handling (App. B): per KV tile a wave classifies itself as fully
// visible (no predicate), beyond its last row (skipped) or on the diagonal /
// window edge (real-position mask on each score); a 32-key half of its first
// or last tile that none of its rows sees is not computed.
#include "logo_internal.h"
#include "plan.h"
#include "attn_common.h"

#include <type_traits>

namespace logo {
namespace {

// Real-position masks of a KV tile (bit set).
constexpr int kMaskNone = 0, kMaskCausal = 1, kMaskWindow = 2;
// Which 32-key halves of a 64-key tile a step computes: both, only the upper
// one (the lower half lies left of every row's window), only the lower one,
// or the lower one and the upper one unless no row reaches it (decided at run
// time: the causal diagonal tiles).
constexpr int kHalfBoth = 0, kHalfUpper = 1, kHalfLower = 2, kHalfDiag = 3;

// LDS tiles, both [key][d].  K rows are padded by 16 B so that the 16-byte
// fragment reads of 8 consecutive rows hit distinct banks.  V rows are not
// padded; instead the 64-byte segments of a row are permuted (segment j of
// row r is stored at j ^ vswz(r)) so that the transpose reads, which take
// one 64-byte segment from each of 4 consecutive rows per half-wave, hit 4
// distinct 64-byte bank groups of the 256-byte bank window.
constexpr int kKPad = 8;
// Output staging of the 8-wave local kernel: each wave's 32 bf16 output rows
// (padded by 16 B) pass through LDS so that every store instruction writes
// whole rows (see attend_item).
constexpr int kStagePad = 8;
template <int D, int STG = 0>
struct alignas(16) Smem {
    uint16_t k[2][kBlockN][D + kKPad];
    uint16_t v[2][kBlockN][D];
    uint16_t ostage[STG > 0 ? STG : 1][kRowsPerWave][STG > 0 ? D + kStagePad : 1];
};
template <int MODE, int W>
constexpr int stage_waves() { return MODE == kModeLocal && W == 8 ? W : 0; }
template <int D>
__device__ __forceinline__ constexpr int vswz(int r) {
    // rows per 256-byte bank window: 128 / D; segments per row: D / 32
    return (r / (128 / D)) % (D / 32);
}

// K/V tiles go global -> LDS directly (buffer_load_dwordx4 ... lds): each
// wave-instruction writes 64 consecutive 16-byte LDS slots (lane i at
// M0 + 16 i), so a padded tile is filled as a sequence of 1 KB slot runs; a
// lane whose slot is row padding re-loads the row's last chunk (never read).
// The per-lane byte offsets inside a tile are fixed and computed once.
template <int D, int W>
struct Dma {
    static constexpr int kSlotsK = (D + kKPad) * 2 / 16;     // 16-byte slots per K row
    static constexpr int kSlotsV = D * 2 / 16;
    static constexpr int kInstK = kSlotsK;                   // 64 rows x slots / 64 lanes
    static constexpr int kInstV = kSlotsV;
    static constexpr int kPerWaveK = (kInstK + W - 1) / W;
    static constexpr int kPerWaveV = (kInstV + W - 1) / W;
    int voff_k[kPerWaveK];
    int voff_v[kPerWaveV];
};

template <int D, int W>
__device__ __forceinline__ void dma_plan(Dma<D, W> &d, int wave, int lane, int row_bytes) {
#pragma unroll
    for (int i = 0; i < Dma<D, W>::kPerWaveK; i++) {
        const int slot = (i * W + wave) * 64 + lane;
        const int row = slot / Dma<D, W>::kSlotsK, col = min(slot % Dma<D, W>::kSlotsK, D / 8 - 1);
        d.voff_k[i] = row * row_bytes + col * 16;
    }
#pragma unroll
    for (int i = 0; i < Dma<D, W>::kPerWaveV; i++) {
        // LDS slot (row, chunk p) receives the chunk whose segment maps to p's
        const int slot = (i * W + wave) * 64 + lane;
        const int row = slot / Dma<D, W>::kSlotsV, p = slot % Dma<D, W>::kSlotsV;
        const int col = ((p >> 2) ^ vswz<D>(row)) * 4 + (p & 3);
        d.voff_v[i] = row * row_bytes + col * 16;
    }
}

// Descriptor of one tile: base = its first key row of this KV head, size =
// the rows that exist, so rows at or past the sequence end read as zeros
// (masked keys with zero values keep masked-out products finite).  Raw
// buffer descriptor words: base address (48 bits, stride 0), size in bytes,
// flags.
__device__ __forceinline__ u32x4 tile_rsrc(const uint16_t *kv, int T, int k0, int row_bytes) {
    const int rows = min(kBlockN, T - k0);
    return raw_rsrc((const char *)kv + (long long)k0 * row_bytes, rows > 0 ? rows * row_bytes : 0);
}

template <int D, int W>
__device__ __forceinline__ void dma_k(uint16_t *dst, const Dma<D, W> &d, const uint16_t *kv_k,
                                      int T, int k0, int row_bytes, int wave) {
    const u32x4 r = tile_rsrc(kv_k, T, k0, row_bytes);
#pragma unroll
    for (int i = 0; i < Dma<D, W>::kPerWaveK; i++) {
        const int inst = i * W + wave;
        if (inst < Dma<D, W>::kInstK)
            lds_load16(r, (char *)dst + inst * 1024, d.voff_k[i]);
    }
}
template <int D, int W>
__device__ __forceinline__ void dma_v(uint16_t *dst, const Dma<D, W> &d, const uint16_t *kv_v,
                                      int T, int k0, int row_bytes, int wave) {
    const u32x4 r = tile_rsrc(kv_v, T, k0, row_bytes);
#pragma unroll
    for (int i = 0; i < Dma<D, W>::kPerWaveV; i++) {
        const int inst = i * W + wave;
        if (inst < Dma<D, W>::kInstV)
            lds_load16(r, (char *)dst + inst * 1024, d.voff_v[i]);
    }
}

// V^T operand of the O^T MFMA straight from the row-major V tile with the
// gfx950 LDS transpose read: within each 16-lane group, lane 4b+e receives
// element e of the 4-element rows addressed by lanes b, b+4, b+8, b+12.
// Lane i of group q addresses row (key0 + 4*(q/2) + i/4), columns
// (c0 + 16*(q%2) + 4*(i%4)) .. +3, so lane l ends up holding column c0 + l%32
// for keys key0 + 4*(l/32) + 0..3 (first read) and, 8 rows further, + 8..11
// (second read): the 8 keys of its MFMA k-slice, in the order the S^T
// accumulator (and so P^T) holds them.
__device__ __forceinline__ bf16x8 read_vt_frag(const uint16_t *vrow_lane, int row_stride) {
    return lds_tr_pair(vrow_lane, vrow_lane + 8 * row_stride);
}

// Attention for one work item: a tile of rows x the heads of one head group.
//   Local / dense: tile jt of sequence b, rows = tokens jt*tpw ...
//   Global: rows = sel_idx[first .. first+nrows), all in sequence b.
//
// Online softmax with a lazily moved reference max: a row's reference m_ref
// only moves (rescaling O and l) when a tile's max exceeds it by more than
// 2^kLazy in the exp2 domain, so probabilities stay <= 2^kLazy and most tiles
// skip the rescale.  The result is the same softmax after the final O / l.
constexpr float kLazy = 8.f;
// 32-row MFMA column blocks per wave: each K / V^T fragment read from LDS
// feeds one MFMA per row group.
constexpr int RG = kRowsPerWave / 32;

// Split-KV partials of the global branch.  Every entry of a split tile
// stores its unnormalised O (relative to its reference m, exp2 domain), m
// and l per lane, releases them, and counts itself done; the entry that
// counts last acquires the others and folds all of them in split order, so
// the result does not depend on which entry finished last.  Returns false
// for the entries that are not last (nothing more to do).
template <int D>
__device__ __forceinline__ bool merge_split(const AttnArgs &a, const SparseTile &t, int hg,
                                            int wave, int lane, f32x16 (&acc)[RG][D / 32],
                                            float (&m)[RG], float (&l)[RG]) {
    __shared__ int s_last;
    constexpr int kLanes = kWavesGlobal * 64;
    constexpr int kAccFloats = kLanes * RG * (D / 2);
    const int sid = uni(t.sid), split = uni(t.split), ns = uni(t.nsplit);
    const int li = wave * 64 + lane;
    const int64_t pf = (int64_t)partial_floats(D);
    float *base = a.partial + (int64_t)sid * a.n_hg * pf;
    const int64_t slot_stride = (int64_t)a.n_hg * pf;
    float *mine = base + split * slot_stride + (int64_t)hg * pf;
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
#pragma unroll
        for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
            for (int qd = 0; qd < 4; qd++) {
                const f32x4 v = {acc[rg][cb][qd * 4 + 0], acc[rg][cb][qd * 4 + 1],
                                 acc[rg][cb][qd * 4 + 2], acc[rg][cb][qd * 4 + 3]};
                *(f32x4 *)(mine + (((rg * (D / 32) + cb) * 4 + qd) * kLanes + li) * 4) = v;
            }
        mine[kAccFloats + rg * kLanes + li] = m[rg];
        mine[kAccFloats + (RG + rg) * kLanes + li] = l[rg];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0)
        s_last = atomicAdd(&a.split_cnt[sid * a.n_hg + hg], 1) == ns - 1;
    __syncthreads();
    const bool last = s_last;
    if (!last)
        return false;
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
        float M = kNegInf, L = 0.f;
#pragma unroll
        for (int cb = 0; cb < D / 32; cb++)
            acc[rg][cb] = f32x16{};
        for (int j = 0; j < ns; j++) {
            const float *pj = base + j * slot_stride + (int64_t)hg * pf;
            const float mj = pj[kAccFloats + rg * kLanes + li];
            const float lj = pj[kAccFloats + (RG + rg) * kLanes + li];
            const float mn = fmaxf(M, mj);
            const float mc = (mn == kNegInf) ? 0.f : mn;
            const float ra = __builtin_amdgcn_exp2f(M - mc), rb = __builtin_amdgcn_exp2f(mj - mc);
#pragma unroll
            for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                for (int qd = 0; qd < 4; qd++) {
                    const f32x4 v = *(const f32x4 *)(
                        pj + (((rg * (D / 32) + cb) * 4 + qd) * kLanes + li) * 4);
#pragma unroll
                    for (int e = 0; e < 4; e++)
                        acc[rg][cb][qd * 4 + e] = fmaf(acc[rg][cb][qd * 4 + e], ra, v[e] * rb);
                }
            L = fmaf(L, ra, lj * rb);
            M = mn;
        }
        l[rg] = L;
        m[rg] = M;
    }
    return true;
}

// Wave-uniform state of one work item.
struct ItemU {
    int b, hg, T, nvalid, wg_pmin, wg_pmax, head, kvh;
    int64_t base;
    int kb_lo, kb_hi, kb_first, kb_last, wpmin, wpmax;
    bool wave_valid;
    SparseTile tile;
};
// This lane's query rows of one item (one per row group) and the inputs of
// the fused epilogue; rows past the tile end repeat the last row and are
// never stored.
struct ItemL {
    int pos[RG];
    int64_t orow[RG], qtok[RG];
    bool row_valid[RG];
    float ep_gate[RG];
    int ep_rank[RG];
};

// Column of the LP matrix that row r of its permuted copy holds: bits 2 and 3
// of r (within its 32-row block) swapped.  With A'[h][r][k] = A[h][k][perm(r)]
// as the A operand of the 32x32x16 MFMA and a lane's Q fragments as the B
// operand, accumulator element 8 j + e of lane (g, m) is output channel
// 16 j + 8 g + e of its 32-channel block for query row m -- the layout of the
// B operand of the next product, so the rounded result replaces the
// fragments directly.
__device__ __forceinline__ int lp_perm(int r) { return (r & ~0xC) | ((r & 4) << 1) | ((r & 8) >> 1); }

// Q^G = phi(Q) on the selected rows as the global kernel loads them (Eq.
// branch-transform): LP q A_h (bf16 MFMA, fp32 accumulation) or SO
// q * s_h + b_h (fp32), one bf16 rounding each.
template <int D>
__device__ __forceinline__ void apply_qphi(const AttnArgs &a, int head,
                                           bf16x8 (&qf)[RG][D / 16]) {
    const int lane = threadIdx.x & 63, g = lane >> 5, m = lane & 31;
    if (a.qphi == 1) {
        const uint16_t *ap = a.aperm + (int64_t)head * D * D;
        bf16x8 qn[RG][D / 16];
#pragma unroll
        for (int cb = 0; cb < D / 32; cb++) {
            f32x16 c[RG];
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
                c[rg] = f32x16{};
#pragma unroll
            for (int ks = 0; ks < D / 16; ks++) {
                const bf16x8 af = *(const bf16x8 *)(ap + (cb * 32 + m) * D + ks * 16 + g * 8);
#pragma unroll
                for (int rg = 0; rg < RG; rg++)
                    c[rg] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, qf[rg][ks], c[rg], 0, 0, 0);
            }
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
#pragma unroll
                for (int h = 0; h < 2; h++)
#pragma unroll
                    for (int e = 0; e < 8; e += 2) {
                        const bf16x2 v = cvt_bf16x2(c[rg][8 * h + e], c[rg][8 * h + e + 1]);
                        qn[rg][2 * cb + h][e] = v[0];
                        qn[rg][2 * cb + h][e + 1] = v[1];
                    }
        }
#pragma unroll
        for (int rg = 0; rg < RG; rg++)
#pragma unroll
            for (int ks = 0; ks < D / 16; ks++)
                qf[rg][ks] = qn[rg][ks];
    } else if (a.qphi == 2) {
#pragma unroll
        for (int ks = 0; ks < D / 16; ks++) {
            const int c0 = head * D + ks * 16 + g * 8;
            const f32x4 s0 = *(const f32x4 *)(a.qphi_s + c0), s1 = *(const f32x4 *)(a.qphi_s + c0 + 4);
            const f32x4 b0 = *(const f32x4 *)(a.qphi_b + c0), b1 = *(const f32x4 *)(a.qphi_b + c0 + 4);
            const float sv[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
            const float bv[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
#pragma unroll
                for (int e = 0; e < 8; e += 2) {
                    const bf16x2 v = cvt_bf16x2(fmaf((float)qf[rg][ks][e], sv[e], bv[e]),
                                                fmaf((float)qf[rg][ks][e + 1], sv[e + 1], bv[e + 1]));
                    qf[rg][ks][e] = v[0];
                    qf[rg][ks][e + 1] = v[1];
                }
        }
    }
}

// The permuted copy of one head's LP matrix (see lp_perm), 16 bytes per
// thread and step: A'[r][k0 .. k0+7] gathers column lp_perm(r) of rows
// k0 .. k0+7 of A.
template <int D, int NT>
__device__ __forceinline__ void permute_lp_head(const uint16_t *A, uint16_t *Ap, int head) {
    const uint16_t *src = A + (int64_t)head * D * D;
    uint16_t *dst = Ap + (int64_t)head * D * D;
    for (int c = threadIdx.x; c < D * D / 8; c += NT) {
        const int r = c / (D / 8), k0 = (c % (D / 8)) * 8;
        const uint16_t *sc = src + k0 * D + lp_perm(r);
        auto pair = [&](int e) { return (uint32_t)sc[e * D] | ((uint32_t)sc[(e + 1) * D] << 16); };
        *(u32x4 *)(dst + r * D + k0) = u32x4{pair(0), pair(2), pair(4), pair(6)};
    }
}

// The tensors of an item's branch: the one-launch layer's global items read
// the global branch's Q / K / V and gain (qg, kg, vg, gain_g); every other
// item, the standalone global launch included, reads q, k, v and gain.
template <int MODE, int EPI>
__device__ __forceinline__ constexpr bool global_tensors() {
    return MODE == kModeGlobal && EPI == kEpiLayer;
}

// An item's indices and rows, and the loads of its Q fragments and fused-
// epilogue inputs (issued here; waited for with the item's first K tile).
//   Local / dense: tile jt of sequence b, rows = tokens jt*tpw ...
//   Global: rows = sel_idx[first .. first+nrows), all in sequence b.
template <int D, int MODE, int EPI>
__device__ __forceinline__ void item_begin(const AttnArgs &a, int b, int hg, int jt,
                                           SparseTile tile, ItemU &u, ItemL &l,
                                           bf16x8 (&qf)[RG][D / 16]) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int g = lane >> 5, m = lane & 31;
    u.b = b = uni(b);
    u.hg = hg = uni(hg);
    const int64_t base = uni(a.cu_seqlens[b]);
    const int T = uni(a.cu_seqlens[b + 1] - (int)base);
    u.base = base;
    u.T = T;
    const int hw = wave % a.hpw, tb = wave / a.hpw;
    u.head = hg * a.hpw + hw;
    u.kvh = (hg * a.hpw) / a.group;

    int nvalid, wg_pmin, wg_pmax;
    if (MODE == kModeGlobal) {
        tile.first = uni(tile.first);
        nvalid = uni(tile.nrows);
        wg_pmax = uni(tile.pos_max);
        wg_pmin = uni(a.sel_idx[tile.first] - (int)base);
    } else {
        const int p0 = jt * a.tpw;
        nvalid = min(a.tpw, T - p0);
        wg_pmin = p0;
        wg_pmax = p0 + nvalid - 1;
    }
    u.tile = tile;
    u.nvalid = nvalid;
    u.wg_pmin = wg_pmin;
    u.wg_pmax = wg_pmax;
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
        const int ri = tb * kRowsPerWave + rg * 32 + m;
        l.row_valid[rg] = ri < nvalid;
        const int ric = l.row_valid[rg] ? ri : nvalid - 1;
        if (MODE == kModeGlobal) {
            const int rank = tile.first + ric;
            l.pos[rg] = a.sel_idx[rank] - (int)base;
            l.orow[rg] = rank;
        } else {
            l.pos[rg] = wg_pmin + ric;
            l.orow[rg] = base + l.pos[rg];
        }
        l.qtok[rg] = base + l.pos[rg];
    }
    u.wave_valid = tb * kRowsPerWave < nvalid;
    u.wpmin = __builtin_amdgcn_readfirstlane(l.pos[0]);
    u.wpmax = __builtin_amdgcn_readlane(l.pos[RG - 1], 31);

#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
        const uint16_t *qp = (global_tensors<MODE, EPI>() ? a.qg : a.q) +
                             (l.qtok[rg] * a.hq + u.head) * (int64_t)D + g * 8;
#pragma unroll
        for (int s = 0; s < D / 16; s++)
            qf[rg][s] = *(const bf16x8 *)(qp + s * 16);
    }
    if constexpr (MODE == kModeGlobal && EPI != kEpiRaw)
        if (a.qphi != 0)
            apply_qphi<D>(a, u.head, qf);
    // Inputs of the fused epilogue, fetched now so that their latency overlaps
    // the KV loop.
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
        l.ep_gate[rg] = 0.f;
        l.ep_rank[rg] = -1;
        if (EPI != kEpiRaw && MODE != kModeDense) {
            l.ep_gate[rg] = a.gate[l.qtok[rg]];
            l.ep_rank[rg] = (MODE == kModeGlobal) ? (int)l.orow[rg] : a.tok2sel[l.qtok[rg]];
        }
    }

    const int w = a.window;
    const int lo = (MODE == kModeLocal) ? max(0, wg_pmin - w + 1) : 0;
    // KV blocks of this item: a global entry covers its own KV range
    u.kb_lo = (MODE == kModeGlobal) ? uni(tile.kb_begin) : lo / kBlockN;
    u.kb_hi = (MODE == kModeGlobal) ? uni(tile.kb_end) : wg_pmax / kBlockN;
    // Tiles this wave computes: a contiguous, wave-uniform sub-range.
    u.kb_first = u.kb_lo;
    u.kb_last = min(u.wpmax / kBlockN, u.kb_hi);
    if (MODE == kModeLocal)
        u.kb_first = max(u.kb_lo, max(0, u.wpmin - w + 1) / kBlockN);
    if (!u.wave_valid) {
        u.kb_first = u.kb_hi + 1;
        u.kb_last = u.kb_hi;
    }
}

// The first K tile of an item into K buffer 0 (the K/V pipeline of attend_item
// starts from it); every earlier read of K buffer 0 must have ended at a
// barrier before this.
template <int D, int MODE, int EPI, int W, int STG>
__device__ __forceinline__ void item_first_k(const AttnArgs &a, Smem<D, STG> &sm, const ItemU &u) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int row_bytes = a.hkv * D * 2;
    Dma<D, W> dma;
    dma_plan<D, W>(dma, wave, lane, row_bytes);
    const uint16_t *kv_k =
        (global_tensors<MODE, EPI>() ? a.kg : a.k) + (u.base * a.hkv + u.kvh) * (int64_t)D;
    dma_k<D, W>(&sm.k[0][0][0], dma, kv_k, u.T, u.kb_lo * kBlockN, row_bytes, wave);
}

// Attention for one work item.  Its item_begin loads and first K tile are
// in flight (waited: false), or every wave has already waited for its own
// share of them (waited: true; then the first step needs only the barrier).
// prefetch() runs once every wave has passed the barrier after the item's
// last K / V tile step -- the K buffers and qf are then free -- and before
// the item's last PV product and epilogue, so the next item's loads overlap
// them; it returns whether it issued loads, and then each wave waits for
// them before its first output store.  So the next item starts without
// waiting for this item's stores, which drain during its first step.
template <int D, int MODE, int EPI, int W, int STG, class Prefetch>
__device__ __forceinline__ void attend_item(const AttnArgs &a, Smem<D, STG> &sm, const ItemU &u,
                                            const ItemL &l, bf16x8 (&qf)[RG][D / 16],
                                            bool waited, Prefetch &&prefetch) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int g = lane >> 5, m = lane & 31;
    const int64_t base = u.base;
    const int T = u.T;
    const int head = u.head, kvh = u.kvh;
    const SparseTile &tile = u.tile;
    const int wpmin = u.wpmin, wpmax = u.wpmax;
    const bool wave_valid = u.wave_valid;
    const int kb_lo = u.kb_lo, kb_hi = u.kb_hi;
    const int kb_first = u.kb_first, kb_last = u.kb_last;
    const int(&pos)[RG] = l.pos;
    const int64_t(&orow)[RG] = l.orow;
    const int64_t(&qtok)[RG] = l.qtok;
    const bool(&row_valid)[RG] = l.row_valid;
    const float(&ep_gate)[RG] = l.ep_gate;
    const int(&ep_rank)[RG] = l.ep_rank;

    // Lane's row / column inside a V tile for the transpose reads.
    const int vt_row = 4 * g + ((lane & 15) >> 2);
    const int vt_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    // Stored column of this lane's read in 32-column block cb (the rows it
    // reads differ from vt_row by multiples of 8, which keep vswz).
    int vt_scol[D / 32];
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++)
        vt_scol[cb] = (cb ^ vswz<D>(vt_row)) * 32 + vt_col;

    const int w = a.window;
    const float c = a.scale_log2;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

    // K/V base of this sequence and KV head, and this thread's fixed byte
    // offsets inside a tile.
    const int row_bytes = a.hkv * D * 2;
    constexpr bool kGT = global_tensors<MODE, EPI>();
    const uint16_t *kv_k = (kGT ? a.kg : a.k) + (base * a.hkv + kvh) * (int64_t)D;
    const uint16_t *kv_v = (kGT ? a.vg : a.v) + (base * a.hkv + kvh) * (int64_t)D;
    Dma<D, W> dma;
    dma_plan<D, W>(dma, wave, lane, row_bytes);

    f32x16 acc[RG][D / 32];
    float m_ref[RG], l_run[RG];
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
#pragma unroll
        for (int cb = 0; cb < D / 32; cb++)
            acc[rg][cb] = f32x16{};
        m_ref[rg] = kNegInf;
        l_run[rg] = 0.f;
    }

    // Software-pipelined KV loop.  Step kb (between two barriers) stages
    // K(kb+1) and V(kb), computes S(kb) = K(kb) Q^T, then interleaves the
    // softmax of tile kb, 16 keys at a time, with the PV MFMAs of tile kb-1
    // (its rounded P kept in registers), so the exps of one tile overlap the
    // PV MFMAs of the previous one.  V is consumed one step after K; two
    // buffers each, and every buffer is rewritten only after the barrier that
    // ends its last read.
    bf16x2 pw[RG][2][8];                      // P of the last softmax-ed tile
    f32x16 s[RG][2];                          // S of the tile being softmax-ed
    auto kidx = [&](int kb_) { return (kb_ - kb_lo) & 1; };
    auto vidx = [&](int kb_) { return (kb_ - kb_lo) & 1; };
    // The item's first K tile (buffer 0) and its Q and epilogue-input loads:
    // this wait covers all of them (inside the loop the only vector-memory
    // loads in flight are the K/V tile loads, which the compiler does not
    // track).  The barrier also ends every wave's reads of the previous
    // item's last V tile before this item's first V load.  When each wave has
    // waited for its loads already, a bare barrier (no memory fence, which
    // would wait for the previous item's output stores) suffices: the K tile
    // is in LDS once every wave's share has arrived.
    if (waited)
        __builtin_amdgcn_s_barrier();
    else
        dma_wait_barrier();

    // Loads of step kb: K(kb+1) and V(kb).
    auto stage = [&](int kb_) {
        if (kb_ < kb_hi)
            dma_k<D, W>(&sm.k[kidx(kb_ + 1)][0][0], dma, kv_k, T, (kb_ + 1) * kBlockN, row_bytes,
                        wave);
        dma_v<D, W>(&sm.v[vidx(kb_)][0][0], dma, kv_v, T, kb_ * kBlockN, row_bytes, wave);
    };
    // S(kb) = K(kb) Q^T into s (the 32-key halves sb0 <= sb < sb1).
    auto op_s = [&](int kb_, auto half) {
        constexpr int hf = decltype(half)::value;
        constexpr int sb0 = hf == kHalfUpper ? 1 : 0, sb1 = hf == kHalfLower ? 1 : 2;
        const uint16_t(*kt)[D + kKPad] = sm.k[kidx(kb_)];
#pragma unroll
        for (int rg = 0; rg < RG; rg++)
#pragma unroll
            for (int sb = sb0; sb < sb1; sb++)
                s[rg][sb] = f32x16{};
#pragma unroll
        for (int ss = 0; ss < D / 16; ss++)
#pragma unroll
            for (int sb = sb0; sb < sb1; sb++) {
                const bf16x8 kf = *(const bf16x8 *)&kt[sb * 32 + m][ss * 16 + g * 8];
#pragma unroll
                for (int rg = 0; rg < RG; rg++)
                    s[rg][sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[rg][ss],
                                                                        s[rg][sb], 0, 0, 0);
            }
        // Schedule: four K-fragment reads ahead, then the MFMAs of one read
        // per read, so LDS latency hides behind the MFMAs of the S blocks.
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);      // DS reads
#pragma unroll
        for (int i = 0; i < (D / 16) * (sb1 - sb0) - 4; i++) {
            __builtin_amdgcn_sched_group_barrier(0x008, RG, 0); // MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * RG, 0);
    };
    // PV of the tile whose P is in pw, V from buffer vi, for one 16-key slice
    // q (0..3) of the 64-key tile.
    auto pv_slice = [&](int vi, int q) {
        const int sb = q >> 1, ss = q & 1;
        bf16x8 pf[RG];
#pragma unroll
        for (int rg = 0; rg < RG; rg++)
#pragma unroll
            for (int j = 0; j < 4; j++) {
                pf[rg][2 * j] = pw[rg][sb][ss * 4 + j][0];
                pf[rg][2 * j + 1] = pw[rg][sb][ss * 4 + j][1];
            }
#pragma unroll
        for (int cb = 0; cb < D / 32; cb++) {
            const bf16x8 vf = read_vt_frag(&sm.v[vi][sb * 32 + ss * 16 + vt_row][vt_scol[cb]], D);
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
                acc[rg][cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[rg], acc[rg][cb], 0, 0,
                                                                      0);
        }
    };
    auto pv = [&](int vi) {
#pragma unroll
        for (int q = 0; q < 4; q++)
            pv_slice(vi, q);
    };
    // Rescale of O decided by the previous softmax, applied before the next
    // PV accumulates into O (deferred so that no branch separates a tile's
    // exps from the PV MFMAs they are interleaved with).
    bool resc_pend = false;
    float alpha_pend[RG];
#pragma unroll
    for (int rg = 0; rg < RG; rg++)
        alpha_pend[rg] = 1.f;
    auto apply_rescale = [&]() {
        if (resc_pend) {
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++)
                    acc[rg][cb] *= alpha_pend[rg];
            resc_pend = false;
        }
    };
    // Softmax of tile kb (s -> pw); with do_pv, each 16-key slice's exps are
    // preceded by that slice's PV MFMAs of tile kb-1 (V(kb-1)), which read
    // the old pw before the exps overwrite it.  masked: the real-position
    // mask of the tile -- kMaskCausal (key <= pos, diagonal tiles),
    // kMaskWindow (key > pos - w, the local window's left edge) or both.
    auto op_sm = [&](int kb_, auto do_pv, auto masked, auto half) {
        constexpr int mk = decltype(masked)::value;
        constexpr int hf = decltype(half)::value;
        constexpr int sb0 = hf == kHalfUpper ? 1 : 0, sb1 = hf == kHalfLower ? 1 : 2;
        if constexpr (mk != kMaskNone) {
            const int k0 = kb_ * kBlockN;
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
#pragma unroll
                for (int sb = sb0; sb < sb1; sb++)
#pragma unroll
                    for (int i = 0; i < 16; i++) {
                        const int key = k0 + sb * 32 + (i >> 2) * 8 + g * 4 + (i & 3);
                        bool ok = true;
                        if constexpr ((mk & kMaskCausal) != 0)
                            ok = key <= pos[rg];
                        if constexpr (MODE == kModeLocal && (mk & kMaskWindow) != 0)
                            ok = ok && (key > pos[rg] - w);
                        if (!ok)
                            s[rg][sb][i] = kNegInf;
                    }
        }
        float alpha[RG], mc[RG], psum[RG];
        bool any_move = false;
#pragma unroll
        for (int rg = 0; rg < RG; rg++) {
            float mx = kNegInf;
#pragma unroll
            for (int sb = sb0; sb < sb1; sb++)
#pragma unroll
                for (int i = 0; i < 16; i++)
                    mx = fmaxf(mx, s[rg][sb][i]);
            mx = pair_max(mx) * c;           // tile max in the exp2 domain
            // The reference moves only when the new max is far above it; a
            // lane whose rows are still fully masked keeps m_ref = -inf.
            const bool move = mx > m_ref[rg] + kLazy;
            const float m_new = move ? mx : m_ref[rg];
            alpha[rg] = move ? __builtin_amdgcn_exp2f(m_ref[rg] - m_new) : 1.f;
            mc[rg] = (m_new == kNegInf) ? 0.f : m_new;
            m_ref[rg] = m_new;
            any_move = any_move || move;
            psum[rg] = 0.f;
        }
        // P = exp2(s*c - m), rounded to bf16 for the PV product; the row sum
        // accumulates the same rounded values (v_dot2 with ones).
        const int vprev = vidx(kb_ - 1);
#pragma unroll
        for (int q = 0; q < 4; q++) {
            if constexpr (decltype(do_pv)::value)
                pv_slice(vprev, q);
            const int sb = q >> 1, i0 = (q & 1) * 8;
            if (sb < sb0 || sb >= sb1) {
                // a half no row sees: P = 0 (read by the next step's PV
                // product only when it is the lower half)
                if (hf == kHalfUpper)
#pragma unroll
                    for (int rg = 0; rg < RG; rg++)
#pragma unroll
                        for (int i = i0; i < i0 + 8; i += 2)
                            pw[rg][sb][i >> 1] = bf16x2{};
                continue;
            }
#pragma unroll
            for (int rg = 0; rg < RG; rg++)
#pragma unroll
                for (int i = i0; i < i0 + 8; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(fmaf(s[rg][sb][i], c, -mc[rg]));
                    const float p1 = __builtin_amdgcn_exp2f(fmaf(s[rg][sb][i + 1], c, -mc[rg]));
                    pw[rg][sb][i >> 1] = cvt_bf16x2(p0, p1);
                    psum[rg] = __builtin_amdgcn_fdot2_f32_bf16(pw[rg][sb][i >> 1], ones, psum[rg],
                                                               false);
                }
        }
#pragma unroll
        for (int rg = 0; rg < RG; rg++) {
            l_run[rg] = fmaf(l_run[rg], alpha[rg], psum[rg]);
            alpha_pend[rg] = alpha[rg];
        }
        resc_pend = __builtin_amdgcn_ballot_w64(any_move) != 0;
    };

    using T_ = std::true_type;
    using F_ = std::false_type;
    using MNone = std::integral_constant<int, kMaskNone>;
    using MCausal = std::integral_constant<int, kMaskCausal>;
    using MWindow = std::integral_constant<int, kMaskWindow>;
    using MBoth = std::integral_constant<int, kMaskCausal | kMaskWindow>;
    using HBoth = std::integral_constant<int, kHalfBoth>;
    using HUpper = std::integral_constant<int, kHalfUpper>;
    using HLower = std::integral_constant<int, kHalfLower>;
    using HDiag = std::integral_constant<int, kHalfDiag>;
    // 32-key halves no row of the wave sees: the lower half of the first
    // computed tile lies left of every row's window (local branch; then that
    // tile is a window-edge tile), the upper half of the last one right of
    // every row's position (then it is a diagonal tile).  Their score MFMAs
    // (and, for the lower half, exps) are skipped, and the upper half's PV
    // product too.
    const bool lo_out = MODE == kModeLocal && kb_first * kBlockN + 31 <= wpmin - w;
    const bool hi_out = kb_last * kBlockN + 32 > wpmax;
    // The last computed tile's upper half was skipped: its PV product covers
    // the lower half only.
    bool last_lower = false;
    auto pv_last = [&](int vi) {
        if (last_lower) {
            pv_slice(vi, 0);
            pv_slice(vi, 1);
        } else {
            pv(vi);
        }
    };
    // One step: S(kb) + softmax(kb) [x PV(kb-1)], or PV(kb-1) alone.
    auto step = [&](int kb_, auto do_s, auto do_pv, auto masked, auto half) {
        stage(kb_);
        if constexpr (decltype(do_pv)::value)
            apply_rescale();
        if constexpr (decltype(do_s)::value) {
            if constexpr (decltype(half)::value == kHalfDiag) {
                // the last tile's upper half is skipped when every row
                // lies below it; its scores are then -inf (P = 0)
                op_s(kb_, HLower{});
                if (hi_out && kb_ == kb_last) {
#pragma unroll
                    for (int rg = 0; rg < RG; rg++)
#pragma unroll
                        for (int i = 0; i < 16; i++)
                            s[rg][1][i] = kNegInf;
                    last_lower = true;
                } else {
                    op_s(kb_, HUpper{});
                }
                op_sm(kb_, do_pv, masked, HBoth{});
            } else {
                op_s(kb_, half);
                op_sm(kb_, do_pv, masked, half);
            }
        } else if constexpr (decltype(do_pv)::value) {
            pv_last(vidx(kb_ - 1));
        }
        dma_wait_barrier();
    };
    // Tiles needing the real-position mask: the causal diagonal (some key past
    // the wave's first row: kb > kb_c) and, for the local branch, the
    // window's left edge (some key at or before the last row's pos - w:
    // kb < kb_w).  The first is a suffix of the wave's tiles, the second a
    // prefix.
    const int kb_c = (wpmin + 1) / kBlockN - 1;
    int kb_w = kb_first;
    if (MODE == kModeLocal) {
        const int edge = wpmax - w + 1;            // keys below this are out for the last row
        if (edge > 0)
            kb_w = max(kb_w, (edge + kBlockN - 1) / kBlockN);
    }

    // Every wave walks all tiles of the workgroup's range (they share the
    // staging and the barriers) but computes only its own sub-range
    // kb_first..kb_last, in loops of a single mask kind each -- window edge,
    // unmasked middle (or both masks where edge and diagonal overlap),
    // diagonal -- so that no loop body switches between instantiations.
    int kb = kb_lo;
    bool pending = false;
    for (; kb < kb_first && kb <= kb_hi; kb++)
        step(kb, F_{}, F_{}, MNone{}, HBoth{});
    if (kb_first <= kb_last) {
        // the first tile computed has no PV of a previous tile
        const bool need_c = kb > kb_c, need_w = kb < kb_w;
        if (need_c && need_w) {
            if (MODE == kModeLocal && lo_out)
                step(kb, T_{}, F_{}, MBoth{}, HUpper{});
            else
                step(kb, T_{}, F_{}, MBoth{}, HBoth{});
        } else if (need_c) {
            step(kb, T_{}, F_{}, MCausal{}, HBoth{});
        } else if (need_w) {
            if (MODE == kModeLocal && lo_out)
                step(kb, T_{}, F_{}, MWindow{}, HUpper{});
            else
                step(kb, T_{}, F_{}, MWindow{}, HBoth{});
        } else {
            step(kb, T_{}, F_{}, MNone{}, HBoth{});
        }
        kb++;
        if (MODE == kModeLocal) {
            for (const int e = min(kb_last, min(kb_w - 1, kb_c)); kb <= e; kb++)
                step(kb, T_{}, T_{}, MWindow{}, HBoth{});
            for (const int e = min(kb_last, kb_w - 1); kb <= e; kb++)
                step(kb, T_{}, T_{}, MBoth{}, HBoth{});
        }
        for (const int e = min(kb_last, kb_c); kb <= e; kb++)
            step(kb, T_{}, T_{}, MNone{}, HBoth{});
        for (; kb <= kb_last; kb++)
            step(kb, T_{}, T_{}, MCausal{}, HDiag{});
        pending = true;
    }
    if (pending && kb <= kb_hi) {
        step(kb, F_{}, T_{}, MNone{}, HBoth{});
        pending = false;
        kb++;
    }
    for (; kb <= kb_hi; kb++)
        step(kb, F_{}, F_{}, MNone{}, HBoth{});
    const bool prefetched = prefetch();
    if (pending) {
        apply_rescale();
        pv_last(vidx(kb_hi));                // V(kb_hi) was staged by the last step
    }

    float l_tot[RG];
#pragma unroll
    for (int rg = 0; rg < RG; rg++)
        l_tot[rg] = pair_sum(l_run[rg]);
    if constexpr (MODE == kModeGlobal) {
        // a split entry: publish the partial, and the last of the tile's
        // entries to finish merges all of them and runs the epilogue
        if (uni(tile.nsplit) > 1 && !merge_split<D>(a, tile, u.hg, wave, lane, acc, m_ref, l_tot))
            return;
    }
#pragma unroll
    for (int rg = 0; rg < RG; rg++) {
        const float inv = 1.f / l_tot[rg];
        if (EPI != kEpiRaw && MODE != kModeDense) {
            // ContextNorm over the row's d values (this lane holds d/2 of them,
            // its partner l^32 the other half), the softmax's 1/l, the fusion
            // weight and the gain folded into one scale per element:
            // Norm(o) = acc * (1/l) / sqrt(mean((acc/l)^2) + eps).
            float ss = 0.f;
#pragma unroll
            for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                for (int i = 0; i < 16; i++)
                    ss = fmaf(acc[rg][cb][i], acc[rg][cb][i], ss);
            ss = pair_sum(ss);
            // the next item's loads have arrived before this item's stores
            // are issued (see above)
            if (rg == 0 && prefetched)
                __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            if (!(wave_valid && row_valid[rg]))
                continue;
            if constexpr (EPI == kEpiFusedTrain) {
                // training forward: also the raw branch output (fp32, token
                // rows for the local branch, rank rows for the global one) and
                // the row's base-2 log-sum-exp of the scaled scores
                if (g == 0)
                    a.lse[(int64_t)head * a.lse_stride + orow[rg]] =
                        (m_ref[rg] == kNegInf ? 0.f : m_ref[rg]) + log2f(l_tot[rg]);
                float *rp = (float *)a.out + (orow[rg] * a.hq + head) * (int64_t)D + g * 4;
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                    for (int qd = 0; qd < 4; qd++) {
                        const f32x4 v = {acc[rg][cb][qd * 4 + 0] * inv, acc[rg][cb][qd * 4 + 1] * inv,
                                         acc[rg][cb][qd * 4 + 2] * inv, acc[rg][cb][qd * 4 + 3] * inv};
                        *(f32x4 *)(rp + cb * 32 + qd * 8) = v;
                    }
            }
            const float rn = 1.f / sqrtf(ss * inv * inv / (float)D + a.eps);
            const int64_t tok = qtok[rg];
            const float p = ep_gate[rg];
            const int r = ep_rank[rg];
            const float *gain = kGT ? a.gain_g : a.gain;
            const float *gp = gain ? gain + head * D + g * 4 : nullptr;
            // selected token in the local branch: keep (1-p) Norm^L in fp32
            const bool keep = MODE == kModeLocal && r >= 0;
            const float wgt = (MODE == kModeGlobal) ? p : (keep ? 1.f - p : 1.f);
            const float scale = inv * rn * wgt;
            auto scaled = [&](int cb, int qd) {
                f32x4 v = {acc[rg][cb][qd * 4 + 0], acc[rg][cb][qd * 4 + 1],
                           acc[rg][cb][qd * 4 + 2], acc[rg][cb][qd * 4 + 3]};
                v *= scale;
                if (gp)
                    v *= *(const f32x4 *)(gp + cb * 32 + qd * 8);
                return v;
            };
            if (keep) {
                float *lp = a.lc + ((int64_t)r * a.hq + head) * D + g * 4;
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                    for (int qd = 0; qd < 4; qd++)
                        *(f32x4 *)(lp + cb * 32 + qd * 8) = scaled(cb, qd);
                continue;
            }
            if constexpr (EPI == kEpiLayer && MODE == kModeGlobal) {
                // one-launch layer: p Norm^G to the compact buffer; the local
                // branch's part may not exist yet, a later pass adds them
                float *cp = a.gc + ((int64_t)r * a.hq + head) * D + g * 4;
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                    for (int qd = 0; qd < 4; qd++)
                        *(f32x4 *)(cp + cb * 32 + qd * 8) = scaled(cb, qd);
                continue;
            }
            const float *lp = (MODE == kModeGlobal)
                                  ? a.lc + ((int64_t)r * a.hq + head) * D + g * 4 : nullptr;
            uint16_t *op = a.out_bf16 + (tok * a.hq + head) * (int64_t)D + g * 4;
#pragma unroll
            for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                for (int qd = 0; qd < 4; qd++) {
                    f32x4 v = scaled(cb, qd);
                    if (MODE == kModeGlobal)
                        v += *(const f32x4 *)(lp + cb * 32 + qd * 8);
                    u32x2 o;
                    o.x = pack_bf16x2(v.x, v.y);
                    o.y = pack_bf16x2(v.z, v.w);
                    if constexpr (STG > 0)
                        *(u32x2 *)&sm.ostage[wave][m][cb * 32 + qd * 8 + g * 4] = o;
                    else
                        *(u32x2 *)(op + cb * 32 + qd * 8) = o;
                }
            continue;
        }
        if (!(wave_valid && row_valid[rg]))
            continue;
        // training forward: the row's base-2 log-sum-exp of the scaled
        // scores, log2(sum_j 2^(c s_j)) = m + log2(l)
        if (a.lse && g == 0)
            a.lse[(int64_t)head * a.lse_stride + orow[rg]] =
                (m_ref[rg] == kNegInf ? 0.f : m_ref[rg]) + log2f(l_tot[rg]);
        if (MODE == kModeDense) {
            uint16_t *op = (uint16_t *)a.out + (orow[rg] * a.hq + head) * (int64_t)D + g * 4;
#pragma unroll
            for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                for (int qd = 0; qd < 4; qd++) {
                    u32x2 v;
                    v.x = pack_bf16x2(acc[rg][cb][qd * 4 + 0] * inv, acc[rg][cb][qd * 4 + 1] * inv);
                    v.y = pack_bf16x2(acc[rg][cb][qd * 4 + 2] * inv, acc[rg][cb][qd * 4 + 3] * inv);
                    *(u32x2 *)(op + cb * 32 + qd * 8) = v;
                }
        } else {
            float *op = (float *)a.out + (orow[rg] * a.hq + head) * (int64_t)D + g * 4;
#pragma unroll
            for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
                for (int qd = 0; qd < 4; qd++) {
                    f32x4 v = {acc[rg][cb][qd * 4 + 0] * inv, acc[rg][cb][qd * 4 + 1] * inv,
                               acc[rg][cb][qd * 4 + 2] * inv, acc[rg][cb][qd * 4 + 3] * inv};
                    *(f32x4 *)(op + cb * 32 + qd * 8) = v;
                }
        }
    }
    if constexpr (STG > 0 && EPI != kEpiRaw && MODE == kModeLocal) {
        // The wave's unselected rows, staged in LDS above (row m at
        // ostage[wave][m]), go out as 16-byte chunks in row order: every
        // store instruction writes 64 lanes x 16 B = whole head slices of
        // 128 / D rows, instead of 16 B in each of 32 rows.  Rows are
        // consecutive tokens (local mode); selected and invalid rows were
        // written elsewhere or not at all and are skipped.
        static_assert(RG == 1, "one row group per wave");
        const bool staged = wave_valid && row_valid[0] && ep_rank[0] < 0;
        const uint32_t smask = (uint32_t)__builtin_amdgcn_ballot_w64(staged && g == 0);
        constexpr int kChunksPerRow = D / 8, kRowsPerStore = 64 / kChunksPerRow;
        // The lane's row and chunk of the first store come from an opaque
        // copy of the lane index, so that the compiler keeps one pointer live
        // instead of hoisting a row index and mask per store out of the
        // persistent item loop (which made the kernel spill).
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int r0 = ln / kChunksPerRow, c8 = (ln % kChunksPerRow) * 8;
        const uint16_t *src = &sm.ostage[wave][r0][c8];
        uint16_t *dst = a.out_bf16 + ((base + wpmin + r0) * a.hq + head) * (int64_t)D + c8;
        const int64_t dstep = (int64_t)kRowsPerStore * a.hq * D;
        const uint32_t lmask = smask >> r0;
#pragma unroll
        for (int i = 0; i < kRowsPerWave / kRowsPerStore; i++) {
            if ((lmask >> (i * kRowsPerStore)) & 1u) {
                const u32x4 v = *(const u32x4 *)(src + i * kRowsPerStore * (D + kStagePad));
                *(u32x4 *)(dst + i * dstep) = v;
            }
        }
    }
}

template <int D, int MODE, int EPI, int W>
__global__ __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(2)))
void attn_kernel(const AttnArgs a) {
    constexpr int STG = stage_waves<MODE, W>();
    __shared__ Smem<D, STG> sm;
    auto no_prefetch = [] { return false; };
    if (MODE == kModeGlobal) {
        // Persistent workgroups pull (tile, head group) items from the queue
        // of their XCD (workgroups are dispatched round-robin over the 8
        // XCDs): queue x holds items x, x+8, x+16, ...  Items are in
        // longest-first order, and items that share a KV head tend to share
        // an XCD and its L2.  Once its own queue is empty a workgroup takes
        // what is left in the other queues (in XCD order), so no XCD idles
        // while another has work.  Wave 0 reads the 8 queue counters at once
        // and takes an item from the first queue that still has one; an
        // index past the end means that queue has just emptied, and the
        // counters only grow, so each retry closes a queue: a workgroup
        // exits after at most 8 empty takes (the loop allows 17), and at
        // once when there is no entry at all.
        __shared__ int s_item;
        const int x0 = blockIdx.x % kQueues;
        const int n_entries = a.queue[0];
        if (n_entries == 0)
            return;
        const int n_items = n_entries * a.n_hg;
        const int lane = threadIdx.x & 63;
        // this lane's queue (lanes 0..7) and its length
        const int xl = (x0 + lane) % kQueues;
        const int len_l = (n_items - xl + kQueues - 1) / kQueues;
        for (;;) {
            if (threadIdx.x < 64) {
                int item = -1;
                for (int tries = 0; tries <= 2 * kQueues; tries++) {
                    const int c = lane < kQueues
                                      ? __hip_atomic_load(&a.queue[1 + xl], __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_AGENT)
                                      : 0;
                    const uint64_t open =
                        __builtin_amdgcn_ballot_w64(lane < kQueues && c < len_l);
                    if (open == 0)
                        break;
                    const int f = __builtin_ctzll(open);
                    const int x = (x0 + f) % kQueues;
                    int got = 0;
                    if (lane == f)
                        got = x + kQueues * atomicAdd(&a.queue[1 + x], 1);
                    got = __builtin_amdgcn_readlane(got, f);
                    if (got < n_items) {
                        item = got;
                        break;
                    }
                }
                if (lane == 0)
                    s_item = item;
            }
            // (these barriers also end every read of the previous item's
            // K / V tiles before the next item's first K tile load)
            __syncthreads();
            const int item = __builtin_amdgcn_readfirstlane(s_item);
            __syncthreads();
            if (item < 0)
                break;
            const SparseTile t = a.tiles[item / a.n_hg];
            ItemU u;
            ItemL l;
            bf16x8 qf[RG][D / 16];
            item_begin<D, MODE, EPI>(a, t.seq, item % a.n_hg, 0, t, u, l, qf);
            item_first_k<D, MODE, EPI, W, STG>(a, sm, u);
            attend_item<D, MODE, EPI, W, STG>(a, sm, u, l, qf, false, no_prefetch);
        }
    } else if (MODE == kModeLocal) {
        const int wid = blockIdx.x;
        if constexpr (EPI != kEpiRaw) {
            // The fused layer's local launch: after the item_stride
            // persistent workgroups come one that builds the global branch's
            // work table (its LDS holds the table) and, for a global branch
            // with an LP query transform, one per head that writes the
            // permuted copy of its matrix.  Being last, they take CUs that
            // the first workgroups to finish leave free, and no item
            // workgroup waits for them.
            if (wid >= a.item_stride) {
                int x = wid - a.item_stride;
                if (a.plan_wg) {
                    if (x == 0) {
                        constexpr int E = D == 128 ? 512 : 256;
                        static_assert(sizeof(plan_detail::PlanLds<E>) <= sizeof(Smem<D, STG>),
                                      "plan table must fit in the K/V staging buffers");
                        build_plan<W * 64, E>(a.cu_seqlens, a.num_seqs, a.plan,
                                              *reinterpret_cast<plan_detail::PlanLds<E> *>(&sm));
                        return;
                    }
                    x -= 1;
                }
                if (x < a.prep_wgs)
                    permute_lp_head<D, W * 64>(a.prep_a, a.aperm, x);
                return;
            }
        }
        // Persistent workgroups: items wid, wid + stride, ...  Item i is head
        // group i % n_hg of token tile i / n_hg, the sequences' tiles back to
        // back (so no workgroup of a ragged batch idles); the valid items are
        // a prefix, so the first invalid one ends the loop.
        auto decode = [&](int item, int &b, int &hg, int &jt) {
            if (item >= a.n_items)
                return false;
            hg = item % a.n_hg;
            int rest = item / a.n_hg;
            for (b = 0; b < a.num_seqs; b++) {
                const int nt = (a.cu_seqlens[b + 1] - a.cu_seqlens[b] + a.tpw - 1) / a.tpw;
                if (rest < nt)
                    break;
                rest -= nt;
            }
            jt = rest;
            return b < a.num_seqs;
        };
        int item = wid, b = 0, hg = 0, jt = 0;
        if (!decode(item, b, hg, jt))
            return;
        ItemU u;
        ItemL l;
        bf16x8 qf[RG][D / 16];
        item_begin<D, MODE, EPI>(a, b, hg, jt, SparseTile{}, u, l, qf);
        item_first_k<D, MODE, EPI, W, STG>(a, sm, u);
        bool waited = false;
        for (;;) {
            // The next item's Q, epilogue inputs and first K tile are loaded
            // while this item finishes its last PV product and epilogue.
            const int next = item + a.item_stride;
            int nb = 0, nhg = 0, njt = 0;
            const bool has_next = decode(next, nb, nhg, njt);
            ItemU nu;
            ItemL nl;
            attend_item<D, MODE, EPI, W, STG>(a, sm, u, l, qf, waited, [&] {
                if (has_next) {
                    item_begin<D, MODE, EPI>(a, nb, nhg, njt, SparseTile{}, nu, nl, qf);
                    item_first_k<D, MODE, EPI, W, STG>(a, sm, nu);
                }
                return has_next;
            });
            if (!has_next)
                break;
            waited = true;
            u = nu;
            l = nl;
            item = next;
        }
    } else {
        const int bid = blockIdx.x;
        const int hg = bid % a.n_hg;
        const int rest = bid / a.n_hg;
        const int b = rest % a.num_seqs;
        const int jt = a.ntile_max - 1 - rest / a.num_seqs;       // longest rows first
        const int T = a.cu_seqlens[b + 1] - a.cu_seqlens[b];
        if (jt * a.tpw >= T)
            return;
        ItemU u;
        ItemL l;
        bf16x8 qf[RG][D / 16];
        item_begin<D, MODE, EPI>(a, b, hg, jt, SparseTile{}, u, l, qf);
        item_first_k<D, MODE, EPI, W, STG>(a, sm, u);
        attend_item<D, MODE, EPI, W, STG>(a, sm, u, l, qf, false, no_prefetch);
    }
}

// One item from per-XCD queues: queue x holds items x, x + 8, ... below
// n_items and ctr[x] counts the takes from it.  The caller's own queue x0
// first, then the others in XCD order; an index past the end means that
// queue has just emptied, and the counters only grow, so each retry closes a
// queue.  Called by all lanes of one wave; returns the item (wave-uniform) or
// -1 once every queue is empty.
__device__ __forceinline__ int queue_take(int32_t *ctr, int n_items, int x0) {
    const int lane = threadIdx.x & 63;
    const int xl = (x0 + lane) % kQueues;
    const int len_l = (n_items - xl + kQueues - 1) / kQueues;
    for (int tries = 0; tries <= 2 * kQueues; tries++) {
        const int c = lane < kQueues
                          ? __hip_atomic_load(&ctr[xl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                          : 0;
        const uint64_t open = __builtin_amdgcn_ballot_w64(lane < kQueues && c < len_l);
        if (open == 0)
            return -1;
        const int f = __builtin_ctzll(open);
        const int x = (x0 + f) % kQueues;
        int got = 0;
        if (lane == f)
            got = x + kQueues * atomicAdd(&ctr[x], 1);
        got = __builtin_amdgcn_readlane(got, f);
        if (got < n_items)
            return got;
    }
    return -1;
}

// A work-table entry written during the same launch by another workgroup:
// device-scope loads, which read the entry where the writer's release put it
// and not a stale cached copy.
__device__ __forceinline__ SparseTile load_tile_coherent(const SparseTile *p) {
    const int32_t *w = reinterpret_cast<const int32_t *>(p);
    auto ld = [&](int i) {
        return __hip_atomic_load(w + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    SparseTile t;
    t.first = ld(0);
    t.nrows = ld(1);
    t.seq = ld(2);
    t.pos_max = ld(3);
    t.kb_begin = ld(4);
    t.kb_end = ld(5);
    t.split = ld(6);
    t.nsplit = ld(7);
    t.sid = ld(8);
    t.pad[0] = t.pad[1] = t.pad[2] = 0;
    return t;
}

// Items left in a local queue below which a workgroup takes its next item
// only when it needs it (the 32 or 64 workgroups of an XCD share its queue;
// switching three items per workgroup before the end measured best).
constexpr int kLateClaimItems = 96;
// Bound of the wait for the work table (s_sleep 8 = 512 cycles per poll:
// ~2 s), so that no workgroup can wait for ever.
constexpr int kPlanSpinMax = 1 << 23;

// The layer's two branches in one persistent launch, when both use W-wave
// workgroups with the same tiles: W = 8 (one per CU) for Hq / Hkv a multiple
// of 4, W = 4 (two per CU) for one query head per KV head.  The local branch's items are short and
// many (every token tile x head group, ~17 KV steps at w = 1024), the global
// branch's few and long (a tile's whole causal prefix), so running them one
// launch after the other leaves the GPU partly idle at each launch's end
// (the workgroups of the global launch end ~10% apart: its long items and the
// XCDs' different speeds).  Here every workgroup takes global items first,
// longest first, and then local items until none is left, so the short local
// items fill in behind the long ones:
//   A. workgroup 0 builds the global work table (and the permuted LP
//      matrices of an LP query transform) and releases it with a flag; every
//      other workgroup meanwhile runs one local item, then waits for the
//      flag.
//   B. global items from the per-XCD queues of the table (longest first,
//      stealing once the own queue is empty), epilogue kEpiLayer: p Norm^G
//      of each selected row to the compact buffer gc.
//   C. local items from per-XCD queues (queue x: items x, x + 8, ..., i.e.
//      the head groups of one XCD share KV heads), the next item's loads
//      issued after the current item's last K / V step as in the local
//      launch; the next item is claimed from the own queue when the current
//      one starts (the atomic's reply has arrived by the prefetch), except
//      near the queue's end, where it is taken at the prefetch so that no
//      workgroup holds an item it cannot start yet while others run dry.
// Selected rows get (1-p) Norm^L in lc from their local item and p Norm^G in
// gc from their global item, in either order; launch_sel_sum then writes
// their output rows.
template <int D, int W>
__global__ __launch_bounds__(W * 64) __attribute__((amdgpu_waves_per_eu(2)))
void layer_kernel(const AttnArgs a) {
    constexpr int STG = stage_waves<kModeLocal, W>();
    __shared__ Smem<D, STG> sm;
    __shared__ int s_item, s_entries;
    const int tid = threadIdx.x, lane = tid & 63;
    const int x0 = blockIdx.x % kQueues;
    int32_t *const lq = a.ctl + 1;
    auto no_prefetch = [] { return false; };
    // Local item -> (sequence, head group, token tile); false past the last
    // valid item (items are head group fastest, then the sequences' token
    // tiles back to back; n_items may exceed the valid ones).
    auto decode = [&](int item, int &b, int &hg, int &jt) {
        if (item < 0 || item >= a.n_items)
            return false;
        hg = item % a.n_hg;
        int rest = item / a.n_hg;
        for (b = 0; b < a.num_seqs; b++) {
            const int nt = (a.cu_seqlens[b + 1] - a.cu_seqlens[b] + a.tpw - 1) / a.tpw;
            if (rest < nt)
                break;
            rest -= nt;
        }
        jt = rest;
        return b < a.num_seqs;
    };
    // wave 0 takes an item, the workgroup learns it (the second barrier ends
    // every wave's read before s_item is written again)
    auto take_wg = [&](int32_t *ctr, int n) {
        if (tid < 64) {
            const int it = queue_take(ctr, n, x0);
            if (lane == 0)
                s_item = it;
        }
        __syncthreads();
        const int it = __builtin_amdgcn_readfirstlane(s_item);
        __syncthreads();
        return it;
    };
    // the next valid local item (any queue), or -1
    auto take_local = [&](int &b, int &hg, int &jt) {
        int it;
        do {
            it = take_wg(lq, a.n_items);
        } while (it >= 0 && !decode(it, b, hg, jt));
        return it;
    };

    // With two workgroups per CU (W = 4) the second half of the grid starts
    // with local items, so that a CU runs a (memory-bound) global item and a
    // (compute-bound) local item side by side rather than two of one kind.
    bool local_first = false;
    if constexpr (W == 4)
        local_first = blockIdx.x >= gridDim.x / 2;

    // A. the work table, or one local item while it is built
    if (blockIdx.x == 0) {
        constexpr int E = D == 128 ? 512 : 256;
        static_assert(sizeof(plan_detail::PlanLds<E>) <= sizeof(Smem<D, STG>),
                      "plan table must fit in the staging buffers");
        build_plan<W * 64, E>(a.cu_seqlens, a.num_seqs, a.plan,
                              *reinterpret_cast<plan_detail::PlanLds<E> *>(&sm));
        for (int h = 0; h < a.prep_wgs; h++)
            permute_lp_head<D, W * 64>(a.prep_a, a.aperm, h);
        // every wave's stores written back to where other XCDs read them,
        // then the flag
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __syncthreads();
        if (tid == 0)
            __hip_atomic_store(&a.ctl[0], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else if (!local_first) {
        int b = 0, hg = 0, jt = 0;
        if (take_local(b, hg, jt) >= 0) {
            ItemU u;
            ItemL l;
            bf16x8 qf[RG][D / 16];
            item_begin<D, kModeLocal, kEpiLayer>(a, b, hg, jt, SparseTile{}, u, l, qf);
            item_first_k<D, kModeLocal, kEpiLayer, W, STG>(a, sm, u);
            attend_item<D, kModeLocal, kEpiLayer, W, STG>(a, sm, u, l, qf, false, no_prefetch);
        }
    }

    // B. global items, once the table is there
    auto global_phase = [&] {
        if (tid == 0) {
            // (no table after the bound: the global items are skipped)
            bool ready = false;
            for (int n = 0; n < kPlanSpinMax && !ready; n++) {
                ready = __hip_atomic_load(&a.ctl[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
                if (!ready)
                    __builtin_amdgcn_s_sleep(8);
            }
            s_entries = ready ? __hip_atomic_load(&a.queue[0], __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT)
                              : 0;
        }
        __syncthreads();
        const int n_entries = __builtin_amdgcn_readfirstlane(s_entries);
        if (n_entries <= 0)
            return;
        const int n_gitems = n_entries * a.n_hg;
        for (;;) {
            const int item = take_wg(a.queue + 1, n_gitems);
            if (item < 0)
                break;
            const SparseTile t = load_tile_coherent(a.tiles + item / a.n_hg);
            ItemU u;
            ItemL l;
            bf16x8 qf[RG][D / 16];
            item_begin<D, kModeGlobal, kEpiLayer>(a, t.seq, item % a.n_hg, 0, t, u, l, qf);
            item_first_k<D, kModeGlobal, kEpiLayer, W, STG>(a, sm, u);
            attend_item<D, kModeGlobal, kEpiLayer, W, STG>(a, sm, u, l, qf, false, no_prefetch);
        }
    };
    // C. local items
    auto local_phase = [&] {
        int b = 0, hg = 0, jt = 0;
        if (take_local(b, hg, jt) < 0)
            return;
        ItemU u;
        ItemL l;
        bf16x8 qf[RG][D / 16];
        item_begin<D, kModeLocal, kEpiLayer>(a, b, hg, jt, SparseTile{}, u, l, qf);
        item_first_k<D, kModeLocal, kEpiLayer, W, STG>(a, sm, u);
        bool waited = false;
        // Claim of the next item from the own queue, issued when an item
        // starts and resolved at its prefetch, so that the atomic's reply
        // has arrived by then; once the own queue's remaining items are fewer
        // than kLateClaimItems, the next item is taken only at the prefetch
        // instead, so that no workgroup holds an item it cannot start yet
        // while the queues run dry.
        bool early = true;
        for (;;) {
            int claim = 0;
            if (early && tid == 0)
                claim = atomicAdd(&lq[x0], 1);
            ItemU nu;
            ItemL nl;
            int nxt = -1;
            attend_item<D, kModeLocal, kEpiLayer, W, STG>(a, sm, u, l, qf, waited, [&] {
                if (tid < 64) {
                    int nb, nhg, njt;
                    int it = early ? x0 + kQueues * __builtin_amdgcn_readfirstlane(claim) : -1;
                    if (!decode(it, nb, nhg, njt)) {
                        do {
                            it = queue_take(lq, a.n_items, x0);
                        } while (it >= 0 && !decode(it, nb, nhg, njt));
                    }
                    if (lane == 0)
                        s_item = it;
                }
                // s_item is written again only at the next item's prefetch,
                // after that item's barriers, or by take_wg after a barrier
                __syncthreads();
                nxt = __builtin_amdgcn_readfirstlane(s_item);
                if (nxt < 0)
                    return false;
                early = nxt + kQueues * kLateClaimItems < a.n_items;
                int nb = 0, nhg = 0, njt = 0;
                decode(nxt, nb, nhg, njt);
                item_begin<D, kModeLocal, kEpiLayer>(a, nb, nhg, njt, SparseTile{}, nu, nl, qf);
                item_first_k<D, kModeLocal, kEpiLayer, W, STG>(a, sm, nu);
                return true;
            });
            if (nxt < 0)
                break;
            waited = true;
            u = nu;
            l = nl;
        }
    };
    if (local_first) {
        local_phase();
        global_phase();
    } else {
        global_phase();
        local_phase();
    }
}

template <int D>
hipError_t launch_layer_d(int waves, const AttnArgs &a, int grid, hipStream_t s) {
    if (waves == 8)
        hipLaunchKernelGGL((layer_kernel<D, 8>), dim3(grid), dim3(512), 0, s, a);
    else
        hipLaunchKernelGGL((layer_kernel<D, 4>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int D>
int layer_blocks_per_cu_d(int waves) {
    int n = 0;
    const hipError_t e =
        waves == 8 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, layer_kernel<D, 8>, 512, 0)
                   : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, layer_kernel<D, 4>, 256, 0);
    if (e != hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}

template <int D, int MODE, int EPI, int W>
hipError_t launch_one(const AttnArgs &a, int grid, hipStream_t s) {
    hipLaunchKernelGGL((attn_kernel<D, MODE, EPI, W>), dim3(grid), dim3(W * 64), 0, s, a);
    return hipGetLastError();
}

template <int D, int MODE, int W>
int blocks_per_cu_one() {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, attn_kernel<D, MODE, kEpiRaw, W>, W * 64,
                                                     0) != hipSuccess)
        return 1;
    return n > 0 ? n : 1;
}

template <int D, int MODE, int W>
hipError_t launch_epi(int epi, const AttnArgs &a, int grid, hipStream_t s) {
    return epi == kEpiFused        ? launch_one<D, MODE, kEpiFused, W>(a, grid, s)
           : epi == kEpiFusedTrain ? launch_one<D, MODE, kEpiFusedTrain, W>(a, grid, s)
                                   : launch_one<D, MODE, kEpiRaw, W>(a, grid, s);
}

template <int D>
hipError_t launch_d(int mode, int epi, int waves, const AttnArgs &a, int grid, hipStream_t s) {
    if (mode == kModeLocal)
        return waves == 8 ? launch_epi<D, kModeLocal, 8>(epi, a, grid, s)
                          : launch_epi<D, kModeLocal, kWavesLocal>(epi, a, grid, s);
    if (mode == kModeGlobal)
        return waves == 8 ? launch_epi<D, kModeGlobal, kWavesGlobal>(epi, a, grid, s)
                          : launch_epi<D, kModeGlobal, kWavesLocal>(epi, a, grid, s);
    return launch_one<D, kModeDense, kEpiRaw, kWavesGlobal>(a, grid, s);
}

template <int D>
int blocks_per_cu_d(int mode, int waves) {
    if (mode == kModeLocal)
        return waves == 8 ? blocks_per_cu_one<D, kModeLocal, 8>()
                          : blocks_per_cu_one<D, kModeLocal, kWavesLocal>();
    if (mode == kModeGlobal)
        return waves == 8 ? blocks_per_cu_one<D, kModeGlobal, kWavesGlobal>()
                          : blocks_per_cu_one<D, kModeGlobal, kWavesLocal>();
    return blocks_per_cu_one<D, kModeDense, kWavesGlobal>();
}

}  // namespace

hipError_t launch_attention(int mode, int epi, int head_dim, int waves, const AttnArgs &a,
                            int grid, hipStream_t s) {
    if (grid <= 0)
        return hipSuccess;
    return head_dim == 128 ? launch_d<128>(mode, epi, waves, a, grid, s)
                           : launch_d<64>(mode, epi, waves, a, grid, s);
}

int attention_blocks_per_cu(int mode, int head_dim, int waves) {
    return head_dim == 128 ? blocks_per_cu_d<128>(mode, waves) : blocks_per_cu_d<64>(mode, waves);
}

hipError_t launch_layer(int head_dim, int waves, const AttnArgs &a, int grid, hipStream_t s) {
    if (grid <= 0)
        return hipSuccess;
    return head_dim == 128 ? launch_layer_d<128>(waves, a, grid, s)
                           : launch_layer_d<64>(waves, a, grid, s);
}

int layer_blocks_per_cu(int head_dim, int waves) {
    return head_dim == 128 ? layer_blocks_per_cu_d<128>(waves) : layer_blocks_per_cu_d<64>(waves);
}

}  // namespace logo
