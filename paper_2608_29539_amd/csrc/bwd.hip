// bwd.hip -- backward pass of the layer with the selection held fixed
// (App. B, backward traversal of the query-sparse global branch; the chain
// rule through Eqs. contextnorm, output-fusion and branch-attention):
//
//   fusion_bwd_kernel  ContextNorm + fusion backward per (token, head): the
//                      gradients of the raw branch outputs dO^L, dO^G (bf16,
//                      the operand of the attention backward), the row sums
//                      Delta = dO . O, each row's term of dL/dp, partial gain
//                      gradients, and a compact copy of the selected rows of
//                      Q^G (so the global branch's query tiles are contiguous).
//   gate_grad_kernel   dL/dp_t = sum over heads of the row terms.
//   gain_grad_kernel   column sums of the gain-gradient partials.
//   bwd_dq_kernel      dQ of one branch.  Rows: local = every token (keys of
//                      its window), global = the selected rows in rank order
//                      (keys 0..pos).  Lane = query: S^T = K Q^T and
//                      dP^T = V dO^T with Q, dO in registers, then
//                      dQ^T += K^T dS^T with K^T read transposed from LDS.
//   bwd_dkv_kernel     dK, dV of one branch over dense KV blocks.  Lane = key:
//                      S = Q K^T, dP = dO V^T with K, V in registers, then
//                      dV^T += dO^T P and dK^T += Q^T dS with dO^T, Q^T read
//                      transposed from LDS.  A KV block of the global branch
//                      starts at the first compacted query row that can see
//                      it (binary search of sel_idx), so its loop covers only
//                      rows at or after the block, and only the first one or
//                      two query tiles need the causal mask.
//
// Softmax recomputation: P = 2^(c s - lse) with c = scale log2(e) and lse
// the forward's base-2 log-sum-exp; dS = P (dP - Delta).  P and dS are
// rounded to bf16 for the MFMAs, accumulation is fp32, and the outputs are
// fp32 (dQ, dK scaled by the softmax scale at the end).
//
// LDS tile layout (Q, dO, K, V tiles of 64 rows x d bf16, unpadded): the
// 16-byte chunk j of row r is stored at chunk j ^ swz(r).  The swizzle makes
// both access patterns conflict-free: the fragment reads (16 lanes read 16
// consecutive rows, one chunk each) and the transpose reads (32 lanes read
// 4 consecutive rows, 64 contiguous bytes each).
#include "logo_internal.h"
#include "attn_common.h"

#include <type_traits>

namespace logo {
namespace {

constexpr int kBwdWaves = 4;
constexpr int kTileRows = 64;   // rows of a staged tile (keys or queries)

template <int D>
__device__ __forceinline__ constexpr int swz(int r) {
    return D == 128 ? (((r & 3) << 2) | ((r >> 2) & 3))
                    : ((((r >> 1) & 1) << 2) | ((r >> 2) & 3));
}
// Byte offset of element col (a multiple of 4) of row r in a swizzled tile.
template <int D>
__device__ __forceinline__ int swz_off(int r, int col) {
    return r * D * 2 + (((col >> 3) ^ swz<D>(r)) << 4) + (col & 7) * 2;
}

// Global -> LDS staging of one swizzled 64-row tile by the 4 waves: LDS slot
// s (16 bytes) holds chunk (s % C) ^ swz(row) of row s / C, C = d / 8.  The
// per-lane byte offsets inside a tile are fixed and computed once.
template <int D>
struct TileDma {
    static constexpr int kInst = kTileRows * (D / 8) / 64;
    static constexpr int kPerWave = kInst / kBwdWaves;
    int voff[kPerWave];
};
template <int D>
__device__ __forceinline__ void tile_dma_plan(TileDma<D> &d, int wave, int lane, int row_bytes) {
#pragma unroll
    for (int i = 0; i < TileDma<D>::kPerWave; i++) {
        const int slot = (i * kBwdWaves + wave) * 64 + lane;
        const int row = slot / (D / 8), p = slot % (D / 8);
        d.voff[i] = row * row_bytes + ((p ^ swz<D>(row)) << 4);
    }
}
template <int D>
__device__ __forceinline__ void tile_dma(void *dst, const TileDma<D> &d, u32x4 r, int wave) {
#pragma unroll
    for (int i = 0; i < TileDma<D>::kPerWave; i++)
        lds_load16(r, (char *)dst + (i * kBwdWaves + wave) * 1024, d.voff[i]);
}

// Per-lane LDS offsets of the two fragment kinds inside a tile:
//   row: A/B operand rows  (row m = lane % 32, columns 16 ss + 8 g .. +7)
//   tr : transposed operand, column block cb, first / second read (rows
//        4 g + (lane % 16) / 4 and 8 further)
template <int D>
struct FragOffsets {
    int row[D / 16];
    int tr0[D / 32], tr1[D / 32];
};
template <int D>
__device__ __forceinline__ void frag_offsets(FragOffsets<D> &o, int lane) {
    const int m = lane & 31, g = lane >> 5;
#pragma unroll
    for (int ss = 0; ss < D / 16; ss++)
        o.row[ss] = swz_off<D>(m, ss * 16 + g * 8);
    const int tr_row = 4 * g + ((lane & 15) >> 2);
    const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++) {
        o.tr0[cb] = swz_off<D>(tr_row, cb * 32 + tr_col);
        o.tr1[cb] = swz_off<D>(tr_row + 8, cb * 32 + tr_col);
    }
}
__device__ __forceinline__ bf16x8 frag_at(const char *tile, int off) {
    return *(const bf16x8 *)(tile + off);
}
// Transposed fragment of rows row0 .. row0+15 (row0 a multiple of 16),
// column block cb: lane l holds column 32 cb + l % 32 of rows
// row0 + 4 g + 0..3 and row0 + 8 + 4 g + 0..3 -- the order in which an
// accumulator's lane holds those rows.
template <int D>
__device__ __forceinline__ bf16x8 frag_tr(const char *tile, const FragOffsets<D> &o, int row0,
                                          int cb) {
    const char *t = tile + row0 * D * 2;
    return lds_tr_pair(t + o.tr0[cb], t + o.tr1[cb]);
}

__device__ __forceinline__ bf16x8 pack8(const bf16x2 (&w)[8], int half) {
    bf16x8 f;
#pragma unroll
    for (int j = 0; j < 4; j++) {
        f[2 * j] = w[half * 4 + j][0];
        f[2 * j + 1] = w[half * 4 + j][1];
    }
    return f;
}

// ---------------------------------------------------------------------------
// dQ
// ---------------------------------------------------------------------------
template <int D, int MODE>
__global__ __launch_bounds__(kBwdWaves * 64) __attribute__((amdgpu_waves_per_eu(2)))
void bwd_dq_kernel(const BwdArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sk[2][kTileRows * D];
    __shared__ __attribute__((aligned(16))) uint16_t sv[2][kTileRows * D];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int g = lane >> 5, m = lane & 31;
    const int bid = blockIdx.x;
    const int hg = bid % a.n_hg, rest = bid / a.n_hg;
    const int b = uni(rest % a.num_seqs);
    const int jt = a.ntile_max - 1 - rest / a.num_seqs;     // longest rows first
    const int base = uni(a.cu_seqlens[b]);
    const int T = uni(a.cu_seqlens[b + 1] - base);
    int row0 = base, nrows = T;
    if (MODE == kModeGlobal) {
        row0 = uni(a.cu_sel[b]);
        nrows = uni(max(0, min(a.cu_sel[b + 1], a.cap) - row0));
    }
    const int t0 = jt * a.tpw;
    if (t0 >= nrows)
        return;
    const int nvalid = min(a.tpw, nrows - t0);
    const int hw = wave % a.hpw, tb = wave / a.hpw;
    const int head = hg * a.hpw + hw;
    const int kvh = (hg * a.hpw) / a.group;
    auto pos_of = [&](int r) { return (MODE == kModeGlobal ? a.sel_idx[r] : r) - base; };
    const int ri = tb * 32 + m;
    const bool valid = ri < nvalid;
    const int r = row0 + t0 + (valid ? ri : nvalid - 1);
    const int pos = pos_of(r);
    const bool wave_valid = tb * 32 < nvalid;
    const int wpmin = __builtin_amdgcn_readfirstlane(pos);
    const int wpmax = __builtin_amdgcn_readlane(pos, 31);
    const int wg_pmin = uni(pos_of(row0 + t0));
    const int wg_pmax = uni(pos_of(row0 + t0 + nvalid - 1));

    bf16x8 qf[D / 16], dof[D / 16];
    {
        const int64_t off = ((int64_t)r * a.hq + head) * D + g * 8;
#pragma unroll
        for (int ss = 0; ss < D / 16; ss++) {
            qf[ss] = *(const bf16x8 *)(a.q + off + ss * 16);
            dof[ss] = *(const bf16x8 *)(a.dout + off + ss * 16);
        }
    }
    const float lse = a.lse[(int64_t)head * a.row_stride + r];
    const float dlt = a.delta[(int64_t)head * a.row_stride + r];
    const float c = a.scale_log2;

    const int w = a.window;
    const int lo = (MODE == kModeLocal) ? max(0, wg_pmin - w + 1) : 0;
    const int kb_lo = lo / kTileRows, kb_hi = wg_pmax / kTileRows;
    int kb_first = kb_lo, kb_last = min(wpmax / kTileRows, kb_hi);
    if (MODE == kModeLocal)
        kb_first = max(kb_lo, max(0, wpmin - w + 1) / kTileRows);
    if (!wave_valid) {
        kb_first = kb_hi + 1;
        kb_last = kb_hi;
    }
    // tiles that need the real-position mask: past the causal edge of the
    // wave's first row, or (local) before the window edge of its last row
    const int kb_c = (wpmin + 1) / kTileRows - 1;
    int kb_w = kb_first;
    if (MODE == kModeLocal && wpmax - w + 1 > 0)
        kb_w = max(kb_w, (wpmax - w + 1 + kTileRows - 1) / kTileRows);

    const int row_bytes = a.hkv * D * 2;
    const uint16_t *kbase = a.k + ((int64_t)base * a.hkv + kvh) * D;
    const uint16_t *vbase = a.v + ((int64_t)base * a.hkv + kvh) * D;
    TileDma<D> dma;
    tile_dma_plan<D>(dma, wave, lane, row_bytes);
    FragOffsets<D> fo;
    frag_offsets<D>(fo, lane);
    auto stage = [&](int kb_, int buf) {
        const int k0 = kb_ * kTileRows;
        const int nb = max(0, min(kTileRows, T - k0)) * row_bytes;
        tile_dma<D>(sk[buf], dma, raw_rsrc(kbase + (int64_t)k0 * a.hkv * D, nb), wave);
        tile_dma<D>(sv[buf], dma, raw_rsrc(vbase + (int64_t)k0 * a.hkv * D, nb), wave);
    };

    f32x16 acc[D / 32];
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++)
        acc[cb] = f32x16{};

    // bufc: the buffer as a compile-time constant, so that every fragment
    // address is a per-lane offset plus an immediate.  masked: a compile-time
    // flag (a runtime one is if-converted into selects on every tile).
    auto compute = [&](int kb_, auto bufc, auto masked) {
        constexpr int B = decltype(bufc)::value;
        const char *kt = (const char *)sk[B];
        const char *vt = (const char *)sv[B];
        const int k0 = kb_ * kTileRows;
#pragma unroll
        for (int sb = 0; sb < 2; sb++) {
            f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
            for (int ss = 0; ss < D / 16; ss++) {
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    frag_at(kt + sb * 32 * D * 2, fo.row[ss]), qf[ss], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    frag_at(vt + sb * 32 * D * 2, fo.row[ss]), dof[ss], dp, 0, 0, 0);
            }
            // Schedule: two fragment reads ahead, then one MFMA per read, so
            // only a few fragments are live at a time (the register budget
            // of two waves per SIMD).
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);       // DS read
#pragma unroll
            for (int i = 0; i < D / 8 - 2; i++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            // lane: query column; register i: key k0 + 32 sb + 8 (i/4) + 4 g + i%4
            bf16x2 dsw[8];
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                float d2[2];
#pragma unroll
                for (int e = 0; e < 2; e++) {
                    float p = __builtin_amdgcn_exp2f(fmaf(s[i + e], c, -lse));
                    if constexpr (decltype(masked)::value) {
                        const int key = k0 + sb * 32 + ((i + e) >> 2) * 8 + g * 4 + ((i + e) & 3);
                        bool ok = key <= pos;
                        if (MODE == kModeLocal)
                            ok = ok && key > pos - w;
                        p = ok ? p : 0.f;
                    }
                    d2[e] = p * (dp[i + e] - dlt);
                }
                dsw[i >> 1] = cvt_bf16x2(d2[0], d2[1]);
            }
#pragma unroll
            for (int half = 0; half < 2; half++) {
                const bf16x8 bf = pack8(dsw, half);
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++)
                    acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag_tr<D>(kt, fo, sb * 32 + half * 16, cb), bf, acc[cb], 0, 0, 0);
            }
            // one transposed fragment (two reads) ahead of each MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
            for (int i = 0; i < D / 16 - 1; i++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    // Step kb (buffer (kb - kb_lo) % 2): stage tile kb+1 into the other
    // buffer, compute tile kb, then wait for the staged loads and barrier.
    auto step = [&](int kb_, auto bufc) {
        constexpr int B = decltype(bufc)::value;
        if (kb_ < kb_hi)
            stage(kb_ + 1, B ^ 1);
        if (kb_ >= kb_first && kb_ <= kb_last) {
            if (kb_ > kb_c || kb_ < kb_w)
                compute(kb_, bufc, std::true_type{});
            else
                compute(kb_, bufc, std::false_type{});
        }
        dma_wait_barrier();
    };
    stage(kb_lo, 0);
    dma_wait_barrier();
    for (int kb = kb_lo; kb <= kb_hi; kb += 2) {
        step(kb, I0{});
        if (kb + 1 <= kb_hi)
            step(kb + 1, I1{});
    }

    if (!(wave_valid && valid))
        return;
    const int tok = pos + base;
    float *op = a.dq + ((int64_t)tok * a.hq + head) * D + g * 4;
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
        for (int qd = 0; qd < 4; qd++) {
            f32x4 v = {acc[cb][qd * 4 + 0], acc[cb][qd * 4 + 1], acc[cb][qd * 4 + 2],
                       acc[cb][qd * 4 + 3]};
            v *= a.scale;
            if (a.acc_q)
                v += *(const f32x4 *)(op + cb * 32 + qd * 8);
            *(f32x4 *)(op + cb * 32 + qd * 8) = v;
        }
}

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
constexpr int kKeysPerWg = kBwdWaves * 32;

template <int D, int MODE>
__global__ __launch_bounds__(kBwdWaves * 64) __attribute__((amdgpu_waves_per_eu(1, 1)))
void bwd_dkv_kernel(const BwdArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sq[2][kTileRows * D];
    __shared__ __attribute__((aligned(16))) uint16_t sd[2][kTileRows * D];
    // per-row lse, Delta and (global) token index of the staged tiles
    __shared__ __attribute__((aligned(16))) float sl[2][kTileRows];
    __shared__ __attribute__((aligned(16))) float sdl[2][kTileRows];
    __shared__ __attribute__((aligned(16))) int32_t sp[2][kTileRows];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = uni(tid >> 6);
    const int g = lane >> 5, m = lane & 31;
    const int bid = blockIdx.x;
    const int kvh = bid % a.hkv, rest = bid / a.hkv;
    const int b = uni(rest % a.num_seqs);
    const int jt = rest / a.num_seqs;                        // early blocks (most rows) first
    const int base = uni(a.cu_seqlens[b]);
    const int T = uni(a.cu_seqlens[b + 1] - base);
    const int k0 = jt * kKeysPerWg;
    if (k0 >= T)
        return;
    const int j0 = k0 + wave * 32;                           // this wave's first key
    const int key = j0 + m;                                  // this lane's key (column)
    const int w = a.window;

    bf16x8 kf[D / 16], vf[D / 16];
    {
        const int jl = min(key, T - 1);
        const int64_t off = ((int64_t)(base + jl) * a.hkv + kvh) * D + g * 8;
#pragma unroll
        for (int ss = 0; ss < D / 16; ss++) {
            kf[ss] = *(const bf16x8 *)(a.k + off + ss * 16);
            vf[ss] = *(const bf16x8 *)(a.v + off + ss * 16);
        }
    }

    // Rows that can see a key of this block: local, positions k0 .. k0+127+w-1;
    // global, the compacted rows from the first one at or after k0.
    int r_begin, r_end;
    if (MODE == kModeGlobal) {
        const int s0 = uni(a.cu_sel[b]);
        const int s1 = uni(max(s0, min(a.cu_sel[b + 1], a.cap)));
        int lo_ = s0, hi_ = s1;
        while (lo_ < hi_) {
            const int mid = (lo_ + hi_) >> 1;
            if (uni(a.sel_idx[mid]) - base < k0)
                lo_ = mid + 1;
            else
                hi_ = mid;
        }
        r_begin = lo_;
        r_end = s1;
    } else {
        r_begin = base + k0;
        r_end = base + (int)min((long long)T, (long long)k0 + kKeysPerWg - 1 + w);
    }
    const int nblk = (r_end - r_begin + kTileRows - 1) / kTileRows;
    const int nsteps = nblk * a.group;                       // every head of the KV group

    const int row_bytes = a.hq * D * 2;
    TileDma<D> dma;
    tile_dma_plan<D>(dma, wave, lane, row_bytes);
    FragOffsets<D> fo;
    frag_offsets<D>(fo, lane);
    auto step_rows = [&](int st, int &head, int &r0, int &nv) {
        const int hh = st / nblk, qb = st % nblk;
        head = kvh * a.group + hh;
        r0 = r_begin + qb * kTileRows;
        nv = min(kTileRows, r_end - r0);
    };
    // Staging of step st into buffer buf: the Q / dO tiles go global -> LDS
    // directly; the per-row scalars are loaded into a register of one lane
    // per row (wave 0: lse, 1: Delta, 2: token index) by stage() and written
    // to LDS by commit() after the current step's compute, so their latency
    // hides behind it.  Rows past the tile's end get values no row uses.
    float row_val = 0.f;
    auto stage = [&](int st, int buf) {
        int head, r0, nv;
        step_rows(st, head, r0, nv);
        const int64_t off = ((int64_t)r0 * a.hq + head) * D;
        tile_dma<D>(sq[buf], dma, raw_rsrc(a.q + off, nv * row_bytes), wave);
        tile_dma<D>(sd[buf], dma, raw_rsrc(a.dout + off, nv * row_bytes), wave);
        const int64_t ro = (int64_t)head * a.row_stride + r0;
        const int rr = min(lane, nv - 1);
        if (wave == 0)
            row_val = a.lse[ro + rr];
        else if (wave == 1)
            row_val = a.delta[ro + rr];
        else if (wave == 2 && MODE == kModeGlobal)
            row_val = __int_as_float(a.sel_idx[r0 + rr]);
    };
    auto commit = [&](int buf) {
        if (wave == 0)
            sl[buf][lane] = row_val;
        else if (wave == 1)
            sdl[buf][lane] = row_val;
        else if (wave == 2 && MODE == kModeGlobal)
            sp[buf][lane] = __float_as_int(row_val);
    };

    f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++)
        dk[cb] = dv[cb] = f32x16{};
    const float c = a.scale_log2;
    const int jmax = min(j0 + 31, T - 1);

    // One 64-row step: two halves of 32 query rows.
    // One MFMA path for masked and unmasked tiles (two instantiations would
    // give the loop-carried dK / dV accumulators different registers on the
    // two paths and copies where they merge); the mask is a uniform branch
    // in the softmax part only.
    auto compute = [&](auto bufc, int r0, int nv, bool masked) {
        constexpr int buf = decltype(bufc)::value;
        const char *qt = (const char *)sq[buf];
        const char *dt = (const char *)sd[buf];
        // Both 32-row halves in one straight-line block (rows past nv are
        // masked), so the scheduler can overlap one half's softmax with the
        // other half's MFMAs.
#pragma unroll
        for (int qh = 0; qh < 2; qh++) {
            f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
            for (int ss = 0; ss < D / 16; ss++) {
                s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    frag_at(qt + qh * 32 * D * 2, fo.row[ss]), kf[ss], s, 0, 0, 0);
                dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    frag_at(dt + qh * 32 * D * 2, fo.row[ss]), vf[ss], dp, 0, 0, 0);
            }
            // six fragment reads ahead, then one MFMA per read
            __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
            for (int i = 0; i < D / 8 - 6; i++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
            // lane: key column; register i: row qh*32 + 8 (i/4) + 4 g + i%4
            float p[16], dl[16];
#pragma unroll
            for (int qd = 0; qd < 4; qd++) {
                const int ro = qh * 32 + qd * 8 + g * 4;
                const f32x4 l4 = *(const f32x4 *)&sl[buf][ro];
                const f32x4 d4 = *(const f32x4 *)&sdl[buf][ro];
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    p[qd * 4 + e] = __builtin_amdgcn_exp2f(fmaf(s[qd * 4 + e], c, -l4[e]));
                    dl[qd * 4 + e] = d4[e];
                }
            }
            if (masked) {
#pragma unroll
                for (int i = 0; i < 16; i++) {
                    const int qi = qh * 32 + (i >> 2) * 8 + g * 4 + (i & 3);
                    const int qpos = (MODE == kModeGlobal ? sp[buf][qi] : r0 + qi) - base;
                    bool ok = qi < nv && key <= qpos;
                    if (MODE == kModeLocal)
                        ok = ok && qpos < key + w;
                    p[i] = ok ? p[i] : 0.f;
                }
            }
            bf16x2 pw[8], dsw[8];
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                pw[i >> 1] = cvt_bf16x2(p[i], p[i + 1]);
                dsw[i >> 1] = cvt_bf16x2(p[i] * (dp[i] - dl[i]), p[i + 1] * (dp[i + 1] - dl[i + 1]));
            }
#pragma unroll
            for (int half = 0; half < 2; half++) {
                const bf16x8 pb = pack8(pw, half), db = pack8(dsw, half);
#pragma unroll
                for (int cb = 0; cb < D / 32; cb++) {
                    dv[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag_tr<D>(dt, fo, qh * 32 + half * 16, cb), pb, dv[cb], 0, 0, 0);
                    dk[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag_tr<D>(qt, fo, qh * 32 + half * 16, cb), db, dk[cb], 0, 0, 0);
                }
            }
            // two transposed fragments (four reads) ahead of the MFMAs
            __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
            for (int i = 0; i < D / 8 - 4; i++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
        }
    };

    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    auto step = [&](int st, auto bufc) {
        constexpr int buf = decltype(bufc)::value;
        const bool next = st + 1 < nsteps;
        if (next)
            stage(st + 1, buf ^ 1);
        int head, r0, nv;
        step_rows(st, head, r0, nv);
        // positions of the tile's first and last rows (ascending)
        const int pmin = (MODE == kModeGlobal ? uni(sp[buf][0]) : r0) - base;
        const int pmax = (MODE == kModeGlobal ? uni(sp[buf][nv - 1]) : r0 + nv - 1) - base;
        // skip: no row of the tile sees a key of this wave
        bool none = j0 >= T || pmax < j0;
        if (MODE == kModeLocal)
            none = none || pmin > jmax + w - 1;
        if (!none) {
            bool full = nv == kTileRows && pmin >= j0 + 31 && j0 + 31 < T;
            if (MODE == kModeLocal)
                full = full && pmax <= j0 + w - 1;
            compute(bufc, r0, nv, !full);
        }
        if (next)
            commit(buf ^ 1);
        dma_wait_barrier();
    };
    if (nsteps > 0) {
        stage(0, 0);
        commit(0);
        dma_wait_barrier();
    }
    for (int st = 0; st < nsteps; st += 2) {
        step(st, I0{});
        if (st + 1 < nsteps)
            step(st + 1, I1{});
    }

    if (key >= T)
        return;
    const int64_t off = ((int64_t)(base + key) * a.hkv + kvh) * D + g * 4;
    float *kp = a.dk + off;
    float *vp = a.dv + off;
#pragma unroll
    for (int cb = 0; cb < D / 32; cb++)
#pragma unroll
        for (int qd = 0; qd < 4; qd++) {
            f32x4 vk = {dk[cb][qd * 4 + 0], dk[cb][qd * 4 + 1], dk[cb][qd * 4 + 2],
                        dk[cb][qd * 4 + 3]};
            f32x4 vv = {dv[cb][qd * 4 + 0], dv[cb][qd * 4 + 1], dv[cb][qd * 4 + 2],
                        dv[cb][qd * 4 + 3]};
            vk *= a.scale;
            const int o = cb * 32 + qd * 8;
            if (a.acc_k)
                vk += *(const f32x4 *)(kp + o);
            if (a.acc_v)
                vv += *(const f32x4 *)(vp + o);
            *(f32x4 *)(kp + o) = vk;
            *(f32x4 *)(vp + o) = vv;
        }
}

// ---------------------------------------------------------------------------
// ContextNorm + fusion backward
// ---------------------------------------------------------------------------
// Slots: a token's Hq x d values are S = Hq d / 8 slots of 8; thread t of a
// workgroup handles slots (t + 256 k) % S of token t0 + (t + 256 k) / S for
// k < KS, so with S <= 256 a pass covers 256 / S tokens and with S > 256 a
// token takes KS = S / 256 slot sets.  A (token, head) row is d / 8
// consecutive lanes; its sums are DPP lane exchanges within them.
template <int Ctrl>
__device__ __forceinline__ float dpp_mov(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), Ctrl, 0xF, 0xF, false));
}
template <int D>
__device__ __forceinline__ float row_sum(float x) {
    // DPP within each group of D / 8 lanes (16 or 8, aligned): the two quad
    // swaps, then the half-row mirror (lane i <- 7 - i of its 8) and, for 16
    // lanes, the row mirror (i <- 15 - i), each pairing the partial sums of
    // disjoint lane sets.
    static_assert(D / 8 == 16 || D / 8 == 8, "row of 8 or 16 lanes");
    x += dpp_mov<0xB1>(x);        // quad_perm [1,0,3,2]
    x += dpp_mov<0x4E>(x);        // quad_perm [2,3,0,1]
    x += dpp_mov<0x141>(x);       // row_half_mirror
    if constexpr (D / 8 == 16)
        x += dpp_mov<0x140>(x);   // row_mirror
    return x;
}

template <int D, int KS>
__global__ __launch_bounds__(256) void fusion_bwd_kernel(const FusionBwdArgs a) {
    const int S = a.hq * (D / 8);
    const int P = S >= 256 ? 1 : 256 / S;                   // tokens per pass
    const int t_begin = blockIdx.x * a.tokens_per_block;
    const int t_end = min(a.n, t_begin + a.tokens_per_block);
    float gl_acc[KS][8], gg_acc[KS][8];
#pragma unroll
    for (int k = 0; k < KS; k++)
#pragma unroll
        for (int e = 0; e < 8; e++)
            gl_acc[k][e] = gg_acc[k][e] = 0.f;

    for (int t0 = t_begin; t0 < t_end; t0 += P) {
#pragma unroll
        for (int k = 0; k < KS; k++) {
            const int v = threadIdx.x + 256 * k;
            const int toff = v / S, slot = v % S;
            const int tok = t0 + toff;
            if (toff >= P || tok >= t_end)
                continue;                                    // uniform over a row's lanes
            const int h = slot / (D / 8), c0 = (slot % (D / 8)) * 8;
            const bool lead = c0 == 0;
            const int64_t e0 = ((int64_t)tok * a.hq + h) * D + c0;
            const float p = a.gate[tok];
            const int rank = a.tok2sel[tok];
            float dr[8];
            {
                const u32x4 w4 = *(const u32x4 *)(a.dout + e0);
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const uint32_t wd = w4[i];
                    dr[2 * i] = __uint_as_float(wd << 16);
                    dr[2 * i + 1] = __uint_as_float(wd & 0xFFFF0000u);
                }
            }
            float side = 0.f;
            // branch 0: local (every token), branch 1: global (selected)
#pragma unroll
            for (int br = 0; br < 2; br++) {
                if (br == 1 && rank < 0)
                    break;
                const float *src = br ? a.og + ((int64_t)rank * a.hq + h) * D + c0 : a.ol + e0;
                const float *gn = br ? a.gain_g : a.gain_l;
                float o[8], gv[8];
                {
                    const f32x4 x0 = *(const f32x4 *)src, x1 = *(const f32x4 *)(src + 4);
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        o[e] = x0[e];
                        o[4 + e] = x1[e];
                    }
                }
#pragma unroll
                for (int e = 0; e < 8; e++)
                    gv[e] = gn ? gn[h * D + c0 + e] : 1.f;
                const float wgt = br ? p : (rank >= 0 ? 1.f - p : 1.f);
                float sq = 0.f, proj = 0.f, sd = 0.f;
#pragma unroll
                for (int e = 0; e < 8; e++) {
                    sq = fmaf(o[e], o[e], sq);
                    proj = fmaf(gv[e] * dr[e], o[e], proj);
                    sd = fmaf(dr[e] * gv[e], o[e], sd);
                }
                sq = row_sum<D>(sq);
                proj = row_sum<D>(proj) * wgt;
                sd = row_sum<D>(sd);
                const float rr = sqrtf(sq / (float)D + a.eps);
                const float ir = 1.f / rr;
                const float k3 = proj * ir * ir * ir / (float)D;
                float dO[8], dl = 0.f;
                float *gacc = br ? gg_acc[k] : gl_acc[k];
#pragma unroll
                for (int e = 0; e < 8; e++) {
                    dO[e] = gv[e] * wgt * dr[e] * ir - o[e] * k3;
                    gacc[e] = fmaf(wgt * dr[e] * ir, o[e], gacc[e]);
                }
                // The attention backward takes dO in bf16 (dP = dO V^T);
                // Delta = dO . O takes the same rounded values, so that
                // sum_j dS_j = sum_j P_j (dP_j - Delta) vanishes as it does
                // in exact arithmetic (with one visible key, dS = 0).
                const u32x4 dob = u32x4{pack_bf16x2(dO[0], dO[1]), pack_bf16x2(dO[2], dO[3]),
                                        pack_bf16x2(dO[4], dO[5]), pack_bf16x2(dO[6], dO[7])};
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    dl = fmaf(__uint_as_float(dob[i] << 16), o[2 * i], dl);
                    dl = fmaf(__uint_as_float(dob[i] & 0xFFFF0000u), o[2 * i + 1], dl);
                }
                dl = row_sum<D>(dl);
                side += (br ? 1.f : -1.f) * sd * ir;
                const int64_t row = br ? rank : tok;
                uint16_t *dst = (br ? a.dog : a.dol) + (row * a.hq + h) * D + c0;
                *(u32x4 *)dst = dob;
                if (lead)
                    (br ? a.delta_g : a.delta_l)[(int64_t)h * (br ? a.cap : a.n) + row] = dl;
                if (br == 1)
                    *(u32x4 *)(a.qc + (row * a.hq + h) * D + c0) = *(const u32x4 *)(a.q_g + e0);
            }
            if (lead)
                a.side[(int64_t)tok * a.hq + h] = rank >= 0 ? side : 0.f;
        }
    }
    // gain-gradient partials: row blockIdx.x * P + toff of [rows][Hq d]
    const int cols = a.hq * D;
#pragma unroll
    for (int k = 0; k < KS; k++) {
        const int v = threadIdx.x + 256 * k;
        const int toff = v / S, slot = v % S;
        if (toff >= P)
            continue;
        const int64_t o = ((int64_t)blockIdx.x * P + toff) * cols + slot * 8;
#pragma unroll
        for (int e = 0; e < 8; e++) {
            if (a.part_l)
                a.part_l[o + e] = gl_acc[k][e];
            if (a.part_g)
                a.part_g[o + e] = gg_acc[k][e];
        }
    }
}

// dL/dp_t: sum over heads of the per-row terms (zero for unselected tokens).
__global__ __launch_bounds__(256) void gate_grad_kernel(int n, int hq, const float *side,
                                                        float *dgate) {
    const int t = blockIdx.x * 256 + threadIdx.x;
    if (t >= n)
        return;
    float s = 0.f;
    for (int h = 0; h < hq; h++)
        s += side[(int64_t)t * hq + h];
    dgate[t] = s;
}

// Column sums of [rows][cols] partials over row chunks of kGainChunk:
// workgroup (x, y) sums rows y*kGainChunk .. +kGainChunk-1 of 64 columns
// (the 4 waves take every 4th row, then a fixed-order sum of the 4) into
// out[y][cols].  Two passes reduce any row count to one row.
constexpr int kGainChunk = 64;
__global__ __launch_bounds__(256) void gain_grad_kernel(int rows, int cols, const float *part,
                                                        float *out) {
    __shared__ float red[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int col = blockIdx.x * 64 + lane;
    const int r0 = blockIdx.y * kGainChunk, r1 = min(rows, r0 + kGainChunk);
    float s = 0.f;
    if (col < cols)
        for (int r = r0 + wave; r < r1; r += 4)
            s += part[(int64_t)r * cols + col];
    red[wave][lane] = s;
    __syncthreads();
    if (wave == 0 && col < cols)
        out[(int64_t)blockIdx.y * cols + col] =
            (red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]);
}

// Delta = rowsum(dO * O) per (token, head) for plain attention (bf16 O and
// dO), written [Hq][N]; one thread per 8 elements, d / 8 lanes per row.
template <int D>
__global__ __launch_bounds__(256) void attn_delta_kernel(int64_t n_rows, int hq, int64_t n,
                                                         const uint16_t *o, const uint16_t *dout,
                                                         float *delta) {
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t row = g / (D / 8);
    const bool ok = row < n_rows;
    float acc = 0.f;
    if (ok) {
        const u32x4 a = *(const u32x4 *)(o + g * 8), b = *(const u32x4 *)(dout + g * 8);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const uint32_t x = a[i], y = b[i];
            acc = fmaf(__uint_as_float(x << 16), __uint_as_float(y << 16), acc);
            acc = fmaf(__uint_as_float(x & 0xFFFF0000u), __uint_as_float(y & 0xFFFF0000u), acc);
        }
    }
    acc = row_sum<D>(acc);
    if (ok && (g % (D / 8)) == 0) {
        const int64_t t = row / hq;
        const int h = (int)(row % hq);
        delta[(int64_t)h * n + t] = acc;
    }
}

// Inputs of the standalone query-sparse backward: per (selected rank < the
// device count, head) row, the compact copy of the row of Q and Delta = dO . O (O fp32,
// dO bf16, both compact), written [Hq][cap].  d / 8 lanes per row.
template <int D>
__global__ __launch_bounds__(256) void sparse_prep_kernel(int64_t n_rows, int hq, int64_t cap,
                                                          const int32_t *n_sel_dev,
                                                          const int32_t *sel_idx,
                                                          const uint16_t *q, const float *o,
                                                          const uint16_t *dout, uint16_t *qc,
                                                          float *delta) {
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t row = g / (D / 8);
    // rows of ranks at or past the selected count (read on the device) are
    // skipped: their sel_idx entries are not written by the selection
    const int64_t live = min((int64_t)n_sel_dev[0], cap) * hq;
    const bool ok = row < n_rows && row < live;
    float acc = 0.f;
    if (ok) {
        const int64_t r = row / hq;
        const int h = (int)(row % hq);
        const int c0 = (int)(g % (D / 8)) * 8;
        const u32x4 b = *(const u32x4 *)(dout + g * 8);
        const f32x4 o0 = *(const f32x4 *)(o + g * 8), o1 = *(const f32x4 *)(o + g * 8 + 4);
        const float of[8] = {o0[0], o0[1], o0[2], o0[3], o1[0], o1[1], o1[2], o1[3]};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const uint32_t y = b[i];
            acc = fmaf(of[2 * i], __uint_as_float(y << 16), acc);
            acc = fmaf(of[2 * i + 1], __uint_as_float(y & 0xFFFF0000u), acc);
        }
        const int64_t tok = sel_idx[r];
        *(u32x4 *)(qc + g * 8) = *(const u32x4 *)(q + (tok * hq + h) * D + c0);
    }
    acc = row_sum<D>(acc);
    if (ok && (g % (D / 8)) == 0)
        delta[(int64_t)(row % hq) * cap + row / hq] = acc;
}

__global__ __launch_bounds__(256) void fill_zero_kernel(int64_t n, float *x) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n)
        x[i] = 0.f;
}

template <int D>
hipError_t launch_fusion_bwd_d(const FusionBwdArgs &a, int grid, hipStream_t s) {
    const int S = a.hq * (D / 8);
    const int ks = S <= 256 ? 1 : S / 256;
    if (ks == 1)
        hipLaunchKernelGGL((fusion_bwd_kernel<D, 1>), dim3(grid), dim3(256), 0, s, a);
    else if (ks == 2)
        hipLaunchKernelGGL((fusion_bwd_kernel<D, 2>), dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((fusion_bwd_kernel<D, 4>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

int fusion_bwd_tokens_per_pass(int hq, int head_dim) {
    const int S = hq * head_dim / 8;
    return S >= 256 ? 1 : 256 / S;
}

bool fusion_bwd_supported(int hq, int head_dim) {
    const int S = hq * head_dim / 8;
    return S <= 256 ? true : (S % 256 == 0 && S / 256 <= 4 && (S / 256) != 3);
}

hipError_t launch_fusion_bwd(const FusionBwdArgs &a, int grid, int head_dim, hipStream_t s) {
    if (grid <= 0)
        return hipSuccess;
    return head_dim == 128 ? launch_fusion_bwd_d<128>(a, grid, s)
                           : launch_fusion_bwd_d<64>(a, grid, s);
}

hipError_t launch_gate_grad(int n, int hq, const float *side, float *dgate, hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(gate_grad_kernel, dim3((n + 255) / 256), dim3(256), 0, s, n, hq, side,
                       dgate);
    return hipGetLastError();
}

int gain_grad_chunks(int rows) { return (rows + kGainChunk - 1) / kGainChunk; }

hipError_t launch_gain_grad(int rows, int cols, const float *part, float *tmp, float *out,
                            hipStream_t s) {
    const int chunks = gain_grad_chunks(rows);
    if (chunks > kGainChunk)
        return hipErrorInvalidValue;               // two passes cover 4096 rows
    const float *src = part;
    if (chunks > 1) {
        hipLaunchKernelGGL(gain_grad_kernel, dim3((cols + 63) / 64, chunks), dim3(256), 0, s, rows,
                           cols, part, tmp);
        src = tmp;
    }
    hipLaunchKernelGGL(gain_grad_kernel, dim3((cols + 63) / 64, 1), dim3(256), 0, s,
                       chunks > 1 ? chunks : rows, cols, src, out);
    return hipGetLastError();
}

hipError_t launch_attn_delta(int64_t n, int hq, int head_dim, const uint16_t *o,
                             const uint16_t *dout, float *delta, hipStream_t s) {
    const int64_t threads = n * hq * (head_dim / 8);
    if (threads <= 0)
        return hipSuccess;
    const dim3 grid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
        hipLaunchKernelGGL((attn_delta_kernel<128>), grid, dim3(256), 0, s, n * hq, hq, n, o, dout,
                           delta);
    else
        hipLaunchKernelGGL((attn_delta_kernel<64>), grid, dim3(256), 0, s, n * hq, hq, n, o, dout,
                           delta);
    return hipGetLastError();
}

hipError_t launch_sparse_prep(int64_t cap, int hq, int head_dim, const int32_t *n_sel_dev,
                              const int32_t *sel_idx, const uint16_t *q, const float *o,
                              const uint16_t *dout, uint16_t *qc, float *delta, hipStream_t s) {
    const int64_t threads = cap * hq * (head_dim / 8);
    if (threads <= 0)
        return hipSuccess;
    const dim3 grid((unsigned)((threads + 255) / 256));
    if (head_dim == 128)
        hipLaunchKernelGGL((sparse_prep_kernel<128>), grid, dim3(256), 0, s, cap * hq, hq, cap,
                           n_sel_dev, sel_idx, q, o, dout, qc, delta);
    else
        hipLaunchKernelGGL((sparse_prep_kernel<64>), grid, dim3(256), 0, s, cap * hq, hq, cap,
                           n_sel_dev, sel_idx, q, o, dout, qc, delta);
    return hipGetLastError();
}

hipError_t launch_fill_zero(int64_t n, float *x, hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, n, x);
    return hipGetLastError();
}

hipError_t launch_bwd_dq(int mode, int head_dim, const BwdArgs &a, int grid, hipStream_t s) {
    if (grid <= 0)
        return hipSuccess;
    if (head_dim == 128) {
        if (mode == kModeLocal)
            hipLaunchKernelGGL((bwd_dq_kernel<128, kModeLocal>), dim3(grid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((bwd_dq_kernel<128, kModeGlobal>), dim3(grid), dim3(256), 0, s, a);
    } else {
        if (mode == kModeLocal)
            hipLaunchKernelGGL((bwd_dq_kernel<64, kModeLocal>), dim3(grid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((bwd_dq_kernel<64, kModeGlobal>), dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

hipError_t launch_bwd_dkv(int mode, int head_dim, const BwdArgs &a, int grid, hipStream_t s) {
    if (grid <= 0)
        return hipSuccess;
    if (head_dim == 128) {
        if (mode == kModeLocal)
            hipLaunchKernelGGL((bwd_dkv_kernel<128, kModeLocal>), dim3(grid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((bwd_dkv_kernel<128, kModeGlobal>), dim3(grid), dim3(256), 0, s, a);
    } else {
        if (mode == kModeLocal)
            hipLaunchKernelGGL((bwd_dkv_kernel<64, kModeLocal>), dim3(grid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((bwd_dkv_kernel<64, kModeGlobal>), dim3(grid), dim3(256), 0, s, a);
    }
    return hipGetLastError();
}

int bwd_keys_per_block() { return kKeysPerWg; }

}  // namespace logo
