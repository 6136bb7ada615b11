// plan.h -- the work table of the query-sparse global branch, built on the
// device by one workgroup of NT threads (NT a multiple of 64, <= 1024).
//
// Each sequence's selected rows (sel_idx[cu_sel[b] .. cu_sel[b+1])) are cut
// into tiles of tpw rows; a tile covers the 64-key KV blocks 0 .. pos_max/64
// of its sequence (App. B: a tile's keys stop at its last row).  Tiles longer
// than a share of one persistent workgroup's mean load are split into up to
// kMaxSplit consecutive KV ranges (partial slots are handed out longest tile
// first while they last); every entry is then ordered longest first
// (bucketed by KV length), and the queue and split counters are reset.
//
// The table is built in LDS when it fits (the caller passes the LDS block and
// its entry capacity) and copied out once; otherwise it is built in the
// global buffers of PlanArgs.  Used by the standalone plan launch, by one
// extra workgroup of the local-branch launch of the fused layer forward and
// by the first workgroup of the one-launch layer.
#pragma once

#include "logo_internal.h"

namespace logo {
namespace plan_detail {

constexpr int kBuckets = 1024;

}  // namespace plan_detail

// Table capacity in LDS of the standalone plan launch (1024 threads, ~71 KB).
constexpr int kPlanLdsEntriesStandalone = 640;

namespace plan_detail {

// LDS of the plan for E table entries.
template <int E>
struct PlanLds {
    SparseTile tmp[E], out[E];
    int32_t scratch[2 * E];
    int32_t hist[kBuckets];
    int32_t wave_part[16];
    int32_t carry;
    unsigned long long total_blocks;
};

// Inclusive scan of one int per thread over the NT threads.
template <int NT>
__device__ __forceinline__ int scan_incl(int v, int32_t *wave_part) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(v, d, 64);
        if (lane >= d)
            v += t;
    }
    if (lane == 63)
        wave_part[wave] = v;
    __syncthreads();
    int before = 0;
    for (int i = 0; i < wave; i++)
        before += wave_part[i];
    __syncthreads();
    return v + before;
}

// Exclusive prefix sum of v[0..n) in place; returns the total.
template <int NT>
__device__ int scan_array(int32_t *v, int n, int32_t *wave_part, int32_t *carry) {
    const int tid = threadIdx.x;
    if (tid == 0)
        *carry = 0;
    __syncthreads();
    for (int c0 = 0; c0 < n; c0 += NT) {
        const int i = c0 + tid;
        const int x = i < n ? v[i] : 0;
        const int c = *carry;
        const int incl = scan_incl<NT>(x, wave_part);
        if (i < n)
            v[i] = c + incl - x;
        __syncthreads();
        if (tid == NT - 1)
            *carry = c + incl;
        __syncthreads();
    }
    const int total = *carry;
    __syncthreads();
    return total;
}

// Largest b in [0, B-1] with cu[b] <= t.
__device__ __forceinline__ int owner(const int32_t *cu, int B, int t) {
    int lo = 0, hi = B - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (cu[mid] <= t)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int blocks_of(const SparseTile &t) { return t.kb_end - t.kb_begin + 1; }

// Entry copies as three 16-byte moves (the tables may live in LDS or in
// global memory, behind generic pointers).
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ SparseTile load_tile(const SparseTile *p) {
    const i32x4 *s = reinterpret_cast<const i32x4 *>(p);
    const i32x4 a = s[0], b = s[1], c = s[2];
    SparseTile t;
    t.first = a.x; t.nrows = a.y; t.seq = a.z; t.pos_max = a.w;
    t.kb_begin = b.x; t.kb_end = b.y; t.split = b.z; t.nsplit = b.w;
    t.sid = c.x; t.pad[0] = c.y; t.pad[1] = c.z; t.pad[2] = c.w;
    return t;
}
__device__ __forceinline__ void store_tile(SparseTile *p, const SparseTile &t) {
    i32x4 *d = reinterpret_cast<i32x4 *>(p);
    d[0] = i32x4{t.first, t.nrows, t.seq, t.pos_max};
    d[1] = i32x4{t.kb_begin, t.kb_end, t.split, t.nsplit};
    d[2] = i32x4{t.sid, t.pad[0], t.pad[1], t.pad[2]};
}

// Longest-first bucket sort of src[0..n) into dst by KV blocks (1 ..
// max_blocks); the order inside a bucket is arbitrary and no result depends
// on it.
template <int NT>
__device__ void sort_desc(const SparseTile *src, SparseTile *dst, int n, int max_blocks,
                          int32_t *hist, int32_t *wave_part) {
    constexpr int kPer = kBuckets / NT;       // buckets owned by each thread
    const int tid = threadIdx.x;
    const long long mw = max_blocks > 0 ? max_blocks : 1;
    auto bucket = [&](const SparseTile &t) {
        const long long bk = ((mw - blocks_of(t)) * kBuckets) / mw;
        return (int)(bk < 0 ? 0 : (bk >= kBuckets ? kBuckets - 1 : bk));
    };
    for (int i = tid; i < kBuckets; i += NT)
        hist[i] = 0;
    __syncthreads();
    for (int u = tid; u < n; u += NT)
        atomicAdd(&hist[bucket(load_tile(src + u))], 1);
    __syncthreads();
    int c[kPer], own = 0;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        c[j] = hist[tid * kPer + j];
        own += c[j];
    }
    int run = scan_incl<NT>(own, wave_part) - own;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
        hist[tid * kPer + j] = run;
        run += c[j];
    }
    __syncthreads();
    for (int u = tid; u < n; u += NT) {
        const SparseTile t = load_tile(src + u);
        store_tile(dst + atomicAdd(&hist[bucket(t)], 1), t);
    }
    __syncthreads();
}

}  // namespace plan_detail

// Build the work table (see the file comment).  cu: device cu_seqlens [B+1].
template <int NT, int E>
__device__ void build_plan(const int32_t *cu, int B, const PlanArgs &p,
                           plan_detail::PlanLds<E> &l) {
    using namespace plan_detail;
    static_assert(NT % 64 == 0 && NT <= 1024 && kBuckets % NT == 0, "plan workgroup size");
    const int32_t *cu_sel = p.cu_sel, *sel_idx = p.sel_idx;
    const int tpw = p.tpw, cap = p.cap, n_hg = p.n_hg;
    const int split_slots = p.split_slots, stride = p.stride;
    const bool in_lds = stride + split_slots <= E && stride <= E;
    SparseTile *tmp = in_lds ? l.tmp : p.tmp, *out = in_lds ? l.out : p.out;
    int32_t *sa = in_lds ? l.scratch : p.scratch;
    int32_t *sb = sa + (in_lds ? E : stride);
    const int tid = threadIdx.x;

    // 1. tiles per sequence -> exclusive prefix
    for (int b = tid; b < B; b += NT) {
        const int s0 = min(cu_sel[b], cap), s1 = min(cu_sel[b + 1], cap);
        sa[b] = (s1 - s0 + tpw - 1) / tpw;
    }
    __syncthreads();
    const int n_tiles = scan_array<NT>(sa, B, l.wave_part, &l.carry);
    if (tid == 0) {
        sa[B] = n_tiles;
        l.total_blocks = 0;
    }
    __syncthreads();

    // 2. whole tiles (unsorted) and their total KV blocks
    unsigned long long my_blocks = 0;
    for (int u = tid; u < n_tiles; u += NT) {
        const int b = owner(sa, B, u);
        const int s0 = min(cu_sel[b], cap), s1 = min(cu_sel[b + 1], cap);
        const int first = s0 + (u - sa[b]) * tpw;
        const int nrows = min(tpw, s1 - first);
        const int pmax = sel_idx[first + nrows - 1] - cu[b];
        SparseTile t;
        t.first = first;
        t.nrows = nrows;
        t.seq = b;
        t.pos_max = pmax;
        t.kb_begin = 0;
        t.kb_end = pmax / kBlockN;
        t.split = 0;
        t.nsplit = 1;
        t.sid = -1;
        t.pad[0] = t.pad[1] = t.pad[2] = 0;
        store_tile(tmp + u, t);
        my_blocks += (unsigned long long)(t.kb_end + 1);
    }
    atomicAdd(&l.total_blocks, my_blocks);
    __syncthreads();
    const int max_blocks = (p.max_seqlen + kBlockN - 1) / kBlockN;
    // 3. longest first
    sort_desc<NT>(tmp, out, n_tiles, max_blocks, l.hist, l.wave_part);

    // 4. KV split: a tile longer than `target` blocks (a 1/kSplitDiv share of
    //    the mean load of one persistent workgroup, other work of the grid
    //    included) becomes ns = ceil(blocks / target) entries (at most
    //    kMaxSplit), while partial slots last.
    const unsigned long long work = l.total_blocks * (unsigned long long)n_hg +
                                    (unsigned long long)(p.extra_blocks > 0 ? p.extra_blocks : 0);
    const unsigned long long div = (unsigned long long)kSplitDiv * (unsigned long long)p.grid_wgs;
    long long target = (long long)((work + div - 1) / div);
    if (target < kMinSplitBlocks)
        target = kMinSplitBlocks;
    auto nsplit_of = [&](const SparseTile &t) {
        const long long nb = blocks_of(t);
        if (nb <= target)
            return 1;
        const long long ns = (nb + target - 1) / target;
        return (int)(ns < kMaxSplit ? ns : kMaxSplit);
    };
    for (int u = tid; u < n_tiles; u += NT) {
        const int ns = nsplit_of(load_tile(out + u));
        sa[u] = ns > 1 ? ns : 0;
    }
    __syncthreads();
    scan_array<NT>(sa, n_tiles, l.wave_part, &l.carry);    // slot base per tile
    for (int u = tid; u < n_tiles; u += NT) {
        SparseTile t = load_tile(out + u);
        const int ns = nsplit_of(t);
        sb[u] = (ns > 1 && sa[u] + ns <= split_slots) ? ns : 1;
        t.pad[0] = sb[u];                                   // entries of tile u
        store_tile(out + u, t);
    }
    __syncthreads();
    const int n_entries = scan_array<NT>(sb, n_tiles, l.wave_part, &l.carry);
    for (int u = tid; u < n_tiles; u += NT) {
        SparseTile t = load_tile(out + u);
        const int ns = t.pad[0];
        t.pad[0] = 0;
        const int nb = t.kb_end + 1;
        const int e0 = sb[u];
        for (int s = 0; s < ns; s++) {
            SparseTile h = t;
            h.kb_begin = (int)(((long long)s * nb) / ns);
            h.kb_end = (int)(((long long)(s + 1) * nb) / ns) - 1;
            h.split = s;
            h.nsplit = ns;
            h.sid = ns > 1 ? sa[u] : -1;
            store_tile(tmp + e0 + s, h);
        }
    }
    __syncthreads();
    // 5. entries longest first
    sort_desc<NT>(tmp, out, n_entries, max_blocks, l.hist, l.wave_part);
    if (in_lds) {
        for (int u = tid; u < n_entries; u += NT)
            store_tile(p.out + u, load_tile(out + u));
    }
    for (int i = tid; i < split_slots * n_hg; i += NT)
        p.split_cnt[i] = 0;
    if (tid == 0) {
        p.queue[0] = n_entries;
        for (int x = 0; x < kQueues; x++)
            p.queue[1 + x] = 0;
    }
}

}  // namespace logo
