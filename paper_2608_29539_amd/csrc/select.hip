// select.hip -- hard routing and stream compaction (Eq. gate-routing;
// Sec. 3.3 / App. B: selected queries packed in ascending order with their
// original positions and compacted sequence offsets), plus the tile plan
// of the query-sparse global branch.
//
//   threshold_kernel  ratio mode: per sequence, k = floor(ratio*T) in IEEE
//                     double; the threshold is the (k+1)-th largest gate, found
//                     by a three-pass radix select (12 + 12 + 8 bits) over
//                     order-preserving uint32 keys with LDS histograms.
//   count_kernel      z_t = gate[t] > thr[b(t)] (strict, fp32); per-chunk counts
//                     from wave ballots.
//   write_kernel      exclusive ranks (chunk offset + ballot/mbcnt prefix),
//                     writes sel_idx, tok2sel and cu_sel.
//   sparse_plan_kernel
//                     cuts each sequence's selected rows into tiles of tpw
//                     rows, splits the longest tiles into KV ranges so that no
//                     work entry exceeds a fraction of one persistent
//                     workgroup's mean load, orders the entries longest-first
//                     (bucketed by KV length), then resets the work queues and
//                     the split counters.
#include "logo_internal.h"

namespace logo {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelPerThread = 16;
constexpr int kSelChunk = kSelThreads * kSelPerThread;   // tokens per workgroup
constexpr int kRadixThreads = 1024;

// Order-preserving map from fp32 to uint32 (-0 is folded onto +0 first).
__device__ __forceinline__ uint32_t float_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u)
        u = 0;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_float(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k;
    return __uint_as_float(u);
}

// Block-wide inclusive scan of one int per thread (blockDim.x <= 1024).
__device__ __forceinline__ int block_inclusive_scan(int v, int *s_wave) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nwaves = (blockDim.x + 63) >> 6;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(v, d, 64);
        if (lane >= d)
            v += t;
    }
    if (lane == 63)
        s_wave[wave] = v;
    __syncthreads();
    int before = 0;
    for (int i = 0; i < wave; i++)
        before += s_wave[i];
    (void)nwaves;
    __syncthreads();
    return v + before;
}

__global__ __launch_bounds__(kRadixThreads) void threshold_kernel(const int32_t *cu,
                                                                  const float *gate,
                                                                  double ratio, float *thr) {
    __shared__ int hist[4096];
    __shared__ int s_wave[16];
    __shared__ uint32_t s_bin;
    __shared__ int s_rank;
    const int b = blockIdx.x, tid = threadIdx.x;
    const int base = cu[b];
    const int T = cu[b + 1] - base;
    const long long k = (long long)floor(ratio * (double)T);
    if (k >= T) {
        if (tid == 0)
            thr[b] = -__builtin_inff();
        return;
    }
    int rank = (int)(T - k - 1);      // ascending rank of the threshold value
    uint32_t prefix = 0, pmask = 0;
    const int shifts[3] = {20, 8, 0};
    const int widths[3] = {12, 12, 8};
    for (int pass = 0; pass < 3; pass++) {
        const int sh = shifts[pass], nb = 1 << widths[pass];
        for (int i = tid; i < 4096; i += kRadixThreads)
            hist[i] = 0;
        __syncthreads();
        for (int t = tid; t < T; t += kRadixThreads) {
            const uint32_t key = float_key(gate[base + t]);
            if ((key & pmask) == prefix)
                atomicAdd(&hist[(key >> sh) & (nb - 1)], 1);
        }
        __syncthreads();
        // Each thread owns 4 consecutive bins (nb <= 4096).
        int own = 0;
        int cnt[4];
#pragma unroll
        for (int j = 0; j < 4; j++) {
            const int bin = tid * 4 + j;
            cnt[j] = bin < nb ? hist[bin] : 0;
            own += cnt[j];
        }
        const int incl = block_inclusive_scan(own, s_wave);
        int run = incl - own;
#pragma unroll
        for (int j = 0; j < 4; j++) {
            if (cnt[j] > 0 && rank >= run && rank < run + cnt[j]) {
                s_bin = (uint32_t)(tid * 4 + j);
                s_rank = rank - run;
            }
            run += cnt[j];
        }
        __syncthreads();
        prefix |= s_bin << sh;
        pmask |= (uint32_t)(nb - 1) << sh;
        rank = s_rank;
        __syncthreads();
    }
    if (tid == 0) {
        float f = key_float(prefix);
        thr[b] = f;
    }
}

__global__ void fill_threshold_kernel(int num_seqs, float value, float *thr) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b < num_seqs)
        thr[b] = value;
}

// Largest b in [0, B-1] with cu[b] <= t (the owner of token t).
__device__ __forceinline__ int owner_seq(const int32_t *cu, int B, int t) {
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

__global__ __launch_bounds__(kSelThreads) void count_kernel(const int32_t *cu, int B, int N,
                                                             const float *gate, const float *thr,
                                                             int32_t *chunk_counts) {
    __shared__ int s_cnt[kSelThreads / 64];
    const int c0 = blockIdx.x * kSelChunk;
    const int tid = threadIdx.x;
    int b = -1, b_end = 0;
    int count = 0;
    for (int i = 0; i < kSelPerThread; i++) {
        const int t = c0 + i * kSelThreads + tid;
        bool z = false;
        if (t < N) {
            if (b < 0 || t >= b_end) {
                b = owner_seq(cu, B, t);
                b_end = cu[b + 1];
            }
            z = gate[t] > thr[b];
        }
        count += __popcll(__ballot(z));
    }
    if ((tid & 63) == 0)
        s_cnt[tid >> 6] = count;
    __syncthreads();
    if (tid == 0) {
        int s = 0;
        for (int w = 0; w < kSelThreads / 64; w++)
            s += s_cnt[w];
        chunk_counts[blockIdx.x] = s;
    }
}

__global__ __launch_bounds__(kSelThreads) void write_kernel(const int32_t *cu, int B, int N,
                                                             const float *gate, const float *thr,
                                                             const int32_t *chunk_counts,
                                                             int32_t *sel_idx, int32_t cap,
                                                             int32_t *cu_sel, int32_t *tok2sel) {
    __shared__ int s_red[kSelThreads / 64];
    __shared__ int s_off;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Offset of this chunk = sum of the counts of all earlier chunks.
    int part = 0;
    for (int i = tid; i < (int)blockIdx.x; i += kSelThreads)
        part += chunk_counts[i];
#pragma unroll
    for (int d = 32; d > 0; d >>= 1)
        part += __shfl_xor(part, d, 64);
    if (lane == 0)
        s_red[wave] = part;
    __syncthreads();
    if (tid == 0) {
        int s = 0;
        for (int w = 0; w < kSelThreads / 64; w++)
            s += s_red[w];
        s_off = s;
    }
    __syncthreads();
    int offset = s_off;
    __syncthreads();

    const int c0 = blockIdx.x * kSelChunk;
    int b = -1, b_end = 0;
    for (int i = 0; i < kSelPerThread; i++) {
        const int t = c0 + i * kSelThreads + tid;
        bool z = false;
        if (t < N) {
            if (b < 0 || t >= b_end) {
                b = owner_seq(cu, B, t);
                b_end = cu[b + 1];
            }
            z = gate[t] > thr[b];
        }
        const unsigned long long mask = __ballot(z);
        const int lane_prefix = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                          __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
        if (lane == 0)
            s_red[wave] = __popcll(mask);
        __syncthreads();
        int before = 0, total = 0;
        for (int w = 0; w < kSelThreads / 64; w++) {
            const int cw = s_red[w];
            if (w < wave)
                before += cw;
            total += cw;
        }
        __syncthreads();
        const int rank = offset + before + lane_prefix;   // exclusive rank of token t
        if (t < N) {
            if (z && rank < cap)
                sel_idx[rank] = t;
            if (tok2sel)
                tok2sel[t] = (z && rank < cap) ? rank : -1;
            // cu_sel[b'] for every sequence b' that starts at token t
            if (cu[b] == t) {
                for (int bb = b; bb >= 0 && cu[bb] == t; bb--)
                    cu_sel[bb] = rank;
            }
        }
        offset += total;
    }
    // Sequences that start at N (the end), including cu_sel[B] = n_sel.
    if (blockIdx.x == gridDim.x - 1 && tid == 0) {
        for (int bb = B; bb >= 0 && cu[bb] == N; bb--)
            cu_sel[bb] = offset;
    }
}

// Exclusive prefix sum, in place, of n ints in global memory by one
// 1024-thread workgroup (chunks of 1024 with a carry); returns the total.
__device__ int block_exclusive_scan_array(int32_t *v, int n, int *s_wave, int *s_carry) {
    const int tid = threadIdx.x;
    if (tid == 0)
        *s_carry = 0;
    __syncthreads();
    for (int c0 = 0; c0 < n; c0 += 1024) {
        const int i = c0 + tid;
        const int x = i < n ? v[i] : 0;
        const int carry = *s_carry;
        const int incl = block_inclusive_scan(x, s_wave);
        if (i < n)
            v[i] = carry + incl - x;
        __syncthreads();
        if (tid == 1023)
            *s_carry = carry + incl;
        __syncthreads();
    }
    const int total = *s_carry;
    __syncthreads();
    return total;
}

constexpr int kBuckets = 1024;

__device__ __forceinline__ int entry_blocks(const SparseTile &t) { return t.kb_end - t.kb_begin + 1; }

// Longest-first bucket sort of n entries of src into dst by their number of
// KV blocks (in [1, max_blocks]); the order inside a bucket is arbitrary and
// no result depends on it.
__device__ void bucket_sort_desc(const SparseTile *src, SparseTile *dst, int n, int max_blocks,
                                 int *hist, int *s_wave) {
    const int tid = threadIdx.x;
    const long long mw = max_blocks > 0 ? max_blocks : 1;
    auto bucket = [&](const SparseTile &t) {
        long long bk = ((mw - entry_blocks(t)) * kBuckets) / mw;
        return (int)(bk < 0 ? 0 : (bk >= kBuckets ? kBuckets - 1 : bk));
    };
    hist[tid] = 0;
    __syncthreads();
    for (int u = tid; u < n; u += 1024)
        atomicAdd(&hist[bucket(src[u])], 1);
    __syncthreads();
    const int hv = hist[tid];
    const int incl = block_inclusive_scan(hv, s_wave);
    hist[tid] = incl - hv;
    __syncthreads();
    for (int u = tid; u < n; u += 1024) {
        const SparseTile t = src[u];
        dst[atomicAdd(&hist[bucket(t)], 1)] = t;
    }
    __syncthreads();
}

// One workgroup of 1024 threads.  scratch holds 2 * (stride) ints with
// stride >= max(B, max_tiles) + 1.
__global__ __launch_bounds__(1024) void sparse_plan_kernel(
    const int32_t *cu, const int32_t *cu_sel, const int32_t *sel_idx, int B, int tpw, int cap,
    int max_seqlen, int n_hg, int grid_wgs, int split_slots, int stride, SparseTile *tmp,
    SparseTile *out, int32_t *scratch, int32_t *queue, int32_t *split_cnt) {
    __shared__ int s_wave[16];
    __shared__ int s_carry;
    __shared__ int hist[kBuckets];
    __shared__ unsigned long long s_total_blocks;
    const int tid = threadIdx.x;
    int32_t *sa = scratch, *sb = scratch + stride;

    // 1. tiles per sequence -> exclusive prefix
    for (int b = tid; b < B; b += 1024) {
        const int s0 = min(cu_sel[b], cap), s1 = min(cu_sel[b + 1], cap);
        sa[b] = (s1 - s0 + tpw - 1) / tpw;
    }
    __syncthreads();
    const int n_tiles = block_exclusive_scan_array(sa, B, s_wave, &s_carry);
    if (tid == 0) {
        sa[B] = n_tiles;
        s_total_blocks = 0;
    }
    __syncthreads();

    // 2. the whole tiles (unsorted) into tmp, and their total KV blocks
    unsigned long long my_blocks = 0;
    for (int u = tid; u < n_tiles; u += 1024) {
        const int b = owner_seq(sa, B, u);
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
        tmp[u] = t;
        my_blocks += (unsigned long long)(t.kb_end + 1);
    }
    atomicAdd(&s_total_blocks, my_blocks);
    __syncthreads();
    const int max_blocks = (max_seqlen + kBlockN - 1) / kBlockN;
    // 3. longest first
    bucket_sort_desc(tmp, out, n_tiles, max_blocks, hist, s_wave);

    // 4. KV split: a tile longer than `target` blocks (a 1/kSplitDiv share of
    //    the mean load of one persistent workgroup) becomes ns = ceil(blocks /
    //    target) entries (at most kMaxSplit) over consecutive KV ranges, while
    //    partial slots last (longest tiles first).
    const unsigned long long work = s_total_blocks * (unsigned long long)n_hg;
    const unsigned long long div = (unsigned long long)kSplitDiv * (unsigned long long)grid_wgs;
    long long target = (long long)((work + div - 1) / div);
    if (target < kMinSplitBlocks)
        target = kMinSplitBlocks;
    auto nsplit_of = [&](const SparseTile &t) {
        const long long nb = entry_blocks(t);
        if (nb <= target)
            return 1;
        const long long ns = (nb + target - 1) / target;
        return (int)(ns < kMaxSplit ? ns : kMaxSplit);
    };
    for (int u = tid; u < n_tiles; u += 1024) {
        const int ns = nsplit_of(out[u]);
        sa[u] = ns > 1 ? ns : 0;
    }
    __syncthreads();
    block_exclusive_scan_array(sa, n_tiles, s_wave, &s_carry);   // slot base
    for (int u = tid; u < n_tiles; u += 1024) {
        const int ns = nsplit_of(out[u]);
        sb[u] = (ns > 1 && sa[u] + ns <= split_slots) ? ns : 1;
    }
    __syncthreads();
    // sb[u] = entries of tile u; keep a copy of the counts in tmp's pad
    for (int u = tid; u < n_tiles; u += 1024)
        out[u].pad[0] = sb[u];
    __syncthreads();
    const int n_entries = block_exclusive_scan_array(sb, n_tiles, s_wave, &s_carry);
    for (int u = tid; u < n_tiles; u += 1024) {
        SparseTile t = out[u];
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
            tmp[e0 + s] = h;
        }
    }
    __syncthreads();
    // 5. entries longest first
    bucket_sort_desc(tmp, out, n_entries, max_blocks, hist, s_wave);
    for (int i = tid; i < split_slots * n_hg; i += 1024)
        split_cnt[i] = 0;
    if (tid == 0) {
        queue[0] = n_entries;
        for (int x = 0; x < kQueues; x++)
            queue[1 + x] = 0;
    }
}

}  // namespace

int select_chunks(int n_tokens) {
    const int c = (n_tokens + kSelChunk - 1) / kSelChunk;
    return c > 0 ? c : 1;
}

hipError_t launch_select(const int32_t *cu_seqlens, int num_seqs, int n_tokens,
                         const float *gate, int mode, float threshold, double ratio,
                         int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                         int32_t *tok2sel, float *thr, int32_t *chunk_counts, hipStream_t s) {
    if (mode == 1) {
        hipLaunchKernelGGL(threshold_kernel, dim3(num_seqs), dim3(kRadixThreads), 0, s,
                           cu_seqlens, gate, ratio, thr);
    } else {
        hipLaunchKernelGGL(fill_threshold_kernel, dim3((num_seqs + 255) / 256), dim3(256), 0, s,
                           num_seqs, threshold, thr);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int chunks = select_chunks(n_tokens);
    hipLaunchKernelGGL(count_kernel, dim3(chunks), dim3(kSelThreads), 0, s, cu_seqlens, num_seqs,
                       n_tokens, gate, (const float *)thr, chunk_counts);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(write_kernel, dim3(chunks), dim3(kSelThreads), 0, s, cu_seqlens, num_seqs,
                       n_tokens, gate, (const float *)thr, (const int32_t *)chunk_counts, sel_idx,
                       sel_capacity, cu_sel, tok2sel);
    return hipGetLastError();
}

hipError_t launch_sparse_plan(const int32_t *cu_seqlens, const int32_t *cu_sel,
                              const int32_t *sel_idx, int num_seqs, int tpw, int sel_capacity,
                              int max_seqlen, int n_hg, int grid_wgs, int split_slots,
                              int stride, SparseTile *tiles_tmp, SparseTile *tiles,
                              int32_t *scratch, int32_t *queue, int32_t *split_cnt,
                              hipStream_t s) {
    hipLaunchKernelGGL(sparse_plan_kernel, dim3(1), dim3(1024), 0, s, cu_seqlens, cu_sel, sel_idx,
                       num_seqs, tpw, sel_capacity, max_seqlen, n_hg, grid_wgs, split_slots,
                       stride, tiles_tmp, tiles, scratch, queue, split_cnt);
    return hipGetLastError();
}

}  // namespace logo
