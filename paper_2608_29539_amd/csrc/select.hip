// select.hip -- hard routing and stream compaction (Eq. gate-routing;
// Sec. 3.3 / App. B: selected queries packed in ascending order with their
// original positions and compacted sequence offsets), plus the tile plan
// of the query-sparse global branch.
//
//   select_seq_kernel one 1024-thread workgroup per sequence.  Threshold:
//                     ratio mode takes k = floor(ratio*T) in IEEE double and
//                     the (k+1)-th largest gate, found by a three-pass radix
//                     select (12 + 12 + 8 bits) over order-preserving uint32
//                     keys with LDS histograms; threshold mode takes the given
//                     value.  Then z_t = gate[t] > thr (strict, fp32, done on
//                     the keys) is counted and, with the sequence's offset
//                     known, compacted: ranks from wave ballots, mbcnt and a
//                     workgroup scan; writes sel_idx, tok2sel and cu_sel.  One
//                     sequence: a single launch does all of it.  Several: a
//                     first launch finds the thresholds and counts, a second
//                     one compacts with offset = sum of the earlier counts.
//   budget_kernel     one step of the global-budget controller (Sec. 3.2, Eq.
//                     threshold-update) from the realized ratio cu_sel[B] / N.
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

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kKeysPerThread = 32;                      // gate keys per thread per chunk
constexpr int kSelChunk = kKeysPerThread * kSelThreads;  // tokens per chunk (32768)

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
// Keys above this one are positive NaNs, which never compare greater.
constexpr uint32_t kPosInfKey = 0xFF800000u;

// Block-wide inclusive scan of one int per thread (blockDim.x <= 1024).
__device__ __forceinline__ int block_inclusive_scan(int v, int *s_wave) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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
    __syncthreads();
    return v + before;
}

// Block-wide sum (every thread gets it).
__device__ __forceinline__ int block_sum(int v, int *s_wave) {
#pragma unroll
    for (int d = 32; d > 0; d >>= 1)
        v += __shfl_xor(v, d, 64);
    if ((threadIdx.x & 63) == 0)
        s_wave[threadIdx.x >> 6] = v;
    __syncthreads();
    int sum = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); i++)
        sum += s_wave[i];
    __syncthreads();
    return sum;
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

// Work tables that fit are built in LDS and copied out once at the end (the
// plan's phases are short, so global-memory round trips would dominate).
constexpr int kPlanLdsEntries = 640;
constexpr int kPlanLdsInts = 1280;

// The tile plan, run by one workgroup of 1024 threads (see PlanArgs).
__device__ void plan_body(const int32_t *cu, int B, const PlanArgs &p) {
    const int32_t *cu_sel = p.cu_sel, *sel_idx = p.sel_idx;
    const int tpw = p.tpw, cap = p.cap, max_seqlen = p.max_seqlen, n_hg = p.n_hg;
    const int grid_wgs = p.grid_wgs, split_slots = p.split_slots, stride = p.stride;
    __shared__ SparseTile l_tmp[kPlanLdsEntries], l_out[kPlanLdsEntries];
    __shared__ int32_t l_scratch[kPlanLdsInts];
    const bool in_lds = stride + split_slots <= kPlanLdsEntries && 2 * stride <= kPlanLdsInts;
    SparseTile *tmp = in_lds ? l_tmp : p.tmp, *out = in_lds ? l_out : p.out;
    int32_t *scratch = in_lds ? l_scratch : p.scratch;
    int32_t *queue = p.queue, *split_cnt = p.split_cnt;
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
    if (in_lds) {
        for (int u = tid; u < n_entries; u += 1024)
            p.out[u] = out[u];
    }
    for (int i = tid; i < split_slots * n_hg; i += 1024)
        split_cnt[i] = 0;
    if (tid == 0) {
        queue[0] = n_entries;
        for (int x = 0; x < kQueues; x++)
            queue[1 + x] = 0;
    }
}

__global__ __launch_bounds__(1024) void sparse_plan_kernel(const int32_t *cu, int B, PlanArgs p) {
    plan_body(cu, B, p);
}

// kThreshold: find thr[b] (ratio mode) or take `fixed` (threshold mode), and
// write thr[b]; otherwise read thr[b].  kWrite: compact (offset = sum of
// cnt[b'] over b' < b, or 0 for a single sequence); otherwise write cnt[b].
// kPlan (one sequence only): then build the global tile plan.
template <bool kThreshold, bool kWrite, bool kPlan>
__global__ __launch_bounds__(kSelThreads) void select_seq_kernel(
    const int32_t *__restrict__ cu, int B, const float *__restrict__ gate, int mode, float fixed,
    double ratio, float *__restrict__ thr, int32_t *__restrict__ cnt, int32_t *__restrict__ sel_idx,
    int32_t cap, int32_t *__restrict__ cu_sel, int32_t *__restrict__ tok2sel, PlanArgs plan) {
    __shared__ int hist[4096];
    __shared__ int s_wave[kSelWaves];
    __shared__ uint32_t s_bin;
    __shared__ int s_rank, s_bincnt;
    __shared__ int s_cnt[kKeysPerThread * kSelWaves];   // selected per (round, wave)
    __shared__ int s_total;
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t base = cu[b];
    const int T = cu[b + 1] - (int)base;

    // Keys of one chunk of kSelChunk tokens (token c0 + j * 1024 + tid in
    // key[j]), loaded with all loads in flight at once; a sequence that fits
    // in one chunk is loaded once.
    const bool resident = T <= kSelChunk;
    uint32_t key[kKeysPerThread];
    auto load_chunk = [&](int c0) {
#pragma unroll
        for (int j = 0; j < kKeysPerThread; j++) {
            const int t = c0 + j * kSelThreads + tid;
            key[j] = t < T ? float_key(gate[base + t]) : 0u;
        }
    };
    if (resident)
        load_chunk(0);

    uint32_t thr_key;
    if constexpr (kThreshold) {
        const long long k = mode == 1 ? (long long)floor(ratio * (double)T) : 0;
        if (mode == 2)
            fixed = thr[0];                   // the device-held threshold
        if (mode != 1) {
            // a NaN threshold (device mode) selects nothing, as gate > NaN
            thr_key = fixed == fixed ? float_key(fixed) : 0xFFFFFFFFu;
        } else if (k >= T) {
            thr_key = float_key(-__builtin_inff());
        } else {
            int rank = (int)(T - k - 1);      // ascending rank of the threshold value
            uint32_t prefix = 0, pmask = 0;
            for (int pass = 0; pass < 3; pass++) {
                const int sh = pass == 0 ? 20 : (pass == 1 ? 8 : 0);
                const int nb = pass == 2 ? 256 : 4096;
                for (int i = tid; i < 4096; i += kSelThreads)
                    hist[i] = 0;
                __syncthreads();
                for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                    if (!resident)
                        load_chunk(c0);
                    // Runs of equal digits are counted in a register and added
                    // in one atomic (concentrated gate distributions put most
                    // keys of a pass into a few bins).
                    int cur = -1, run_len = 0;
#pragma unroll
                    for (int j = 0; j < kKeysPerThread; j++) {
                        const int t = c0 + j * kSelThreads + tid;
                        if (t < T && (key[j] & pmask) == prefix) {
                            const int d = (int)((key[j] >> sh) & (uint32_t)(nb - 1));
                            if (d != cur) {
                                if (run_len > 0)
                                    atomicAdd(&hist[cur], run_len);
                                cur = d;
                                run_len = 0;
                            }
                            run_len++;
                        }
                    }
                    if (run_len > 0)
                        atomicAdd(&hist[cur], run_len);
                }
                __syncthreads();
                // Each thread owns 4 consecutive bins.
                int own = 0;
                int c4[4];
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    const int bin = tid * 4 + j;
                    c4[j] = bin < nb ? hist[bin] : 0;
                    own += c4[j];
                }
                const int incl = block_inclusive_scan(own, s_wave);
                int run = incl - own;
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    if (c4[j] > 0 && rank >= run && rank < run + c4[j]) {
                        s_bin = (uint32_t)(tid * 4 + j);
                        s_rank = rank - run;
                        s_bincnt = c4[j];
                    }
                    run += c4[j];
                }
                __syncthreads();
                prefix |= s_bin << sh;
                pmask |= (uint32_t)(nb - 1) << sh;
                rank = s_rank;
                const bool unique = s_bincnt == 1;
                __syncthreads();
                if (pass < 2 && unique && resident) {
                    // one key left in the bin: it is the threshold
#pragma unroll
                    for (int j = 0; j < kKeysPerThread; j++) {
                        const int t = j * kSelThreads + tid;
                        if (t < T && (key[j] & pmask) == prefix)
                            s_bin = key[j];
                    }
                    __syncthreads();
                    prefix = s_bin;
                    break;
                }
            }
            thr_key = prefix;
        }
        if (tid == 0)
            thr[b] = mode == 1 ? key_float(thr_key) : fixed;
    } else {
        const float v = thr[b];
        thr_key = v == v ? float_key(v) : 0xFFFFFFFFu;   // NaN: nothing passes
    }
    // z = gate > thr on the keys: -0 and +0 share a key, and NaN gates (keys
    // above +inf, or below -inf) never pass.
    auto pass_z = [&](uint32_t kj, int t) { return t < T && kj > thr_key && kj <= kPosInfKey; };

    if constexpr (!kWrite) {
        int mine = 0;
        for (int c0 = 0; c0 < T; c0 += kSelChunk) {
            if (!resident)
                load_chunk(c0);
#pragma unroll
            for (int j = 0; j < kKeysPerThread; j++)
                mine += pass_z(key[j], c0 + j * kSelThreads + tid) ? 1 : 0;
        }
        const int total = block_sum(mine, s_wave);
        if (tid == 0)
            cnt[b] = total;
    } else {
        int offset = 0;
        if (B > 1) {
            int part = 0;
            for (int i = tid; i < b; i += kSelThreads)
                part += cnt[i];
            offset = block_sum(part, s_wave);
        }
        if (tid == 0)
            cu_sel[b] = offset;
        int running = offset;
        for (int c0 = 0; c0 < T; c0 += kSelChunk) {
            if (!resident)
                load_chunk(c0);
            uint64_t mask[kKeysPerThread];
#pragma unroll
            for (int j = 0; j < kKeysPerThread; j++) {
                mask[j] = __ballot(pass_z(key[j], c0 + j * kSelThreads + tid));
                if (lane == 0)
                    s_cnt[j * kSelWaves + wave] = (int)__popcll(mask[j]);
            }
            __syncthreads();
            // exclusive scan of the (round, wave) counts in token order
            const int n_cnt = kKeysPerThread * kSelWaves;   // 512 <= 1024
            const int v = tid < n_cnt ? s_cnt[tid] : 0;
            const int incl = block_inclusive_scan(v, s_wave);
            if (tid < n_cnt)
                s_cnt[tid] = incl - v;
            if (tid == kSelThreads - 1)
                s_total = incl;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < kKeysPerThread; j++) {
                const int t = c0 + j * kSelThreads + tid;
                if (t < T) {
                    const uint64_t m = mask[j];
                    const bool z = (m >> lane) & 1ull;
                    const int r = running + s_cnt[j * kSelWaves + wave] +
                                  (int)__builtin_amdgcn_mbcnt_hi(
                                      (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
                    if (z && r < cap)
                        sel_idx[r] = (int32_t)(base + t);
                    if (tok2sel)
                        tok2sel[base + t] = (z && r < cap) ? r : -1;
                }
            }
            running += s_total;
            __syncthreads();
        }
        if (b == B - 1 && tid == 0)
            cu_sel[B] = running;
        if constexpr (kPlan) {
            // one sequence: this workgroup wrote all of sel_idx and cu_sel
            __syncthreads();
            plan_body(cu, B, plan);
        }
    }
}

// F = cu_sel[B] / N (Eq. realized-ratio), compared with rho in double;
// b_th <- b_th + gamma sign(F - rho) in fp32 (Eq. threshold-update).
__global__ void budget_kernel(const int32_t *cu_sel, int B, int N, double rho, float gamma,
                              float *b_th, float *realized) {
    if (threadIdx.x != 0)
        return;
    if (N <= 0) {
        if (realized)
            *realized = 0.f;
        return;
    }
    const double f = (double)cu_sel[B] / (double)N;
    const float b = *b_th;
    *b_th = f > rho ? b + gamma : (f < rho ? b - gamma : b);
    if (realized)
        *realized = (float)f;
}

}  // namespace

hipError_t launch_budget_update(const int32_t *cu_sel, int num_seqs, int n_tokens, double rho,
                                float gamma, float *b_th, float *realized, hipStream_t s) {
    hipLaunchKernelGGL(budget_kernel, dim3(1), dim3(64), 0, s, cu_sel, num_seqs, n_tokens, rho,
                       gamma, b_th, realized);
    return hipGetLastError();
}

hipError_t launch_select(const int32_t *cu_seqlens, int num_seqs, int n_tokens,
                         const float *gate, int mode, float threshold, double ratio,
                         int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                         int32_t *tok2sel, float *thr, int32_t *seq_counts,
                         const PlanArgs *plan, hipStream_t s) {
    (void)n_tokens;
    const PlanArgs none{};
    if (num_seqs == 1) {
        if (plan)
            hipLaunchKernelGGL((select_seq_kernel<true, true, true>), dim3(1), dim3(kSelThreads), 0,
                               s, cu_seqlens, 1, gate, mode, threshold, ratio, thr, seq_counts,
                               sel_idx, sel_capacity, cu_sel, tok2sel, *plan);
        else
            hipLaunchKernelGGL((select_seq_kernel<true, true, false>), dim3(1), dim3(kSelThreads),
                               0, s, cu_seqlens, 1, gate, mode, threshold, ratio, thr, seq_counts,
                               sel_idx, sel_capacity, cu_sel, tok2sel, none);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((select_seq_kernel<true, false, false>), dim3(num_seqs), dim3(kSelThreads),
                       0, s, cu_seqlens, num_seqs, gate, mode, threshold, ratio, thr, seq_counts,
                       sel_idx, sel_capacity, cu_sel, tok2sel, none);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((select_seq_kernel<false, true, false>), dim3(num_seqs), dim3(kSelThreads),
                       0, s, cu_seqlens, num_seqs, gate, mode, threshold, ratio, thr, seq_counts,
                       sel_idx, sel_capacity, cu_sel, tok2sel, none);
    e = hipGetLastError();
    if (e != hipSuccess || !plan)
        return e;
    return launch_sparse_plan(cu_seqlens, num_seqs, *plan, s);
}

hipError_t launch_sparse_plan(const int32_t *cu_seqlens, int num_seqs, const PlanArgs &plan,
                              hipStream_t s) {
    hipLaunchKernelGGL(sparse_plan_kernel, dim3(1), dim3(1024), 0, s, cu_seqlens, num_seqs, plan);
    return hipGetLastError();
}

}  // namespace logo
