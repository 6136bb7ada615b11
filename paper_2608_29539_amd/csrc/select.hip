// select.hip -- hard routing and stream compaction (Eq. gate-routing;
// Sec. 3.3 / App. B: selected queries packed in ascending order with their
// original positions and compacted sequence offsets), plus the tile plan
// of the query-sparse global branch.
//
//   select_kernel     up to 16 workgroups of 1024 threads per sequence (more
//                     for sequences over 512K tokens), each compacting one
//                     part of it.  Threshold: ratio mode takes
//                     k = floor(ratio*T) in IEEE double and the (k+1)-th
//                     largest gate, found by every part: an LDS histogram
//                     of 4096 equal-width probability bins, then the gates
//                     of the bin that holds it are gathered and ranked among
//                     themselves (radix passes of at most 12 bits over
//                     order-preserving uint32 keys when that bin is too
//                     full); threshold mode takes the given value.  Then
//                     z_t = gate[t] > thr (strict, fp32, on the gates held
//                     in registers) and the part's ranks follow from wave
//                     ballots, one scan of per-block counts and the lane
//                     prefix (mbcnt); writes sel_idx, tok2sel and cu_sel.
//                     One sequence: a single launch.
//                     Several: a first launch finds the thresholds and
//                     counts, a second one compacts with offset = sum of the
//                     earlier counts.
//   budget_kernel     one step of the global-budget controller (Sec. 3.2, Eq.
//                     threshold-update) from the realized ratio cu_sel[B] / N.
//   sparse_plan_kernel
//                     the global branch's work table (plan.h) for the
//                     standalone query-sparse entry point; the fused layer
//                     builds it inside its local-branch launch instead.
#include "logo_internal.h"
#include "plan.h"

namespace logo {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kKeysPerThread = 32;                      // gates per thread per chunk
constexpr int kSelChunk = kKeysPerThread * kSelThreads;  // tokens per chunk (32768)
constexpr int kPartUnit = 4 * kSelThreads;              // smallest part (4096 tokens)
constexpr int kMaxParts = 16;                           // parts per sequence while parts fit a chunk
// Word 3 of a raw (untyped, stride 0) buffer descriptor.
constexpr int kRawBufferWord3 = 0x00020000;

// Order-preserving map from fp32 to uint32 (-0 is folded onto +0 first); the
// radix passes of the threshold search work on these keys.
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
// First-pass bins of the ratio-mode search: kProbBins equal-width bins over
// the probability range [0, 1].  prob_bin is non-decreasing in the value:
// values below 1/4096 (and -inf) go to bin 0, values from 4095/4096 up (and
// +inf) to the last bin; a NaN lands in the last bin (ratio mode requires
// finite gates, so this only keeps the index in range).  v * 4096 is exact,
// so bin b holds exactly the values in [b/4096, (b+1)/4096) (open-ended for
// the end bins), which is how the gather pass tests membership.
constexpr int kProbBins = 4096;
constexpr int kMaxCand = 1024;          // values of one bin ranked directly
__device__ __forceinline__ int prob_bin(float v) {
    return (int)fmaxf(fminf(v * (float)kProbBins, (float)(kProbBins - 1)), 0.f);
}

// Inclusive prefix sum over the 64 lanes of a wave with DPP row shifts and
// row broadcasts (lanes that a step does not write add zero).
__device__ __forceinline__ int wave_incl_scan(int x) {
    int s = x + __builtin_amdgcn_update_dpp(0, x, 0x111, 0xf, 0xf, true);   // row_shr:1
    s += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xf, 0xf, true);          // row_shr:2
    s += __builtin_amdgcn_update_dpp(0, x, 0x113, 0xf, 0xf, true);          // row_shr:3
    s += __builtin_amdgcn_update_dpp(0, s, 0x114, 0xf, 0xe, false);         // row_shr:4
    s += __builtin_amdgcn_update_dpp(0, s, 0x118, 0xf, 0xc, false);         // row_shr:8
    s += __builtin_amdgcn_update_dpp(0, s, 0x142, 0xa, 0xf, false);         // row_bcast:15
    s += __builtin_amdgcn_update_dpp(0, s, 0x143, 0xc, 0xf, false);         // row_bcast:31
    return s;
}

// Block-wide exclusive prefix sum of one int per thread, and the block total
// (blockDim.x = kSelThreads).  s_wave: kSelWaves ints of LDS.
__device__ __forceinline__ int block_excl_scan(int v, int *s_wave, int &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int incl = wave_incl_scan(v);
    if (lane == 63)
        s_wave[wave] = incl;
    __syncthreads();
    const int wt = wave_incl_scan(lane < kSelWaves ? s_wave[lane] : 0);
    total = __builtin_amdgcn_readlane(wt, kSelWaves - 1);
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int before = wv > 0 ? __builtin_amdgcn_readlane(wt, wv - 1) : 0;
    __syncthreads();
    return before + incl - v;
}

// Block-wide sum (every thread gets it).
__device__ __forceinline__ int block_sum(int v, int *s_wave) {
    int total;
    block_excl_scan(v, s_wave, total);
    return total;
}

// Block-wide minimum and maximum of the keys (every thread gets both).
__device__ __forceinline__ void block_min_max(uint32_t &mn, uint32_t &mx, uint32_t *s_u) {
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) {
        mn = min(mn, (uint32_t)__shfl_xor((int)mn, d, 64));
        mx = max(mx, (uint32_t)__shfl_xor((int)mx, d, 64));
    }
    if ((threadIdx.x & 63) == 0) {
        s_u[threadIdx.x >> 6] = mn;
        s_u[kSelWaves + (threadIdx.x >> 6)] = mx;
    }
    __syncthreads();
    for (int i = 0; i < kSelWaves; i++) {
        mn = min(mn, s_u[i]);
        mx = max(mx, s_u[kSelWaves + i]);
    }
    __syncthreads();
}

// Selection, one 1024-thread workgroup per (part, sequence): blockIdx.y is
// the sequence, blockIdx.x the part, and part p writes the tokens
// [p * part_tokens, (p + 1) * part_tokens) of the sequence.  part_tokens is
// 4096 times a power of two up to kSelChunk, or a multiple of kSelChunk, so
// a part never straddles two chunks.
//
// kThreshold: find thr[b] (ratio mode, every part of the sequence finds the
// same value) or take the given one, and part 0 writes thr[b]; otherwise read
// thr[b].  kWrite: compact the part (offset = the counts of the earlier
// sequences in cnt, plus the selected tokens of the sequence before the
// part); otherwise (one part per sequence) write the sequence's count to
// cnt[b].
//
// The gates of one chunk of kSelChunk tokens stay in registers: slot j of
// thread tid holds token c0 + 1024 j + tid, so the lanes of wave w hold the
// 64 consecutive tokens of block 16 j + w of the chunk.  Slots past the
// chunk's end hold -inf, which is never selected (gate > thr is false for
// every thr), and a wave skips the slots none of its lanes holds a token in.
//
// Ratio mode: the threshold is the gate of ascending rank T-k-1.  A histogram
// over kProbBins probability bins finds the bin that holds it (the -inf
// fillers of the visited slots rank first, so the rank is shifted by their
// count); when that bin holds at most kMaxCand values they are gathered into
// LDS and the threshold is the one with the right number of smaller values.
// Otherwise radix passes of at most 12 bits over order-preserving uint32 keys
// start below the bits all of the sequence's keys share (the common prefix of
// the smallest and the largest key), so that gates spread over a narrow range
// still spread over the histogram bins; a pass whose chosen bin holds a
// single key ends the search.
//
// Compaction: z = gate > thr in fp32 (NaN never passes, -0 equals +0).  One
// ballot per slot gives each block's selected count (kept in LDS), one scan
// of the 512 block counts gives each block's first rank, and a token's rank
// adds the selected lanes below it (mbcnt).
template <bool kThreshold, bool kWrite>
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const int32_t *__restrict__ cu, int B, const float *__restrict__ gate, int mode, float fixed,
    double ratio, float *__restrict__ thr, int32_t *__restrict__ cnt, int32_t *__restrict__ sel_idx,
    int32_t cap, int32_t *__restrict__ cu_sel, int32_t *__restrict__ tok2sel, int part_tokens,
    int32_t *__restrict__ zero_words, int n_zero) {
    __shared__ int hist[kProbBins];           // histogram, then the block counts
    __shared__ int s_wave[kSelWaves];
    __shared__ uint32_t s_u[2 * kSelWaves];
    __shared__ int s_bin, s_rank, s_bincnt, s_ncand;
    __shared__ float s_thr;
    __shared__ float cand[kMaxCand];          // values of the threshold's probability bin
    const int b = blockIdx.y, part = blockIdx.x, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // the control words of the launch that follows (first workgroup)
    if (kWrite && b == 0 && part == 0 && tid < n_zero)
        zero_words[tid] = 0;
    const int64_t base = cu[b];
    const int T = cu[b + 1] - (int)base;
    const int p0 = part * part_tokens;
    if (part > 0 && p0 >= T)
        return;                               // an empty part (the whole workgroup)

    const long long k = (kThreshold && mode == 1) ? (long long)floor(ratio * (double)T) : 0;
    const bool search = kThreshold && mode == 1 && k < T;   // ratio mode, k < T
    // Gates of one chunk (token c0 + j * 1024 + tid in g[j]); a sequence
    // that fits in one chunk is loaded once.
    const bool resident = T <= kSelChunk;
    float g[kKeysPerThread];
    // The chunk is read through a buffer descriptor that covers exactly its
    // tokens, with each load's whole offset in the bounds-checked VGPR
    // offset, so the loads need no condition and are all in flight at once.
    auto load_chunk = [&](int c0) {
        const int n = min(T - c0, kSelChunk);
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(gate + base + c0), (short)0, n * 4, kRawBufferWord3);
#pragma unroll
        for (int j = 0; j < kKeysPerThread; j++) {
            const float v = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(r, (j * kSelThreads + tid) * 4, 0, 0));
            g[j] = j * kSelThreads < n - tid ? v : -__builtin_inff();
        }
    };
    // Slots of the chunk at c0 in which some lane of wave w holds a token.
    auto wave_slots = [&](int c0, int w) {
        const int n = min(T - c0, kSelChunk) - w * 64;
        return n > 0 ? min(kKeysPerThread, (n + kSelThreads - 1) / kSelThreads) : 0;
    };
    if (resident)
        load_chunk(0);

    float thr_v;
    if constexpr (kThreshold) {
        if (mode == 2)
            fixed = thr[0];                   // the device-held threshold
        if (mode != 1) {
            thr_v = fixed;                    // a NaN threshold selects nothing
        } else if (!search) {
            thr_v = -__builtin_inff();
        } else {
            // ascending rank of the threshold among the visited values:
            // T - k - 1 among the gates, after the -inf fillers
            int rank0 = (int)(T - k - 1);
            for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                int visited = 0;
                for (int w = 0; w < kSelWaves; w++)
                    visited += wave_slots(c0, w) * 64;
                rank0 += visited - min(T - c0, kSelChunk);
            }
            // The bin that holds the value of ascending rank `rank`, of nb
            // counted bins (4 per thread): s_bin, the rank within it
            // (s_rank) and its count (s_bincnt).
            auto pick_bin = [&](int nb, int rank) {
                int own = 0;
                int c4[4];
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    const int bin = tid * 4 + j;
                    c4[j] = bin < nb ? hist[bin] : 0;
                    own += c4[j];
                }
                int total;
                int run = block_excl_scan(own, s_wave, total);
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    if (c4[j] > 0 && rank >= run && rank < run + c4[j]) {
                        s_bin = tid * 4 + j;
                        s_rank = rank - run;
                        s_bincnt = c4[j];
                    }
                    run += c4[j];
                }
                __syncthreads();
            };
            // First pass: kProbBins bins of equal width over the probability
            // range [0, 1].  Gates are probabilities, so the bins split them
            // finely; the values in the threshold's bin are gathered and
            // ranked among themselves.
            for (int i = tid; i < kProbBins; i += kSelThreads)
                hist[i] = 0;
            if (tid == 0) {
                s_ncand = 0;
                s_thr = -__builtin_inff();
            }
            __syncthreads();
            for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                if (!resident)
                    load_chunk(c0);
                const int ns = __builtin_amdgcn_readfirstlane(wave_slots(c0, wave));
#pragma unroll
                for (int j = 0; j < kKeysPerThread; j++)
                    if (j < ns)
                        atomicAdd(&hist[prob_bin(g[j])], 1);
            }
            __syncthreads();
            pick_bin(kProbBins, rank0);
            const int pbin = s_bin, prank = s_rank, pcnt = s_bincnt;
            if (pcnt <= kMaxCand) {
                // gather the bin's values: min(v, 1) in [lo, hi) is the same
                // test as prob_bin(v) == pbin (NaN: min gives 1, last bin)
                const float lo = pbin == 0 ? -__builtin_inff() : (float)pbin * (1.f / kProbBins);
                const float hi = pbin == kProbBins - 1 ? 2.f : (float)(pbin + 1) * (1.f / kProbBins);
                for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                    if (!resident)
                        load_chunk(c0);
                    const int ns = __builtin_amdgcn_readfirstlane(wave_slots(c0, wave));
#pragma unroll
                    for (int j = 0; j < kKeysPerThread; j++)
                        if (j < ns && fminf(g[j], 1.f) >= lo && fminf(g[j], 1.f) < hi) {
                            const int at = atomicAdd(&s_ncand, 1);
                            if (at < kMaxCand)
                                cand[at] = g[j];
                        }
                }
                __syncthreads();
                // the value with prank values below it (ties: the one whose
                // run of equal values covers prank); -0 is reported as +0
                if (tid < pcnt) {
                    const float x = cand[tid];
                    int lt = 0, le = 0;
                    for (int i = 0; i < pcnt; i++) {
                        const float y = cand[i];
                        lt += y < x;
                        le += y <= x;
                    }
                    if (lt <= prank && prank < le)
                        s_thr = x + 0.f;
                }
                __syncthreads();
                thr_v = s_thr;
            } else {
                // A bin too full to rank directly (gates outside [0, 1], or
                // many close or equal values): radix passes over the keys.
                int rank = rank0;
                uint32_t mn = 0xFFFFFFFFu, mx = 0u;
                for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                    if (!resident)
                        load_chunk(c0);
                    const int ns = __builtin_amdgcn_readfirstlane(wave_slots(c0, wave));
#pragma unroll
                    for (int j = 0; j < kKeysPerThread; j++)
                        if (j < ns) {
                            mn = min(mn, float_key(g[j]));
                            mx = max(mx, float_key(g[j]));
                        }
                }
                block_min_max(mn, mx, s_u);
                uint32_t prefix = mn;
                if (mn != mx) {
                    int hi = 31 - __clz(mn ^ mx);           // highest bit that differs
                    uint32_t pmask = ~((2u << hi) - 1u);    // bits every key shares
                    prefix = mn & pmask;
                    while (hi >= 0) {
                        const int nbits = min(12, hi + 1);
                        const int sh = hi + 1 - nbits;
                        const int nb = 1 << nbits;
                        for (int i = tid; i < nb; i += kSelThreads)
                            hist[i] = 0;
                        __syncthreads();
                        for (int c0 = 0; c0 < T; c0 += kSelChunk) {
                            if (!resident)
                                load_chunk(c0);
                            const int ns = __builtin_amdgcn_readfirstlane(wave_slots(c0, wave));
                            // Consecutive slots of a thread are 1024 tokens
                            // apart, so their digits are unrelated: one
                            // atomic per key.
#pragma unroll
                            for (int j = 0; j < kKeysPerThread; j++) {
                                const uint32_t key = float_key(g[j]);
                                if (j < ns && (key & pmask) == prefix)
                                    atomicAdd(&hist[(key >> sh) & (uint32_t)(nb - 1)], 1);
                            }
                        }
                        __syncthreads();
                        pick_bin(nb, rank);
                        prefix |= (uint32_t)s_bin << sh;
                        pmask |= (uint32_t)(nb - 1) << sh;
                        rank = s_rank;
                        const bool unique = s_bincnt == 1;
                        __syncthreads();
                        hi = sh - 1;
                        if (hi >= 0 && unique && resident) {
                            // one key left in the bin: it is the threshold
                            const int ns = __builtin_amdgcn_readfirstlane(wave_slots(0, wave));
#pragma unroll
                            for (int j = 0; j < kKeysPerThread; j++)
                                if (j < ns && (float_key(g[j]) & pmask) == prefix)
                                    s_u[0] = float_key(g[j]);
                            __syncthreads();
                            prefix = s_u[0];
                            break;
                        }
                    }
                }
                thr_v = key_float(prefix);
            }
        }
        if (part == 0 && tid == 0)
            thr[b] = thr_v;
    } else {
        thr_v = thr[b];
    }
    // selected tokens of the chunk in registers (per wave)
    auto chunk_count = [&](int c0) {
        const int ns = __builtin_amdgcn_readfirstlane(wave_slots(c0, wave));
        int n = 0;
#pragma unroll
        for (int j = 0; j < kKeysPerThread; j++)
            if (j < ns)
                n += __builtin_popcountll(__builtin_amdgcn_ballot_w64(g[j] > thr_v));
        return n;                              // wave-uniform
    };

    if constexpr (!kWrite) {
        int mine = 0;
        for (int c0 = 0; c0 < T; c0 += kSelChunk) {
            if (!resident)
                load_chunk(c0);
            mine += chunk_count(c0);
        }
        const int total = block_sum(lane == 0 ? mine : 0, s_wave);
        if (tid == 0)
            cnt[b] = total;
    } else {
        int offset = 0;
        if (B > 1) {
            int mine = 0;
            for (int i = tid; i < b; i += kSelThreads)
                mine += cnt[i];
            offset = block_sum(mine, s_wave);
        }
        if (part == 0 && tid == 0)
            cu_sel[b] = offset;
        const int p1 = part == (int)gridDim.x - 1 ? T : min(T, p0 + part_tokens);
        int end_count = offset;               // selected tokens before p1 (with the offset)
        if (p0 < p1) {
            // the chunk that holds the part, and the selected tokens before it
            const int cs = (p0 / kSelChunk) * kSelChunk;
            int before = 0;
            for (int c0 = 0; c0 < cs; c0 += kSelChunk) {
                load_chunk(c0);
                before += chunk_count(c0);
            }
            before = offset + (cs > 0 ? block_sum(lane == 0 ? before : 0, s_wave) : 0);
            if (!resident)
                load_chunk(cs);
            // selected count of each 64-token block of the chunk: lane j of
            // the wave collects slot j's count, one LDS write per wave
            const int ns = __builtin_amdgcn_readfirstlane(wave_slots(cs, wave));
            int bc = 0;
#pragma unroll
            for (int j = 0; j < kKeysPerThread; j++)
                if (j < ns) {
                    const int nj = __builtin_popcountll(__builtin_amdgcn_ballot_w64(g[j] > thr_v));
                    bc = lane == j ? nj : bc;
                }
            if (lane < kKeysPerThread)
                hist[lane * kSelWaves + wave] = bc;
            __syncthreads();
            // exclusive scan of the 512 block counts in token order (block
            // 16 j + w at hist[16 j + w])
            constexpr int kBlocks = kKeysPerThread * kSelWaves;
            int chunk_total;
            const int v = tid < kBlocks ? hist[tid] : 0;
            const int ex = block_excl_scan(v, s_wave, chunk_total);
            if (tid < kBlocks)
                hist[tid] = ex;
            __syncthreads();
            // ranks and writes of the part's tokens
#pragma unroll
            for (int j = 0; j < kKeysPerThread; j++) {
                const int j0 = cs + j * kSelThreads;      // first token of slot j
                if (j0 + kSelThreads <= p0 || j0 >= p1 || j >= ns)
                    continue;                             // (wave-uniform)
                const bool z = g[j] > thr_v;
                const uint64_t bal = __builtin_amdgcn_ballot_w64(z);
                const int r = before + hist[j * kSelWaves + wave] +
                              (int)__builtin_amdgcn_mbcnt_hi(
                                  (uint32_t)(bal >> 32),
                                  __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
                const int t = j0 + tid;
                if (t >= p0 && t < p1) {
                    const bool keep = z && r < cap;
                    if (keep)
                        sel_idx[r] = (int32_t)(base + t);
                    if (tok2sel)
                        tok2sel[base + t] = keep ? r : -1;
                }
            }
            end_count = before + chunk_total;
        }
        // the part holding the last token of the last sequence closes cu_sel
        if (b == B - 1 && p1 == T && tid == 0)
            cu_sel[B] = end_count;
    }
}

__global__ __launch_bounds__(1024) void sparse_plan_kernel(const int32_t *cu, int B, PlanArgs p) {
    __shared__ plan_detail::PlanLds<kPlanLdsEntriesStandalone> lds;
    build_plan<1024>(cu, B, p, lds);
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

hipError_t launch_select(const int32_t *cu_seqlens, int num_seqs, int max_seqlen,
                         const float *gate, int mode, float threshold, double ratio,
                         int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                         int32_t *tok2sel, float *thr, int32_t *seq_counts, hipStream_t s,
                         int32_t *zero_words, int n_zero) {
    // parts of 4096 * 2^i tokens, at most kMaxParts per sequence unless a
    // part would exceed one chunk (then one part per chunk)
    int part_tokens = kPartUnit;
    while (part_tokens < kSelChunk &&
           ((long long)max_seqlen + part_tokens - 1) / part_tokens > kMaxParts)
        part_tokens *= 2;
    const int parts = (int)std::max(1LL, ((long long)max_seqlen + part_tokens - 1) / part_tokens);
    if (num_seqs == 1) {
        hipLaunchKernelGGL((select_kernel<true, true>), dim3(parts, 1), dim3(kSelThreads), 0, s,
                           cu_seqlens, 1, gate, mode, threshold, ratio, thr, seq_counts, sel_idx,
                           sel_capacity, cu_sel, tok2sel, part_tokens, zero_words, n_zero);
        return hipGetLastError();
    }
    hipLaunchKernelGGL((select_kernel<true, false>), dim3(1, num_seqs), dim3(kSelThreads), 0, s,
                       cu_seqlens, num_seqs, gate, mode, threshold, ratio, thr, seq_counts,
                       sel_idx, sel_capacity, cu_sel, tok2sel, part_tokens, nullptr, 0);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((select_kernel<false, true>), dim3(parts, num_seqs), dim3(kSelThreads), 0,
                       s, cu_seqlens, num_seqs, gate, mode, threshold, ratio, thr, seq_counts,
                       sel_idx, sel_capacity, cu_sel, tok2sel, part_tokens, zero_words, n_zero);
    return hipGetLastError();
}

hipError_t launch_sparse_plan(const int32_t *cu_seqlens, int num_seqs, const PlanArgs &plan,
                              hipStream_t s) {
    hipLaunchKernelGGL(sparse_plan_kernel, dim3(1), dim3(1024), 0, s, cu_seqlens, num_seqs, plan);
    return hipGetLastError();
}

}  // namespace logo
