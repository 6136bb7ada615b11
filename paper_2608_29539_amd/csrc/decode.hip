// decode.hip -- one autoregressive decoding step of the layer (Sec. 3.3 and
// App. B, Autoregressive Decoding).  Each of B sequences appends one token
// whose key and value are already the last row of its cache.  The token's
// query attends to the last min(L, w) cached keys (local branch); when its
// gate passes the threshold it also attends to the whole cache (global
// branch), and the two outputs are ContextNorm-ed and fused as in the layer.
//
// Only selected tokens do global work: every global work item tests its
// sequence's routing decision z_b = gate[b] > thr (fp32, strict) and an
// unselected one exits at once, so an unselected token costs one window of
// the cache (the paper's batched decoding instead launches the dense kernel
// for every row and masks).
//
//   decode_attn_kernel    split-KV attention, one workgroup per (branch,
//                         sequence, KV head, head group, chunk of keys):
//                         the GH query heads of one KV head share every K/V
//                         row read, sixteen lanes (one DPP row) cover one
//                         2d-byte row, and each of the 16 streams keeps two
//                         rows in flight.  Writes the chunk's unnormalised
//                         (O, m, l) per head.  One extra workgroup writes
//                         the compacted list of selected sequences, each
//                         sequence's rank and the count.
//   decode_combine_kernel merges the chunks of each (sequence, head) in chunk
//                         order, applies ContextNorm to each branch and the
//                         fusion, and rounds once to bf16.
//
// The cache is read once per branch (HBM-bound); the arithmetic is fp32
// (bf16 dot products accumulate in fp32 with v_dot2), so no MFMA is needed.
#include "logo_internal.h"

namespace logo {
namespace {

constexpr int kDecThreads = 256;
constexpr int kLanesPerRow = 16;            // lanes that share one cached K / V row
constexpr int kStreams = kDecThreads / kLanesPerRow;   // keys per workgroup step
constexpr int kPrefetch = 2;                // rows in flight per stream
constexpr float kNegInfD = -__builtin_inff();
constexpr float kLazyD = 8.f;               // exp2-domain headroom of the running max

typedef uint32_t u32x4d __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2d __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// One lane's slice of a cached row: N 32-bit words (one 16- or 8-byte load).
// A struct rather than a dependent-size ext_vector_type: element reads of
// such a vector passed by value into a lambda compiled to element 0.
template <int N>
struct alignas(4 * N) Words {
    uint32_t w[N];
};

// Sum over the 16 lanes of a DPP row, returned in every lane: rotations by 8
// and 4 within the row, then the two quad swaps.
template <int Ctrl>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), Ctrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f<0x128>(x);   // row_ror:8
    x += dpp_f<0x124>(x);   // row_ror:4
    x += dpp_f<0x4E>(x);    // quad_perm [2,3,0,1]
    x += dpp_f<0xB1>(x);    // quad_perm [1,0,3,2]
    return x;
}

// The token's routing decision z_b = gate[b] > thr (fp32, strict: a NaN
// gate or threshold selects nothing), taken identically by every workgroup
// that needs it.
__device__ __forceinline__ float decode_threshold(const DecodeArgs &a) {
    return a.sel_mode == 2 ? a.thr_dev[0] : a.thr_host;
}

// The compacted list of selected sequences (ascending), each sequence's rank
// (-1 if unselected) and the count: one workgroup, ballot + mbcnt ranks and
// a carry over chunks of kDecThreads sequences.
__device__ void build_active_list(const DecodeArgs &a) {
    __shared__ int s_cnt[kDecThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const float thr = decode_threshold(a);
    int carry = 0;
    for (int c0 = 0; c0 < a.num_seqs; c0 += kDecThreads) {
        const int b = c0 + tid;
        const bool z = b < a.num_seqs && a.gate[b] > thr;
        const uint64_t m = __ballot(z);
        const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0));
        if (lane == 0)
            s_cnt[wave] = (int)__popcll(m);
        __syncthreads();
        int before = carry, total = 0;
        for (int i = 0; i < kDecThreads / 64; i++) {
            if (i < wave)
                before += s_cnt[i];
            total += s_cnt[i];
        }
        if (b < a.num_seqs) {
            const int r = before + below;
            a.rank_of[b] = z ? r : -1;
            if (z)
                a.act[r] = b;
        }
        carry += total;
        __syncthreads();                         // s_cnt is rewritten by the next chunk
    }
    if (tid == 0)
        a.n_act[0] = carry;
}

// (m, l, acc) of stream b merged into stream a (exp2 domain).
__device__ __forceinline__ void merge_into(float &ma, float &la, float &mb, float &lb, float *aa,
                                           const float *ab, int n) {
    const float M = fmaxf(ma, mb);
    const float Mc = M == kNegInfD ? 0.f : M;
    const float fa = __builtin_amdgcn_exp2f(ma - Mc), fb = __builtin_amdgcn_exp2f(mb - Mc);
    la = la * fa + lb * fb;
    for (int i = 0; i < n; i++)
        aa[i] = aa[i] * fa + ab[i] * fb;
    ma = M;
}

template <int D, int GH>
__global__ __launch_bounds__(kDecThreads) void decode_attn_kernel(const DecodeArgs a) {
    constexpr int DE = D / kLanesPerRow;  // d values per lane
    constexpr int DW = DE / 2;            // 32-bit words per lane (2 bf16 each)
    typedef Words<DW> frag_t;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int e = lane % kLanesPerRow, sid = tid / kLanesPerRow;

    // work item -> (branch, sequence, kv head, head group, chunk); the last
    // workgroup builds the list of selected sequences instead
    const int per_row = a.hkv * a.nhg;
    int item = blockIdx.x;
    if (item == a.n_local_items + a.n_global_items) {
        build_active_list(a);
        return;
    }
    const bool global = item >= a.n_local_items;
    if (global)
        item -= a.n_local_items;
    const int nch = global ? a.chunks_global : a.chunks_local;
    const int c = item % nch;
    const int rest = item / nch;
    const int hgi = rest % a.nhg;
    const int kvh = (rest / a.nhg) % a.hkv;
    const int b = rest / per_row;                // sequence
    if (global && !(a.gate[b] > decode_threshold(a)))
        return;                                  // an unselected token: window only
    const int64_t base = a.cu[b];
    const int L = a.cu[b + 1] - (int)base;
    const int lo = global ? 0 : max(0, L - a.window);
    const int k0 = lo + c * a.kc;
    const int k1 = min(L, k0 + a.kc);
    if (k0 >= k1)
        return;                                  // a chunk past this sequence's keys
    // this item's partials: [item][GH][m, l, acc[D]]
    float *out_part = (global ? a.part_global : a.part_local) + (int64_t)item * GH * (D + 2);
    const uint16_t *kc_ = global ? a.k_g : a.k;
    const uint16_t *vc_ = global ? a.v_g : a.v;
    const uint16_t *qv = global ? a.q_g : a.q;
    const int h0 = kvh * a.group + hgi * GH;     // first query head of the group

    // Query slices (bf16 pairs) of the GH heads.
    uint32_t q2[GH][DW];
#pragma unroll
    for (int hh = 0; hh < GH; hh++) {
        const uint32_t *qp = (const uint32_t *)(qv + ((int64_t)b * a.hq + h0 + hh) * D + e * DE);
#pragma unroll
        for (int i = 0; i < DW; i++)
            q2[hh][i] = qp[i];
    }
    float m[GH], l[GH], acc[GH][DE];
#pragma unroll
    for (int hh = 0; hh < GH; hh++) {
        m[hh] = kNegInfD;
        l[hh] = 0.f;
#pragma unroll
        for (int i = 0; i < DE; i++)
            acc[hh][i] = 0.f;
    }

    const int64_t row_stride = (int64_t)a.hkv * D;    // elements between cached tokens
    const uint16_t *kbase = kc_ + (base * a.hkv + kvh) * (int64_t)D + e * DE;
    const uint16_t *vbase = vc_ + (base * a.hkv + kvh) * (int64_t)D + e * DE;
    auto load_row = [&](const uint16_t *p, int j) {
        return *(const frag_t *)(p + (int64_t)j * row_stride);
    };
    // Online softmax update with key row (kw, vw).
    auto consume = [&](const frag_t kw, const frag_t vw) {
        float s[GH];
#pragma unroll
        for (int hh = 0; hh < GH; hh++) {
            float d0 = 0.f;
#pragma unroll
            for (int i = 0; i < DW; i++)
                d0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2d, q2[hh][i]),
                                                    __builtin_bit_cast(bf16x2d, kw.w[i]), d0, false);
            s[hh] = row16_sum(d0) * a.scale_log2;
        }
        float vf[DE];
#pragma unroll
        for (int i = 0; i < DW; i++) {
            vf[2 * i] = bf16_lo(vw.w[i]);
            vf[2 * i + 1] = bf16_hi(vw.w[i]);
        }
#pragma unroll
        for (int hh = 0; hh < GH; hh++) {
            if (s[hh] > m[hh] + kLazyD) {
                // the running max moves (always on the first key)
                const float alpha = __builtin_amdgcn_exp2f(m[hh] - s[hh]);
                l[hh] *= alpha;
#pragma unroll
                for (int i = 0; i < DE; i++)
                    acc[hh][i] *= alpha;
                m[hh] = s[hh];
            }
            const float p = __builtin_amdgcn_exp2f(s[hh] - m[hh]);
            l[hh] += p;
#pragma unroll
            for (int i = 0; i < DE; i++)
                acc[hh][i] = fmaf(p, vf[i], acc[hh][i]);
        }
    };

    // Each stream (16 lanes) walks keys k0 + sid, k0 + sid + kStreams, ...,
    // with kPrefetch rows in flight in a ring of registers (the ring index is
    // a compile-time constant: the loop body covers kPrefetch keys).
    int j = k0 + sid;
    frag_t kr[kPrefetch], vr[kPrefetch];
#pragma unroll
    for (int p = 0; p < kPrefetch; p++) {
        const int jp = j + p * kStreams;
        if (jp < k1) {
            kr[p] = load_row(kbase, jp);
            vr[p] = load_row(vbase, jp);
        }
    }
    for (; j < k1; j += kPrefetch * kStreams) {
#pragma unroll
        for (int p = 0; p < kPrefetch; p++) {
            const int jc = j + p * kStreams;
            if (jc < k1) {
                const frag_t kw = kr[p], vw = vr[p];
                const int jn = jc + kPrefetch * kStreams;
                if (jn < k1) {
                    kr[p] = load_row(kbase, jn);
                    vr[p] = load_row(vbase, jn);
                }
                consume(kw, vw);
            }
        }
    }

    // Merge the streams of the wave (lanes with the same e), then the waves.
#pragma unroll
    for (int hh = 0; hh < GH; hh++) {
#pragma unroll
        for (int sh = kLanesPerRow; sh < 64; sh <<= 1) {
            float mo = __shfl_xor(m[hh], sh, 64), lo_ = __shfl_xor(l[hh], sh, 64);
            float ao[DE];
#pragma unroll
            for (int i = 0; i < DE; i++)
                ao[i] = __shfl_xor(acc[hh][i], sh, 64);
            merge_into(m[hh], l[hh], mo, lo_, acc[hh], ao, DE);
        }
    }
    __shared__ float s_m[4][GH], s_l[4][GH];
    __shared__ float s_acc[4][GH][D];
    if (lane < kLanesPerRow) {
#pragma unroll
        for (int hh = 0; hh < GH; hh++) {
            if (lane == 0) {
                s_m[wave][hh] = m[hh];
                s_l[wave][hh] = l[hh];
            }
#pragma unroll
            for (int i = 0; i < DE; i++)
                s_acc[wave][hh][e * DE + i] = acc[hh][i];
        }
    }
    __syncthreads();
    // thread t < GH * D: head t / D, element t % D
    for (int t = tid; t < GH * D; t += kDecThreads) {
        const int hh = t / D, x = t % D;
        float M = s_m[0][hh], Lw = s_l[0][hh], A = s_acc[0][hh][x];
        for (int w2 = 1; w2 < 4; w2++) {
            float mb = s_m[w2][hh], lb = s_l[w2][hh];
            const float ab = s_acc[w2][hh][x];
            merge_into(M, Lw, mb, lb, &A, &ab, 1);
        }
        float *op = out_part + hh * (D + 2);
        op[2 + x] = A;
        if (x == 0) {
            op[0] = M;
            op[1] = Lw;
        }
    }
}

// One wave per (sequence, query head), four per workgroup.  A branch's
// chunks are merged in one pass: the largest chunk maximum first (lane c
// holds chunk c), then every chunk's weight 2^(m_c - M), then the weighted
// sum, in which the wave's lanes are 4 chunk groups x 16 element groups
// (lane = 16 cg + eg: chunks cg, cg+4, ..., elements D/16 eg ..), so each
// lane's dependent chain is a quarter of the chunks; two shuffle steps add
// the chunk groups.  Lanes 0..15 then hold the row (D/16 elements each) for
// ContextNorm, the fusion and the store.  At most 128 chunks per branch.
constexpr int kMaxChunks = 128;

template <int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(const DecodeArgs a) {
    constexpr int EL = D / 16;                    // elements per lane
    __shared__ float s_w[4][kMaxChunks];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int cg = lane >> 4, eg = lane & 15;
    const int job = blockIdx.x * 4 + wave;
    if (job >= a.num_seqs * a.hq)
        return;                                   // whole wave: no barrier below
    const int b = job / a.hq, h = job % a.hq;
    const int L = a.cu[b + 1] - a.cu[b];
    // chunks of this sequence (clamped to the planned slots: max_seqlen bounds L)
    const int n_loc = min((min(L, a.window) + a.kc - 1) / a.kc, a.chunks_local);
    const int n_glb = min((L + a.kc - 1) / a.kc, a.chunks_global);
    const int r = a.rank_of[b];
    const float p = a.gate[b];
    const int kvh = h / a.group, hg = (h % a.group) / a.gh, hh = (h % a.group) % a.gh;
    float *w = s_w[wave];
    // O / l of one branch of sequence `row`; lane eg's elements
    auto branch = [&](const float *parts, int row, int nch, int chunks_stride, float (&o)[EL]) {
        const int64_t item0 = (((int64_t)row * a.hkv + kvh) * a.nhg + hg) * chunks_stride;
        auto slot = [&](int c) { return parts + ((item0 + c) * a.gh + hh) * (D + 2); };
        float mc[2], lc[2];
        float M = kNegInfD;
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int c = lane + 64 * i;
            mc[i] = c < nch ? slot(c)[0] : kNegInfD;
            lc[i] = c < nch ? slot(c)[1] : 0.f;
            M = fmaxf(M, mc[i]);
        }
#pragma unroll
        for (int sh = 1; sh < 64; sh <<= 1)
            M = fmaxf(M, __shfl_xor(M, sh, 64));
        const float Mc = M == kNegInfD ? 0.f : M;
        float lsum = 0.f;
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int c = lane + 64 * i;
            const float wc = c < nch ? __builtin_amdgcn_exp2f(mc[i] - Mc) : 0.f;
            if (c < nch)
                w[c] = wc;
            lsum = fmaf(wc, lc[i], lsum);
        }
#pragma unroll
        for (int sh = 1; sh < 64; sh <<= 1)
            lsum += __shfl_xor(lsum, sh, 64);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        float A[EL];
#pragma unroll
        for (int i = 0; i < EL; i++)
            A[i] = 0.f;
#pragma unroll 2
        for (int c = cg; c < nch; c += 4) {
            const float wc = w[c];
            const float *pp = slot(c) + 2 + eg * EL;
#pragma unroll
            for (int i = 0; i < EL; i++)
                A[i] = fmaf(wc, pp[i], A[i]);
        }
#pragma unroll
        for (int i = 0; i < EL; i++) {
            A[i] += __shfl_xor(A[i], 16, 64);
            A[i] += __shfl_xor(A[i], 32, 64);
        }
        __builtin_amdgcn_wave_barrier();
        const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
#pragma unroll
        for (int i = 0; i < EL; i++)
            o[i] = A[i] * inv;
    };
    auto norm = [&](float (&o)[EL], const float *gain) {
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < EL; i++)
            ss = fmaf(o[i], o[i], ss);
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1)
            ss += __shfl_xor(ss, sh, 64);
        const float rn = 1.f / sqrtf(ss / (float)D + a.eps);
#pragma unroll
        for (int i = 0; i < EL; i++)
            o[i] = o[i] * rn * (gain ? gain[h * D + eg * EL + i] : 1.f);
    };
    float ol[EL];
    branch(a.part_local, b, n_loc, a.chunks_local, ol);
    norm(ol, a.gain_local);
    if (r >= 0) {
        float og[EL];
        branch(a.part_global, b, n_glb, a.chunks_global, og);
        norm(og, a.gain_global);
#pragma unroll
        for (int i = 0; i < EL; i++)
            ol[i] = (1.f - p) * ol[i] + p * og[i];
    }
    if (cg != 0)
        return;
    uint16_t *op = a.out + ((int64_t)b * a.hq + h) * D + eg * EL;
#pragma unroll
    for (int i = 0; i < EL; i++)
        op[i] = __builtin_bit_cast(uint16_t, (__bf16)ol[i]);
}

template <int D, int GH>
hipError_t launch_attn_gh(const DecodeArgs &a, hipStream_t s) {
    const int grid = a.n_local_items + a.n_global_items + 1;   // + the list builder
    hipLaunchKernelGGL((decode_attn_kernel<D, GH>), dim3(grid), dim3(kDecThreads), 0, s, a);
    return hipGetLastError();
}

template <int D>
hipError_t launch_attn_d(const DecodeArgs &a, hipStream_t s) {
    if (a.gh == 4)
        return launch_attn_gh<D, 4>(a, s);
    if (a.gh == 2)
        return launch_attn_gh<D, 2>(a, s);
    return launch_attn_gh<D, 1>(a, s);
}

}  // namespace

hipError_t launch_decode(const DecodeArgs &a, hipStream_t s) {
    hipError_t e = a.head_dim == 128 ? launch_attn_d<128>(a, s) : launch_attn_d<64>(a, s);
    if (e != hipSuccess)
        return e;
    const int grid = (a.num_seqs * a.hq + 3) / 4;
    if (a.head_dim == 128)
        hipLaunchKernelGGL((decode_combine_kernel<128>), dim3(grid), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((decode_combine_kernel<64>), dim3(grid), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace logo
