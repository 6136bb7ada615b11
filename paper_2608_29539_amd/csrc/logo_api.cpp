// logo_api.cpp -- the C ABI of liblogo (include/logo.h): argument validation,
// workspace carving and stream-ordered kernel launches.  Every argument is
// checked on the host before the first launch, so an error status means that
// nothing was enqueued.  The library holds no device memory and never
// synchronises (unless LOGO_DEBUG_SYNC=1 is set, which synchronises the
// stream after each launch to localise device faults).
#include "../../include/logo.h"
#include "logo_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>

using namespace logo;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

bool debug_sync() {
    static const bool on = [] {
        const char *e = std::getenv("LOGO_DEBUG_SYNC");
        return e && e[0] == '1';
    }();
    return on;
}

logo_status hip_status(hipError_t e, hipStream_t s) {
    if (e != hipSuccess)
        return LOGO_ERR_HIP;
    if (debug_sync() && hipStreamSynchronize(s) != hipSuccess)
        return LOGO_ERR_HIP;
    return LOGO_OK;
}

logo_status check_problem(const logo_problem *p) {
    if (!p || !p->cu_seqlens)
        return LOGO_ERR_NULL;
    if (p->num_seqs < 1 || p->total_tokens < 0 || p->max_seqlen < 0)
        return LOGO_ERR_SHAPE;
    if (p->total_tokens > 0 && p->max_seqlen < 1)
        return LOGO_ERR_SHAPE;
    if (p->num_q_heads < 1 || p->num_kv_heads < 1 || p->num_q_heads % p->num_kv_heads != 0)
        return LOGO_ERR_SHAPE;
    if (p->head_dim != 64 && p->head_dim != 128)
        return LOGO_ERR_UNSUPPORTED;
    if (p->window < 1)
        return LOGO_ERR_ARG;
    if (std::isnan(p->softmax_scale) || std::isinf(p->softmax_scale))
        return LOGO_ERR_ARG;
    // element offsets are 64-bit in the kernels; token and row indices are 32-bit
    if ((long long)p->total_tokens * p->num_q_heads >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    if (p->cu_seqlens_host) {
        const int32_t *cu = p->cu_seqlens_host;
        if (cu[0] != 0 || cu[p->num_seqs] != p->total_tokens)
            return LOGO_ERR_SHAPE;
        for (int b = 0; b < p->num_seqs; b++) {
            const long long T = (long long)cu[b + 1] - cu[b];
            if (T < 0 || T > p->max_seqlen)
                return LOGO_ERR_SHAPE;
        }
    }
    return LOGO_OK;
}

double softmax_scale(const logo_problem *p) {
    return p->softmax_scale > 0.f ? (double)p->softmax_scale : 1.0 / std::sqrt((double)p->head_dim);
}

float scale_log2(const logo_problem *p) {
    return (float)(softmax_scale(p) * 1.4426950408889634);   // log2(e)
}

AttnArgs make_args(const logo_problem *p, const TilePlan &tp) {
    AttnArgs a;
    std::memset(&a, 0, sizeof a);
    a.cu_seqlens = p->cu_seqlens;
    a.num_seqs = p->num_seqs;
    a.hq = p->num_q_heads;
    a.hkv = p->num_kv_heads;
    a.group = p->num_q_heads / p->num_kv_heads;
    a.hpw = tp.hpw;
    a.tpw = tp.tpw;
    a.n_hg = tp.n_hg;
    a.window = p->window;
    a.ntile_max = (p->max_seqlen + tp.tpw - 1) / tp.tpw;
    a.scale_log2 = scale_log2(p);
    return a;
}

// --- workspace layouts ------------------------------------------------------
struct SelectWs {
    size_t thr, counts, total;
};
SelectWs select_ws(const logo_problem *p) {
    SelectWs w;
    size_t off = 0;
    w.thr = off;
    off += align_up(sizeof(float) * (size_t)p->num_seqs);
    w.counts = off;
    off += align_up(sizeof(int32_t) * (size_t)p->num_seqs);
    w.total = off;
    return w;
}

struct GlobalWs {
    size_t tiles, tiles_tmp, scratch, queue, split_cnt, partial, total;
    int max_tiles, slots, stride;
};
GlobalWs global_ws(const logo_problem *p, int32_t cap) {
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads,
                                       global_waves(p->num_q_heads, p->num_kv_heads));
    GlobalWs w;
    w.max_tiles = (int)((cap + tp.tpw - 1) / tp.tpw + p->num_seqs);
    w.slots = split_slots(w.max_tiles, tp.n_hg);
    w.stride = (w.max_tiles > p->num_seqs ? w.max_tiles : p->num_seqs) + 1;
    const size_t entries = (size_t)w.max_tiles + (size_t)w.slots;
    size_t off = 0;
    w.tiles = off;
    off += align_up(sizeof(SparseTile) * entries);
    w.tiles_tmp = off;
    off += align_up(sizeof(SparseTile) * entries);
    w.scratch = off;
    off += align_up(sizeof(int32_t) * 2 * (size_t)w.stride);
    w.queue = off;
    off += align_up(sizeof(int32_t) * (1 + kQueues));
    w.split_cnt = off;
    off += align_up(sizeof(int32_t) * (size_t)w.slots * tp.n_hg);
    w.partial = off;
    off += align_up(sizeof(float) * partial_floats(p->head_dim) * (size_t)w.slots * tp.n_hg);
    w.total = off;
    return w;
}

// logo_attn_fwd runs the fused epilogues, so its only large buffers are the
// compact fp32 (1-p) Norm^L and p Norm^G of the selected rows.
struct FwdWs {
    size_t sel_ws, glob_ws, lc, gc, ctl, sel_idx, cu_sel, tok2sel, thr, aperm, total;
};
// aperm: room for the permuted copy of the LP query transform's matrices
// (logo_attn_fwd_qphi with LOGO_PHI_LP).
FwdWs fwd_ws(const logo_problem *p, int32_t cap, bool aperm = false) {
    const size_t row = (size_t)p->num_q_heads * p->head_dim * sizeof(float);
    FwdWs w;
    size_t off = 0;
    w.sel_ws = off;
    off += align_up(select_ws(p).total);
    w.glob_ws = off;
    off += align_up(global_ws(p, cap).total);
    w.lc = off;
    off += align_up(row * (size_t)cap);
    // the one-launch layer: p Norm^G of the selected rows, control words
    w.gc = off;
    off += align_up(row * (size_t)cap);
    w.ctl = off;
    off += align_up(sizeof(int32_t) * kLayerCtlWords);
    w.sel_idx = off;
    off += align_up(sizeof(int32_t) * (size_t)cap);
    w.cu_sel = off;
    off += align_up(sizeof(int32_t) * ((size_t)p->num_seqs + 1));
    w.tok2sel = off;
    off += align_up(sizeof(int32_t) * (size_t)p->total_tokens);
    w.thr = off;
    off += align_up(sizeof(float) * (size_t)p->num_seqs);
    w.aperm = off;
    if (aperm)
        off += align_up(2 * (size_t)p->num_q_heads * p->head_dim * p->head_dim);
    w.total = off;
    return w;
}

// Decoding: keys per chunk (a multiple of 32, at least 256, at most 128
// chunks per cache), query heads per work item (the largest of 4, 2, 1
// dividing the group), and the workspace of the partial results.
// logo_attn_bwd: dO^L / dO^G (bf16), the compact Q^G rows, the row sums
// Delta, the per-row gate terms and the gain-gradient partials.
constexpr int kFusionBwdMaxBlocks = 2048;
struct BwdWs {
    size_t dol, dog, qc, delta_l, delta_g, side, part_l, part_g, part_tmp, total;
    int blocks, tokens_per_block, part_rows;
};
BwdWs bwd_ws(const logo_problem *p, int32_t cap) {
    const size_t N = (size_t)p->total_tokens, H = (size_t)p->num_q_heads, d = p->head_dim;
    const int P = fusion_bwd_tokens_per_pass(p->num_q_heads, p->head_dim);
    const long long passes = ((long long)N + P - 1) / P;
    BwdWs w;
    // at most 4096 partial rows (the two-pass column sum's reach)
    const long long max_blocks = std::min<long long>(kFusionBwdMaxBlocks, 4096 / P);
    w.blocks = (int)(passes < max_blocks ? passes : max_blocks);
    if (w.blocks < 1)
        w.blocks = 1;
    w.tokens_per_block = (int)((passes + w.blocks - 1) / w.blocks) * P;
    w.part_rows = w.blocks * P;
    size_t off = 0;
    w.dol = off;
    off += align_up(2 * N * H * d);
    w.dog = off;
    off += align_up(2 * (size_t)cap * H * d);
    w.qc = off;
    off += align_up(2 * (size_t)cap * H * d);
    w.delta_l = off;
    off += align_up(4 * H * N);
    w.delta_g = off;
    off += align_up(4 * H * (size_t)cap);
    w.side = off;
    off += align_up(4 * N * H);
    w.part_l = off;
    off += align_up(4 * (size_t)w.part_rows * H * d);
    w.part_g = off;
    off += align_up(4 * (size_t)w.part_rows * H * d);
    w.part_tmp = off;
    off += align_up(4 * (size_t)gain_grad_chunks(w.part_rows) * H * d);
    w.total = off;
    return w;
}

// standalone query-sparse backward: compact Q rows and Delta
struct GlobalBwdWs {
    size_t qc, delta, total;
};
GlobalBwdWs global_bwd_ws(const logo_problem *p, int32_t cap) {
    GlobalBwdWs w;
    const size_t H = (size_t)p->num_q_heads, d = p->head_dim;
    w.qc = 0;
    w.delta = align_up(2 * (size_t)cap * H * d);
    w.total = w.delta + align_up(4 * H * (size_t)cap);
    return w;
}

size_t dense_bwd_ws(const logo_problem *p) {
    return align_up(sizeof(float) * (size_t)p->num_q_heads * (size_t)p->total_tokens);
}

BwdArgs make_bwd_args(const logo_problem *p) {
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, kWavesLocal);
    BwdArgs a;
    std::memset(&a, 0, sizeof a);
    a.cu_seqlens = p->cu_seqlens;
    a.num_seqs = p->num_seqs;
    a.hq = p->num_q_heads;
    a.hkv = p->num_kv_heads;
    a.group = p->num_q_heads / p->num_kv_heads;
    a.hpw = tp.hpw;
    a.tpw = tp.tpw;
    a.n_hg = tp.n_hg;
    a.window = p->window;
    a.ntile_max = (p->max_seqlen + tp.tpw - 1) / tp.tpw;
    a.scale_log2 = scale_log2(p);
    a.scale = (float)softmax_scale(p);
    return a;
}

struct DecodePlan {
    int kc, gh, nhg, chunks_local, chunks_global;
    long long n_local_items, n_global_items;
    size_t act, rank_of, n_act, part_local, part_global, total;
};
DecodePlan decode_plan(const logo_problem *p) {
    DecodePlan d;
    const long long maxL = p->max_seqlen > 0 ? p->max_seqlen : 1;
    // Keys per chunk: at least 512 (a workgroup's fixed cost -- query loads,
    // stream and wave merges, the partial's store -- is then small next to
    // its 256 KiB of K / V per KV head at d = 128), at most 128 chunks per
    // cache, a multiple of 32.
    long long kc = (maxL + 127) / 128;
    kc = ((kc + 31) / 32) * 32;
    d.kc = (int)(kc < 512 ? 512 : kc);
    const int g = p->num_q_heads / p->num_kv_heads;
    d.gh = g % 4 == 0 ? 4 : (g % 2 == 0 ? 2 : 1);
    d.nhg = g / d.gh;
    const long long wl = maxL < p->window ? maxL : p->window;
    d.chunks_local = (int)((wl + d.kc - 1) / d.kc);
    d.chunks_global = (int)((maxL + d.kc - 1) / d.kc);
    const long long per_row = (long long)p->num_kv_heads * d.nhg;
    d.n_local_items = (long long)p->num_seqs * per_row * d.chunks_local;
    d.n_global_items = (long long)p->num_seqs * per_row * d.chunks_global;
    const size_t slot = sizeof(float) * (size_t)d.gh * (p->head_dim + 2);
    size_t off = 0;
    d.act = off;
    off += align_up(sizeof(int32_t) * (size_t)p->num_seqs);
    d.rank_of = off;
    off += align_up(sizeof(int32_t) * (size_t)p->num_seqs);
    d.n_act = off;
    off += align_up(sizeof(int32_t));
    d.part_local = off;
    off += align_up(slot * (size_t)d.n_local_items);
    d.part_global = off;
    off += align_up(slot * (size_t)d.n_global_items);
    d.total = off;
    return d;
}

logo_status check_ws(void *ws, size_t ws_bytes, size_t need) {
    if (need == 0)
        return LOGO_OK;
    if (!ws || ((uintptr_t)ws % kAlign) != 0 || ws_bytes < need)
        return LOGO_ERR_WORKSPACE;
    return LOGO_OK;
}

int64_t ratio_capacity(const logo_problem *p, double ratio) {
    if (!p->cu_seqlens_host)
        return p->total_tokens;
    int64_t s = 0;
    for (int b = 0; b < p->num_seqs; b++) {
        const int64_t T = (int64_t)p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b];
        int64_t k = (int64_t)std::floor(ratio * (double)T);
        s += k < T ? k : T;
    }
    return s;
}

logo_status check_select_args(const logo_problem *p, const float *gate, logo_sel_mode mode,
                              float threshold, double ratio, const int32_t *sel_idx,
                              int32_t cap, const int32_t *cu_sel, const float *thr_out) {
    if ((!gate && p->total_tokens > 0) || !cu_sel)
        return LOGO_ERR_NULL;
    if (cap < 0)
        return LOGO_ERR_SHAPE;
    if (cap > 0 && !sel_idx)
        return LOGO_ERR_NULL;
    if (mode == LOGO_SEL_THRESHOLD) {
        if (std::isnan(threshold))
            return LOGO_ERR_ARG;
    } else if (mode == LOGO_SEL_THRESHOLD_DEVICE) {
        if (!thr_out)
            return LOGO_ERR_NULL;
    } else if (mode == LOGO_SEL_RATIO) {
        if (!(ratio >= 0.0 && ratio <= 1.0))
            return LOGO_ERR_ARG;
        if ((int64_t)cap < ratio_capacity(p, ratio))
            return LOGO_ERR_SHAPE;
    } else {
        return LOGO_ERR_ARG;
    }
    return LOGO_OK;
}

logo_status run_select(const logo_problem *p, const float *gate, logo_sel_mode mode,
                       float threshold, double ratio, int32_t *sel_idx, int32_t cap,
                       int32_t *cu_sel, int32_t *tok2sel, float *thr_out, char *ws,
                       hipStream_t s, int32_t *zero_words = nullptr, int n_zero = 0) {
    const SelectWs w = select_ws(p);
    float *thr = thr_out ? thr_out : (float *)(ws + w.thr);
    return hip_status(launch_select(p->cu_seqlens, p->num_seqs, p->max_seqlen, gate, (int)mode,
                                    threshold, ratio, sel_idx, cap, cu_sel, tok2sel, thr,
                                    (int32_t *)(ws + w.counts), s, zero_words, n_zero),
                      s);
}

// Persistent grid of the global kernel on the current device: its CUs times
// the kernel's resident workgroups per CU, rounded up to a multiple of the
// work queues.  The CU count is queried once per device and the occupancy
// once per head dim (std::call_once); a call only asks which device is
// current.
constexpr int kMaxDevices = 64;
struct DeviceCache {
    std::once_flag once;
    int cus = 0;
};
DeviceCache g_devices[kMaxDevices];

// Scratch memory of logo_decode_noalloc: a fixed device array instead of a
// caller workspace (see that entry point).  Every GPU the library runs on
// holds its own copy from the module's load until the process ends.  In host
// code the array's name is only a host-side stand-in; its address on each
// device is looked up once, with that device current, and only that address
// is passed to kernels.
static __device__ __align__(256) unsigned char scratch[LOGO_NOALLOC_SCRATCH_BYTES];

struct ScratchSlot {
    std::once_flag once;
    void *ptr = nullptr;
};
ScratchSlot g_scratch[kMaxDevices];

logo_status device_scratch(void **ptr) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return LOGO_ERR_HIP;
    ScratchSlot &sl = g_scratch[dev];
    std::call_once(sl.once, [&] {
        void *a = nullptr;
        if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) == hipSuccess)
            sl.ptr = a;
    });
    if (!sl.ptr)
        return LOGO_ERR_HIP;
    *ptr = sl.ptr;
    return LOGO_OK;
}

logo_status device_cus(int &cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return LOGO_ERR_HIP;
    DeviceCache &c = g_devices[dev];
    std::call_once(c.once, [&] {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
            c.cus = n;
    });
    cus = c.cus;
    return cus > 0 ? LOGO_OK : LOGO_ERR_HIP;
}

// Resident workgroups per CU of an attention kernel (mode x head dim x
// waves), queried once each.
std::once_flag g_occ_once[3][2][2];
int g_occ[3][2][2];

int blocks_per_cu(int mode, int head_dim, int waves) {
    const int di = head_dim == 128 ? 1 : 0, wi = waves == 8 ? 1 : 0;
    std::call_once(g_occ_once[mode][di][wi],
                   [&] { g_occ[mode][di][wi] = attention_blocks_per_cu(mode, head_dim, waves); });
    return g_occ[mode][di][wi];
}

// Persistent grid of the one-launch layer (occupancy queried once per head
// dim and workgroup size), a multiple of the work queues.
std::once_flag g_layer_occ_once[2][2];
int g_layer_occ[2][2];

logo_status layer_grid(int head_dim, int waves, int &grid) {
    int cus = 0;
    const logo_status st = device_cus(cus);
    if (st != LOGO_OK)
        return st;
    const int di = head_dim == 128 ? 1 : 0, wi = waves == 8 ? 1 : 0;
    std::call_once(g_layer_occ_once[di][wi],
                   [&] { g_layer_occ[di][wi] = layer_blocks_per_cu(head_dim, waves); });
    grid = cus * g_layer_occ[di][wi];
    grid = ((grid + kQueues - 1) / kQueues) * kQueues;
    return LOGO_OK;
}

logo_status global_grid(int head_dim, int waves, int &grid) {
    int cus = 0;
    const logo_status st = device_cus(cus);
    if (st != LOGO_OK)
        return st;
    grid = cus * blocks_per_cu(kModeGlobal, head_dim, waves);
    grid = ((grid + kQueues - 1) / kQueues) * kQueues;
    return LOGO_OK;
}

// The arguments of the global branch's tile plan (work table in the global
// workspace `ws`) and the persistent grid that consumes it.
logo_status global_plan(const logo_problem *p, const int32_t *sel_idx, const int32_t *cu_sel,
                        int32_t cap, char *ws, PlanArgs &pa, int &grid) {
    const int waves = global_waves(p->num_q_heads, p->num_kv_heads);
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, waves);
    const GlobalWs w = global_ws(p, cap);
    const logo_status st = global_grid(p->head_dim, waves, grid);
    if (st != LOGO_OK)
        return st;
    // no more persistent workgroups than the plan can make items (tiles,
    // each split at most kMaxSplit ways, times head groups): a small
    // selection does not pay for draining the queues of a full grid
    const long long most = (long long)w.max_tiles * kMaxSplit * tp.n_hg;
    if (most < grid)
        grid = (int)(((most + kQueues - 1) / kQueues) * kQueues);
    pa.cu_sel = cu_sel;
    pa.sel_idx = sel_idx;
    pa.tpw = tp.tpw;
    pa.cap = cap;
    pa.max_seqlen = p->max_seqlen;
    pa.n_hg = tp.n_hg;
    pa.grid_wgs = grid;
    pa.split_slots = w.slots;
    pa.stride = w.stride;
    pa.extra_blocks = 0;
    pa.tmp = (SparseTile *)(ws + w.tiles_tmp);
    pa.out = (SparseTile *)(ws + w.tiles);
    pa.scratch = (int32_t *)(ws + w.scratch);
    pa.queue = (int32_t *)(ws + w.queue);
    pa.split_cnt = (int32_t *)(ws + w.split_cnt);
    return LOGO_OK;
}

// Fused-epilogue inputs (logo_attn_fwd only).
// qphi: the global branch's query transform applied by the global kernel as
// it loads the selected rows (0 none, 1 LP from the permuted copy aperm of
// lp_a, which the local launch writes, 2 SO with qs / qb).
struct FusedEpi {
    const int32_t *tok2sel;
    const float *gate;
    const float *gain;
    float eps;
    float *lc;
    logo_bf16 *out;
    int qphi;
    const logo_bf16 *lp_a;
    uint16_t *aperm;
    const float *qs, *qb;
};

void set_fused(AttnArgs &a, const FusedEpi *f, const float *gain) {
    a.tok2sel = f->tok2sel;
    a.gate = f->gate;
    a.gain = gain;
    a.eps = f->eps;
    a.lc = f->lc;
    a.out_bf16 = f->out;
}

// o: raw fp32 O^L (f == NULL) or the fused epilogue (f != NULL).  plan:
// with the fused epilogue, one extra workgroup of the launch builds the
// global branch's work table.
logo_status run_local(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                      const logo_bf16 *v, float *o, const FusedEpi *f, const float *gain,
                      hipStream_t s, const PlanArgs *plan = nullptr, float *lse = nullptr) {
    if (p->total_tokens == 0)
        return LOGO_OK;
    const int waves = local_waves(p->num_q_heads, p->num_kv_heads);
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, waves);
    AttnArgs a = make_args(p, tp);
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = o;
    a.lse = lse;
    a.lse_stride = p->total_tokens;
    if (f)
        set_fused(a, f, gain);
    if (f && plan) {
        a.plan_wg = 1;
        a.plan = *plan;
    }
    if (f && f->qphi == 1) {
        a.prep_wgs = p->num_q_heads;
        a.prep_a = f->lp_a;
        a.aperm = f->aperm;
    }
    // items: head groups x the sequences' tiles back to back (sum_b
    // ceil(T_b / tpw) <= ceil(N / tpw) + B - 1); persistent workgroups, a
    // multiple of the 8 XCDs, take every item_stride-th item
    const long long items =
        (long long)tp.n_hg * ((p->total_tokens + tp.tpw - 1) / tp.tpw + p->num_seqs);
    if (items >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    int cus = 0;
    logo_status st = device_cus(cus);
    if (st != LOGO_OK)
        return st;
    long long wgs = (long long)cus * blocks_per_cu(kModeLocal, p->head_dim, waves);
    wgs = ((wgs + kQueues - 1) / kQueues) * kQueues;
    if (wgs > items)
        wgs = items;
    a.n_items = (int32_t)items;
    a.item_stride = (int32_t)wgs;
    return hip_status(launch_attention(kModeLocal, f ? (o ? kEpiFusedTrain : kEpiFused) : kEpiRaw,
                                       p->head_dim, waves, a,
                                       (int)wgs + a.plan_wg + a.prep_wgs, s),
                      s);
}

// built: the plan of a fused launch whose extra workgroup has already
// written the work table (its arguments and grid from global_plan); NULL
// builds the table with a launch of its own first.
logo_status run_global(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                       const logo_bf16 *v, const int32_t *sel_idx, const int32_t *cu_sel,
                       int32_t cap, float *o, const FusedEpi *f, const float *gain, char *ws,
                       hipStream_t s, hipEvent_t after_plan = nullptr,
                       const PlanArgs *built = nullptr, int built_grid = 0,
                       float *lse = nullptr) {
    if (p->total_tokens == 0 || cap == 0)
        return after_plan ? hip_status(hipEventRecord(after_plan, s), s) : LOGO_OK;
    const int waves = global_waves(p->num_q_heads, p->num_kv_heads);
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, waves);
    const GlobalWs w = global_ws(p, cap);
    PlanArgs pa;
    int grid = 0;
    logo_status st;
    if (built) {
        pa = *built;
        grid = built_grid;
    } else {
        if ((st = global_plan(p, sel_idx, cu_sel, cap, ws, pa, grid)) != LOGO_OK)
            return st;
        st = hip_status(launch_sparse_plan(p->cu_seqlens, p->num_seqs, pa, s), s);
        if (st != LOGO_OK)
            return st;
    }
    if (after_plan && hipEventRecord(after_plan, s) != hipSuccess)
        return LOGO_ERR_HIP;
    AttnArgs a = make_args(p, tp);
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = o;
    a.sel_idx = sel_idx;
    a.tiles = pa.out;
    a.queue = pa.queue;
    a.split_cnt = pa.split_cnt;
    a.partial = (float *)(ws + w.partial);
    a.lse = lse;
    a.lse_stride = cap;
    if (f) {
        set_fused(a, f, gain);
        a.qphi = f->qphi;
        a.aperm = f->aperm;
        a.qphi_s = f->qs;
        a.qphi_b = f->qb;
    }
    return hip_status(
        launch_attention(kModeGlobal, f ? (o ? kEpiFusedTrain : kEpiFused) : kEpiRaw, p->head_dim,
                         waves, a, grid, s),
        s);
}

// logo_attn_fwd's launches: both branches in one launch (layer_kernel) when
// their workgroups have the same waves and the local branch gives each
// persistent workgroup at least kLayerMinLocalBlocks KV blocks of work --
// enough to cover the work table, which the launch's first workgroup builds
// (~15-20 us) while the others run local items; otherwise the local launch,
// then the global one.  LOGO_FWD_LAUNCHES=1 or 2 picks one or the other where
// both are possible (tests run both).
constexpr long long kLayerMinLocalBlocks = 8;
struct LayerPlan {
    int waves = 0, grid = 0;
    long long items = 0;          // local items (an upper bound; the valid ones a prefix)
    long long extra_blocks = 0;   // their KV blocks, ~(w + tpw) / 64 + 1 each
};

logo_status layer_plan(const logo_problem *p, LayerPlan &lp) {
    lp = LayerPlan{};
    const int waves = layer_waves(p->num_q_heads, p->num_kv_heads);
    if (waves == 0 || p->total_tokens == 0)
        return LOGO_OK;
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, waves);
    int grid = 0;
    const logo_status st = layer_grid(p->head_dim, waves, grid);
    if (st != LOGO_OK)
        return st;
    const long long tiles = (p->total_tokens + tp.tpw - 1) / tp.tpw;
    const long long span = std::min<long long>(p->window, p->max_seqlen) + tp.tpw;
    lp.waves = waves;
    lp.grid = grid;
    lp.items = (long long)tp.n_hg * (tiles + p->num_seqs);
    lp.extra_blocks = (long long)tp.n_hg * tiles * ((span + kBlockN - 1) / kBlockN + 1);
    return LOGO_OK;
}

bool use_one_launch(const LayerPlan &lp) {
    if (lp.waves == 0)
        return false;
    const char *e = std::getenv("LOGO_FWD_LAUNCHES");
    if (e && e[0] == '1')
        return true;
    if (e && e[0] == '2')
        return false;
    return lp.extra_blocks >= kLayerMinLocalBlocks * lp.grid;
}

// The one-launch layer: the local items and the global work table's items in
// one persistent grid, whose first workgroup builds the table
// (layer_kernel).  gc / ctl: the compact p Norm^G buffer and the launch's
// control words (cleared by the selection kernel before it).  The selected
// rows' output is written afterwards by launch_sel_sum.
logo_status run_layer(const logo_problem *p, const LayerPlan &lp, const logo_bf16 *q,
                      const logo_bf16 *k, const logo_bf16 *v, const logo_bf16 *qg,
                      const logo_bf16 *kg, const logo_bf16 *vg, const int32_t *sel_idx,
                      const int32_t *cu_sel, int32_t cap, const FusedEpi *f,
                      const float *gain_local, const float *gain_global, float *gc, int32_t *ctl,
                      char *glob_ws, hipStream_t s) {
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, lp.waves);
    PlanArgs pa;
    int grid_g = 0;
    const logo_status st = global_plan(p, sel_idx, cu_sel, cap, glob_ws, pa, grid_g);
    if (st != LOGO_OK)
        return st;
    if (lp.items >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    // the local items count into the table's split threshold as the grid's
    // other work
    pa.grid_wgs = lp.grid;
    pa.extra_blocks = (int64_t)lp.extra_blocks;
    AttnArgs a = make_args(p, tp);
    a.q = q;
    a.k = k;
    a.v = v;
    a.qg = qg;
    a.kg = kg;
    a.vg = vg;
    set_fused(a, f, gain_local);
    a.gain_g = gain_global;
    a.gc = gc;
    a.ctl = ctl;
    a.sel_idx = sel_idx;
    a.plan = pa;
    a.tiles = pa.out;
    a.queue = pa.queue;
    a.split_cnt = pa.split_cnt;
    a.partial = (float *)(glob_ws + global_ws(p, cap).partial);
    a.n_items = (int32_t)lp.items;
    a.qphi = f->qphi;
    a.aperm = f->aperm;
    a.qphi_s = f->qs;
    a.qphi_b = f->qb;
    if (f->qphi == 1) {
        a.prep_wgs = p->num_q_heads;
        a.prep_a = f->lp_a;
    }
    return hip_status(launch_layer(p->head_dim, lp.waves, a, lp.grid, s), s);
}

logo_status fwd_impl(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                     const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                     const logo_bf16 *v_g, const float *gate, logo_sel_mode mode, float threshold,
                     double ratio, const float *gain_local, const float *gain_global, float eps,
                     logo_bf16 *out, int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                     int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                     logo_stream stream, void *const *events, int qphi = 0,
                     const logo_bf16 *lp_a = nullptr, const float *so_s = nullptr,
                     const float *so_b = nullptr) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (p->total_tokens > 0 && (!q || !k || !v || !gate || !out))
        return LOGO_ERR_NULL;
    if ((qphi == 1 && !lp_a) || (qphi == 2 && (!so_s || !so_b)))
        return LOGO_ERR_NULL;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    if (sel_idx && sel_capacity == 0 && p->total_tokens > 0)
        return LOGO_ERR_SHAPE;
    int32_t cap = sel_capacity;
    if (!sel_idx && cap == 0)
        cap = mode == LOGO_SEL_RATIO && ratio >= 0.0 && ratio <= 1.0
                  ? (int32_t)ratio_capacity(p, ratio)
                  : p->total_tokens;
    if (!(eps >= 0.f) || std::isinf(eps))
        return LOGO_ERR_ARG;
    const FwdWs w = fwd_ws(p, cap, qphi == 1);
    st = check_ws(ws, ws_bytes, w.total);
    if (st != LOGO_OK)
        return st;
    char *base = (char *)ws;
    int32_t *sel = sel_idx ? sel_idx : (int32_t *)(base + w.sel_idx);
    int32_t *cus = cu_sel ? cu_sel : (int32_t *)(base + w.cu_sel);
    int32_t *t2s = tok2sel ? tok2sel : (int32_t *)(base + w.tok2sel);
    float *thr = thr_out ? thr_out : (float *)(base + w.thr);
    st = check_select_args(p, gate, mode, threshold, ratio, sel, cap, cus, thr_out);
    if (st != LOGO_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    const FusedEpi fe{t2s, gate, nullptr, eps, (float *)(base + w.lc), out,
                      qphi, lp_a, (uint16_t *)(base + w.aperm), so_s, so_b};
    auto mark = [&](int i) -> logo_status {
        if (events && hipEventRecord((hipEvent_t)events[i], s) != hipSuccess)
            return LOGO_ERR_HIP;
        return LOGO_OK;
    };

    if ((st = mark(0)) != LOGO_OK)
        return st;
    // Selection, then the local branch with the fused epilogue: Norm^L(O^L)
    // straight to `out` for unselected tokens, (1-p) Norm^L(O^L) to the
    // compact buffer for selected ones; one extra workgroup of that launch
    // builds the global branch's tile plan.  Then the global branch finishes
    // the selected rows.
    const bool with_plan = p->total_tokens > 0 && cap > 0;
    LayerPlan lp;
    if (with_plan && (st = layer_plan(p, lp)) != LOGO_OK)
        return st;
    if (with_plan && use_one_launch(lp)) {
        // both branches in one launch, then the selected rows' sums
        int32_t *ctl = (int32_t *)(base + w.ctl);
        float *lc = (float *)(base + w.lc), *gc = (float *)(base + w.gc);
        st = run_select(p, gate, mode, threshold, ratio, sel, cap, cus, t2s, thr, base + w.sel_ws,
                        s, ctl, kLayerCtlWords);
        if (st != LOGO_OK || (st = mark(1)) != LOGO_OK)
            return st;
        st = run_layer(p, lp, q, k, v, q_g ? q_g : q, k_g ? k_g : k, v_g ? v_g : v, sel, cus, cap,
                       &fe, gain_local, gain_global, gc, ctl, base + w.glob_ws, s);
        if (st != LOGO_OK || (st = mark(2)) != LOGO_OK || (st = mark(3)) != LOGO_OK)
            return st;
        st = hip_status(launch_sel_sum(cap, p->num_q_heads, p->head_dim, cus, p->num_seqs, sel, lc,
                                       gc, out, s),
                        s);
        if (st != LOGO_OK)
            return st;
        return mark(4);
    }
    PlanArgs plan;
    int grid_g = 0;
    if (with_plan && (st = global_plan(p, sel, cus, cap, base + w.glob_ws, plan, grid_g)) != LOGO_OK)
        return st;
    st = run_select(p, gate, mode, threshold, ratio, sel, cap, cus, t2s, thr, base + w.sel_ws, s);
    if (st != LOGO_OK || (st = mark(1)) != LOGO_OK)
        return st;
    st = run_local(p, q, k, v, nullptr, &fe, gain_local, s, with_plan ? &plan : nullptr);
    if (st != LOGO_OK || (st = mark(2)) != LOGO_OK)
        return st;
    st = run_global(p, q_g ? q_g : q, k_g ? k_g : k, v_g ? v_g : v, sel, cus, cap, nullptr, &fe,
                    gain_global, base + w.glob_ws, s, events ? (hipEvent_t)events[3] : nullptr,
                    &plan, grid_g);
    if (st != LOGO_OK)
        return st;
    return mark(4);
}

}  // namespace

extern "C" {

const char *logo_status_str(logo_status s) {
    switch (s) {
    case LOGO_OK: return "LOGO_OK";
    case LOGO_ERR_NULL: return "LOGO_ERR_NULL";
    case LOGO_ERR_SHAPE: return "LOGO_ERR_SHAPE";
    case LOGO_ERR_UNSUPPORTED: return "LOGO_ERR_UNSUPPORTED";
    case LOGO_ERR_ARG: return "LOGO_ERR_ARG";
    case LOGO_ERR_WORKSPACE: return "LOGO_ERR_WORKSPACE";
    case LOGO_ERR_HIP: return "LOGO_ERR_HIP";
    case LOGO_ERR_SCRATCH_LIMIT: return "LOGO_ERR_SCRATCH_LIMIT";
    }
    return "LOGO_ERR_UNKNOWN";
}

const char *logo_version(void) { return "0.1.0"; }

int logo_attn_fwd_launches(const logo_problem *p) {
    if (check_problem(p) != LOGO_OK)
        return -1;
    LayerPlan lp;
    if (layer_plan(p, lp) != LOGO_OK)
        return -1;
    return use_one_launch(lp) ? 1 : 2;
}

int64_t logo_ratio_capacity(const logo_problem *p, double ratio) {
    if (check_problem(p) != LOGO_OK || !(ratio >= 0.0 && ratio <= 1.0))
        return -1;
    return ratio_capacity(p, ratio);
}

logo_status logo_budget_update(const logo_problem *p, const int32_t *cu_sel, double rho,
                               float gamma, float *b_th, float *realized, logo_stream stream) {
    if (!p)
        return LOGO_ERR_NULL;
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (!cu_sel || !b_th)
        return LOGO_ERR_NULL;
    if (!(rho >= 0.0 && rho <= 1.0) || !(gamma >= 0.f) || std::isinf(gamma))
        return LOGO_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    return hip_status(launch_budget_update(cu_sel, p->num_seqs, p->total_tokens, rho, gamma,
                                           b_th, realized, s),
                      s);
}

float logo_pmask_initial_threshold(float gamma, int64_t pmask_steps) {
    return (float)(0.5 - (double)gamma * (double)pmask_steps);
}

size_t logo_workspace_bytes(const logo_problem *p, int entry, int32_t sel_capacity) {
    if (check_problem(p) != LOGO_OK || sel_capacity < 0)
        return 0;
    const int32_t cap = sel_capacity > 0 ? sel_capacity : p->total_tokens;
    switch (entry) {
    case LOGO_ENTRY_SELECT: return select_ws(p).total;
    case LOGO_ENTRY_GLOBAL: return global_ws(p, cap).total;
    case LOGO_ENTRY_FWD: return fwd_ws(p, cap).total;
    case LOGO_ENTRY_FWD_QPHI: return fwd_ws(p, cap, true).total;
    case LOGO_ENTRY_DECODE: return decode_plan(p).total;
    case LOGO_ENTRY_FWD_TRAIN: return fwd_ws(p, cap).total;
    case LOGO_ENTRY_BWD: return bwd_ws(p, cap).total;
    case LOGO_ENTRY_DENSE_BWD: return dense_bwd_ws(p);
    case LOGO_ENTRY_GLOBAL_BWD: return global_bwd_ws(p, cap).total;
    case LOGO_ENTRY_LOCAL:
    case LOGO_ENTRY_COMBINE:
    case LOGO_ENTRY_DENSE: return 0;
    }
    return 0;
}

logo_status logo_select(const logo_problem *p, const float *gate, logo_sel_mode mode,
                        float threshold, double ratio, int32_t *sel_idx, int32_t sel_capacity,
                        int32_t *cu_sel, int32_t *tok2sel, float *thr_out, void *ws,
                        size_t ws_bytes, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    st = check_select_args(p, gate, mode, threshold, ratio, sel_idx, sel_capacity, cu_sel,
                           thr_out);
    if (st != LOGO_OK)
        return st;
    st = check_ws(ws, ws_bytes, select_ws(p).total);
    if (st != LOGO_OK)
        return st;
    return run_select(p, gate, mode, threshold, ratio, sel_idx, sel_capacity, cu_sel, tok2sel,
                      thr_out, (char *)ws, (hipStream_t)stream);
}

logo_status logo_local_attn(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                            const logo_bf16 *v, float *o_local, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (p->total_tokens > 0 && (!q || !k || !v || !o_local))
        return LOGO_ERR_NULL;
    return run_local(p, q, k, v, o_local, nullptr, nullptr, (hipStream_t)stream);
}

logo_status logo_global_attn_sparse_q(const logo_problem *p, const logo_bf16 *q,
                                      const logo_bf16 *k, const logo_bf16 *v,
                                      const int32_t *sel_idx, const int32_t *cu_sel,
                                      int32_t sel_capacity, float *o_global, void *ws,
                                      size_t ws_bytes, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    if (!cu_sel)
        return LOGO_ERR_NULL;
    if (sel_capacity > 0 && p->total_tokens > 0 && (!q || !k || !v || !sel_idx || !o_global))
        return LOGO_ERR_NULL;
    if (sel_capacity > 0 && p->total_tokens > 0) {
        st = check_ws(ws, ws_bytes, global_ws(p, sel_capacity).total);
        if (st != LOGO_OK)
            return st;
    }
    return run_global(p, q, k, v, sel_idx, cu_sel, sel_capacity, o_global, nullptr, nullptr,
                      (char *)ws, (hipStream_t)stream);
}

logo_status logo_combine(const logo_problem *p, const float *o_local, const float *o_global,
                         const float *gate, const int32_t *tok2sel, const float *gain_local,
                         const float *gain_global, float eps, int apply_norm, logo_bf16 *out,
                         logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (p->total_tokens > 0 && (!o_local || !gate || !tok2sel || !out))
        return LOGO_ERR_NULL;
    if (!(eps >= 0.f) || std::isinf(eps))
        return LOGO_ERR_ARG;
    hipStream_t s = (hipStream_t)stream;
    return hip_status(launch_combine(p->total_tokens, p->num_q_heads, p->head_dim, o_local,
                                     o_global, gate, tok2sel, gain_local, gain_global, eps,
                                     apply_norm ? 1 : 0, out, s),
                      s);
}

logo_status logo_attn_fwd(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                          const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                          const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                          float threshold, double ratio, const float *gain_local,
                          const float *gain_global, float eps, logo_bf16 *out,
                          int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                          int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                          logo_stream stream) {
    return fwd_impl(p, q, k, v, q_g, k_g, v_g, gate, mode, threshold, ratio, gain_local,
                    gain_global, eps, out, sel_idx, sel_capacity, cu_sel, tok2sel, thr_out, ws,
                    ws_bytes, stream, nullptr);
}

logo_status logo_attn_fwd_qphi(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                               const logo_bf16 *v, logo_phi_kind q_phi, const logo_bf16 *A,
                               const float *s, const float *b, const logo_bf16 *k_g,
                               const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                               float threshold, double ratio, const float *gain_local,
                               const float *gain_global, float eps, logo_bf16 *out,
                               int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                               int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                               logo_stream stream) {
    if (q_phi != LOGO_PHI_LP && q_phi != LOGO_PHI_SO)
        return LOGO_ERR_ARG;
    return fwd_impl(p, q, k, v, nullptr, k_g, v_g, gate, mode, threshold, ratio, gain_local,
                    gain_global, eps, out, sel_idx, sel_capacity, cu_sel, tok2sel, thr_out, ws,
                    ws_bytes, stream, nullptr, q_phi == LOGO_PHI_LP ? 1 : 2, A, s, b);
}

logo_status logo_attn_fwd_profiled(const logo_problem *p, const logo_bf16 *q,
                                   const logo_bf16 *k, const logo_bf16 *v,
                                   const logo_bf16 *q_g, const logo_bf16 *k_g,
                                   const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                   float threshold, double ratio, const float *gain_local,
                                   const float *gain_global, float eps, logo_bf16 *out,
                                   int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                                   int32_t *tok2sel, float *thr_out, void *ws, size_t ws_bytes,
                                   logo_stream stream, void *const *events) {
    if (!events)
        return LOGO_ERR_NULL;
    for (int i = 0; i < 5; i++)
        if (!events[i])
            return LOGO_ERR_NULL;
    return fwd_impl(p, q, k, v, q_g, k_g, v_g, gate, mode, threshold, ratio, gain_local,
                    gain_global, eps, out, sel_idx, sel_capacity, cu_sel, tok2sel, thr_out, ws,
                    ws_bytes, stream, events);
}

logo_status logo_dense_causal_attn(const logo_problem *p, const logo_bf16 *q,
                                   const logo_bf16 *k, const logo_bf16 *v, logo_bf16 *out,
                                   logo_stream stream) {
    return logo_dense_causal_attn_fwd_train(p, q, k, v, out, nullptr, stream);
}

logo_status logo_dense_causal_attn_fwd_train(const logo_problem *p, const logo_bf16 *q,
                                             const logo_bf16 *k, const logo_bf16 *v,
                                             logo_bf16 *out, float *lse, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (p->total_tokens == 0)
        return LOGO_OK;
    if (!q || !k || !v || !out)
        return LOGO_ERR_NULL;
    const TilePlan tp = make_tile_plan(p->num_q_heads, p->num_kv_heads, kWavesGlobal);
    AttnArgs a = make_args(p, tp);
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = out;
    a.lse = lse;
    a.lse_stride = p->total_tokens;
    const long long grid = (long long)tp.n_hg * p->num_seqs * a.ntile_max;
    if (grid >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    hipStream_t s = (hipStream_t)stream;
    return hip_status(launch_attention(kModeDense, kEpiRaw, p->head_dim, kWavesGlobal, a, (int)grid, s), s);
}

}  // extern "C"

namespace {

// One decoding step.  noalloc: the scratch is the library's fixed device
// array (ws and ws_bytes are ignored), after the same argument checks.
logo_status decode_run(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                       const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                       const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                       float threshold, const float *thr_dev, const float *gain_local,
                       const float *gain_global, float eps, logo_bf16 *out, int32_t *active,
                       int32_t *n_active, void *ws, size_t ws_bytes, logo_stream stream,
                       bool noalloc) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (!q || !k || !v || !gate || !out)
        return LOGO_ERR_NULL;
    if (mode == LOGO_SEL_THRESHOLD) {
        if (std::isnan(threshold))
            return LOGO_ERR_ARG;
    } else if (mode == LOGO_SEL_THRESHOLD_DEVICE) {
        if (!thr_dev)
            return LOGO_ERR_NULL;
    } else {
        return LOGO_ERR_ARG;
    }
    if (!(eps >= 0.f) || std::isinf(eps))
        return LOGO_ERR_ARG;
    if (p->cu_seqlens_host)
        for (int b = 0; b < p->num_seqs; b++)
            if (p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b] < 1)
                return LOGO_ERR_SHAPE;
    if ((long long)p->num_seqs * p->num_q_heads >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    const DecodePlan d = decode_plan(p);
    if (d.n_local_items + d.n_global_items >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    if (noalloc) {
        if (d.total > (size_t)LOGO_NOALLOC_SCRATCH_BYTES)
            return LOGO_ERR_SCRATCH_LIMIT;
        if ((st = device_scratch(&ws)) != LOGO_OK)
            return st;
        ws_bytes = (size_t)LOGO_NOALLOC_SCRATCH_BYTES;
    }
    st = check_ws(ws, ws_bytes, d.total);
    if (st != LOGO_OK)
        return st;
    char *base = (char *)ws;
    DecodeArgs a;
    std::memset(&a, 0, sizeof a);
    a.q = q;
    a.k = k;
    a.v = v;
    a.q_g = q_g ? q_g : q;
    a.k_g = k_g ? k_g : k;
    a.v_g = v_g ? v_g : v;
    a.cu = p->cu_seqlens;
    a.gate = gate;
    a.gain_local = gain_local;
    a.gain_global = gain_global;
    a.eps = eps;
    a.scale_log2 = scale_log2(p);
    a.num_seqs = p->num_seqs;
    a.hq = p->num_q_heads;
    a.hkv = p->num_kv_heads;
    a.group = p->num_q_heads / p->num_kv_heads;
    a.head_dim = p->head_dim;
    a.window = p->window;
    a.gh = d.gh;
    a.nhg = d.nhg;
    a.kc = d.kc;
    a.chunks_local = d.chunks_local;
    a.chunks_global = d.chunks_global;
    a.n_local_items = (int32_t)d.n_local_items;
    a.n_global_items = (int32_t)d.n_global_items;
    a.act = active ? active : (int32_t *)(base + d.act);
    a.rank_of = (int32_t *)(base + d.rank_of);
    a.n_act = n_active ? n_active : (int32_t *)(base + d.n_act);
    a.part_local = (float *)(base + d.part_local);
    a.part_global = (float *)(base + d.part_global);
    a.out = out;
    a.sel_mode = (int32_t)mode;
    a.thr_host = threshold;
    a.thr_dev = thr_dev;
    hipStream_t s = (hipStream_t)stream;
    return hip_status(launch_decode(a, s), s);
}

}  // namespace

extern "C" {

logo_status logo_decode(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                        const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                        const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                        float threshold, const float *thr_dev, const float *gain_local,
                        const float *gain_global, float eps, logo_bf16 *out, int32_t *active,
                        int32_t *n_active, void *ws, size_t ws_bytes, logo_stream stream) {
    return decode_run(p, q, k, v, q_g, k_g, v_g, gate, mode, threshold, thr_dev, gain_local,
                      gain_global, eps, out, active, n_active, ws, ws_bytes, stream, false);
}

logo_status logo_decode_noalloc(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                                const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                                const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                float threshold, const float *thr_dev, const float *gain_local,
                                const float *gain_global, float eps, logo_bf16 *out,
                                int32_t *active, int32_t *n_active, logo_stream stream) {
    return decode_run(p, q, k, v, q_g, k_g, v_g, gate, mode, threshold, thr_dev, gain_local,
                      gain_global, eps, out, active, n_active, nullptr, 0, stream, true);
}

logo_status logo_gate_proj(int64_t n_tokens, int32_t d_model, const logo_bf16 *x,
                           const logo_bf16 *w_g, float *gate_out, logo_stream stream) {
    if (n_tokens < 0 || d_model < 1)
        return LOGO_ERR_SHAPE;
    if (d_model % 8 != 0)
        return LOGO_ERR_UNSUPPORTED;
    if (n_tokens == 0)
        return LOGO_OK;
    if (!x || !w_g || !gate_out)
        return LOGO_ERR_NULL;
    if ((uintptr_t)x % 16 != 0 || (uintptr_t)w_g % 16 != 0)
        return LOGO_ERR_ARG;
    if (n_tokens / 4 >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    hipStream_t s = (hipStream_t)stream;
    return hip_status(launch_gate_proj(n_tokens, d_model, x, w_g, gate_out, s), s);
}

logo_status logo_branch_transform(int64_t n_tokens, int32_t num_heads, int32_t head_dim,
                                  logo_phi_kind kind, const logo_bf16 *u, const logo_bf16 *A,
                                  const float *s, const float *b, const int32_t *rows,
                                  int64_t n_rows, const int32_t *n_rows_dev, logo_bf16 *u_g,
                                  logo_stream stream) {
    if (n_tokens < 0 || num_heads < 1 || n_rows < 0)
        return LOGO_ERR_SHAPE;
    if (head_dim != 64 && head_dim != 128)
        return LOGO_ERR_UNSUPPORTED;
    if (kind != LOGO_PHI_LP && kind != LOGO_PHI_SO)
        return LOGO_ERR_ARG;
    if (!rows && n_rows != n_tokens)
        return LOGO_ERR_SHAPE;
    if (n_rows == 0 || n_tokens == 0)
        return LOGO_OK;
    if (!u || !u_g || (kind == LOGO_PHI_LP && !A) || (kind == LOGO_PHI_SO && (!s || !b)))
        return LOGO_ERR_NULL;
    if ((uintptr_t)u % 16 != 0 || (uintptr_t)u_g % 16 != 0 || (A && (uintptr_t)A % 16 != 0))
        return LOGO_ERR_ARG;
    if (n_rows * num_heads * head_dim / 8 / 256 >= (1LL << 31) ||
        (n_rows + 255) / 256 >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    hipStream_t st = (hipStream_t)stream;
    return hip_status(launch_branch_transform((int)kind, n_rows, num_heads, head_dim, u, A, s, b,
                                              rows, n_rows_dev, u_g, st),
                      st);
}

logo_status logo_attn_fwd_train(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                                const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                                const logo_bf16 *v_g, const float *gate, logo_sel_mode mode,
                                float threshold, double ratio, const float *gain_local,
                                const float *gain_global, float eps, logo_bf16 *out,
                                int32_t *sel_idx, int32_t sel_capacity, int32_t *cu_sel,
                                int32_t *tok2sel, float *thr_out, float *o_local,
                                float *lse_local, float *o_global, float *lse_global, void *ws,
                                size_t ws_bytes, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if ((!gate && p->total_tokens > 0) || !cu_sel)
        return LOGO_ERR_NULL;
    if (p->total_tokens > 0 &&
        (!q || !k || !v || !out || !tok2sel || !o_local || !lse_local))
        return LOGO_ERR_NULL;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    if (sel_capacity > 0 && (!sel_idx || !o_global || !lse_global))
        return LOGO_ERR_NULL;
    if (!(eps >= 0.f) || std::isinf(eps))
        return LOGO_ERR_ARG;
    const int32_t cap = sel_capacity;
    const FwdWs w = fwd_ws(p, cap);
    st = check_ws(ws, ws_bytes, w.total);
    if (st != LOGO_OK)
        return st;
    char *base = (char *)ws;
    float *thr = thr_out ? thr_out : (float *)(base + w.thr);
    st = check_select_args(p, gate, mode, threshold, ratio, sel_idx, cap, cu_sel, thr_out);
    if (st != LOGO_OK)
        return st;
    hipStream_t s = (hipStream_t)stream;
    // The inference path's launches (selection; local branch whose extra
    // workgroup builds the global branch's tile plan; global branch), with
    // epilogues that also keep the raw branch outputs and their LSEs.
    const FusedEpi fe{tok2sel, gate, nullptr, eps, (float *)(base + w.lc), out,
                      0, nullptr, nullptr, nullptr, nullptr};
    PlanArgs plan;
    int grid_g = 0;
    const bool with_plan = p->total_tokens > 0 && cap > 0;
    if (with_plan &&
        (st = global_plan(p, sel_idx, cu_sel, cap, base + w.glob_ws, plan, grid_g)) != LOGO_OK)
        return st;
    st = run_select(p, gate, mode, threshold, ratio, sel_idx, cap, cu_sel, tok2sel, thr,
                    base + w.sel_ws, s);
    if (st != LOGO_OK)
        return st;
    st = run_local(p, q, k, v, o_local, &fe, gain_local, s, with_plan ? &plan : nullptr,
                   lse_local);
    if (st != LOGO_OK)
        return st;
    return run_global(p, q_g ? q_g : q, k_g ? k_g : k, v_g ? v_g : v, sel_idx, cu_sel, cap,
                      o_global, &fe, gain_global, base + w.glob_ws, s, nullptr, &plan, grid_g,
                      lse_global);
}

logo_status logo_attn_bwd(const logo_problem *p, const logo_bf16 *q, const logo_bf16 *k,
                          const logo_bf16 *v, const logo_bf16 *q_g, const logo_bf16 *k_g,
                          const logo_bf16 *v_g, const float *gate, const float *gain_local,
                          const float *gain_global, float eps, const int32_t *sel_idx,
                          int32_t sel_capacity, const int32_t *cu_sel, const int32_t *tok2sel,
                          const float *o_local, const float *lse_local, const float *o_global,
                          const float *lse_global, const logo_bf16 *dout, float *dq, float *dk,
                          float *dv, float *dq_g, float *dk_g, float *dv_g, float *dgate,
                          float *dgain_local, float *dgain_global, void *ws, size_t ws_bytes,
                          logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (!cu_sel)
        return LOGO_ERR_NULL;
    if ((q_g == nullptr) != (dq_g == nullptr) || (k_g == nullptr) != (dk_g == nullptr) ||
        (v_g == nullptr) != (dv_g == nullptr))
        return LOGO_ERR_ARG;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    const int32_t N = p->total_tokens;
    if (N > 0 && (!q || !k || !v || !gate || !tok2sel || !o_local || !lse_local || !dout ||
                  !dq || !dk || !dv))
        return LOGO_ERR_NULL;
    if (N > 0 && sel_capacity > 0 && (!sel_idx || !o_global || !lse_global))
        return LOGO_ERR_NULL;
    if (!(eps >= 0.f) || std::isinf(eps))
        return LOGO_ERR_ARG;
    if (!fusion_bwd_supported(p->num_q_heads, p->head_dim))
        return LOGO_ERR_UNSUPPORTED;
    const int32_t cap = sel_capacity;
    const BwdWs w = bwd_ws(p, cap);
    st = check_ws(ws, ws_bytes, w.total);
    if (st != LOGO_OK)
        return st;
    if (N == 0)
        return LOGO_OK;
    char *base = (char *)ws;
    hipStream_t s = (hipStream_t)stream;
    const int H = p->num_q_heads, d = p->head_dim;
    const logo_bf16 *qg = q_g ? q_g : q;

    // 1. ContextNorm + fusion backward (and the compact Q^G rows)
    FusionBwdArgs f;
    std::memset(&f, 0, sizeof f);
    f.ol = o_local;
    f.og = o_global;
    f.dout = dout;
    f.q_g = qg;
    f.gate = gate;
    f.tok2sel = tok2sel;
    f.gain_l = gain_local;
    f.gain_g = gain_global;
    f.eps = eps;
    f.n = N;
    f.hq = H;
    f.cap = cap;
    f.tokens_per_block = w.tokens_per_block;
    f.dol = (uint16_t *)(base + w.dol);
    f.dog = (uint16_t *)(base + w.dog);
    f.qc = (uint16_t *)(base + w.qc);
    f.delta_l = (float *)(base + w.delta_l);
    f.delta_g = (float *)(base + w.delta_g);
    f.side = (float *)(base + w.side);
    f.part_l = dgain_local ? (float *)(base + w.part_l) : nullptr;
    f.part_g = dgain_global ? (float *)(base + w.part_g) : nullptr;
    st = hip_status(launch_fusion_bwd(f, w.blocks, d, s), s);
    if (st == LOGO_OK && dgate)
        st = hip_status(launch_gate_grad(N, H, f.side, dgate, s), s);
    float *gtmp = (float *)(base + w.part_tmp);
    if (st == LOGO_OK && dgain_local)
        st = hip_status(launch_gain_grad(w.part_rows, H * d, f.part_l, gtmp, dgain_local, s), s);
    if (st == LOGO_OK && dgain_global)
        st = hip_status(launch_gain_grad(w.part_rows, H * d, f.part_g, gtmp, dgain_global, s), s);
    if (st != LOGO_OK)
        return st;

    // 2. local branch: dQ, dK, dV (overwrite)
    BwdArgs a = make_bwd_args(p);
    a.cap = cap;
    a.q = q;
    a.k = k;
    a.v = v;
    a.dout = f.dol;
    a.lse = lse_local;
    a.delta = f.delta_l;
    a.row_stride = N;
    a.sel_idx = sel_idx;
    a.cu_sel = cu_sel;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    const long long grid_q = (long long)a.n_hg * p->num_seqs * a.ntile_max;
    const int kpb = bwd_keys_per_block();
    const long long grid_kv =
        (long long)((p->max_seqlen + kpb - 1) / kpb) * p->num_seqs * p->num_kv_heads;
    if (grid_q >= (1LL << 31) || grid_kv >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    st = hip_status(launch_bwd_dq(kModeLocal, d, a, (int)grid_q, s), s);
    if (st == LOGO_OK)
        st = hip_status(launch_bwd_dkv(kModeLocal, d, a, (int)grid_kv, s), s);
    if (st != LOGO_OK)
        return st;

    // 3. global branch: selected rows (compact), dense K/V; added into the
    //    local gradients where the branch shares the tensor
    if (dq_g)
        st = hip_status(launch_fill_zero((int64_t)N * H * d, dq_g, s), s);
    if (st != LOGO_OK)
        return st;
    a.q = f.qc;
    a.k = k_g ? k_g : k;
    a.v = v_g ? v_g : v;
    a.dout = f.dog;
    a.lse = lse_global;
    a.delta = f.delta_g;
    a.row_stride = cap;
    a.dq = dq_g ? dq_g : dq;
    a.dk = dk_g ? dk_g : dk;
    a.dv = dv_g ? dv_g : dv;
    a.acc_q = dq_g ? 0 : 1;
    a.acc_k = dk_g ? 0 : 1;
    a.acc_v = dv_g ? 0 : 1;
    if (cap > 0)
        st = hip_status(launch_bwd_dq(kModeGlobal, d, a, (int)grid_q, s), s);
    if (st == LOGO_OK)
        st = hip_status(launch_bwd_dkv(kModeGlobal, d, a, (int)grid_kv, s), s);
    return st;
}

logo_status logo_dense_causal_attn_bwd(const logo_problem *p, const logo_bf16 *q,
                                       const logo_bf16 *k, const logo_bf16 *v,
                                       const logo_bf16 *out, const float *lse,
                                       const logo_bf16 *dout, float *dq, float *dk, float *dv,
                                       void *ws, size_t ws_bytes, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    const int32_t N = p->total_tokens;
    if (N > 0 && (!q || !k || !v || !out || !lse || !dout || !dq || !dk || !dv))
        return LOGO_ERR_NULL;
    st = check_ws(ws, ws_bytes, dense_bwd_ws(p));
    if (st != LOGO_OK)
        return st;
    if (N == 0)
        return LOGO_OK;
    hipStream_t s = (hipStream_t)stream;
    float *delta = (float *)ws;
    st = hip_status(launch_attn_delta(N, p->num_q_heads, p->head_dim, out, dout, delta, s), s);
    if (st != LOGO_OK)
        return st;
    // plain causal attention is the local kernels' row set with a window that
    // covers every sequence
    BwdArgs a = make_bwd_args(p);
    a.window = p->max_seqlen > 0 ? p->max_seqlen : 1;
    a.q = q;
    a.k = k;
    a.v = v;
    a.dout = dout;
    a.lse = lse;
    a.delta = delta;
    a.row_stride = N;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    const long long grid_q = (long long)a.n_hg * p->num_seqs * a.ntile_max;
    const int kpb = bwd_keys_per_block();
    const long long grid_kv =
        (long long)((p->max_seqlen + kpb - 1) / kpb) * p->num_seqs * p->num_kv_heads;
    if (grid_q >= (1LL << 31) || grid_kv >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    st = hip_status(launch_bwd_dq(kModeLocal, p->head_dim, a, (int)grid_q, s), s);
    if (st == LOGO_OK)
        st = hip_status(launch_bwd_dkv(kModeLocal, p->head_dim, a, (int)grid_kv, s), s);
    return st;
}

logo_status logo_global_attn_sparse_q_fwd_train(const logo_problem *p, const logo_bf16 *q,
                                                const logo_bf16 *k, const logo_bf16 *v,
                                                const int32_t *sel_idx, const int32_t *cu_sel,
                                                int32_t sel_capacity, float *o_global,
                                                float *lse_global, void *ws, size_t ws_bytes,
                                                logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    if (!cu_sel)
        return LOGO_ERR_NULL;
    if (sel_capacity > 0 && p->total_tokens > 0 &&
        (!q || !k || !v || !sel_idx || !o_global || !lse_global))
        return LOGO_ERR_NULL;
    if (sel_capacity > 0 && p->total_tokens > 0) {
        st = check_ws(ws, ws_bytes, global_ws(p, sel_capacity).total);
        if (st != LOGO_OK)
            return st;
    }
    return run_global(p, q, k, v, sel_idx, cu_sel, sel_capacity, o_global, nullptr, nullptr,
                      (char *)ws, (hipStream_t)stream, nullptr, nullptr, 0, lse_global);
}

logo_status logo_global_attn_sparse_q_bwd(const logo_problem *p, const logo_bf16 *q,
                                          const logo_bf16 *k, const logo_bf16 *v,
                                          const int32_t *sel_idx, const int32_t *cu_sel,
                                          int32_t sel_capacity, const float *o_global,
                                          const float *lse_global, const logo_bf16 *dout,
                                          float *dq, float *dk, float *dv, void *ws,
                                          size_t ws_bytes, logo_stream stream) {
    logo_status st = check_problem(p);
    if (st != LOGO_OK)
        return st;
    if (sel_capacity < 0)
        return LOGO_ERR_SHAPE;
    const int32_t N = p->total_tokens, cap = sel_capacity;
    if (!cu_sel)
        return LOGO_ERR_NULL;
    if (N > 0 && (!q || !k || !v || !dq || !dk || !dv))
        return LOGO_ERR_NULL;
    if (N > 0 && cap > 0 && (!sel_idx || !o_global || !lse_global || !dout))
        return LOGO_ERR_NULL;
    const GlobalBwdWs w = global_bwd_ws(p, cap);
    st = check_ws(ws, ws_bytes, w.total);
    if (st != LOGO_OK)
        return st;
    if (N == 0)
        return LOGO_OK;
    hipStream_t s = (hipStream_t)stream;
    const int H = p->num_q_heads, d = p->head_dim;
    char *base = (char *)ws;
    uint16_t *qc = (uint16_t *)(base + w.qc);
    float *delta = (float *)(base + w.delta);
    st = hip_status(launch_fill_zero((int64_t)N * H * d, dq, s), s);
    if (st == LOGO_OK && cap > 0)
        st = hip_status(launch_sparse_prep(cap, H, d, cu_sel + p->num_seqs, sel_idx, q, o_global,
                                           dout, qc, delta, s),
                        s);
    if (st != LOGO_OK)
        return st;
    BwdArgs a = make_bwd_args(p);
    a.cap = cap;
    a.q = qc;
    a.k = k;
    a.v = v;
    a.dout = dout;
    a.lse = lse_global;
    a.delta = delta;
    a.row_stride = cap;
    a.sel_idx = sel_idx;
    a.cu_sel = cu_sel;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    const long long grid_q = (long long)a.n_hg * p->num_seqs * a.ntile_max;
    const int kpb = bwd_keys_per_block();
    const long long grid_kv =
        (long long)((p->max_seqlen + kpb - 1) / kpb) * p->num_seqs * p->num_kv_heads;
    if (grid_q >= (1LL << 31) || grid_kv >= (1LL << 31))
        return LOGO_ERR_UNSUPPORTED;
    if (cap > 0)
        st = hip_status(launch_bwd_dq(kModeGlobal, d, a, (int)grid_q, s), s);
    if (st == LOGO_OK)
        st = hip_status(launch_bwd_dkv(kModeGlobal, d, a, (int)grid_kv, s), s);
    return st;
}

}  // extern "C"
