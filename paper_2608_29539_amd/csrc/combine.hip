// combine.hip -- ContextNorm and output fusion, back in token order
// (Eq. contextnorm: head-wise RMSNorm of each branch; Eq. output-fusion:
// (1-p) Norm^L + p Norm^G for selected tokens, Norm^L otherwise).
//
// HBM-bound streaming kernels.  combine_kernel (logo_combine): one (token,
// head) row of d fp32 values is handled by d/4 lanes with 16-byte loads; the
// row's sum of squares is a butterfly over those lanes, and unselected rows
// never touch o_global.  sel_sum_kernel: the selected rows' output of the
// one-launch layer, from its two weighted branch parts.
#include "logo_internal.h"

#include <algorithm>

namespace logo {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    __bf16 x = (__bf16)a, y = (__bf16)b;   // round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

template <int D>
__global__ __launch_bounds__(256) void combine_kernel(long long n_rows, int hq,
                                                      const float *__restrict__ ol,
                                                      const float *__restrict__ og,
                                                      const float *__restrict__ gate,
                                                      const int32_t *__restrict__ tok2sel,
                                                      const float *__restrict__ gl,
                                                      const float *__restrict__ gg, float eps,
                                                      int apply_norm, uint16_t *__restrict__ out) {
    constexpr int kLanesPerRow = D / 4;
    constexpr int kRowsPerBlock = 256 / kLanesPerRow;
    const int sub = threadIdx.x % kLanesPerRow;
    long long row = (long long)blockIdx.x * kRowsPerBlock + threadIdx.x / kLanesPerRow;
    const bool valid = row < n_rows;
    if (!valid)
        row = n_rows - 1;
    const long long t = row / hq;
    const int h = (int)(row % hq);
    const int c0 = sub * 4;

    const f32x4 xl = *(const f32x4 *)(ol + row * D + c0);
    const int r = tok2sel[t];
    f32x4 xg = {0.f, 0.f, 0.f, 0.f};
    if (r >= 0)
        xg = *(const f32x4 *)(og + ((long long)r * hq + h) * D + c0);

    float sl = xl.x * xl.x + xl.y * xl.y + xl.z * xl.z + xl.w * xl.w;
    float sg = xg.x * xg.x + xg.y * xg.y + xg.z * xg.z + xg.w * xg.w;
#pragma unroll
    for (int d = kLanesPerRow / 2; d > 0; d >>= 1) {
        sl += __shfl_xor(sl, d, kLanesPerRow);
        sg += __shfl_xor(sg, d, kLanesPerRow);
    }
    float il = 1.f, ig = 1.f;
    if (apply_norm) {
        il = 1.f / sqrtf(sl / (float)D + eps);
        ig = 1.f / sqrtf(sg / (float)D + eps);
    }
    f32x4 wl = {1.f, 1.f, 1.f, 1.f}, wg = {1.f, 1.f, 1.f, 1.f};
    if (apply_norm && gl)
        wl = *(const f32x4 *)(gl + h * D + c0);
    if (apply_norm && gg)
        wg = *(const f32x4 *)(gg + h * D + c0);
    f32x4 y = xl * il * wl;
    if (r >= 0) {
        const float p = gate[t];
        y = (1.f - p) * y + p * (xg * ig * wg);
    }
    if (valid) {
        u32x2 o;
        o.x = pack_bf16x2(y.x, y.y);
        o.y = pack_bf16x2(y.z, y.w);
        *(u32x2 *)(out + row * D + c0) = o;
    }
}

// Output rows of the selected tokens from the two branch parts of the
// one-launch layer (Eq. output-fusion): out[sel_idx[r]][h] = bf16(lc[r][h] +
// gc[r][h]), lc = (1-p) Norm^L and gc = p Norm^G already weighted.  Eight
// values per thread (two 16-byte loads of each part, one 16-byte store),
// grid-stride over the selected count read on the device.
template <int D>
__global__ __launch_bounds__(256) void sel_sum_kernel(int32_t cap, int hq,
                                                      const int32_t *__restrict__ cu_sel, int B,
                                                      const int32_t *__restrict__ sel_idx,
                                                      const float *__restrict__ lc,
                                                      const float *__restrict__ gc,
                                                      uint16_t *__restrict__ out) {
    constexpr int kVecPerRow = D / 8;
    const int n = min(cu_sel[B], cap);
    const long long nvec = (long long)n * hq * kVecPerRow;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < nvec;
         i += (long long)gridDim.x * 256) {
        const long long rh = i / kVecPerRow;           // r * hq + h
        const int c = (int)(i % kVecPerRow) * 8;
        const long long r = rh / hq;
        const int h = (int)(rh % hq);
        const float *pl = lc + rh * D + c, *pg = gc + rh * D + c;
        const f32x4 a0 = *(const f32x4 *)pl, a1 = *(const f32x4 *)(pl + 4);
        const f32x4 b0 = *(const f32x4 *)pg, b1 = *(const f32x4 *)(pg + 4);
        const f32x4 y0 = a0 + b0, y1 = a1 + b1;
        typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
        u32x4v o;
        o.x = pack_bf16x2(y0.x, y0.y);
        o.y = pack_bf16x2(y0.z, y0.w);
        o.z = pack_bf16x2(y1.x, y1.y);
        o.w = pack_bf16x2(y1.z, y1.w);
        *(u32x4v *)(out + ((long long)sel_idx[r] * hq + h) * D + c) = o;
    }
}

}  // namespace

hipError_t launch_sel_sum(int32_t cap, int hq, int head_dim, const int32_t *cu_sel, int num_seqs,
                          const int32_t *sel_idx, const float *lc, const float *gc,
                          uint16_t *out, hipStream_t s) {
    const long long vecs = (long long)cap * hq * (head_dim / 8);
    if (vecs == 0)
        return hipSuccess;
    const long long grid = std::min((vecs + 255) / 256, 8192LL);
    if (head_dim == 128)
        hipLaunchKernelGGL(sel_sum_kernel<128>, dim3((unsigned)grid), dim3(256), 0, s, cap, hq,
                           cu_sel, num_seqs, sel_idx, lc, gc, out);
    else
        hipLaunchKernelGGL(sel_sum_kernel<64>, dim3((unsigned)grid), dim3(256), 0, s, cap, hq,
                           cu_sel, num_seqs, sel_idx, lc, gc, out);
    return hipGetLastError();
}

hipError_t launch_combine(int n_tokens, int hq, int head_dim, const float *o_local,
                          const float *o_global, const float *gate, const int32_t *tok2sel,
                          const float *gain_local, const float *gain_global, float eps,
                          int apply_norm, uint16_t *out, hipStream_t s) {
    const long long rows = (long long)n_tokens * hq;
    if (rows == 0)
        return hipSuccess;
    if (head_dim == 128) {
        const long long grid = (rows + 7) / 8;
        hipLaunchKernelGGL(combine_kernel<128>, dim3((unsigned)grid), dim3(256), 0, s, rows, hq,
                           o_local, o_global, gate, tok2sel, gain_local, gain_global, eps,
                           apply_norm, out);
    } else {
        const long long grid = (rows + 15) / 16;
        hipLaunchKernelGGL(combine_kernel<64>, dim3((unsigned)grid), dim3(256), 0, s, rows, hq,
                           o_local, o_global, gate, tok2sel, gain_local, gain_global, eps,
                           apply_norm, out);
    }
    return hipGetLastError();
}

}  // namespace logo
