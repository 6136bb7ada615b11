// transform.hip -- the steps on either side of the attention: the gate
// projection p = sigmoid(x . w_g) (Sec. 3.2, Eq. gate-routing) and the
// lightweight branch transforms that produce the global-branch Q/K/V from the
// local ones (Sec. 3.2, Eq. branch-transform):
//   LP: U^G_h = U^L_h A_h  (A_h a d x d matrix per head)
//   SO: U^G_h = U^L_h * s_h + b_h
//
//   gate_proj_kernel      one wave per token: 16-byte loads of x and w_g,
//                         v_dot2 products accumulated in fp32, a wave sum,
//                         the sigmoid in fp32.  HBM-bound (2 dm bytes/token).
//   so_transform_kernel   elementwise fp32 fma, one bf16 rounding.
//   lp_transform_kernel   per head a GEMM [rows x d] x [d x d] on bf16 MFMA
//                         (v_mfma_f32_32x32x16_bf16), computed transposed:
//                         (U A_h)^T = A_h^T U^T, so the U operand is read
//                         straight from row-major memory (16 bytes per lane,
//                         like the attention kernels' Q) and each lane's
//                         output column is one token row (stores of 4 bf16).
//                         A_h is staged once per workgroup in LDS, transposed,
//                         so its fragments are 16-byte LDS reads.
// Rows may be a list of token indices (the selected queries of the global
// branch); outputs go to the token's own row of a [N][H][d] tensor.
#include "logo_internal.h"

namespace logo {
namespace {

typedef __bf16 bf16x8t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2t __attribute__((ext_vector_type(2)));
typedef float f32x16t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    typedef float f2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, bf16x2t));
}

// p[t] = sigmoid(x[t] . w_g); 4 tokens per 256-thread workgroup, d_model a
// multiple of 8.
__global__ __launch_bounds__(256) void gate_proj_kernel(int64_t n, int dm, const uint16_t *x,
                                                        const uint16_t *w, float *p) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= n)
        return;
    const uint16_t *xr = x + t * dm;
    float acc = 0.f;
    for (int c = lane * 8; c < dm; c += 64 * 8) {
        const u32x4t xv = *(const u32x4t *)(xr + c);
        const u32x4t wv = *(const u32x4t *)(w + c);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            // through named words: a bit_cast applied to a vector element
            // expression reads element 0 with this compiler
            const uint32_t xw = xv[i], ww = wv[i];
            acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2t, xw),
                                                  __builtin_bit_cast(bf16x2t, ww), acc, false);
        }
    }
#pragma unroll
    for (int sh = 1; sh < 64; sh <<= 1)
        acc += __shfl_xor(acc, sh, 64);
    if (lane == 0)
        p[t] = 1.f / (1.f + expf(-acc));
}

// SO: one thread per 8 elements of a (row, head) slice.
__global__ __launch_bounds__(256) void so_transform_kernel(int64_t n_rows, int H, int d,
                                                           const uint16_t *u, const float *s,
                                                           const float *b, const int32_t *rows,
                                                           const int32_t *n_rows_dev,
                                                           uint16_t *out) {
    const int per_row = H * d / 8;
    const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t r = g / per_row;
    const int64_t nr = n_rows_dev ? min((int64_t)n_rows_dev[0], n_rows) : n_rows;
    if (r >= nr)
        return;
    const int e0 = (int)(g % per_row) * 8;          // element in [H * d)
    const int64_t t = rows ? rows[r] : r;
    const u32x4t v = *(const u32x4t *)(u + t * H * d + e0);
    u32x4t o;
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const float lo = __uint_as_float(v[i] << 16), hi = __uint_as_float(v[i] & 0xFFFF0000u);
        const int e = e0 + 2 * i;
        o[i] = pack2(fmaf(lo, s[e], b[e]), fmaf(hi, s[e + 1], b[e + 1]));
    }
    *(u32x4t *)(out + t * H * d + e0) = o;
}

// LP: workgroup = (head h, block of kLpRows rows); 4 waves, each 32 rows at
// a time with the next 32 rows' operands prefetched.  LDS holds A_h^T
// [d][d + 8] (bf16, rows padded by 16 bytes), filled by 8 x 8 blocks: eight
// coalesced 16-byte row reads per thread, a transpose in registers, eight
// 16-byte writes.
constexpr int kLpRows = 512;

template <int D>
__global__ __launch_bounds__(256) void lp_transform_kernel(int64_t n_rows, int H, const uint16_t *u,
                                                           const uint16_t *A, const int32_t *rows,
                                                           const int32_t *n_rows_dev,
                                                           uint16_t *out) {
    constexpr int KP = D + 8;
    __shared__ __attribute__((aligned(16))) uint16_t at[D][KP];   // at[j][c] = A_h[c][j]
    const int h = blockIdx.y;
    const int64_t r0 = (int64_t)blockIdx.x * kLpRows;
    const int64_t nr = n_rows_dev ? min((int64_t)n_rows_dev[0], n_rows) : n_rows;
    if (r0 >= nr)
        return;                                     // whole workgroup
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m = lane & 31, g = lane >> 5;
    // stage A_h transposed: a thread takes one 8 x 8 block (rows c0..c0+7,
    // columns j0..j0+7) of A_h with eight 16-byte row reads (lanes take
    // consecutive column blocks: coalesced), transposes it in registers and
    // writes at[j0 + e][c0..c0+7] with one 16-byte store per column e
    const uint16_t *Ah = A + (int64_t)h * D * D;
    constexpr int NB = D / 8;                       // 8 x 8 blocks per row
    for (int idx = tid; idx < NB * NB; idx += 256) {
        const int j0 = (idx % NB) * 8, c0 = (idx / NB) * 8;
        u32x4t r[8];
#pragma unroll
        for (int i = 0; i < 8; i++)
            r[i] = *(const u32x4t *)(Ah + (int64_t)(c0 + i) * D + j0);
#pragma unroll
        for (int e = 0; e < 8; e++) {
            // element e of rows 2 i2 and 2 i2 + 1 -> the low / high half of word i2
            uint32_t w[4];
#pragma unroll
            for (int i2 = 0; i2 < 4; i2++) {
                const uint32_t a0 = r[2 * i2][e >> 1], a1 = r[2 * i2 + 1][e >> 1];
                w[i2] = (e & 1) ? ((a0 >> 16) | (a1 & 0xFFFF0000u))
                                : ((a0 & 0xFFFFu) | (a1 << 16));
            }
            *(u32x4t *)&at[j0 + e][c0] = u32x4t{w[0], w[1], w[2], w[3]};
        }
    }
    __syncthreads();
    const int64_t r_end = min(r0 + kLpRows, nr);
    // this lane's operand row of the block starting at rb (rows past the end
    // repeat the last one and are not stored)
    auto load_block = [&](int64_t rb, bf16x8t (&uf)[D / 16], int64_t &t) {
        const int64_t r = min(rb + m, nr - 1);
        t = rows ? rows[r] : r;
        const uint16_t *ur = u + (t * H + h) * (int64_t)D + g * 8;
#pragma unroll
        for (int cb = 0; cb < D / 16; cb++)
            uf[cb] = *(const bf16x8t *)(ur + cb * 16);
    };
    int64_t rb = r0 + wave * 32;
    if (rb >= r_end)
        return;
    bf16x8t uf[D / 16];
    int64_t t;
    load_block(rb, uf, t);
    for (; rb < r_end; rb += 4 * 32) {
        bf16x8t un[D / 16];
        int64_t tn = t;
        const bool more = rb + 4 * 32 < r_end;
        if (more)
            load_block(rb + 4 * 32, un, tn);
        uint16_t *op = out + (t * H + h) * (int64_t)D + g * 4;
        const bool store = rb + m < r_end;
#pragma unroll
        for (int jb = 0; jb < D / 32; jb++) {
            f32x16t acc = f32x16t{};
#pragma unroll
            for (int cb = 0; cb < D / 16; cb++) {
                const bf16x8t af = *(const bf16x8t *)&at[jb * 32 + m][cb * 16 + g * 8];
                acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, uf[cb], acc, 0, 0, 0);
            }
            // lane holds out[t][h][j] for j = 32 jb + 8 q + 4 g + (0..3)
            if (store) {
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    u32x2t o;
                    o.x = pack2(acc[q * 4 + 0], acc[q * 4 + 1]);
                    o.y = pack2(acc[q * 4 + 2], acc[q * 4 + 3]);
                    *(u32x2t *)(op + jb * 32 + q * 8) = o;
                }
            }
        }
        if (more) {
#pragma unroll
            for (int cb = 0; cb < D / 16; cb++)
                uf[cb] = un[cb];
            t = tn;
        }
    }
}

}  // namespace

hipError_t launch_gate_proj(int64_t n, int dm, const uint16_t *x, const uint16_t *w, float *p,
                            hipStream_t s) {
    if (n <= 0)
        return hipSuccess;
    hipLaunchKernelGGL(gate_proj_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s, n, dm, x,
                       w, p);
    return hipGetLastError();
}

hipError_t launch_branch_transform(int kind, int64_t n_rows, int H, int d, const uint16_t *u,
                                   const uint16_t *A, const float *sc, const float *bi,
                                   const int32_t *rows, const int32_t *n_rows_dev, uint16_t *out,
                                   hipStream_t s) {
    if (n_rows <= 0)
        return hipSuccess;
    if (kind == 1) {
        const int64_t threads = n_rows * H * d / 8;
        hipLaunchKernelGGL(so_transform_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256),
                           0, s, n_rows, H, d, u, sc, bi, rows, n_rows_dev, out);
        return hipGetLastError();
    }
    const dim3 grid((unsigned)((n_rows + kLpRows - 1) / kLpRows), (unsigned)H);
    if (d == 128)
        hipLaunchKernelGGL((lp_transform_kernel<128>), grid, dim3(256), 0, s, n_rows, H, u, A,
                           rows, n_rows_dev, out);
    else
        hipLaunchKernelGGL((lp_transform_kernel<64>), grid, dim3(256), 0, s, n_rows, H, u, A,
                           rows, n_rows_dev, out);
    return hipGetLastError();
}

}  // namespace logo
