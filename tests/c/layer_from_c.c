/* A C99 host program that runs one LoGo layer forward through liblogo on the
 * GPU with no Python in the process: it reads a problem and its inputs from
 * a file, allocates device memory with the HIP runtime, calls
 * logo_attn_fwd in ratio mode, and writes the selection and the bf16 output
 * to a file for the test to compare against the oracle.
 *
 * Input file (little-endian): int32 B, N, Hq, Hkv, d, window, max_seqlen,
 * pad; float64 ratio; int32 cu_seqlens[B+1]; uint16 q[N][Hq][d],
 * k[N][Hkv][d], v[N][Hkv][d] (bf16 bits); float32 gate[N].
 * Output file: int32 cu_sel[B+1]; int32 capacity; int32 sel_idx[capacity];
 * uint16 out[N][Hq][d].
 * Exit status: 0 on success, 2 on a file error, 3 on a HIP error, 4 on a
 * library status other than LOGO_OK. */
#include "logo.h"

#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#define HIP_OK(call)                                                              \
    do {                                                                          \
        hipError_t e_ = (call);                                                   \
        if (e_ != hipSuccess) {                                                   \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));            \
            return 3;                                                             \
        }                                                                         \
    } while (0)

static int read_all(FILE *f, void *dst, size_t bytes) {
    return bytes == 0 || fread(dst, 1, bytes, f) == bytes;
}

static int write_all(FILE *f, const void *src, size_t bytes) {
    return bytes == 0 || fwrite(src, 1, bytes, f) == bytes;
}

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s <input> <output>\n", argv[0]);
        return 2;
    }
    FILE *fin = fopen(argv[1], "rb");
    if (!fin) {
        perror(argv[1]);
        return 2;
    }
    int32_t hdr[8];
    double ratio;
    if (!read_all(fin, hdr, sizeof hdr) || !read_all(fin, &ratio, sizeof ratio)) {
        fprintf(stderr, "short header\n");
        return 2;
    }
    const int32_t B = hdr[0], N = hdr[1], Hq = hdr[2], Hkv = hdr[3], d = hdr[4];
    const size_t nq = (size_t)N * Hq * d, nkv = (size_t)N * Hkv * d;
    int32_t *cu = malloc(sizeof(int32_t) * (size_t)(B + 1));
    uint16_t *q = malloc(2 * nq), *k = malloc(2 * nkv), *v = malloc(2 * nkv);
    float *gate = malloc(sizeof(float) * (size_t)(N > 0 ? N : 1));
    uint16_t *out = malloc(2 * (nq > 0 ? nq : 1));
    if (!cu || !q || !k || !v || !gate || !out) {
        fprintf(stderr, "host allocation failed\n");
        return 2;
    }
    if (!read_all(fin, cu, sizeof(int32_t) * (size_t)(B + 1)) || !read_all(fin, q, 2 * nq) ||
        !read_all(fin, k, 2 * nkv) || !read_all(fin, v, 2 * nkv) ||
        !read_all(fin, gate, sizeof(float) * (size_t)N)) {
        fprintf(stderr, "short input\n");
        return 2;
    }
    fclose(fin);

    int32_t *d_cu, *d_sel, *d_cu_sel, *d_tok2sel;
    uint16_t *d_q, *d_k, *d_v, *d_out;
    float *d_gate, *d_thr;
    void *d_ws = NULL;
    HIP_OK(hipMalloc((void **)&d_cu, sizeof(int32_t) * (size_t)(B + 1)));
    HIP_OK(hipMemcpy(d_cu, cu, sizeof(int32_t) * (size_t)(B + 1), hipMemcpyHostToDevice));

    logo_problem p;
    memset(&p, 0, sizeof p);
    p.num_seqs = B;
    p.total_tokens = N;
    p.max_seqlen = hdr[6];
    p.cu_seqlens = d_cu;
    p.cu_seqlens_host = cu;
    p.num_q_heads = Hq;
    p.num_kv_heads = Hkv;
    p.head_dim = d;
    p.window = hdr[5];
    p.softmax_scale = 0.0f;

    int64_t cap64 = logo_ratio_capacity(&p, ratio);
    if (cap64 < 0) {
        fprintf(stderr, "logo_ratio_capacity: %lld\n", (long long)cap64);
        return 4;
    }
    const int32_t cap = cap64 > 0 ? (int32_t)cap64 : 1;
    const size_t ws_bytes = logo_workspace_bytes(&p, LOGO_ENTRY_FWD, cap);

    HIP_OK(hipMalloc((void **)&d_q, 2 * nq));
    HIP_OK(hipMalloc((void **)&d_k, 2 * nkv));
    HIP_OK(hipMalloc((void **)&d_v, 2 * nkv));
    HIP_OK(hipMalloc((void **)&d_out, 2 * nq));
    HIP_OK(hipMalloc((void **)&d_gate, sizeof(float) * (size_t)N));
    HIP_OK(hipMalloc((void **)&d_thr, sizeof(float) * (size_t)B));
    HIP_OK(hipMalloc((void **)&d_sel, sizeof(int32_t) * (size_t)cap));
    HIP_OK(hipMalloc((void **)&d_cu_sel, sizeof(int32_t) * (size_t)(B + 1)));
    HIP_OK(hipMalloc((void **)&d_tok2sel, sizeof(int32_t) * (size_t)N));
    if (ws_bytes)
        HIP_OK(hipMalloc(&d_ws, ws_bytes));      /* 256-byte aligned, as required */
    HIP_OK(hipMemcpy(d_q, q, 2 * nq, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_k, k, 2 * nkv, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_v, v, 2 * nkv, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(d_gate, gate, sizeof(float) * (size_t)N, hipMemcpyHostToDevice));

    const logo_status st = logo_attn_fwd(&p, d_q, d_k, d_v, NULL, NULL, NULL, d_gate,
                                         LOGO_SEL_RATIO, 0.0f, ratio, NULL, NULL, 1e-6f, d_out,
                                         d_sel, cap, d_cu_sel, d_tok2sel, d_thr, d_ws, ws_bytes,
                                         NULL);
    if (st != LOGO_OK) {
        fprintf(stderr, "logo_attn_fwd: %s\n", logo_status_str(st));
        return 4;
    }
    HIP_OK(hipDeviceSynchronize());

    int32_t *cu_sel = malloc(sizeof(int32_t) * (size_t)(B + 1));
    int32_t *sel = malloc(sizeof(int32_t) * (size_t)cap);
    if (!cu_sel || !sel) {
        fprintf(stderr, "host allocation failed\n");
        return 2;
    }
    HIP_OK(hipMemcpy(cu_sel, d_cu_sel, sizeof(int32_t) * (size_t)(B + 1), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(sel, d_sel, sizeof(int32_t) * (size_t)cap, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(out, d_out, 2 * nq, hipMemcpyDeviceToHost));

    FILE *fout = fopen(argv[2], "wb");
    if (!fout) {
        perror(argv[2]);
        return 2;
    }
    if (!write_all(fout, cu_sel, sizeof(int32_t) * (size_t)(B + 1)) ||
        !write_all(fout, &cap, sizeof cap) ||
        !write_all(fout, sel, sizeof(int32_t) * (size_t)cap) || !write_all(fout, out, 2 * nq)) {
        fprintf(stderr, "short write\n");
        return 2;
    }
    fclose(fout);
    printf("layer_from_c: N=%d n_sel=%d capacity=%d workspace=%zu bytes\n", N, cu_sel[B], cap,
           ws_bytes);

    hipFree(d_cu);
    hipFree(d_q);
    hipFree(d_k);
    hipFree(d_v);
    hipFree(d_out);
    hipFree(d_gate);
    hipFree(d_thr);
    hipFree(d_sel);
    hipFree(d_cu_sel);
    hipFree(d_tok2sel);
    hipFree(d_ws);
    free(cu);
    free(q);
    free(k);
    free(v);
    free(gate);
    free(out);
    free(cu_sel);
    free(sel);
    return 0;
}
