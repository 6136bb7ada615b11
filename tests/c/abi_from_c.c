/* A C99 caller of liblogo: the header compiles as plain C and the library's
 * host-side paths answer from C (version and status strings, workspace
 * sizing, and argument validation before any launch or device query).
 * No call here reaches the GPU.  Prints one line per check; exit status 0
 * when every check holds. */
#include "logo.h"

#include <stdio.h>
#include <string.h>

static int failures = 0;

static void check(int ok, const char *what) {
    printf("%s %s\n", ok ? "ok  " : "FAIL", what);
    if (!ok)
        failures++;
}

int main(void) {
    static const int32_t cu_host[3] = {0, 1000, 1500};
    /* a stand-in device address: validation never dereferences it */
    void *const dev = (void *)(uintptr_t)0x1000;
    logo_problem p;
    memset(&p, 0, sizeof p);
    p.num_seqs = 2;
    p.total_tokens = 1500;
    p.max_seqlen = 1000;
    p.cu_seqlens = (const int32_t *)dev;
    p.cu_seqlens_host = cu_host;
    p.num_q_heads = 8;
    p.num_kv_heads = 2;
    p.head_dim = 128;
    p.window = 64;
    p.softmax_scale = 0.0f;

    const char *ver = logo_version();
    check(ver != NULL && ver[0] != '\0', "logo_version");
    check(strlen(logo_status_str(LOGO_OK)) > 0, "logo_status_str(LOGO_OK)");
    check(strlen(logo_status_str(LOGO_ERR_NULL)) > 0, "logo_status_str(LOGO_ERR_NULL)");

    check(logo_workspace_bytes(&p, LOGO_ENTRY_FWD, 400) > 0, "logo_workspace_bytes(FWD)");
    check(logo_ratio_capacity(&p, 0.25) >= 375, "logo_ratio_capacity >= floor(0.25 T) summed");
    check(logo_attn_fwd_launches(NULL) == -1, "logo_attn_fwd_launches(NULL) -> -1");

    /* invalid arguments come back as their documented statuses */
    check(logo_local_attn(&p, NULL, (const logo_bf16 *)dev, (const logo_bf16 *)dev,
                          (float *)dev, NULL) == LOGO_ERR_NULL,
          "logo_local_attn(q = NULL) -> LOGO_ERR_NULL");
    logo_problem bad = p;
    bad.head_dim = 96;
    check(logo_local_attn(&bad, (const logo_bf16 *)dev, (const logo_bf16 *)dev,
                          (const logo_bf16 *)dev, (float *)dev, NULL) == LOGO_ERR_UNSUPPORTED,
          "logo_local_attn(d = 96) -> LOGO_ERR_UNSUPPORTED");
    bad = p;
    bad.num_kv_heads = 3;
    check(logo_local_attn(&bad, (const logo_bf16 *)dev, (const logo_bf16 *)dev,
                          (const logo_bf16 *)dev, (float *)dev, NULL) == LOGO_ERR_SHAPE,
          "logo_local_attn(Hq % Hkv != 0) -> LOGO_ERR_SHAPE");
    bad = p;
    bad.window = 0;
    check(logo_local_attn(&bad, (const logo_bf16 *)dev, (const logo_bf16 *)dev,
                          (const logo_bf16 *)dev, (float *)dev, NULL) == LOGO_ERR_ARG,
          "logo_local_attn(window = 0) -> LOGO_ERR_ARG");

    printf("%d failure(s)\n", failures);
    return failures == 0 ? 0 : 1;
}
