/*
 * A plain C11 caller of the library: the header must compile as C and every
 * function it declares must resolve at link time.  The calls made here all
 * fail host-side validation, so the program needs no GPU.
 */
#include <stdio.h>
#include <string.h>

#include "gt_attn.h"

typedef void (*any_fn)(void);

static int check(int ok, const char* what) {
    if (!ok) fprintf(stderr, "c_caller: %s\n", what);
    return ok ? 0 : 1;
}

int main(void) {
    /* every declared entry point, resolved by the linker */
    const any_fn fns[] = {
        (any_fn)gt_attn_fwd,          (any_fn)gt_attn_fwd_bf16,  (any_fn)gt_attn_fwd_ex,
        (any_fn)gt_attn_fwd_noalloc,  (any_fn)gt_gatv2_fwd,      (any_fn)gt_attn_bwd,
        (any_fn)gt_segment_reduce,    (any_fn)gt_dot_aggr,       (any_fn)gt_csr_validate,
        (any_fn)gt_status_string,     (any_fn)gt_last_error_message, (any_fn)gt_profile_enable,
        (any_fn)gt_profile_collect,   (any_fn)gt_workspace_pool_stats, (any_fn)gt_workspace_release,
    };
    int bad = 0;
    for (size_t i = 0; i < sizeof fns / sizeof fns[0]; ++i) bad |= check(fns[i] != NULL, "null entry point");

    /* the tuning struct is six 32-bit fields, as the binding lays it out */
    bad |= check(sizeof(gt_tuning) == 6 * sizeof(int32_t), "gt_tuning size");
    gt_tuning tu;
    memset(&tu, 0, sizeof tu);
    tu.chunk_edges = 2147483647;

    /* host validation: negative N, and an oversized tuning field */
    gt_status s = gt_attn_fwd(NULL, NULL, NULL, NULL, NULL, NULL, -1, 0, 1, 32, 1.0f, NULL);
    bad |= check(s == GT_ERROR_INVALID_VALUE, "gt_attn_fwd(N = -1) must be GT_ERROR_INVALID_VALUE");
    const char* msg = gt_last_error_message();
    bad |= check(msg != NULL && msg[0] != '\0', "no error message");
    s = gt_attn_fwd_ex(GT_DTYPE_F32, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 10, 10, 1, 32, 1.0f, &tu, NULL);
    bad |= check(s == GT_ERROR_INVALID_VALUE, "an oversized chunk_edges must be GT_ERROR_INVALID_VALUE");
    bad |= check(strlen(gt_status_string(GT_ERROR_NOT_SUPPORTED)) > 0, "gt_status_string");
    if (!bad) printf("c_caller ok: %zu entry points, %s\n", sizeof fns / sizeof fns[0], gt_status_string(s));
    return bad;
}
