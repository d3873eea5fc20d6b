/* Plain C11 caller of the library's C ABI: the header must compile as C and
 * the entry points must be callable without any C++ or Python in between.
 * Only host-side behaviour is exercised (argument checking, error codes,
 * the thread-local message, model parsing), so no GPU is needed.
 * Exit status 0 = every check passed; otherwise the number of failures. */
#include <stdio.h>
#include <string.h>

#include "gnnspmm.h"

static int failures = 0;

static void expect(int cond, const char *what)
{
    if (!cond) {
        fprintf(stderr, "FAIL: %s (last error: %s)\n", what, gs_last_error());
        failures++;
    }
}

int main(int argc, char **argv)
{
    expect(gs_abi_version() == GS_ABI_VERSION, "ABI version matches the header");
    expect(GS_NUM_FORMATS == 6 && GS_CSC == 5, "format enumeration");

    gs_matrix m = (gs_matrix)&failures; /* must be reset to NULL on error */
    expect(gs_build_format(NULL, GS_CSR, NULL, NULL, &m, NULL) == GS_ERR_INVALID_ARG, "null COO rejected");
    expect(m == NULL, "output handle cleared on error");
    expect(strlen(gs_last_error()) > 0, "error message set");

    gs_coo bad = {4, 4, 1, NULL, NULL, NULL};
    expect(gs_build_format(&bad, GS_CSR, NULL, NULL, &m, NULL) == GS_ERR_INVALID_ARG, "nnz > 0 with null arrays");
    gs_coo empty = {4, 4, 0, NULL, NULL, NULL};
    expect(gs_build_format(&empty, 42, NULL, NULL, &m, NULL) == GS_ERR_INVALID_ARG, "unknown format");
    gs_build_opts opts = {65, 0, 0};
    expect(gs_build_format(&empty, GS_BSR, &opts, NULL, &m, NULL) == GS_ERR_INVALID_ARG, "BSR block 65");

    expect(gs_spmm(NULL, NULL, 1, NULL, 1, 1, NULL) == GS_ERR_INVALID_ARG, "spmm on a null handle");
    expect(gs_spmm_noalloc(NULL, NULL, 1, NULL, 1, 1, NULL) == GS_ERR_INVALID_ARG,
           "allocation-free spmm on a null handle");
    expect(GS_NOALLOC_SCRATCH_BYTES >= (1u << 20), "scratch size is declared");
    gs_matrix_info info;
    expect(gs_get_info(NULL, &info) == GS_ERR_INVALID_ARG, "info on a null handle");

    gs_selector_opts so = {GS_SEL_MODEL, GS_CSR, NULL, 0, 16, 3, 1u << 9, 0.0};
    gs_ctx ctx = NULL;
    expect(gs_ctx_create(&so, &ctx) == GS_ERR_INVALID_ARG && ctx == NULL, "candidate mask with an unknown format");
    so.formats = 0;
    so.mode = 7;
    expect(gs_ctx_create(&so, &ctx) == GS_ERR_INVALID_ARG, "unknown selector mode");
    so.mode = GS_SEL_PROFILE;
    so.mem_weight = 1.5;
    expect(gs_ctx_create(&so, &ctx) == GS_ERR_INVALID_ARG, "memory weight above 1");
    so.mem_weight = 0.25;
    expect(gs_ctx_create(&so, &ctx) == GS_OK && ctx != NULL, "profiling context");
    gs_select_stats st;
    expect(gs_ctx_stats(ctx, &st) == GS_OK, "stats of a fresh context");
    gs_ctx_destroy(ctx);
    if (argc > 1) { /* a model file to parse */
        so.mode = GS_SEL_MODEL;
        so.model_path = argv[1];
        ctx = NULL;
        expect(gs_ctx_create(&so, &ctx) == GS_ERR_MODEL && ctx == NULL, "model trained for another w");
        so.mem_weight = 0.0;
        expect(gs_ctx_create(&so, &ctx) == GS_OK && ctx != NULL, "shipped model parses");
        gs_ctx_destroy(ctx);
    }
    if (failures == 0) printf("abi_check: all checks passed\n");
    return failures;
}
