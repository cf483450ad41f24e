/* A plain C99 caller of the library, built by tests/test_abi.py with gcc against
 * include/resispec.h and linked to libresispec.so.  It calls only host-side functions
 * and argument checks that return before any device work, so it runs without a GPU.
 * Prints "ok" and exits 0 when every check holds; otherwise names the first failure. */
#include <stdio.h>
#include <string.h>

#include "resispec.h"

#define CHECK(cond)                                        \
    do {                                                   \
        if (!(cond)) {                                     \
            printf("failed: %s (line %d)\n", #cond, __LINE__); \
            return 1;                                      \
        }                                                  \
    } while (0)

int main(void) {
    CHECK(resispec_abi_version() == RESISPEC_ABI_VERSION);
    CHECK(strcmp(resispec_status_string(RS_OK), resispec_status_string(RS_ERR_INVALID_ARG)) != 0);
    CHECK(resispec_workspace_bytes(0, 5) == 0);
    CHECK(resispec_workspace_bytes(4, 33) >= 3 * 4 * 33 * sizeof(int32_t));
    CHECK(resispec_path_workspace_bytes(8, 1000) > 0);

    /* two trees of five nodes: a valid batch, then a parent that is not earlier */
    int32_t parent[10] = {-1, 0, 0, 1, 1, -1, 0, 1, 2, 3};
    int32_t token[10] = {0, 1, 2, 3, 4, 0, 5, 6, 7, 8};
    int64_t first_bad = 123;
    CHECK(resispec_validate_tree_host(parent, token, 2, 5, 16, &first_bad) == RS_OK);
    CHECK(first_bad == -1);
    parent[8] = 3;
    CHECK(resispec_validate_tree_host(parent, token, 2, 5, 16, &first_bad) == RS_ERR_INVALID_ARG);
    CHECK(first_bad == 8);

    /* device entry points: invalid arguments come back before any launch */
    rs_params prm;
    memset(&prm, 0, sizeof prm);
    prm.mode = RS_MODE_RESISPEC;
    prm.logits_dtype = RS_F32;
    prm.temperature = 1.0f;
    prm.bonus = 1;
    int32_t out_tok[4], out_len[4];
    CHECK(resispec_verify(NULL, NULL, NULL, NULL, NULL, 4, 100, 2, &prm, out_tok, out_len, NULL,
                          NULL) == RS_ERR_INVALID_ARG);
    prm.temperature = 0.0f;
    CHECK(resispec_verify((const void*)16, (const void*)16, (const int32_t*)16, (const float*)16,
                          (const float*)16, 4, 100, 2, &prm, out_tok, out_len, NULL,
                          NULL) == RS_ERR_INVALID_ARG);
    printf("ok\n");
    return 0;
}
