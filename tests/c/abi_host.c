/* Host-only use of the C ABI from C (no GPU): plan a small block-CSR weight
 * with host_only = 1, read it back, convert a dense weight, and check the
 * error reporting.  Prints "ok" and returns 0 on success. */
#include <stdio.h>
#include <string.h>

#include "spconv.h"

#define CHECK(cond)                                                                  \
    do {                                                                             \
        if (!(cond)) {                                                               \
            printf("failed: %s (line %d): %s\n", #cond, __LINE__, spconv_last_error()); \
            return 1;                                                                \
        }                                                                            \
    } while (0)

int main(void) {
    /* W (4 x 6), 1x2 blocks: rows {0,1} at channels 1 and 4, rows {2,3} at channel 5 */
    const int32_t row_ptr[3] = {0, 2, 3};
    const int32_t col_idx[3] = {1, 4, 5};
    const float values[6] = {1.0f, 2.0f, 3.0f, 4.0f, 5.0f, 6.0f};
    const float bias[4] = {0.5f, -0.5f, 0.25f, 0.0f};
    spconv_options o;
    spconv_options_init(&o);
    CHECK(o.struct_size == (int32_t)sizeof(spconv_options) && o.reorder == 1);
    o.host_only = 1;
    spconv_plan plan = NULL;
    CHECK(spconv_plan_create_ex(&plan, 4, 6, 2, row_ptr, col_idx, values, bias, SPCONV_ACT_RELU, SPCONV_F32, &o) ==
          SPCONV_OK);
    spconv_plan_info info;
    CHECK(spconv_plan_get_info(plan, &info) == SPCONV_OK);
    CHECK(info.cout == 4 && info.cin == 6 && info.block_rows == 2 && info.nnzb == 3 && info.block_cols == 1);
    int32_t rp[3], ci[3], perm[2];
    float va[6];
    CHECK(spconv_plan_unpack(plan, rp, ci, va, perm) == SPCONV_OK);
    CHECK(memcmp(rp, row_ptr, sizeof rp) == 0 && memcmp(ci, col_idx, sizeof ci) == 0);
    CHECK(memcmp(va, values, sizeof va) == 0);
    /* a host-only plan cannot run */
    CHECK(spconv_run(plan, (void *)16, (void *)4096, 1, 1, 1, NULL) == SPCONV_E_ARG);
    CHECK(strstr(spconv_last_error(), "host_only") != NULL);
    CHECK(spconv_destroy(plan) == SPCONV_OK);
    CHECK(spconv_destroy(NULL) == SPCONV_OK);

    /* malformed input: a column out of range names the entry */
    const int32_t bad_col[3] = {1, 6, 5};
    CHECK(spconv_plan_create_ex(&plan, 4, 6, 2, row_ptr, bad_col, values, bias, SPCONV_ACT_NONE, SPCONV_F32, &o) ==
          SPCONV_E_FORMAT);
    CHECK(plan == NULL && strstr(spconv_last_error(), "col_idx[1]") != NULL);

    /* dense weight with 2 x 2 blocks: detection and conversion */
    float dense[4 * 4] = {0};
    dense[0 * 4 + 2] = 1.0f; dense[0 * 4 + 3] = 2.0f;
    dense[1 * 4 + 2] = 3.0f; dense[1 * 4 + 3] = 4.0f;
    int32_t kr = 0, kc = 0;
    CHECK(spconv_detect_blocks(4, 4, dense, &kr, &kc) == SPCONV_OK && kr == 2 && kc == 2);
    int32_t brp[3], bci[1];
    float bva[4];
    int64_t nnzb = -1;
    CHECK(spconv_dense_to_bcsr_blocked(4, 4, dense, 2, 2, brp, bci, bva, 1, &nnzb) == SPCONV_OK && nnzb == 1);
    CHECK(brp[0] == 0 && brp[1] == 1 && brp[2] == 1 && bci[0] == 2);
    CHECK(bva[0] == 1.0f && bva[1] == 2.0f && bva[2] == 3.0f && bva[3] == 4.0f);
    CHECK(spconv_dense_to_bcsr_blocked(4, 4, dense, 2, 2, brp, bci, bva, 0, &nnzb) == SPCONV_E_ARG && nnzb == 1);

    puts("ok");
    return 0;
}
