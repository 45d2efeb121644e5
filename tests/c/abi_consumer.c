/* A plain C99 consumer of include/noble.h, linked against libnoble.so.  It
 * makes only host-side calls, and fwd / bwd calls with a bad descriptor,
 * which the library rejects before any HIP call, so it runs without a GPU.
 * Prints "ok" and returns 0 when every check holds. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "noble.h"

static int failures = 0;

#define CHECK(cond)                                                     \
    do {                                                                \
        if (!(cond)) {                                                  \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__,      \
                    __LINE__, #cond);                                   \
            ++failures;                                                 \
        }                                                               \
    } while (0)

static noble_linear_desc desc(int64_t T, int64_t d_in, int64_t d_out, int64_t r, int32_t dtype) {
    noble_linear_desc d;
    memset(&d, 0, sizeof d);
    d.T = T;
    d.d_in = d_in;
    d.d_out = d_out;
    d.r = r;
    d.dtype = dtype;
    return d;
}

int main(void) {
    size_t reserve = 1, scratch = 1;
    noble_linear_desc d = desc(8192, 2048, 2048, 128, NOBLE_BF16);
    noble_linear_desc bad;
    noble_recipe rc;
    noble_lr_mults lr;
    int code;

    CHECK(noble_abi_version() == NOBLE_ABI_VERSION);
    for (code = NOBLE_OK; code <= NOBLE_ERR_BAD_ACTIVATION; ++code)
        CHECK(noble_status_string(code) != NULL && strlen(noble_status_string(code)) > 0);
    CHECK(noble_status_string(1000) != NULL);

    /* workspace sizes: the reserve holds H, float32 [T, G r] */
    CHECK(noble_linear_workspace_size(&d, &reserve, &scratch) == NOBLE_OK);
    CHECK(reserve == (size_t)4 * 8192 * 128);
    CHECK(scratch > 0);
    CHECK(noble_linear_workspace_size(&d, NULL, NULL) == NOBLE_OK);
    d.groups = 4;
    CHECK(noble_linear_workspace_size(&d, &reserve, NULL) == NOBLE_OK);
    CHECK(reserve == (size_t)4 * 8192 * 4 * 128);
    d = desc(64, 64, 64, 0, NOBLE_F32);
    CHECK(noble_linear_workspace_size(&d, &reserve, &scratch) == NOBLE_OK);
    CHECK(reserve == 0);

    /* every validation error */
    CHECK(noble_linear_workspace_size(NULL, &reserve, &scratch) == NOBLE_ERR_NULL_ARG);
    bad = desc(64, 64, 64, 8, 7);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_DTYPE);
    bad = desc(64, 60, 64, 8, NOBLE_BF16);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(-1, 64, 64, 8, NOBLE_BF16);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(64, 64, 64, 264, NOBLE_BF16);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(64, 64, 64, 8, NOBLE_BF16);
    bad.reserved = 1;
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(64, 64, 72, 8, NOBLE_BF16);
    bad.groups = 2;   /* 72 / 2 = 36 is not a multiple of 8 */
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(64, 64, 64, 8, NOBLE_BF16);
    bad.activation = NOBLE_ACT_COSNET3 + 1;
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_ACTIVATION);
    /* a forward product past one dispatch: 8388592 token tiles x 2 column tiles */
    bad = desc(2147483648LL - 4096, 8, 264, 8, NOBLE_BF16);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_ERR_BAD_SHAPE);
    bad = desc(2147483648LL - 4096, 8, 256, 8, NOBLE_BF16);
    CHECK(noble_linear_workspace_size(&bad, &reserve, &scratch) == NOBLE_OK);

    /* the compute calls reject a bad descriptor before any HIP call */
    bad = desc(64, 60, 64, 8, NOBLE_BF16);
    CHECK(noble_linear_fwd(NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0,
                           NULL) == NOBLE_ERR_NULL_ARG);
    CHECK(noble_linear_fwd(&bad, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0,
                           NULL) == NOBLE_ERR_BAD_SHAPE);
    CHECK(noble_linear_bwd(&bad, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                           NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) == NOBLE_ERR_BAD_SHAPE);

    /* training recipe: defaults of Sec. 3.3 / App. A and the Eq. 3-4 rates */
    noble_recipe_defaults(&rc);
    noble_recipe_defaults(NULL);
    CHECK(rc.alpha == 0.01 && rc.w_scale == 0.5 && rc.omega_min == 0.8 && rc.omega_max == 1.2);
    CHECK(rc.phi_std == 0.1 && rc.gamma == 0.3 && rc.gamma_M == 0.45 && rc.omega_lr == 3.0 && rc.phi_lr == 5.0);
    d = desc(8192, 2048, 2048, 128, NOBLE_BF16);
    CHECK(noble_lr_multipliers(&d, &rc, &lr) == NOBLE_OK);
    CHECK(lr.W == 1.0 && lr.b == 1.0 && lr.W_down == 1.0 && lr.omega == 3.0 && lr.phi == 5.0);
    CHECK(fabs(lr.W_up - pow(16.0, 0.6)) < 1e-12 && fabs(lr.M - pow(16.0, 0.45)) < 1e-12);
    d.groups = 2;   /* widths of one group: min(2048, 1024) / 128 = 8 */
    CHECK(noble_lr_multipliers(&d, &rc, &lr) == NOBLE_OK);
    CHECK(fabs(lr.W_up - pow(8.0, 0.6)) < 1e-12);
    CHECK(noble_lr_multipliers(&d, NULL, &lr) == NOBLE_ERR_NULL_ARG);
    CHECK(noble_lr_multipliers(&bad, &rc, &lr) == NOBLE_ERR_BAD_SHAPE);
    CHECK(noble_init_params(&bad, &rc, 1, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL) ==
          NOBLE_ERR_BAD_SHAPE);

    if (failures == 0) printf("ok\n");
    return failures == 0 ? 0 : 1;
}
