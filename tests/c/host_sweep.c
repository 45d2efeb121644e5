/* Host-side sweep of libnoble for the sanitizer build (tests/
 * test_host_sanitizers.py): workspace sizing and weight-gradient planning
 * over a grid of shapes up to the ABI's limits, the learning-rate
 * multipliers, and every fwd / bwd / static-forward call with one required
 * pointer missing, which validation rejects before any HIP call.  Under
 * AddressSanitizer and UndefinedBehaviorSanitizer any out-of-bounds access,
 * signed overflow or other undefined behaviour in that host code aborts the
 * run.  Prints "ok <calls>" when every call returned a valid status. */
#include <stdio.h>
#include <string.h>

#include "noble.h"

static int bad = 0;
static long calls = 0;

static void check_status(int code) {
    ++calls;
    if (code < NOBLE_OK || code > NOBLE_ERR_BAD_ACTIVATION) {
        fprintf(stderr, "unexpected status %d\n", code);
        ++bad;
    }
}

int main(void) {
    static const int64_t Ts[] = {0, 1, 3, 255, 8192, 32768, (int64_t)1 << 20, ((int64_t)1 << 31) - 4096,
                                 (int64_t)1 << 31};
    static const int64_t ds[] = {8, 64, 264, 2048, 8192, (int64_t)1 << 20, ((int64_t)1 << 20) + 8};
    static const int64_t rs[] = {0, 8, 40, 128, 136, 256, 264};
    static const int32_t gs[] = {0, 1, 3, 4, 5};
    void* p[24];
    noble_recipe rc;
    noble_lr_mults lr;
    size_t i, a, b, c, e, f, g;
    for (i = 0; i < 24; ++i) p[i] = (void*)(uintptr_t)(0x100000u + 0x1000u * (unsigned)i);
    noble_recipe_defaults(&rc);
    for (a = 0; a < sizeof Ts / sizeof Ts[0]; ++a)
        for (b = 0; b < sizeof ds / sizeof ds[0]; ++b)
            for (c = 0; c < sizeof ds / sizeof ds[0]; ++c)
                for (e = 0; e < sizeof rs / sizeof rs[0]; ++e)
                    for (f = 0; f < sizeof gs / sizeof gs[0]; ++f)
                        for (g = 0; g < 2; ++g) {
                            noble_linear_desc d;
                            size_t res = 0, scr = 0, fs = 0;
                            memset(&d, 0, sizeof d);
                            d.T = Ts[a];
                            d.d_in = ds[b];
                            d.d_out = ds[c] * (gs[f] > 1 ? gs[f] : 1);
                            d.r = rs[e];
                            d.dtype = (int32_t)g;
                            d.groups = gs[f];
                            d.activation = (int32_t)((a + b + c + e) % (NOBLE_ACT_COSNET3 + 2));   /* and one past */
                            check_status(noble_linear_workspace_size(&d, &res, &scr));
                            check_status(noble_linear_fwd_scratch_size(&d, &fs));
                            check_status(noble_lr_multipliers(&d, &rc, &lr));
                            /* x missing (required when T > 0), else W missing */
                            check_status(noble_linear_fwd(&d, d.T > 0 ? NULL : p[0], d.T > 0 ? p[1] : NULL, NULL,
                                                          p[3], (const float*)p[4], (const float*)p[5], p[6],
                                                          (const float*)p[7], (const float*)p[8], p[9], p[10], p[11],
                                                          p[12], scr, NULL));
                            check_status(noble_linear_fwd_static(&d, p[0], NULL, NULL, p[3], (const float*)p[4],
                                                                 (const float*)p[5], p[6], (const float*)p[7],
                                                                 (const float*)p[8], p[9], p[10], p[11], NULL));
                            /* dy missing (required when T > 0), else W missing */
                            check_status(noble_linear_bwd(&d, d.T > 0 ? NULL : p[0], p[1], d.T > 0 ? p[2] : NULL,
                                                          p[3], (const float*)p[4],
                                                          (const float*)p[5], p[6], (const float*)p[7],
                                                          (const float*)p[8], p[9], p[10], p[11], NULL, NULL,
                                                          (float*)p[14], (float*)p[15], (float*)p[16],
                                                          (float*)p[17], (float*)p[18], (float*)p[19],
                                                          (float*)p[20], p[21], scr, NULL));
                        }
    for (i = 0; i < 12; ++i) {
        const char* s = noble_status_string((int)i - 2);
        if (!s || !s[0]) ++bad;
    }
    check_status(noble_profile_next_wgrad(NULL, NULL, NULL));
    if (bad) return 1;
    printf("ok %ld\n", calls);
    return 0;
}
