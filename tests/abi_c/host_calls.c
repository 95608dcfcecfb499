/*
 * A plain C11 client of the C-ABI: the header must compile as C, and the
 * host-only entry points (version, Eq. 3 trimmed mean, the Eq. 4 check,
 * argument validation and the error string) must behave without a GPU.
 * Exit status 0 = all checks passed.
 */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "mep.h"

static int failures = 0;
#define CHECK(c, msg) do { if (!(c)) { fprintf(stderr, "FAIL: %s\n", msg); ++failures; } } while (0)

int main(void)
{
    const char* v = mep_version();
    CHECK(v != NULL && strlen(v) > 0, "version string");

    /* Eq. 3: samples 1..30, k = 3 -> mean of 4..27 = 15.5 */
    double s[30];
    for (int i = 0; i < 30; ++i)
        s[i] = (double)(30 - i);
    CHECK(mep_trimmed_mean(s, 30, 3) == 15.5, "trimmed mean of 1..30, k = 3");
    CHECK(isnan(mep_trimmed_mean(s, 6, 3)), "R <= 2k gives NaN");

    /* Eq. 4 on host buffers: normwise relative error */
    const float out[4] = {1.0f, 2.0f, 3.0f, 4.0f};
    const double ref[4] = {1.0, 2.0, 3.0, 4.0004};
    double err = -1.0;
    int pass = -1;
    CHECK(mep_check_fe(MEP_F32, out, ref, 4, 1e-4, &err, &pass) == MEP_OK, "check_fe returns OK");
    /* max |out - ref| / max |ref| = (4.0004 - 4) / 4.0004, just below 1e-4 */
    CHECK(fabs(err - (ref[3] - 4.0) / ref[3]) < 1e-15 && pass == 1, "normwise error passes at 1e-4");
    CHECK(mep_check_fe(MEP_F32, out, ref, 4, 5e-5, &err, &pass) == MEP_OK && pass == 0, "fails at 5e-5");

    /* argument validation happens before anything touches the GPU */
    CHECK(mep_matvec(7, 4, 4, NULL, NULL, NULL, NULL, 0, NULL) == MEP_EINVAL, "bad dtype");
    CHECK(strlen(mep_last_error()) > 0, "error string set");
    CHECK(mep_matvec(MEP_F32, -1, 4, NULL, NULL, NULL, NULL, 0, NULL) == MEP_EINVAL, "negative m");
    CHECK(mep_matvec(MEP_F32, 4, 4, NULL, NULL, NULL, NULL, 0, NULL) == MEP_EINVAL, "NULL matrix");
    CHECK(mep_workspace_bytes(MEP_OP_ATA_X, MEP_F32, 16384, 16384) > 0, "ATAX needs a workspace");
    CHECK(mep_workspace_bytes(MEP_OP_MATVEC, MEP_F32, 0, 16) == 0, "empty matrix needs none");
    CHECK(mep_variant_count(MEP_OP_BICG, MEP_F64, 4096, 4096) >= 1, "candidates exist");
    char info[256];
    CHECK(mep_variant_info(MEP_OP_ATA_X, MEP_F32, 16384, 16384, 0, info, sizeof info) == MEP_OK &&
              strstr(info, "G=512") != NULL, "default shape of the headline workload");
    CHECK(mep_profile_begin_sampled(4, 0, 1) == MEP_EINVAL, "sampled profiling rejects group 0");

    if (failures) {
        fprintf(stderr, "%d check(s) failed\n", failures);
        return 1;
    }
    printf("C client: all checks passed (%s)\n", v);
    return 0;
}
