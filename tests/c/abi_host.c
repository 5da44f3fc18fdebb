/* C99 client of the C ABI on host-only plans: builds a constant-Q plan and a
 * band-list plan from the Table 1 preset, queries them and checks error
 * paths. Exit status 0 on success; prints the first failed check. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include "nsgcqt.h"

#define CHECK(cond)                                                       \
    do {                                                                  \
        if (!(cond)) {                                                    \
            fprintf(stderr, "check failed: %s (line %d): %s\n", #cond,   \
                    __LINE__, nsgcqt_last_error());                       \
            return 1;                                                     \
        }                                                                 \
    } while (0)

int main(void) {
    nsgcqt_plan p = NULL;
    nsgcqt_info info;
    nsgcqt_band band;

    /* constant-Q plan of the stress workload's layout */
    CHECK(nsgcqt_plan_create_host(&p, 22050.0, 55.0, 11025.0, 36, 88200, 128) == NSGCQT_OK);
    CHECK(nsgcqt_plan_info(p, &info) == NSGCQT_OK);
    CHECK(info.n_bands == 278 && info.total_coeffs == 88835 && info.packed_len == 44100);
    CHECK(info.device_tables == 0 && info.ws_analyse > 0);
    long long sum = 0;
    for (int i = 0; i < info.n_bands; ++i) {
        CHECK(nsgcqt_band_info(p, i, &band) == NSGCQT_OK);
        CHECK(band.offset == sum && band.length == band.k_hi - band.k_lo + 1);
        sum += band.length;
    }
    CHECK(sum == info.total_coeffs);
    CHECK(nsgcqt_band_info(p, (int)info.n_bands, &band) == NSGCQT_EINVAL);
    float* g = malloc(sizeof(float) * (size_t)info.total_coeffs);
    CHECK(g && nsgcqt_plan_weights(p, 0, g, sizeof(float) * (size_t)info.total_coeffs) == NSGCQT_OK);
    for (long long i = 0; i < info.total_coeffs; ++i) CHECK(g[i] >= 0.f && g[i] <= 1.f);
    free(g);
    CHECK(nsgcqt_plan_destroy(p) == NSGCQT_OK);

    /* the Table 1 preset through an explicit band list */
    int n = 0;
    double fs = 0.0;
    int64_t N = 0;
    CHECK(nsgcqt_layout_table1(NULL, 0, &n, &fs, &N) == NSGCQT_OK && n == 154);
    nsgcqt_band_spec* specs = malloc(sizeof(nsgcqt_band_spec) * (size_t)n);
    CHECK(specs && nsgcqt_layout_table1(specs, n, &n, NULL, NULL) == NSGCQT_OK);
    CHECK(nsgcqt_plan_create_bands_host(&p, fs, N, 4, n, specs) == NSGCQT_OK);
    CHECK(nsgcqt_plan_info(p, &info) == NSGCQT_OK && info.total_coeffs == 132992);
    CHECK(nsgcqt_plan_destroy(p) == NSGCQT_OK);
    /* a length below its support width is rejected */
    specs[5].length = 2;
    p = NULL;
    CHECK(nsgcqt_plan_create_bands_host(&p, fs, N, 4, n, specs) == NSGCQT_EINVAL && p == NULL);
    free(specs);

    /* argument errors */
    CHECK(nsgcqt_plan_create_host(&p, 22050.0, 55.0, 11025.0, 36, 88201, 1) == NSGCQT_EINVAL);
    CHECK(nsgcqt_plan_create_host(NULL, 22050.0, 55.0, 11025.0, 36, 88200, 1) == NSGCQT_EINVAL);
    CHECK(nsgcqt_plan_destroy(NULL) == NSGCQT_OK);
    printf("ok\n");
    return 0;
}
