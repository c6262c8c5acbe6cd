/*
 * Drives the C oracle and the seeded input generator under AddressSanitizer
 * and UndefinedBehaviorSanitizer (built by tests/test_sanitize.py with gcc
 * -fsanitize=address,undefined).  Every direction mask on small ragged
 * shapes, one-pixel grids and single-line scans; every output must come back
 * finite.  Exit status 0 when all calls ran clean.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_scan_fwd(const double *x, const double *w, const double *lam, const double *u,
                     double *y, int dirmask, int B, int C, int G, int H, int W);
void oracle_scan_bwd(const double *x, const double *w, const double *lam, const double *u,
                     const double *dy, double *dx, double *dw, double *dlam, double *du,
                     int dirmask, int B, int C, int G, int H, int W);
void oracle_norm_w(const double *wt, double *w, int dirmask, int B, int G, int H, int W);
void oracle_norm_w_bwd(const double *wt, const double *dw, double *dwt, int dirmask, int B,
                       int G, int H, int W);
void gspn_gen_normal(float *out, int64_t n, uint64_t seed, int tensor_id, int slot,
                     double mean, double sigma, int transform, int bf16);
void gspn_gen_taps(float *w, int B, int G, int H, int W, int vertical, uint64_t seed,
                   int tensor_id, int slot, double sigma, int bf16);

static int failures = 0;

/* exact-size heap buffers, so that any access past the end is reported */
static double *filled(int64_t n, uint64_t seed)
{
    double *p = malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    uint64_t s = seed * 0x9E3779B97F4A7C15ull + 1;
    for (int64_t i = 0; i < n; ++i) {
        s = s * 6364136223846793005ull + 1442695040888963407ull;
        p[i] = (double)(s >> 11) / 9007199254740992.0 - 0.5;
    }
    return p;
}

static void check_finite(const char *what, const double *p, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        if (!isfinite(p[i])) {
            fprintf(stderr, "%s: entry %lld not finite\n", what, (long long)i);
            ++failures;
            return;
        }
}

static int popcount4(int m) { return (m & 1) + ((m >> 1) & 1) + ((m >> 2) & 1) + ((m >> 3) & 1); }

static void run_case(int dirs, int B, int C, int G, int H, int W)
{
    const int D = popcount4(dirs);
    const int64_t n = (int64_t)B * C * H * W, nw = (int64_t)D * B * G * 3 * H * W;
    double *x = filled(n, 1), *lam = filled(D * n, 2), *u = filled(D * n, 3);
    double *wt = filled(nw, 4), *dy = filled(n, 5), *dwn = filled(nw, 6);
    double *w = malloc(sizeof(double) * (size_t)nw), *dwt = malloc(sizeof(double) * (size_t)nw);
    double *y = malloc(sizeof(double) * (size_t)n), *dx = malloc(sizeof(double) * (size_t)n);
    double *dw = malloc(sizeof(double) * (size_t)nw);
    double *dlam = malloc(sizeof(double) * (size_t)(D * n)), *du = malloc(sizeof(double) * (size_t)(D * n));
    oracle_norm_w(wt, w, dirs, B, G, H, W);
    check_finite("norm_w", w, nw);
    oracle_scan_fwd(x, w, lam, u, y, dirs, B, C, G, H, W);
    check_finite("scan_fwd", y, n);
    oracle_scan_bwd(x, w, lam, u, dy, dx, dw, dlam, du, dirs, B, C, G, H, W);
    check_finite("scan_bwd dx", dx, n);
    check_finite("scan_bwd dw", dw, nw);
    check_finite("scan_bwd dlam", dlam, D * n);
    check_finite("scan_bwd du", du, D * n);
    oracle_norm_w_bwd(wt, dwn, dwt, dirs, B, G, H, W);
    check_finite("norm_w_bwd", dwt, nw);
    free(x); free(lam); free(u); free(wt); free(dy); free(dwn); free(w); free(dwt);
    free(y); free(dx); free(dw); free(dlam); free(du);
}

int main(void)
{
    static const int shapes[][5] = {   /* B, C, G, H, W */
        {1, 1, 1, 1, 1}, {1, 2, 1, 1, 6}, {1, 2, 2, 6, 1}, {2, 4, 2, 3, 5},
        {1, 6, 3, 7, 4}, {2, 3, 1, 9, 9}, {1, 8, 8, 2, 11},
    };
    const int nshapes = (int)(sizeof(shapes) / sizeof(shapes[0]));
    for (int s = 0; s < nshapes; ++s)
        for (int dirs = 1; dirs <= 15; ++dirs)
            run_case(dirs, shapes[s][0], shapes[s][1], shapes[s][2], shapes[s][3], shapes[s][4]);

    /* the generator: ragged lengths, both transforms, both storage types,
       taps of both orientations on one-line and one-pixel grids */
    for (int64_t n = 0; n < 40; n += 13) {
        float *o = malloc(sizeof(float) * (size_t)(n > 0 ? n : 1));
        for (int t = 0; t < 2; ++t)
            for (int bf = 0; bf < 2; ++bf)
                gspn_gen_normal(o, n, 7, 1, 2, 0.1, 1.5, t, bf);
        free(o);
    }
    static const int tshapes[][4] = {{1, 1, 1, 1}, {2, 3, 1, 7}, {1, 2, 5, 1}, {2, 1, 4, 6}};
    for (int s = 0; s < 4; ++s)
        for (int v = 0; v < 2; ++v) {
            const int B = tshapes[s][0], G = tshapes[s][1], H = tshapes[s][2], W = tshapes[s][3];
            float *t = malloc(sizeof(float) * (size_t)B * G * 3 * H * W);
            gspn_gen_taps(t, B, G, H, W, v, 11, 3, 4, 1.0, 1);
            free(t);
        }
    if (failures)
        fprintf(stderr, "%d failures\n", failures);
    else
        printf("oracle driver: all cases clean\n");
    return failures ? 1 : 0;
}
