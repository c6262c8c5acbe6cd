/*
 * Drives the host side of libgspn's C ABI under AddressSanitizer and
 * UndefinedBehaviorSanitizer, on a host without a GPU (tests/test_sanitize.py
 * builds the library's sources for the host only, with the sanitizers, and
 * links them with this file).  It takes every path that runs before the first
 * device call: argument checks of every entry point, overlap and alignment
 * checks, the workspace size queries (the dispatch in counting mode, which
 * launches nothing) for one shape of every kernel family and for sizes near
 * the limits, and the status strings.  Pointers are fake device addresses
 * that the host never dereferences.  Exit status 0 when every call returned
 * the expected status with no sanitizer report.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "gspn.h"

static int failures = 0;

#define EXPECT(got, want)                                                                    \
    do {                                                                                     \
        const int g_ = (got), w_ = (want);                                                   \
        if (g_ != w_) {                                                                      \
            fprintf(stderr, "line %d: %s returned %d, expected %d\n", __LINE__, #got, g_,    \
                    w_);                                                                     \
            ++failures;                                                                      \
        }                                                                                    \
    } while (0)

/* fake, 16-byte aligned device addresses, `step` bytes apart */
static void *fake(int i, uint64_t step, uint64_t off)
{
    return (void *)(uintptr_t)(0x7F0000000000ull + (uint64_t)i * step + off);
}

typedef int (*fwd_fn)(const void *, const void *, const void *, const void *, void *, int, int,
                      int, int, int, int, int, void *, int64_t, void *);
typedef int (*bwd_fn)(const void *, const void *, const void *, const void *, const void *,
                      void *, void *, void *, void *, int, int, int, int, int, int, int, void *,
                      int64_t, void *);

static void check_fwd(fwd_fn f)
{
    void *p[5];
    for (int i = 0; i < 5; ++i)
        p[i] = fake(i, 1u << 20, 0);
#define CALLF(P0, P1, P2, P3, P4, DIR, B, C, G, H, W, DT) \
    f(P0, P1, P2, P3, P4, DIR, B, C, G, H, W, DT, NULL, 0, NULL)
    for (int k = 0; k < 5; ++k) {
        void *q[5];
        memcpy(q, p, sizeof(q));
        q[k] = NULL;
        EXPECT(CALLF(q[0], q[1], q[2], q[3], q[4], 15, 1, 4, 2, 8, 8, GSPN_BF16), GSPN_ERR_NULL);
        q[k] = fake(k, 1u << 20, 8);
        EXPECT(CALLF(q[0], q[1], q[2], q[3], q[4], 15, 1, 4, 2, 8, 8, GSPN_BF16), GSPN_ERR_ALIGN);
    }
    const int bad_dirs[] = {0, 16, -1, 31};
    for (int k = 0; k < 4; ++k)
        EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], bad_dirs[k], 1, 4, 2, 8, 8, GSPN_BF16),
               GSPN_ERR_DIRECTION);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 1, 4, 2, 8, 8, 7), GSPN_ERR_DTYPE);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 0, 4, 2, 8, 8, GSPN_BF16), GSPN_ERR_DIM);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 1, 6, 4, 8, 8, GSPN_BF16), GSPN_ERR_DIM);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 1, 4, 2, -3, 8, GSPN_BF16), GSPN_ERR_DIM);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 1, 4, 2, 4097, 8, GSPN_BF16),
           GSPN_ERR_UNSUPPORTED);
    /* sizes whose element counts overflow 32 and 64 bits */
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 1 << 20, 1 << 10, 1, 4096, 4096, GSPN_BF16),
           GSPN_ERR_UNSUPPORTED);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[4], 15, 2147483647, 2147483646, 2, 4096, 4096,
                 GSPN_F32),
           GSPN_ERR_UNSUPPORTED);
    /* output over an input */
    EXPECT(CALLF(p[0], p[1], p[2], p[3], p[0], 15, 1, 4, 2, 8, 8, GSPN_BF16), GSPN_ERR_ALIAS);
    EXPECT(CALLF(p[0], p[1], p[2], p[3], fake(0, 1, 256), 15, 1, 4, 2, 8, 8, GSPN_BF16),
           GSPN_ERR_ALIAS);
#undef CALLF
}

static int bwd_slots4_as_bwd(const void *x, const void *w, const void *lam, const void *u,
                             const void *dy, void *dx, void *dw, void *dlam, void *du, int dir,
                             int B, int C, int G, int H, int W, int dt, void *ws, int64_t wsb,
                             void *s)
{
    return gspn_scan_bwd_slots(4, x, w, lam, u, dy, dx, dw, dlam, du, dir, B, C, G, H, W, dt, ws,
                               wsb, s);
}

static void check_bwd(bwd_fn f)
{
    void *p[9];
    for (int i = 0; i < 9; ++i)
        p[i] = fake(i, 1u << 20, 0);
#define CALLB(Q, DIR, B, C, G, H, W, DT, WS, WSB) \
    f(Q[0], Q[1], Q[2], Q[3], Q[4], Q[5], Q[6], Q[7], Q[8], DIR, B, C, G, H, W, DT, WS, WSB, NULL)
    for (int k = 0; k < 9; ++k) {
        void *q[9];
        memcpy(q, p, sizeof(q));
        q[k] = NULL;
        EXPECT(CALLB(q, 15, 1, 4, 2, 8, 8, GSPN_BF16, NULL, 0), GSPN_ERR_NULL);
        q[k] = fake(k, 1u << 20, 8);
        EXPECT(CALLB(q, 15, 1, 4, 2, 8, 8, GSPN_BF16, NULL, 0), GSPN_ERR_ALIGN);
    }
    EXPECT(CALLB(p, 0, 1, 4, 2, 8, 8, GSPN_BF16, NULL, 0), GSPN_ERR_DIRECTION);
    EXPECT(CALLB(p, 15, 1, 4, 2, 8, 8, -1, NULL, 0), GSPN_ERR_DTYPE);
    EXPECT(CALLB(p, 15, 1, 4, 2, 8, 0, GSPN_BF16, NULL, 0), GSPN_ERR_DIM);
    {
        void *q[9];
        memcpy(q, p, sizeof(q));
        q[7] = q[8];   /* two outputs on one buffer */
        EXPECT(CALLB(q, 15, 1, 4, 2, 8, 8, GSPN_BF16, NULL, 0), GSPN_ERR_ALIAS);
    }
    /* a shape with workspace: missing, short, misaligned, overlapping */
    int64_t need = -1;
    EXPECT(gspn_workspace_size(GSPN_OP_BWD, 5, 1, 4, 2, 70, 100, GSPN_BF16, &need), GSPN_OK);
    void *b[9];
    for (int i = 0; i < 9; ++i)
        b[i] = fake(i + 16, 1u << 26, 0);
    void *ws = fake(32, 1u << 26, 0);
    if (f == gspn_scan_bwd || f == gspn_scan_bwd_blocked || f == bwd_slots4_as_bwd) {
        EXPECT(CALLB(b, 5, 1, 4, 2, 70, 100, GSPN_BF16, NULL, 0), GSPN_ERR_WORKSPACE);
        EXPECT(CALLB(b, 5, 1, 4, 2, 70, 100, GSPN_BF16, ws, need - 1), GSPN_ERR_WORKSPACE);
        EXPECT(CALLB(b, 5, 1, 4, 2, 70, 100, GSPN_BF16, ws, -1), GSPN_ERR_WORKSPACE);
        EXPECT(CALLB(b, 5, 1, 4, 2, 70, 100, GSPN_BF16, (char *)ws + 8, need), GSPN_ERR_ALIGN);
        EXPECT(CALLB(b, 5, 1, 4, 2, 70, 100, GSPN_BF16, b[0], need), GSPN_ERR_ALIAS);
    }
#undef CALLB
}

static int bwd_static_as_bwd(const void *x, const void *w, const void *lam, const void *u,
                             const void *dy, void *dx, void *dw, void *dlam, void *du, int dir,
                             int B, int C, int G, int H, int W, int dt, void *ws, int64_t wsb,
                             void *s)
{
    (void)ws;
    (void)wsb;
    return gspn_scan_bwd_static(x, w, lam, u, dy, dx, dw, dlam, du, dir, B, C, G, H, W, dt, s);
}

static void check_queries(void)
{
    /* one shape of every kernel family, both storage types */
    static const int shapes[][3] = {
        {1, 1, GSPN_BF16},    {5, 7, GSPN_BF16},    {8, 8, GSPN_BF16},     {14, 14, GSPN_BF16},
        {40, 24, GSPN_BF16},  {40, 24, GSPN_F32},   {64, 64, GSPN_BF16},   {56, 56, GSPN_BF16},
        {72, 136, GSPN_BF16}, {256, 256, GSPN_BF16}, {70, 100, GSPN_BF16}, {3, 130, GSPN_F32},
        {4096, 8, GSPN_BF16}, {8, 4096, GSPN_F32},
    };
    static const int groups[][2] = {{4, 1}, {64, 2}, {8, 8}, {768, 24}, {768, 768}};
    static const int dirs[] = {15, 1, 2, 4, 8, 6, 9};
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        for (int c = 0; c < 5; ++c)
            for (int op = 0; op <= GSPN_OP_BWD_NORM_RESERVE; ++op)
                for (size_t d = 0; d < sizeof(dirs) / sizeof(dirs[0]); ++d) {
                    int64_t n1 = -1, n2 = -2;
                    const int st = gspn_workspace_size(op, dirs[d], 2, groups[c][0], groups[c][1],
                                                       shapes[s][0], shapes[s][1], shapes[s][2],
                                                       &n1);
                    EXPECT(st, GSPN_OK);
                    gspn_workspace_size(op, dirs[d], 2, groups[c][0], groups[c][1], shapes[s][0],
                                        shapes[s][1], shapes[s][2], &n2);
                    if (n1 < 0 || n1 != n2) {
                        fprintf(stderr, "query %dx%d op %d: %lld then %lld\n", shapes[s][0],
                                shapes[s][1], op, (long long)n1, (long long)n2);
                        ++failures;
                    }
                }
    int64_t n = 0;
    EXPECT(gspn_workspace_size(GSPN_OP_BWD_NORM_RESERVE + 1, 15, 1, 4, 2, 8, 8, GSPN_BF16, &n),
           GSPN_ERR_UNSUPPORTED);
    /* the training pairs' reserves: sizes and host checks */
    for (size_t s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s)
        for (int c = 0; c < 5; ++c) {
            int64_t r1 = -1, r2 = -1;
            EXPECT(gspn_reserve_size(15, 2, groups[c][0], groups[c][1], shapes[s][0],
                                     shapes[s][1], shapes[s][2], &r1),
                   GSPN_OK);
            EXPECT(gspn_reserve_size_norm(15, 2, groups[c][0], groups[c][1], shapes[s][0],
                                          shapes[s][1], shapes[s][2], &r2),
                   GSPN_OK);
            if (r1 < 0 || r2 < r1) {
                fprintf(stderr, "reserve %dx%d: %lld, norm %lld\n", shapes[s][0], shapes[s][1],
                        (long long)r1, (long long)r2);
                ++failures;
            }
        }
    {
        int64_t rn = 0, wn = 0;
        EXPECT(gspn_reserve_size(15, 1, 64, 2, 64, 64, GSPN_BF16, &rn), GSPN_OK);
        EXPECT(gspn_workspace_size(GSPN_OP_BWD_RESERVE, 15, 1, 64, 2, 64, 64, GSPN_BF16, &wn),
               GSPN_OK);
        void *t[12];
        for (int i = 0; i < 12; ++i)
            t[i] = fake(i + 128, 1u << 26, 0);
        EXPECT(gspn_scan_fwd_train(t[0], t[1], t[2], t[3], t[4], 15, 1, 64, 2, 64, 64, GSPN_BF16,
                                   NULL, 0, NULL, 0, NULL),
               GSPN_ERR_WORKSPACE);
        EXPECT(gspn_scan_fwd_train(t[0], t[1], t[2], t[3], t[4], 15, 1, 64, 2, 64, 64, GSPN_BF16,
                                   t[0], rn, NULL, 0, NULL),
               GSPN_ERR_ALIAS);
        EXPECT(gspn_scan_bwd_reserve(t[0], t[1], t[2], t[3], t[4], t[5], t[6], t[7], t[8], 15, 1,
                                     64, 2, 64, 64, GSPN_BF16, t[9], rn - 16, t[10], wn, NULL),
               GSPN_ERR_WORKSPACE);
        EXPECT(gspn_scan_bwd_norm_reserve(t[0], t[1], t[2], t[3], t[4], t[5], t[6], t[7], t[8],
                                          15, 1, 64, 2, 64, 64, GSPN_BF16, t[9], -1, t[10], wn,
                                          NULL),
               GSPN_ERR_WORKSPACE);
    }
    EXPECT(gspn_workspace_size(GSPN_OP_FWD, 15, 1, 4, 2, 8, 8, GSPN_BF16, NULL), GSPN_ERR_NULL);
    EXPECT(gspn_workspace_size(GSPN_OP_BWD, 15, 1 << 20, 1 << 10, 1, 4096, 4096, GSPN_BF16, &n),
           GSPN_ERR_UNSUPPORTED);
    /* the latent sublayer */
    static const int lat[][2] = {{5, 7}, {37, 37}, {74, 74}, {185, 185}, {300, 9}};
    for (int s = 0; s < 5; ++s) {
        const int st = gspn_latent_workspace_size(15, 32, 1152, 64, lat[s][0], lat[s][1],
                                                  GSPN_BF16, &n);
        if (st != GSPN_OK && st != GSPN_ERR_UNSUPPORTED) {
            fprintf(stderr, "latent query %dx%d: status %d\n", lat[s][0], lat[s][1], st);
            ++failures;
        }
    }
    EXPECT(gspn_latent_workspace_size(15, 32, 1152, 64, 37, 37, GSPN_F32, &n),
           GSPN_ERR_UNSUPPORTED);
    EXPECT(gspn_latent_workspace_size(0, 32, 1152, 64, 37, 37, GSPN_BF16, &n),
           GSPN_ERR_DIRECTION);
    void *p[8];
    for (int i = 0; i < 8; ++i)
        p[i] = fake(i, 1u << 24, 0);
    EXPECT(gspn_latent_fwd(p[0], p[1], p[2], p[3], p[4], p[5], p[6], 15, 1, 32, 16, 8, 8,
                           GSPN_BF16, NULL, 0, NULL),
           GSPN_ERR_WORKSPACE);
    EXPECT(gspn_latent_fwd(p[0], p[1], p[2], p[3], p[4], p[5], p[0], 15, 1, 32, 16, 8, 8,
                           GSPN_BF16, p[7], 1 << 20, NULL),
           GSPN_ERR_ALIAS);
    EXPECT(gspn_project(p[0], p[1], p[2], 1, 8, 12, 8, 8, GSPN_BF16, NULL), GSPN_ERR_UNSUPPORTED);
    EXPECT(gspn_project(p[0], NULL, p[2], 1, 8, 8, 8, 8, GSPN_BF16, NULL), GSPN_ERR_NULL);
    EXPECT(gspn_latent_params(p[0], p[1], p[2], p[3], p[4], p[5], p[6], 15, 1, 12, 8, 8,
                              GSPN_BF16, NULL),
           GSPN_ERR_UNSUPPORTED);
    /* the allocation-free backward refuses a need above its fixed array */
    int64_t need = 0;
    EXPECT(gspn_workspace_size(GSPN_OP_BWD, 15, 16, 64, 2, 70, 100, GSPN_BF16, &need), GSPN_OK);
    if (need <= GSPN_STATIC_SCRATCH_BYTES) {
        fprintf(stderr, "static limit case needs only %lld bytes\n", (long long)need);
        ++failures;
    }
    void *b[9];
    for (int i = 0; i < 9; ++i)
        b[i] = fake(i + 64, 1ull << 32, 0);
    EXPECT(gspn_scan_bwd_static(b[0], b[1], b[2], b[3], b[4], b[5], b[6], b[7], b[8], 15, 16, 64,
                                2, 70, 100, GSPN_BF16, NULL),
           GSPN_ERR_WORKSPACE);
}

int main(void)
{
    check_fwd(gspn_scan_fwd);
    check_fwd(gspn_scan_fwd_blocked);
    check_fwd(gspn_scan_fwd_norm);
    check_bwd(gspn_scan_bwd);
    check_bwd(gspn_scan_bwd_blocked);
    check_bwd(gspn_scan_bwd_norm);
    check_bwd(bwd_static_as_bwd);
    check_bwd(bwd_slots4_as_bwd);
    {
        int64_t n4 = 0, n8 = 0;
        EXPECT(gspn_workspace_size_slots(4, 15, 1, 64, 2, 64, 64, GSPN_BF16, &n4), GSPN_OK);
        EXPECT(gspn_workspace_size_slots(8, 15, 1, 64, 2, 64, 64, GSPN_BF16, &n8), GSPN_OK);
        EXPECT(n4 > n8, 1);
        EXPECT(gspn_workspace_size_slots(3, 15, 1, 64, 2, 64, 64, GSPN_BF16, &n4),
               GSPN_ERR_UNSUPPORTED);
    }
    check_queries();
    for (int s = -20; s < 3; ++s)
        if (gspn_strerror(s) == NULL || gspn_strerror(s)[0] == '\0') {
            fprintf(stderr, "strerror(%d) empty\n", s);
            ++failures;
        }
    EXPECT(gspn_version() >= 200, 1);
    if (failures)
        fprintf(stderr, "%d failures\n", failures);
    else
        printf("abi driver: all checks clean\n");
    return failures ? 1 : 0;
}
