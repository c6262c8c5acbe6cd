/*
 * GSPN line-scan oracle: TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU implementation of the 2D line-scan
 * propagation, written from the paper's definitions:
 *
 *   Sec. 3, Eq. (gspn_recurrence):   h_i = w_i h_{i-1} + Diag(lambda_i) x_i
 *   Sec. 3, Eq. (gspn_output):       y_i = u_i (.) h_i
 *   Sec. 3, Eq. (row_stochastic_norm) and the paragraph after it:
 *       w_i is tridiagonal -- every pixel reads three neighbours of the
 *       previous line (top-left, top-center, top-right) -- and four passes
 *       (top-to-bottom, bottom-to-top, left-to-right, right-to-left) are run.
 *   Sec. 4.2, Eq. (2dsp): one w_i shared by several channels.
 *
 * Only tests/, the smoke check and the benchmark's CPU-baseline leg may call
 * this file.  It shares no code, header or table with the GPU library.
 *
 * Readings where the paper is silent (each one is listed in the design notes):
 *  - the state before the first line is zero, so h_0 = lambda_0 (.) x_0 (this
 *    matches the first block row of the paper's block lower-triangular form,
 *    Eq. (global));
 *  - tap k of the weight stored at a target pixel reads the previous line at
 *    perpendicular offset k-1 (column offset for vertical scans, row offset
 *    for horizontal ones); taps leaving the grid, and every tap on the first
 *    scanned line, are ignored;
 *  - the four directional outputs are summed: y = sum_d u_d (.) h_d;
 *  - each direction has its own w_d, lambda_d, u_d; x is shared;
 *  - channel c uses weight group c / (C/G);
 *  - in the normalization of Eq. (row_stochastic_norm), sigma is the logistic
 *    sigmoid, N(j) holds the taps whose neighbour lies on the grid (the
 *    others get weight 0), and the denominator is clamped below at
 *    NORM_EPS = 1e-30 (the paper's fused normalization clamps but gives no
 *    constant; this one changes nothing unless every sigmoid of N(j) is
 *    below 1e-30, i.e. all logits are below about -69).
 *
 * All arithmetic is double precision.  Layouts (row-major):
 *   x, y, dy, dx       [B][C][H][W]
 *   w, dw              [D][B][G][3][H][W]
 *   lam, u, dlam, du   [D][B][C][H][W]
 * where D is the number of directions in the mask, stacked in increasing
 * direction-bit order (1 = T2B, 2 = B2T, 4 = L2R, 8 = R2L).
 */
#include <stdint.h>
#include <stdlib.h>
#include <math.h>
#include <string.h>

#define NORM_EPS 1e-30

enum { DIR_T2B = 1, DIR_B2T = 2, DIR_L2R = 4, DIR_R2L = 8 };

/* Scan length L and line length P of direction d. */
static int scan_len(int d, int H, int W) { return (d == DIR_T2B || d == DIR_B2T) ? H : W; }
static int line_len(int d, int H, int W) { return (d == DIR_T2B || d == DIR_B2T) ? W : H; }

/* Storage (row, col) of frame position (step i, line position j). */
static void to_storage(int d, int i, int j, int H, int W, int *row, int *col)
{
    switch (d) {
    case DIR_T2B: *row = i;         *col = j;         break;
    case DIR_B2T: *row = H - 1 - i; *col = j;         break;
    case DIR_L2R: *row = j;         *col = i;         break;
    default:      *row = j;         *col = W - 1 - i; break; /* DIR_R2L */
    }
}

/* Flat offsets into the layouts above. */
static int64_t at_x(int b, int c, int r, int col, int C, int H, int W)
{
    return (((int64_t)b * C + c) * H + r) * W + col;
}
static int64_t at_dir(int s, int b, int c, int r, int col, int B, int C, int H, int W)
{
    return ((((int64_t)s * B + b) * C + c) * H + r) * W + col;
}
static int64_t at_w(int s, int b, int g, int k, int r, int col, int B, int G, int H, int W)
{
    return (((((int64_t)s * B + b) * G + g) * 3 + k) * H + r) * W + col;
}

/*
 * Hidden states of one (direction slot s, batch b, channel c) scan:
 * hist[i*P + j] = h_i[j].
 */
static void scan_states(const double *x, const double *w, const double *lam,
                        int d, int s, int b, int c, int B, int C, int G,
                        int H, int W, double *hist)
{
    int L = scan_len(d, H, W), P = line_len(d, H, W);
    int g = c / (C / G);
    for (int i = 0; i < L; ++i) {
        for (int j = 0; j < P; ++j) {
            int r, col;
            to_storage(d, i, j, H, W, &r, &col);
            double acc = 0.0;
            if (i > 0) {
                for (int k = 0; k < 3; ++k) {
                    int jj = j + k - 1;              /* neighbour on line i-1 */
                    if (jj < 0 || jj >= P)
                        continue;
                    acc += w[at_w(s, b, g, k, r, col, B, G, H, W)] * hist[(int64_t)(i - 1) * P + jj];
                }
            }
            acc += lam[at_dir(s, b, c, r, col, B, C, H, W)] * x[at_x(b, c, r, col, C, H, W)];
            hist[(int64_t)i * P + j] = acc;
        }
    }
}

/* y = sum over the directions in dirmask of u_d (.) h_d. */
void oracle_scan_fwd(const double *x, const double *w, const double *lam,
                     const double *u, double *y, int dirmask,
                     int B, int C, int G, int H, int W)
{
    int64_t n = (int64_t)B * C * H * W;
    memset(y, 0, sizeof(double) * (size_t)n);
    int maxlp = H > W ? H : W;
    double *hist = malloc(sizeof(double) * (size_t)maxlp * (size_t)maxlp);
    int s = 0;
    for (int d = 1; d <= 8; d <<= 1) {
        if (!(dirmask & d))
            continue;
        int L = scan_len(d, H, W), P = line_len(d, H, W);
        for (int b = 0; b < B; ++b) {
            for (int c = 0; c < C; ++c) {
                scan_states(x, w, lam, d, s, b, c, B, C, G, H, W, hist);
                for (int i = 0; i < L; ++i) {
                    for (int j = 0; j < P; ++j) {
                        int r, col;
                        to_storage(d, i, j, H, W, &r, &col);
                        y[at_x(b, c, r, col, C, H, W)] +=
                            u[at_dir(s, b, c, r, col, B, C, H, W)] * hist[(int64_t)i * P + j];
                    }
                }
            }
        }
        ++s;
    }
    free(hist);
}

/*
 * Gradients of a loss l(y) given dy = dl/dy.
 *
 * With a_i = dl/dh_i (the adjoint state), the recurrence above gives
 *   a_i[j] = u_i[j] dy_i[j] + sum_k w_{i+1}[j-k+1, k] a_{i+1}[j-k+1]
 * (the targets on line i+1 that read position j), a_L = 0, and
 *   du_i[j]      = dy_i[j] h_i[j]
 *   dlam_i[j]    = a_i[j] x_i[j]
 *   dx_i[j]     += a_i[j] lam_i[j]                 (summed over directions)
 *   dw_i[j, k]  += a_i[j] h_{i-1}[j+k-1]           (i > 0, tap inside the grid;
 *                                                   summed over the group's channels)
 * Every other dw entry is 0.
 */
void oracle_scan_bwd(const double *x, const double *w, const double *lam,
                     const double *u, const double *dy, double *dx, double *dw,
                     double *dlam, double *du, int dirmask,
                     int B, int C, int G, int H, int W)
{
    int D = 0;
    for (int d = 1; d <= 8; d <<= 1)
        D += (dirmask & d) ? 1 : 0;
    int64_t n = (int64_t)B * C * H * W;
    memset(dx, 0, sizeof(double) * (size_t)n);
    memset(dw, 0, sizeof(double) * (size_t)D * B * G * 3 * H * W);
    int maxlp = H > W ? H : W;
    double *hist = malloc(sizeof(double) * (size_t)maxlp * (size_t)maxlp);
    double *a_next = malloc(sizeof(double) * (size_t)maxlp);
    double *a_cur = malloc(sizeof(double) * (size_t)maxlp);
    int s = 0;
    for (int d = 1; d <= 8; d <<= 1) {
        if (!(dirmask & d))
            continue;
        int L = scan_len(d, H, W), P = line_len(d, H, W);
        for (int b = 0; b < B; ++b) {
            for (int c = 0; c < C; ++c) {
                int g = c / (C / G);
                scan_states(x, w, lam, d, s, b, c, B, C, G, H, W, hist);
                for (int j = 0; j < P; ++j)
                    a_next[j] = 0.0;
                for (int i = L - 1; i >= 0; --i) {
                    for (int j = 0; j < P; ++j) {
                        int r, col;
                        to_storage(d, i, j, H, W, &r, &col);
                        int64_t ox = at_x(b, c, r, col, C, H, W);
                        int64_t od = at_dir(s, b, c, r, col, B, C, H, W);
                        double a = u[od] * dy[ox];
                        if (i + 1 < L) {
                            for (int k = 0; k < 3; ++k) {
                                int jt = j - k + 1;      /* target on line i+1 */
                                if (jt < 0 || jt >= P)
                                    continue;
                                int r2, c2;
                                to_storage(d, i + 1, jt, H, W, &r2, &c2);
                                a += w[at_w(s, b, g, k, r2, c2, B, G, H, W)] * a_next[jt];
                            }
                        }
                        a_cur[j] = a;
                        du[od] = dy[ox] * hist[(int64_t)i * P + j];
                        dlam[od] = a * x[ox];
                        dx[ox] += a * lam[od];
                        if (i > 0) {
                            for (int k = 0; k < 3; ++k) {
                                int jj = j + k - 1;
                                if (jj < 0 || jj >= P)
                                    continue;
                                dw[at_w(s, b, g, k, r, col, B, G, H, W)] +=
                                    a * hist[(int64_t)(i - 1) * P + jj];
                            }
                        }
                    }
                    double *t = a_next;
                    a_next = a_cur;
                    a_cur = t;
                }
            }
        }
        ++s;
    }
    free(hist);
    free(a_next);
    free(a_cur);
}

/* Logistic sigmoid. */
static double sigmoid(double t) { return 1.0 / (1.0 + exp(-t)); }

/* Whether tap k of the weight at storage (r, col) reads a neighbour on the grid. */
static int tap_on_grid(int d, int k, int r, int col, int H, int W)
{
    if (d == DIR_T2B || d == DIR_B2T) {
        int c2 = col + k - 1;
        return c2 >= 0 && c2 < W;
    }
    int r2 = r + k - 1;
    return r2 >= 0 && r2 < H;
}

/*
 * Sec. 3, Eq. (row_stochastic_norm): the weights from their logits wt,
 *   w(j, k) = sigma(wt(j, k)) / max(sum_{k' in N(j)} sigma(wt(j, k')), NORM_EPS)
 * for k in N(j), and 0 for the taps outside the grid.  Layout of wt and w:
 * [D][B][G][3][H][W].
 */
void oracle_norm_w(const double *wt, double *w, int dirmask, int B, int G, int H, int W)
{
    int s = 0;
    for (int d = 1; d <= 8; d <<= 1) {
        if (!(dirmask & d))
            continue;
        for (int b = 0; b < B; ++b)
            for (int g = 0; g < G; ++g)
                for (int r = 0; r < H; ++r)
                    for (int col = 0; col < W; ++col) {
                        double sg[3], sum = 0.0;
                        for (int k = 0; k < 3; ++k) {
                            sg[k] = tap_on_grid(d, k, r, col, H, W)
                                        ? sigmoid(wt[at_w(s, b, g, k, r, col, B, G, H, W)])
                                        : 0.0;
                            sum += sg[k];
                        }
                        if (sum < NORM_EPS)
                            sum = NORM_EPS;
                        for (int k = 0; k < 3; ++k)
                            w[at_w(s, b, g, k, r, col, B, G, H, W)] = sg[k] / sum;
                    }
        ++s;
    }
}

/*
 * Gradient of a loss with respect to the logits, given dw = dl/dw of the
 * normalized weights.  With s_k = sigma(wt_k) and S the sum over N(j):
 *   dl/dwt_m = s_m (1 - s_m) (dw_m - sum_{k in N(j)} w_k dw_k) / S
 * for m in N(j), and 0 outside it; where the clamp holds S at NORM_EPS the
 * sum term drops (S no longer depends on the logits).
 */
void oracle_norm_w_bwd(const double *wt, const double *dw, double *dwt, int dirmask, int B,
                       int G, int H, int W)
{
    int s = 0;
    for (int d = 1; d <= 8; d <<= 1) {
        if (!(dirmask & d))
            continue;
        for (int b = 0; b < B; ++b)
            for (int g = 0; g < G; ++g)
                for (int r = 0; r < H; ++r)
                    for (int col = 0; col < W; ++col) {
                        double sg[3], gw[3], sum = 0.0;
                        int on[3];
                        for (int k = 0; k < 3; ++k) {
                            int64_t o = at_w(s, b, g, k, r, col, B, G, H, W);
                            on[k] = tap_on_grid(d, k, r, col, H, W);
                            sg[k] = on[k] ? sigmoid(wt[o]) : 0.0;
                            gw[k] = dw[o];
                            sum += sg[k];
                        }
                        int clamped = sum < NORM_EPS;
                        double den = clamped ? NORM_EPS : sum;
                        double inner = 0.0;
                        if (!clamped)
                            for (int k = 0; k < 3; ++k)
                                if (on[k])
                                    inner += sg[k] / den * gw[k];
                        for (int k = 0; k < 3; ++k)
                            dwt[at_w(s, b, g, k, r, col, B, G, H, W)] =
                                on[k] ? sg[k] * (1.0 - sg[k]) * (gw[k] - inner) / den : 0.0;
                    }
        ++s;
    }
}
