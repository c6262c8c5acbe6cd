/*
 * Seeded synthetic inputs for the GSPN line scan.
 *
 * This module only draws numbers: it holds none of the scan's arithmetic.
 * Both the CPU oracle and the GPU library are fed from the arrays written
 * here, so the two sides always see bit-identical inputs.
 *
 * Random numbers are counter based, so every element is a pure function of
 * (seed, tensor id, direction slot, flat index) and the result does not
 * depend on thread count or evaluation order:
 *
 *   key     = seed << 56 | tensor_id << 48 | slot << 40
 *   r(n)    = splitmix64_mix((key + n + 1) * GAMMA)     n = 2*idx + {0,1}
 *   u1      = ((r(2 idx) >> 11) + 1) * 2^-53            in (0, 1]
 *   u2      =  (r(2 idx + 1) >> 11)  * 2^-53            in [0, 1)
 *   z       = sqrt(-2 ln u1) cos(2 pi u2)               Box-Muller, N(0,1)
 *
 * splitmix64_mix is the output function of Steele, Lea and Flood's
 * SplitMix64 generator (constants as published by Vigna); Box-Muller is the
 * textbook polar-free form.  Values are computed in double, rounded to fp32,
 * and optionally rounded again to bfloat16 (round to nearest even) so that a
 * bf16 tensor and its fp32/fp64 copy hold the same numbers.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GAMMA 0x9E3779B97F4A7C15ull

static uint64_t splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static uint64_t stream_key(uint64_t seed, uint64_t tensor_id, uint64_t slot)
{
    return (seed << 56) | (tensor_id << 48) | (slot << 40);
}

static double std_normal(uint64_t key, uint64_t idx)
{
    uint64_t r1 = splitmix64_mix((key + 2 * idx + 1) * GAMMA);
    uint64_t r2 = splitmix64_mix((key + 2 * idx + 2) * GAMMA);
    double u1 = ((double)(r1 >> 11) + 1.0) * 0x1.0p-53;
    double u2 = (double)(r2 >> 11) * 0x1.0p-53;
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925 * u2);
}

/* double -> fp32 -> (optionally) bf16, returned as fp32. */
static float to_storage(double v, int bf16)
{
    float f = (float)v;
    if (!bf16)
        return f;
    uint32_t b;
    memcpy(&b, &f, 4);
    uint32_t lsb = (b >> 16) & 1u;
    b = (b + 0x7FFFu + lsb) & 0xFFFF0000u;
    memcpy(&f, &b, 4);
    return f;
}

/*
 * out[idx] = transform(mean + sigma * z(idx)), idx in [0, n).
 * transform: 0 = identity, 1 = logistic sigmoid.
 */
void gspn_gen_normal(float *out, int64_t n, uint64_t seed, int tensor_id,
                     int slot, double mean, double sigma, int transform,
                     int bf16)
{
    uint64_t key = stream_key(seed, (uint64_t)tensor_id, (uint64_t)slot);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) {
        double v = mean + sigma * std_normal(key, (uint64_t)i);
        if (transform == 1)
            v = 1.0 / (1.0 + exp(-v));
        out[i] = to_storage(v, bf16);
    }
}

/*
 * Neighbour weights for one scan direction, layout [B][G][3][H][W].
 *
 * Per pixel and group, three logits ~ N(0, sigma^2) are drawn (counter index
 * ((b*G + g)*H*W + pixel)*3 + k).  Tap k names the neighbour at offset k-1
 * along the axis perpendicular to the scan: the column for vertical scans
 * (vertical != 0), the row for horizontal ones.  Taps whose neighbour lies
 * outside the grid get weight 0; the remaining ones get a softmax over their
 * logits (max subtracted, in double).
 */
void gspn_gen_taps(float *w, int B, int G, int H, int W, int vertical,
                   uint64_t seed, int tensor_id, int slot, double sigma,
                   int bf16)
{
    uint64_t key = stream_key(seed, (uint64_t)tensor_id, (uint64_t)slot);
    int64_t HW = (int64_t)H * W;
    int64_t units = (int64_t)B * G;
#pragma omp parallel for schedule(static)
    for (int64_t bg = 0; bg < units; ++bg) {
        for (int64_t p = 0; p < HW; ++p) {
            int row = (int)(p / W), col = (int)(p % W);
            int perp = vertical ? col : row;
            int plen = vertical ? W : H;
            double logit[3], e[3];
            int valid[3];
            double mx = -INFINITY;
            for (int k = 0; k < 3; ++k) {
                int nb = perp + k - 1;
                valid[k] = nb >= 0 && nb < plen;
                logit[k] = sigma * std_normal(key, (uint64_t)((bg * HW + p) * 3 + k));
                if (valid[k] && logit[k] > mx)
                    mx = logit[k];
            }
            double s = 0.0;
            for (int k = 0; k < 3; ++k) {
                e[k] = valid[k] ? exp(logit[k] - mx) : 0.0;
                s += e[k];
            }
            for (int k = 0; k < 3; ++k)
                w[(bg * 3 + k) * HW + p] = to_storage(e[k] / s, bf16);
        }
    }
}
