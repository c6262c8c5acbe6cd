// Device-side helpers shared by the libgspn kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gspn {

// Storage types: fp32 is stored as float, bf16 as its 16-bit pattern.
using bf16_t = uint16_t;

__device__ __forceinline__ float load_f(const float *p) { return *p; }
__device__ __forceinline__ float load_f(const bf16_t *p)
{
    // bf16 -> fp32 is exact: the pattern becomes the high half of the float.
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
}

__device__ __forceinline__ void store_f(float *p, float v) { *p = v; }
__device__ __forceinline__ void store_f(bf16_t *p, float v)
{
    // fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
    __bf16 b = static_cast<__bf16>(v);
    *p = __builtin_bit_cast(bf16_t, b);
}

// Sec. 3, Eq. (row_stochastic_norm) for one pixel: s_k = sigmoid(t_k) on the
// taps whose neighbour lies on the grid (on0, on2; tap 1 always), 0 on the
// others, and w_k = s_k / max(s_0 + s_1 + s_2, kNormEps).  The reciprocals
// are the hardware's (v_rcp_f32, within one fp32 ulp): a correctly rounded
// division takes about ten instructions, and every kernel that normalizes
// (the weights, their gradient, separately or inside a scan) calls these
// same functions, so all of them agree bit for bit.
constexpr float kNormEps = 1e-30f;

__device__ __forceinline__ float sigmoid(float t)
{
    return __builtin_amdgcn_rcpf(1.f + __expf(-t));
}

__device__ __forceinline__ void norm3(const float (&t)[3], bool on0, bool on2, float (&w)[3])
{
    const float s0 = on0 ? sigmoid(t[0]) : 0.f;
    const float s1 = sigmoid(t[1]);
    const float s2 = on2 ? sigmoid(t[2]) : 0.f;
    const float inv = __builtin_amdgcn_rcpf(fmaxf((s0 + s1) + s2, kNormEps));
    w[0] = s0 * inv;
    w[1] = s1 * inv;
    w[2] = s2 * inv;
}

// Gradient with respect to the logits t of one pixel, from the gradient g
// with respect to its weights: dt_m = s_m (1 - s_m) (g_m - sum_k w_k g_k) / S
// (the sum term drops where the clamp holds S at kNormEps); 0 on the taps
// off the grid.
__device__ __forceinline__ void norm3_bwd(const float (&t)[3], const float (&g)[3], bool on0,
                                          bool on2, float (&dt)[3])
{
    const float s[3] = {on0 ? sigmoid(t[0]) : 0.f, sigmoid(t[1]), on2 ? sigmoid(t[2]) : 0.f};
    const float sum = (s[0] + s[1]) + s[2];
    const bool clamped = sum < kNormEps;
    const float inv = __builtin_amdgcn_rcpf(clamped ? kNormEps : sum);
    const float inner = clamped ? 0.f : ((s[0] * inv) * g[0] + (s[1] * inv) * g[1]) + (s[2] * inv) * g[2];
    const bool on[3] = {on0, true, on2};
#pragma unroll
    for (int k = 0; k < 3; ++k)
        dt[k] = on[k] ? s[k] * (1.f - s[k]) * (g[k] - inner) * inv : 0.f;
}

// DPP lane shifts along a line of T lanes (T = 16, 32 or 64).  from_left(v)
// returns v of lane-1 and from_right(v) v of lane+1; lanes without a source
// read 0 (bound_ctrl).  For T = 16 the shift stays inside each 16-lane row,
// so every row is one line.  For T = 32 the whole-wave shift crosses from one
// 32-lane line into the next; callers zero the weights that would read across.
template <int T>
__device__ __forceinline__ float from_left(float v)
{
    constexpr int ctrl = (T == 16) ? 0x111 /* row_shr:1 */ : 0x138 /* wave_shr:1 */;
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, 0xf, 0xf, true));
}

template <int T>
__device__ __forceinline__ float from_right(float v)
{
    constexpr int ctrl = (T == 16) ? 0x101 /* row_shl:1 */ : 0x130 /* wave_shl:1 */;
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), ctrl, 0xf, 0xf, true));
}

// Per-direction planes (lam, u, w and their gradients) are blocked
// line-major: the lines a direction scans (storage rows for vertical
// directions, storage columns for horizontal ones) are grouped in blocks of
// 8 consecutive lines, and inside a block the 8 values of one line position
// are adjacent.  Offset of (line l, position p) in a plane of L lines of P
// positions; the last block holds L - 8*(L/8) lines when L is not a multiple
// of 8.
constexpr int kLineBlock = 8;

__host__ __device__ __forceinline__ int lm_offset(int l, int p, int L, int P)
{
    const int q = l >> 3;
    const int n = L - 8 * q < 8 ? L - 8 * q : 8;
    return 8 * P * q + n * p + (l & 7);
}

// Offset of (storage line l, line position p) in a per-direction plane of L
// lines of P positions, in either layout of the per-direction tensors:
// pixel-major (pm: the plane is the H x W image, row-major, a line being a
// row for vertical directions and a column for horizontal ones) or blocked
// line-major.  W: the image's row length.
__host__ __device__ __forceinline__ int dir_offset(bool pm, bool vert, int l, int p, int L, int P,
                                                   int W)
{
    return pm ? (vert ? l * W + p : p * W + l) : lm_offset(l, p, L, P);
}

// Direction index d (direction bit 1 << d), frame position (step i, line
// position j):
//   pixel offset  e0 + i * es  in an H x W plane whose rows are `pitch`
//                              elements apart (pitch = W in global memory,
//                              padded in LDS);
//   lm(i)                      offset in a per-direction plane (pixel-major
//                              or blocked line-major, see dir_offset).
struct Frame {
    int L;        // scan length
    int P;        // line length
    int e0, es;   // pixel offset of (0, j), change per step
    int j;        // line position
    int W;        // image row length (pixel-major per-direction planes)
    bool rev;     // the scan visits storage lines in decreasing order
    bool vert;    // the lines are storage rows
    bool pm;      // per-direction planes are pixel-major
    __device__ __forceinline__ int line(int i) const { return rev ? L - 1 - i : i; }
    __device__ __forceinline__ int lm(int i) const { return dir_offset(pm, vert, line(i), j, L, P, W); }
    __device__ __forceinline__ int lm_at(int i, int jj) const
    {
        return dir_offset(pm, vert, line(i), jj, L, P, W);
    }
};

__device__ __forceinline__ Frame make_frame(int d, int j, int H, int W, int pitch, bool pm = false)
{
    Frame f;
    f.j = j;
    f.W = W;
    f.pm = pm;
    f.vert = d < 2;
    f.rev = d == 1 || d == 3;
    switch (d) {
    case 0:  f.L = H; f.P = W; f.e0 = j;                   f.es = pitch; break;  // T2B
    case 1:  f.L = H; f.P = W; f.e0 = (H - 1) * pitch + j; f.es = -pitch; break; // B2T
    case 2:  f.L = W; f.P = H; f.e0 = j * pitch;           f.es = 1;     break;  // L2R
    default: f.L = W; f.P = H; f.e0 = j * pitch + (W - 1); f.es = -1;    break;  // R2L
    }
    return f;
}

// Division of a non-negative int below 2^31 by a fixed divisor d as a
// multiply-high and shift (Granlund and Montgomery, "Division by invariant
// integers using multiplication", 1994): with s = ceil(log2 d) and
// m = ceil(2^(31+s) / d), n / d = (n * m) >> (31 + s).  Built on the host;
// on the device a uniform n divides in scalar instructions, where a plain
// division would be expanded on the vector unit.
struct Magic {
    uint32_t m, s;
};

inline Magic make_magic(uint32_t d)
{
    uint32_t l = 0;
    while ((1ull << l) < d)
        ++l;
    const uint64_t num = 1ull << (31 + l);
    return Magic{static_cast<uint32_t>((num + d - 1) / d), l};
}

__device__ __forceinline__ int mdiv(int n, Magic q)
{
    return static_cast<int>(
        static_cast<uint32_t>((static_cast<uint64_t>(static_cast<uint32_t>(n)) * q.m) >> (31 + q.s)));
}

__device__ __forceinline__ int scan_len(int d, int H, int W) { return d < 2 ? H : W; }
__device__ __forceinline__ int line_len(int d, int H, int W) { return d < 2 ? W : H; }

// Slot of direction bit `bit` in the stacked per-direction tensors.
__device__ __forceinline__ int dir_slot(int mask, int bit) { return __popc(mask & (bit - 1)); }

}  // namespace gspn
