// Forward line scans for bf16 planes whose lines are longer than a wave
// (sides up to 256, multiples of 8), with per-direction tensors in the
// blocked line-major layout.
//
// One workgroup per channel plane, one wave per direction (Sec. 3,
// Eqs. (gspn_recurrence), (gspn_output)):
//  * the x plane is loaded once, coalesced, into LDS (132 KB at 256 x 256);
//  * lane l of a wave owns the line positions l + 64 m (m < NPL); the line
//    state stays in NPL VGPRs for the whole scan; the tridiagonal step takes
//    neighbours from the adjacent lanes by DPP wave shifts, and across the
//    boundary between position groups (lane 0 and lane 63) by DPP wave
//    rotates;
//  * lam, u and w come in 8-line blocks of 16-byte coalesced loads, one
//    block ahead of use.
// A 256 x 256 fp32 merge plane does not fit in LDS, so each direction writes
// u_d * h_d to an fp32 plane in its own line-major order (whole lines per
// store) and a tiled kernel sums the directions in direction-bit order,
// transposing the horizontal ones through LDS, and stores y once.  The scan
// and the sum alternate in rounds of planes, so that the sum finds much of
// its round's planes still in the Infinity Cache (wide_round).
//
// Pixel-major per-direction tensors are first copied into the blocked order
// of their direction in the caller's workspace (pieces_kernel: whole rows in
// through LDS, whole 8-line blocks out), and the scan then runs as on blocked
// tensors.  Read in place, a vertical scan would take 2 bytes of a row per
// lane and load (8 loads per 16-byte piece, 40 per block of 8 lines and
// position group), a horizontal one 16 bytes from each of 64 rows; the copy
// costs one read and one write of lam, u and w at full bandwidth instead.
//
// With few channel planes the same direction pass runs on chunks of the scan
// (fwd_wide_chunk_kernel, wide_carry_kernel): end states from zero, carries
// through w alone, then every chunk again from its carry; wide_chunks picks
// the chunk count from the shape.
#include <algorithm>

#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;

constexpr int kMaxNpl = 4;   // positions per lane: lines of up to 256 positions
constexpr int kTile = 64;    // tile side of the direction sum

// bf16 x plane in LDS, rows of an odd number of dwords: a row walk (lanes on
// consecutive columns) and a column walk (lanes on consecutive rows) are both
// free of bank conflicts.
__host__ __device__ inline int wide_pitch_dw(int W) { return (W / 2) | 1; }

template <int NPL>
struct Pieces {
    uint4 l[NPL], u[NPL], w0[NPL], w1[NPL], w2[NPL];
};

// The neighbours of h[m] on the line, over all NPL position groups: lanes
// take lane-1 / lane+1 of their own group by a DPP wave shift; lane 0 and
// lane 63 take the last / first lane of the adjacent group, which a DPP wave
// rotate of that group's value brings to them and the shift leaves in place
// (a shift writes nothing where it has no source).  The line ends read 0.
template <int NPL>
__device__ __forceinline__ void neighbours(const float (&h)[NPL], float (&left)[NPL],
                                           float (&right)[NPL])
{
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
        const int hv = __float_as_int(h[m]);
        if (m == 0) {
            left[m] = from_left<64>(h[m]);
        } else {
            const int rot =
                __builtin_amdgcn_mov_dpp(__float_as_int(h[m - 1]), 0x13C /* wave_ror:1 */, 0xf, 0xf, false);
            left[m] = __int_as_float(
                __builtin_amdgcn_update_dpp(rot, hv, 0x138 /* wave_shr:1 */, 0xf, 0xf, false));
        }
        if (m + 1 == NPL) {
            right[m] = from_right<64>(h[m]);
        } else {
            const int rot =
                __builtin_amdgcn_mov_dpp(__float_as_int(h[m + 1]), 0x134 /* wave_rol:1 */, 0xf, 0xf, false);
            right[m] = __int_as_float(
                __builtin_amdgcn_update_dpp(rot, hv, 0x130 /* wave_shl:1 */, 0xf, 0xf, false));
        }
    }
}

// What a pass over a range of line blocks does (Sec. 3 recurrence; the chunk
// split follows the block lower-triangular form of Eq. (global)):
//   kStore  the recurrence, u * h written to the direction's fp32 plane;
//   kEnd    the recurrence, nothing written: the caller keeps the end state;
//   kHomog  the recurrence without the injection lam * x (only w is read):
//           it carries a state across the blocks, h -> Phi h.
enum PassMode { kStore, kEnd, kHomog };

// One direction of one channel plane over the scan's line blocks fb0 .. fb1-1
// (blocks of 8 lines in scan order), starting from state h (0 before the
// first line) and leaving the state after the last one in h.  HC, WC: the
// plane's sides when they are compile-time constants (0: taken from H, W at
// run time); L, P: scan and line length; the x plane sits in LDS with pitch
// (W / 2) | 1 dwords; ys receives u * h as fp32 in the direction's
// line-major order (line l, position p at l * P + p).
template <int NPL, bool VERT, bool REV, int HC, int WC, int MODE>
__device__ __forceinline__ void wide_dir(int lane, int H_, int W_, rsrc_t lam, rsrc_t u, rsrc_t w,
                                         const uint8_t *xs, u32x4 ys, int fb0, int fb1,
                                         float (&h)[NPL])
{
    const int H = HC ? HC : H_, W = WC ? WC : W_;
    const int L = VERT ? H : W, P = VERT ? W : H;
    const int pdw = wide_pitch_dw(W);
    const uint32_t wplane = (uint32_t)(2 * H * W);
    Sel s[NPL];
    int jc[NPL];
    bool valid[NPL];
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
        const int p = lane + 64 * m;
        valid[m] = p < P;
        s[m] = make_sel(p, P);
        jc[m] = p < P ? p : P - 1;
    }
    const int NB = L / 8;
    auto load = [&](Pieces<NPL> &pc, int fb) {
        const int sq = REV ? NB - 1 - fb : fb;   // storage block of frame block fb
#pragma unroll
        for (int m = 0; m < NPL; ++m) {
            if (MODE != kHomog)
                pc.l[m] = ld_piece<false, VERT, true>(lam, jc[m], sq, P, W);
            if (MODE == kStore)
                pc.u[m] = ld_piece<false, VERT, true>(u, jc[m], sq, P, W);
            pc.w0[m] = ld_piece<false, VERT, false>(w, jc[m], sq, P, W);
            pc.w1[m] = ld_piece<false, VERT, false>(w, jc[m], sq, P, W, wplane);
            pc.w2[m] = ld_piece<false, VERT, false>(w, jc[m], sq, P, W, 2u * wplane);
        }
    };

    auto run_block = [&](const Pieces<NPL> &pc, int fb) {
        // this lane's x at the block's lowest storage line: each step adds a
        // small constant, which the LDS read takes as its offset
        const int l0 = REV ? L - 8 - 8 * fb : 8 * fb;
        uint32_t xb[NPL];
#pragma unroll
        for (int m = 0; m < NPL; ++m)
            xb[m] = VERT ? 4u * (uint32_t)(l0 * pdw) + 2u * (uint32_t)jc[m]
                         : 4u * (uint32_t)(jc[m] * pdw) + 2u * (uint32_t)l0;
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const int e = REV ? 7 - t : t;              // element of the 8-line piece
            const int ln = REV ? L - 1 - i : i;         // storage line of step i
            const uint32_t dx = VERT ? 4u * (uint32_t)(pdw * e) : 2u * (uint32_t)e;   // ln - l0 = e
            float left[NPL], right[NPL];
            neighbours<NPL>(h, left, right);
#pragma unroll
            for (int m = 0; m < NPL; ++m) {
                float hn = 0.f;
                if (MODE != kHomog) {
                    const float xv = bf_lo(lds_u16(xs, xb[m] + dx));
                    hn = elem(pc.l[m], e, s[m].lo1, s[m].hi1) * xv;
                }
                if (i > 0) {
                    hn = fmaf(elem(pc.w1[m], e, s[m].lo1, s[m].hi1), h[m], hn);
                    hn = fmaf(elem(pc.w0[m], e, s[m].lo0, s[m].hi0), left[m], hn);
                    hn = fmaf(elem(pc.w2[m], e, s[m].lo2, s[m].hi2), right[m], hn);
                }
                h[m] = hn;
            }
            if (MODE == kStore) {
#pragma unroll
                for (int m = 0; m < NPL; ++m) {
                    // the lane's part in the address register, the line's in soffset
                    if (valid[m])
                        st32_nt(ys, 4u * (uint32_t)lane, 4u * (uint32_t)(ln * P + 64 * m),
                                __float_as_uint(elem(pc.u[m], e) * h[m]));
                }
            }
        }
        step_fence();
    };

    Pieces<NPL> A, B;
    load(A, fb0);
#pragma unroll 1
    for (int fb = fb0; fb < fb1; fb += 2) {
        if (fb + 1 < fb1)
            load(B, fb + 1);
        run_block(A, fb);
        if (fb + 1 < fb1) {
            if (fb + 2 < fb1)
                load(A, fb + 2);
            run_block(B, fb + 1);
        }
    }
}

template <int AUX>
__device__ __forceinline__ uint2 ld64(rsrc_t r, uint32_t voff, uint32_t soff)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, AUX);
    return make_uint2(v[0], v[1]);
}

// 8 rows of the five streams of a vertical direction, 4 adjacent columns each.
struct VRows {
    uint2 l[8], u[8], w0[8], w1[8], w2[8];
};

// A vertical direction of pixel-major planes (no copy into the blocked
// order), lane l owning the 4 adjacent columns 4l .. 4l+3 of the row (W up
// to 256): a step reads 8 bytes per lane of a row of lambda, u and each tap
// plane (whole rows across the wave), takes the neighbours beyond the lane's
// 4 columns from lanes l-1 and l+1 by DPP wave shifts, and writes u * h as
// 16 bytes of the direction's fp32 row.  The same operations in the same
// order as wide_dir, so the same bits.  Rows come 8 at a time, one block
// ahead of use.
template <bool REV, int HC, int WC>
__device__ __forceinline__ void wide_vert_pm(int lane, int H_, int W_, rsrc_t lam, rsrc_t u,
                                             rsrc_t w, const uint8_t *xs, u32x4 ys)
{
    const int H = HC ? HC : H_, W = WC ? WC : W_;
    const int pdw = wide_pitch_dw(W);
    const uint32_t wplane = (uint32_t)(2 * H * W);
    const int c0 = 4 * lane;
    const bool act = c0 < W;                         // W is a multiple of 8
    // idle lanes read column 0 with every weight and lambda selected to 0:
    // their h stays 0, which is what the last active lane's right neighbour
    // needs (its tap 2 is ignored anyway)
    const uint32_t voff = act ? 2u * (uint32_t)c0 : 0u;
    const uint32_t slo = act ? kSelLo : kSelZero, shi = act ? kSelHi : kSelZero;
    const uint32_t s0lo = (act && c0 > 0) ? kSelLo : kSelZero;          // tap 0, column c0
    const uint32_t s2hi = (act && c0 + 4 < W) ? kSelHi : kSelZero;      // tap 2, column c0+3
    const uint32_t xoff = act ? 2u * (uint32_t)c0 : 0u;
    auto load = [&](VRows &r, int fb) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const uint32_t ro = 2u * (uint32_t)((REV ? H - 1 - i : i) * W);
            r.l[t] = ld64<2 /* nt */>(lam, voff, ro);
            r.u[t] = ld64<2>(u, voff, ro);
            r.w0[t] = ld64<0>(w, voff, ro);
            r.w1[t] = ld64<0>(w, voff, ro + wplane);
            r.w2[t] = ld64<0>(w, voff, ro + 2u * wplane);
        }
    };
    float h[4] = {0.f, 0.f, 0.f, 0.f};
    auto run = [&](const VRows &r, int fb) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const int ln = REV ? H - 1 - i : i;
            const uint32_t xa = 4u * (uint32_t)(ln * pdw) + xoff;
            const uint32_t xw0 = lds_u32(xs, xa), xw1 = lds_u32(xs, xa + 4);
            const float xv[4] = {bf_lo(xw0), bf_hi(xw0), bf_lo(xw1), bf_hi(xw1)};
            const float lv[4] = {widen(r.l[t].x, slo), widen(r.l[t].x, shi), widen(r.l[t].y, slo),
                                 widen(r.l[t].y, shi)};
            const float left = from_left<64>(h[3]), right = from_right<64>(h[0]);
            float hn[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                hn[e] = lv[e] * xv[e];
            if (i > 0) {
                const float w1v[4] = {widen(r.w1[t].x, slo), widen(r.w1[t].x, shi),
                                      widen(r.w1[t].y, slo), widen(r.w1[t].y, shi)};
                const float w0v[4] = {widen(r.w0[t].x, s0lo), widen(r.w0[t].x, shi),
                                      widen(r.w0[t].y, slo), widen(r.w0[t].y, shi)};
                const float w2v[4] = {widen(r.w2[t].x, slo), widen(r.w2[t].x, shi),
                                      widen(r.w2[t].y, slo), widen(r.w2[t].y, s2hi)};
                const float lf[4] = {left, h[0], h[1], h[2]};
                const float rt[4] = {h[1], h[2], h[3], right};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    hn[e] = fmaf(w1v[e], h[e], hn[e]);
                    hn[e] = fmaf(w0v[e], lf[e], hn[e]);
                    hn[e] = fmaf(w2v[e], rt[e], hn[e]);
                }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e)
                h[e] = hn[e];
            if (act) {
                const uint2 uu = r.u[t];
                st128_nt(ys, 4u * (uint32_t)c0, 4u * (uint32_t)(ln * W),
                         make_uint4(__float_as_uint(bf_lo(uu.x) * h[0]),
                                    __float_as_uint(bf_hi(uu.x) * h[1]),
                                    __float_as_uint(bf_lo(uu.y) * h[2]),
                                    __float_as_uint(bf_hi(uu.y) * h[3])));
            }
        }
        step_fence();
    };
    const int NB = H / 8;
    VRows A, B;
    load(A, 0);
#pragma unroll 1
    for (int fb = 0; fb < NB; fb += 2) {
        if (fb + 1 < NB)
            load(B, fb + 1);
        run(A, fb);
        if (fb + 1 < NB) {
            if (fb + 2 < NB)
                load(A, fb + 2);
            run(B, fb + 1);
        }
    }
}

// Direction d's pass over blocks fb0 .. fb1-1 (direction-uniform dispatch).
template <int NPL, int HC, int WC, int MODE>
__device__ __forceinline__ void wide_pass(int d, int lane, int H, int W, rsrc_t rl, rsrc_t ru,
                                          rsrc_t rw, const uint8_t *xs, u32x4 yd, int fb0,
                                          int fb1, float (&h)[NPL])
{
    if (d == 0)
        wide_dir<NPL, true, false, HC, WC, MODE>(lane, H, W, rl, ru, rw, xs, yd, fb0, fb1, h);
    else if (d == 1)
        wide_dir<NPL, true, true, HC, WC, MODE>(lane, H, W, rl, ru, rw, xs, yd, fb0, fb1, h);
    else if (d == 2)
        wide_dir<NPL, false, false, HC, WC, MODE>(lane, H, W, rl, ru, rw, xs, yd, fb0, fb1, h);
    else
        wide_dir<NPL, false, true, HC, WC, MODE>(lane, H, W, rl, ru, rw, xs, yd, fb0, fb1, h);
}

// x plane of channel plane pc -> LDS: coalesced 16-byte pieces into padded rows.
template <int WC>
__device__ __forceinline__ void stage_x_plane(const bf16_t *x, int64_t pc, int H, int W,
                                              Magic divNq, uint32_t *xs32)
{
    const int64_t HW = (int64_t)H * W;
    const int pdw = wide_pitch_dw(W);
    const rsrc_t xr = make_rsrc(x + pc, (uint32_t)(2 * HW));
    const int nq = W / 8;
    const int n = H * nq;
    for (int t = threadIdx.x; t < n; t += 256) {
        const uint4 v = ld128(xr, 16u * (uint32_t)t, 0);
        const int r = WC ? t / (WC / 8) : mdiv(t, divNq), q = t - r * nq;
        uint32_t *dst = xs32 + r * pdw + 4 * q;
        dst[0] = v.x;
        dst[1] = v.y;
        dst[2] = v.z;
        dst[3] = v.w;
    }
}

// VPM: the call is pixel-major and lam, u, w hold blocked copies of the
// horizontal directions only ([nh][B][C][plane], [nh][B][G][3][plane]); the
// vertical ones are read in place from lam_v, u_v, w_v (the call's tensors).
template <int NPL, int HC, int WC, bool VPM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void fwd_wide_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, float *__restrict__ ys, int mask, int B, int C, int G, int H_,
    int W_, Magic divC, Magic divCpg, Magic divNq, int plane0, const bf16_t *__restrict__ lam_v,
    const bf16_t *__restrict__ u_v, const bf16_t *__restrict__ w_v)
{
    const int H = HC ? HC : H_, W = WC ? WC : W_;
    extern __shared__ uint32_t xs32[];
    uint8_t *xs = reinterpret_cast<uint8_t *>(xs32);
    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = plane0 + xcd_remap(blockIdx.x, gridDim.x);
    const int b = mdiv(blk, divC);
    const int c = blk - b * C;
    const int g = mdiv(c, divCpg);
    const int64_t HW = (int64_t)H * W;
    const int64_t pc = ((int64_t)b * C + c) * HW;

    stage_x_plane<WC>(x, pc, H, W, divNq, xs32);
    lds_barrier();

    if ((mask >> d) & 1) {
        const int s = __popc(mask & ((1 << d) - 1));
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const u32x4 yd = make_sdesc(ys + pd, (uint32_t)(4 * HW));
        if (VPM && d < 2) {
            const int64_t pw = (((int64_t)s * B + b) * G + g) * 3 * HW;
            const rsrc_t rl = make_rsrc(lam_v + pd, (uint32_t)(2 * HW));
            const rsrc_t ru = make_rsrc(u_v + pd, (uint32_t)(2 * HW));
            const rsrc_t rw = make_rsrc(w_v + pw, (uint32_t)(6 * HW));
            if (d == 0)
                wide_vert_pm<false, HC, WC>(lane, H, W, rl, ru, rw, xs, yd);
            else
                wide_vert_pm<true, HC, WC>(lane, H, W, rl, ru, rw, xs, yd);
        } else {
            const int sc = VPM ? s - __popc(mask & 3) : s;   // slot among the copies
            const int64_t pdc = (((int64_t)sc * B + b) * C + c) * HW;
            const int64_t pw = (((int64_t)sc * B + b) * G + g) * 3 * HW;
            const rsrc_t rl = make_rsrc(lam + pdc, (uint32_t)(2 * HW));
            const rsrc_t ru = make_rsrc(u + pdc, (uint32_t)(2 * HW));
            const rsrc_t rw = make_rsrc(w + pw, (uint32_t)(6 * HW));
            float h[NPL];
#pragma unroll
            for (int m = 0; m < NPL; ++m)
                h[m] = 0.f;
            const int NB = (d < 2 ? H : W) / 8;
            wide_pass<NPL, HC, WC, kStore>(d, lane, H, W, rl, ru, rw, xs, yd, 0, NB, h);
        }
    }
}

// Scan-axis chunks, for when few channel planes leave most CUs idle under the
// single-pass kernel: every direction's scan is cut into K chunks of whole
// line blocks.  By the block lower-triangular form of Eq. (global) the state
// after chunk k from carry c is Phi_k c + e_k, with e_k the chunk's end state
// from a zero carry and Phi_k the chunk's product of tridiagonal steps.
//  1. fwd_wide_chunk_kernel<kEnd>: every (plane, chunk) -- e_k, stored;
//  2. wide_carry_kernel: per plane, c_1 = e_0, c_{k+1} = Phi_k c_k + e_k, the
//     Phi_k c_k by the recurrence without injection (w only);
//  3. fwd_wide_chunk_kernel<kStore>: every (plane, chunk) from its carry,
//     u * h to the fp32 direction planes; then sum_wide_kernel as usual.
// States are fp32 [plane][direction slot][chunk][max(H, W)], the first P
// (the direction's line length) of each slot used.
template <int NPL, int HC, int WC, int MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void fwd_wide_chunk_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, float *__restrict__ ys, float *__restrict__ st, int mask, int B,
    int C, int G, int H_, int W_, int K, Magic divC, Magic divCpg, Magic divNq, Magic divK)
{
    const int H = HC ? HC : H_, W = WC ? WC : W_;
    extern __shared__ uint32_t xs32[];
    uint8_t *xs = reinterpret_cast<uint8_t *>(xs32);
    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int plane = mdiv(blk, divK);                                 // b * C + c
    const int k = blk - plane * K;                                     // chunk, in scan order
    const int b = mdiv(plane, divC);
    const int c = plane - b * C;
    const int g = mdiv(c, divCpg);
    const int64_t HW = (int64_t)H * W;
    const int64_t pc = ((int64_t)b * C + c) * HW;
    const int D = __popc(mask);
    const int P = d < 2 ? W : H, NBc = (d < 2 ? H : W) / 8 / K;

    stage_x_plane<WC>(x, pc, H, W, divNq, xs32);
    lds_barrier();

    if ((mask >> d) & 1) {
        const int s = __popc(mask & ((1 << d) - 1));
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const int64_t pw = (((int64_t)s * B + b) * G + g) * 3 * HW;
        const rsrc_t rl = make_rsrc(lam + pd, (uint32_t)(2 * HW));
        const rsrc_t ru = make_rsrc(u + pd, (uint32_t)(2 * HW));
        const rsrc_t rw = make_rsrc(w + pw, (uint32_t)(6 * HW));
        const u32x4 yd = make_sdesc(ys + pd, (uint32_t)(4 * HW));
        // this direction's states: chunk k's slot (every slot max(H, W) long)
        float *sk = st + (((int64_t)plane * D + s) * K + k) * (H > W ? H : W);
        float h[NPL];
#pragma unroll
        for (int m = 0; m < NPL; ++m) {
            const int p = lane + 64 * m;
            h[m] = (MODE == kStore && k > 0 && p < P) ? sk[p] : 0.f;
        }
        wide_pass<NPL, HC, WC, MODE>(d, lane, H, W, rl, ru, rw, xs, yd, k * NBc,
                                          (k + 1) * NBc, h);
        if (MODE == kEnd) {
#pragma unroll
            for (int m = 0; m < NPL; ++m) {
                const int p = lane + 64 * m;
                if (p < P)
                    sk[p] = h[m];
            }
        }
    }
}

// The carries: for each plane and direction, c_{k+1} = Phi_k c_k + e_k,
// written over e_{k+1}'s slot neighbour: the state array holds e_k after
// the first pass and c_k (k >= 1; slot 0 unused) after this one.
template <int NPL, int HC, int WC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void wide_carry_kernel(
    const bf16_t *__restrict__ w, float *__restrict__ st, int mask, int B, int C, int G, int H_,
    int W_, int K, Magic divC, Magic divCpg)
{
    const int H = HC ? HC : H_, W = WC ? WC : W_;
    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int plane = xcd_remap(blockIdx.x, gridDim.x);
    const int b = mdiv(plane, divC);
    const int c = plane - b * C;
    const int g = mdiv(c, divCpg);
    const int64_t HW = (int64_t)H * W;
    const int D = __popc(mask);
    if (!((mask >> d) & 1))
        return;
    const int s = __popc(mask & ((1 << d) - 1));
    const int64_t pw = (((int64_t)s * B + b) * G + g) * 3 * HW;
    const rsrc_t rw = make_rsrc(w + pw, (uint32_t)(6 * HW));
    const int P = d < 2 ? W : H, NBc = (d < 2 ? H : W) / 8 / K;
    const int SL = H > W ? H : W;   // every slot is max(H, W) long
    float *sp = st + ((int64_t)plane * D + s) * K * SL;
    float h[NPL], e[NPL];
    // c_1 = e_0
#pragma unroll
    for (int m = 0; m < NPL; ++m) {
        const int p = lane + 64 * m;
        h[m] = p < P ? sp[p] : 0.f;
    }
    for (int k = 1; k < K; ++k) {
        // e_k is read before c_k takes its slot
#pragma unroll
        for (int m = 0; m < NPL; ++m) {
            const int p = lane + 64 * m;
            e[m] = p < P ? sp[(int64_t)k * SL + p] : 0.f;
            if (p < P)
                sp[(int64_t)k * SL + p] = h[m];
        }
        if (k + 1 < K) {
            wide_pass<NPL, HC, WC, kHomog>(d, lane, H, W, rw, rw, rw, nullptr, u32x4{},
                                                k * NBc, (k + 1) * NBc, h);
#pragma unroll
            for (int m = 0; m < NPL; ++m)
                h[m] += e[m];
        }
    }
}

// y = sum over the directions, in direction-bit order, of the fp32 planes
// written by fwd_wide_kernel.  One workgroup per 64 x 64 tile of one channel
// plane.  Thread (wave v, lane l) owns columns 4 (l % 16) .. +3 of rows
// 16 k + 4 v + l / 16 (k < 4): each global access of a wave reads 16 bytes
// per lane, four 256-byte row segments.  Vertical planes are read in place;
// horizontal ones are stored transposed ([column][row]) and turned around
// through LDS (pitch 65: the transposed reads are conflict-free).
__global__ __launch_bounds__(256) void sum_wide_kernel(const float *__restrict__ ys,
                                                       bf16_t *__restrict__ y, int mask, int B,
                                                       int C, int H, int W, int tiles_w,
                                                       int tiles_hw, Magic divTilesW,
                                                       Magic divTilesHW, Magic divC, int plane0)
{
    __shared__ float T[kTile][kTile + 1];
    const int64_t HW = (int64_t)H * W;
    const int pl = mdiv((int)blockIdx.x, divTilesHW);
    const int local = (int)blockIdx.x - pl * tiles_hw;
    const int plane = plane0 + pl;                                     // b * C + c
    const int tr = mdiv(local, divTilesW);
    const int tc = local - tr * tiles_w;
    const int R0 = tr * kTile, C0 = tc * kTile;
    const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int l = threadIdx.x & 63;
    const int b = mdiv(plane, divC);
    const int c = plane - b * C;
    const int c4 = 4 * (l & 15);                    // first of this lane's 4 columns
    const int r1 = 4 * v + (l >> 4);                // row within a 16-row band
    float acc[4][4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            acc[k][e] = 0.f;
    int s = 0;
    for (int d = 0; d < 4; ++d) {
        if (!((mask >> d) & 1))
            continue;
        const float *src = ys + (((int64_t)s * B + b) * C + c) * HW;
        if (d < 2) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int row = R0 + 16 * k + r1, col = C0 + c4;
                if (row < H && col < W) {   // W is a multiple of 8: 4 columns in or out
                    const float4 q = *reinterpret_cast<const float4 *>(src + (int64_t)row * W + col);
                    acc[k][0] += q.x;
                    acc[k][1] += q.y;
                    acc[k][2] += q.z;
                    acc[k][3] += q.w;
                }
            }
        } else {
            // transposed plane: line (column) C0 + 16 k + r1, positions R0 + c4 .. +3
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int tcol = C0 + 16 * k + r1, trow = R0 + c4;
                float4 q = make_float4(0.f, 0.f, 0.f, 0.f);
                if (tcol < W && trow < H)   // H is a multiple of 8
                    q = *reinterpret_cast<const float4 *>(src + (int64_t)tcol * H + trow);
                float *t = &T[16 * k + r1][c4];
                t[0] = q.x;
                t[1] = q.y;
                t[2] = q.z;
                t[3] = q.w;
            }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    acc[k][e] += T[c4 + e][16 * k + r1];
            __syncthreads();
        }
        ++s;
    }
    bf16_t *dst = y + ((int64_t)b * C + c) * HW;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int row = R0 + 16 * k + r1, col = C0 + c4;
        if (row < H && col < W)
            gst64(reinterpret_cast<uint2 *>(dst + (int64_t)row * W + col),
                  pack2(acc[k][0], acc[k][1]), pack2(acc[k][2], acc[k][3]));
    }
}

// v: with the vertical directions read in place, the call's pixel-major
// tensors (p then holds the horizontal directions' blocked copies).
template <int NPL, int HC, int WC, bool VPM>
hipError_t fwd_wide_t(const Problem &p, hipStream_t st, float *ys, size_t lds, int plane0,
                      int nplanes, const Problem *v)
{
    hipError_t e = hipFuncSetAttribute((const void *)fwd_wide_kernel<NPL, HC, WC, VPM>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((fwd_wide_kernel<NPL, HC, WC, VPM>), dim3((unsigned)nplanes), dim3(256),
                       lds, st, (const bf16_t *)p.x, (const bf16_t *)p.w, (const bf16_t *)p.lam,
                       (const bf16_t *)p.u, ys, p.mask, p.B, p.C, p.G, p.H, p.W,
                       make_magic((uint32_t)p.C), make_magic((uint32_t)(p.C / p.G)),
                       make_magic((uint32_t)(p.W / 8)), plane0,
                       (const bf16_t *)(v ? v->lam : nullptr), (const bf16_t *)(v ? v->u : nullptr),
                       (const bf16_t *)(v ? v->w : nullptr));
    return hipGetLastError();
}

// The three launches of the chunked forward (see fwd_wide_chunk_kernel).
template <int NPL, int HC, int WC>
hipError_t fwd_wide_chunked_t(const Problem &p, hipStream_t st, float *ys, float *states,
                              size_t lds, int K)
{
    hipError_t e = hipFuncSetAttribute((const void *)fwd_wide_chunk_kernel<NPL, HC, WC, kEnd>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess)
        e = hipFuncSetAttribute((const void *)fwd_wide_chunk_kernel<NPL, HC, WC, kStore>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    const Magic divC = make_magic((uint32_t)p.C), divCpg = make_magic((uint32_t)(p.C / p.G));
    const Magic divNq = make_magic((uint32_t)(p.W / 8)), divK = make_magic((uint32_t)K);
    const unsigned planes = (unsigned)(p.B * p.C);
    const bf16_t *x = (const bf16_t *)p.x, *w = (const bf16_t *)p.w;
    const bf16_t *lam = (const bf16_t *)p.lam, *u = (const bf16_t *)p.u;
    hipLaunchKernelGGL((fwd_wide_chunk_kernel<NPL, HC, WC, kEnd>), dim3(planes * K), dim3(256),
                       lds, st, x, w, lam, u, ys, states, p.mask, p.B, p.C, p.G, p.H, p.W, K, divC,
                       divCpg, divNq, divK);
    hipLaunchKernelGGL((wide_carry_kernel<NPL, HC, WC>), dim3(planes), dim3(256), 0, st, w,
                       states, p.mask, p.B, p.C, p.G, p.H, p.W, K, divC, divCpg);
    hipLaunchKernelGGL((fwd_wide_chunk_kernel<NPL, HC, WC, kStore>), dim3(planes * K), dim3(256),
                       lds, st, x, w, lam, u, ys, states, p.mask, p.B, p.C, p.G, p.H, p.W, K, divC,
                       divCpg, divNq, divK);
    return hipGetLastError();
}

// The direction sum of planes plane0 .. plane0 + nplanes - 1.
hipError_t launch_sum_wide(const Problem &p, const float *ys, hipStream_t st, int plane0,
                           int nplanes)
{
    const int tiles_w = (p.W + kTile - 1) / kTile;
    const int tiles_h = (p.H + kTile - 1) / kTile;
    const int64_t nblk = (int64_t)nplanes * tiles_w * tiles_h;
    hipLaunchKernelGGL(sum_wide_kernel, dim3((unsigned)nblk), dim3(256), 0, st, ys,
                       (bf16_t *)p.y, p.mask, p.B, p.C, p.H, p.W, tiles_w, tiles_w * tiles_h,
                       make_magic((uint32_t)tiles_w), make_magic((uint32_t)(tiles_w * tiles_h)),
                       make_magic((uint32_t)p.C), plane0);
    return hipGetLastError();
}

size_t wide_lds_bytes(int H, int W) { return (size_t)H * 4 * wide_pitch_dw(W); }

// Pixel-major planes -> blocked line-major.  A row of an H x W plane is nq =
// W / 8 pieces of 16 bytes (piece q: columns 8q..8q+7).  One workgroup per
// band of 32 rows of one plane copies the band's rows into LDS with direct
// 16-byte loads (no registers; rows of nq | 1 pieces, the padding slots
// skipped), then writes the band's part of the blocked plane:
//  * vertical direction (lines are rows, positions columns): piece (q, p) of
//    the output, at q * W + p, holds column p of rows 8q..8q+7, gathered from
//    8 LDS rows (lanes on consecutive columns: no bank conflict);
//  * horizontal direction (lines are columns, positions rows): piece (q, p),
//    at q * H + p, is input piece q of row p, a transpose of 16-byte pieces
//    (a wave reads one piece column; with an odd pitch 16 consecutive lanes
//    hit distinct banks).
// Consecutive lanes write consecutive output pieces.
constexpr int kBand = 32;
constexpr int kBandSlots = kBand * ((64 * kMaxNpl / 8) | 1);   // LDS pieces (W <= 256)

typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glb_void;

__global__ __launch_bounds__(256) void pieces_kernel(const uint4 *__restrict__ src,
                                                     uint4 *__restrict__ dst, int H, int W,
                                                     int bands, int vert, Magic divBands,
                                                     Magic divPitch, Magic divW)
{
    __shared__ uint4 T[kBandSlots];
    const int nq = W / 8, pitch = nq | 1;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int bid = xcd_remap(blockIdx.x, gridDim.x);
    const int pl = mdiv(bid, divBands);
    const int r0 = (bid - pl * bands) * kBand;
    const int rows = H - r0 < kBand ? H - r0 : kBand;     // a multiple of 8
    const int64_t base = (int64_t)pl * H * nq;
    const uint4 *band = src + base + (int64_t)r0 * nq;
    // wave-instruction k fills LDS slots 64k .. 64k+63 (slot: row s / pitch,
    // piece s % pitch)
    const int nslots = rows * pitch;
    for (int k = wave; 64 * k < nslots; k += 4) {
        const int sl = 64 * k + lane;
        const int r = mdiv(sl, divPitch), q = sl - r * pitch;
        if (sl < nslots && q < nq)
            __builtin_amdgcn_global_load_lds((glb_void *)(band + r * nq + q),
                                             (lds_void *)(T + 64 * k), 16, 0, 0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (vert) {
        const uint16_t *T16 = reinterpret_cast<const uint16_t *>(T);
        for (int t = threadIdx.x; t < (rows / 8) * W; t += 256) {
            const int q = mdiv(t, divW), p = t - q * W;
            uint32_t e[8];
#pragma unroll
            for (int k = 0; k < 8; ++k)
                e[k] = T16[(8 * q + k) * (8 * pitch) + p];
            gst128(dst + base + (int64_t)(r0 / 8 + q) * W + p,
                   make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                              e[6] | (e[7] << 16)));
        }
    } else {
        for (int t = threadIdx.x; t < kBand * nq; t += 256) {
            const int q = t / kBand, r = t - q * kBand;
            if (r < rows)
                gst128(dst + base + (int64_t)q * H + r0 + r, T[r * pitch + q]);
        }
    }
}

// nv vertical planes, then nh horizontal ones, of H x W at src -> dst.
hipError_t launch_pieces(const void *src, void *dst, int64_t nv, int64_t nh, int H, int W,
                         hipStream_t st)
{
    const int bands = (H + kBand - 1) / kBand;
    const Magic divB = make_magic((uint32_t)bands), divP = make_magic((uint32_t)((W / 8) | 1));
    const Magic divW = make_magic((uint32_t)W);
    const int64_t HW = (int64_t)H * W;
    const uint4 *s = (const uint4 *)src;
    uint4 *d = (uint4 *)dst;
    if (nv > 0)
        hipLaunchKernelGGL(pieces_kernel, dim3((unsigned)(nv * bands)), dim3(256), 0, st, s, d, H,
                           W, bands, 1, divB, divP, divW);
    if (nh > 0)
        hipLaunchKernelGGL(pieces_kernel, dim3((unsigned)(nh * bands)), dim3(256), 0, st,
                           s + nv * HW / 8, d + nv * HW / 8, H, W, bands, 0, divB, divP, divW);
    return hipGetLastError();
}

// Workgroups of the single-pass forward that the device runs at once (LDS
// bound), 0 if the device cannot be queried (then neither chunks nor rounds).
int64_t wide_fit(size_t lds)
{
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    const int64_t per_cu =
        std::max<int64_t>(1, (int64_t)kLdsBytes / (int64_t)std::max<size_t>(lds, 1));
    return (int64_t)ncu * std::min<int64_t>(per_cu, 8);
}

// Chunks per scan for the chunked forward, or 1 for the single pass.  The
// chunked forward does more than twice the single pass's work (both passes
// over every line, and the carries), and its carry chain still takes every
// line block of a scan in turn, each step bound by issue latency at one wave
// per SIMD (about 380 cycles for the w-only step against about 890 for the
// full one at 256 positions).  It is chosen only where it measured faster:
// scans of at least 256 lines in both orientations, and at least 8 chunks,
// the count doubling while B*C*K workgroups still fit the device at once and
// every chunk keeps at least 2 line blocks.
int wide_chunks(const Problem &p, int64_t fit)
{
    if (fit == 0)
        return 1;
    const int64_t planes = (int64_t)p.B * p.C;
    const int nbh = p.H / 8, nbw = p.W / 8;
    int K = 1;
    while (K < 16 && planes * 2 * K <= fit && nbh % (2 * K) == 0 && nbw % (2 * K) == 0 &&
           nbh / (2 * K) >= 2 && nbw / (2 * K) >= 2)
        K *= 2;
    return (K >= 8 && nbh >= 32 && nbw >= 32) ? K : 1;
}

// The forward of planes plane0 .. plane0 + nplanes - 1 (single pass; the
// chunked forward takes every plane).
hipError_t fwd_wide_l(const Problem &p, hipStream_t st, float *ys, float *states, size_t lds, int K,
                      int plane0, int nplanes, const Problem *v = nullptr)
{
    const int side = p.H > p.W ? p.H : p.W;
    const int npl = (side + 63) / 64;
    // the square planes of 256 and 128 get kernels with their shape built in
    if (K > 1) {
        if (p.H == 256 && p.W == 256)
            return fwd_wide_chunked_t<4, 256, 256>(p, st, ys, states, lds, K);
        if (p.H == 128 && p.W == 128)
            return fwd_wide_chunked_t<2, 128, 128>(p, st, ys, states, lds, K);
        return npl <= 2 ? fwd_wide_chunked_t<2, 0, 0>(p, st, ys, states, lds, K)
               : npl == 3 ? fwd_wide_chunked_t<3, 0, 0>(p, st, ys, states, lds, K)
                          : fwd_wide_chunked_t<4, 0, 0>(p, st, ys, states, lds, K);
    }
    const int p0 = plane0, n = nplanes;
    if (v != nullptr) {
        if (p.H == 256 && p.W == 256)
            return fwd_wide_t<4, 256, 256, true>(p, st, ys, lds, p0, n, v);
        return npl <= 2 ? fwd_wide_t<2, 0, 0, true>(p, st, ys, lds, p0, n, v)
               : npl == 3 ? fwd_wide_t<3, 0, 0, true>(p, st, ys, lds, p0, n, v)
                          : fwd_wide_t<4, 0, 0, true>(p, st, ys, lds, p0, n, v);
    }
    if (p.H == 256 && p.W == 256)
        return fwd_wide_t<4, 256, 256, false>(p, st, ys, lds, p0, n, nullptr);
    if (p.H == 128 && p.W == 128)
        return fwd_wide_t<2, 128, 128, false>(p, st, ys, lds, p0, n, nullptr);
    return npl <= 2 ? fwd_wide_t<2, 0, 0, false>(p, st, ys, lds, p0, n, nullptr)
           : npl == 3 ? fwd_wide_t<3, 0, 0, false>(p, st, ys, lds, p0, n, nullptr)
                      : fwd_wide_t<4, 0, 0, false>(p, st, ys, lds, p0, n, nullptr);
}

// Planes per round of the single-pass forward.  Each round's direction sum
// runs right after its scan, while much of the round's fp32 direction planes
// is still in the 256 MB Infinity Cache: a round holds a whole number of
// device-fulls of planes (so that no round leaves CUs idle) whose planes fit
// that size.  Where one device-full does not fit, the rounds measured slower
// (their drains cost more than the cache saves: the latent grids of 147 and
// 185, 300 MB per device-full, 2% slower) and the forward runs as one pass.
// At 256 x 256, B = 1, C = 1024: rounds of 256 planes (1 MB each), the
// pixel-major forward 1064 -> 958 us, the blocked one 862 -> 721 us.
int wide_round(const Problem &p, int64_t fit)
{
    const int64_t planes = (int64_t)p.B * p.C;
    const int64_t bytes = (int64_t)__builtin_popcount(p.mask) * p.H * p.W * 4;
    const int64_t budget = (int64_t)256 << 20;
    if (fit == 0 || fit >= planes || fit * bytes > budget)
        return (int)planes;
    return (int)std::min(planes, fit * (budget / (fit * bytes)));
}

}  // namespace

hipError_t launch_planes_pieces(const void *src, void *dst, int64_t nv, int64_t nh, int H, int W,
                                hipStream_t st)
{
    return launch_pieces(src, dst, nv, nh, H, W, st);
}

bool wide_supported(const Problem &p)
{
    if (p.dtype != 1 || p.H % 8 != 0 || p.W % 8 != 0)
        return false;
    const int side = p.H > p.W ? p.H : p.W;
    if (side > 64 * kMaxNpl)
        return false;
    return wide_lds_bytes(p.H, p.W) <= (size_t)kLdsBytes;
}

hipError_t launch_fwd_wide(const Problem &p, hipStream_t st)
{
    const int D = __builtin_popcount(p.mask);
    const int64_t n = (int64_t)p.B * p.C * p.H * p.W;
    const size_t lds = wide_lds_bytes(p.H, p.W);
    const int64_t fit = wide_fit(lds);     // one device query per call
    const int K = wide_chunks(p, fit);
    // fp32 direction planes, then (chunked) the chunk states
    const int64_t nst = K > 1 ? (int64_t)p.B * p.C * D * K * std::max(p.H, p.W) : 0;
    float *ys = nullptr;
    hipError_t e = p.ws->take((void **)&ys, (size_t)(D * n + nst) * sizeof(float));
    if (e != hipSuccess)
        return e;
    const int planes = p.B * p.C;
    // the single pass in rounds of planes, each followed by its direction sum
    auto rounds = [&](const Problem &q, const Problem *v) -> hipError_t {
        const int R = wide_round(p, fit);
        hipError_t r = hipSuccess;
        for (int r0 = 0; r0 < planes && r == hipSuccess; r0 += R) {
            const int nr = std::min(R, planes - r0);
            r = fwd_wide_l(q, st, ys, nullptr, lds, 1, r0, nr, v);
            if (r == hipSuccess)
                r = launch_sum_wide(p, ys, st, r0, nr);
        }
        return r;
    };
    if (p.layout != kPixelMajor) {
        if (p.ws->counting)
            return hipSuccess;
        if (K == 1)
            return rounds(p, nullptr);
        e = fwd_wide_l(p, st, ys, ys + D * n, lds, K, 0, planes);
    } else {
        // Blocked copies (workspace) of lam, u and w, then the blocked scan.
        // The single pass reads the vertical directions in place (whole rows,
        // wide_vert_pm), so only the horizontal ones are copied; the chunked
        // passes take every direction from copies.
        const int nv = __builtin_popcount(p.mask & 3), nh = D - nv;
        const int nc = K > 1 ? D : nh;                    // directions copied
        const int64_t bc = (int64_t)p.B * p.C, bg3 = (int64_t)p.B * p.G * 3;
        const int64_t HW = (int64_t)p.H * p.W;
        void *cl = nullptr, *cu = nullptr, *cw = nullptr;
        if (nc > 0) {
            e = p.ws->take(&cl, (size_t)(nc * bc * HW) * 2);
            if (e == hipSuccess)
                e = p.ws->take(&cu, (size_t)(nc * bc * HW) * 2);
            if (e == hipSuccess)
                e = p.ws->take(&cw, (size_t)(nc * bg3 * HW) * 2);
        }
        if (e != hipSuccess || p.ws->counting)
            return e;
        const int cv = nc - nh;                           // vertical directions copied
        const int64_t skip = (int64_t)(nv - cv);          // vertical slots not copied
        if (nc > 0) {
            e = launch_pieces(static_cast<const bf16_t *>(p.lam) + skip * bc * HW, cl, cv * bc,
                              nh * bc, p.H, p.W, st);
            if (e == hipSuccess)
                e = launch_pieces(static_cast<const bf16_t *>(p.u) + skip * bc * HW, cu, cv * bc,
                                  nh * bc, p.H, p.W, st);
            if (e == hipSuccess)
                e = launch_pieces(static_cast<const bf16_t *>(p.w) + skip * bg3 * HW, cw,
                                  cv * bg3, nh * bg3, p.H, p.W, st);
            if (e != hipSuccess)
                return e;
        }
        Problem q = p;
        q.lam = cl;
        q.u = cu;
        q.w = cw;
        q.layout = kBlocked;
        if (K == 1)
            return rounds(q, &p);
        e = fwd_wide_l(q, st, ys, ys + D * n, lds, K, 0, planes);
    }
    if (e == hipSuccess)
        e = launch_sum_wide(p, ys, st, 0, planes);
    return e;
}

}  // namespace gspn
