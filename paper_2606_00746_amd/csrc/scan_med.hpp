#pragma once
// Line scans for bf16 square planes of a compile-time side (24 to 64, a
// multiple of 8), with
// per-direction tensors in blocked line-major layout (8-line blocks, the 8
// values of one line position adjacent) and x, y, dx, dy pixel-major.
//
// Lane layout: one lane per position of a line (the perpendicular axis), one
// line per wave, h in a VGPR for the whole scan, DPP for the two neighbours of
// the tridiagonal step (Sec. 3, Eq. (gspn_recurrence)).  bf16 is widened with
// one v_perm_b32 whose per-lane selector also zeroes the taps that leave the
// grid, so ignored taps may hold any value.
//
// Every global access reads or writes whole 128-byte lines: on this GPU the
// cost of a load is set by the lines it touches, not by its bytes.  With the
// blocked layout one coalesced 16-byte load gives a lane its position on 8
// consecutive lines of a tensor, so each per-direction stream costs one load
// (or store) instruction per 8 steps.
//
// Forward (one workgroup = one channel plane, one wave per direction):
//  * the x plane is loaded once, coalesced, into LDS and read from there by
//    all four directions (rows for vertical scans, columns for horizontal);
//  * each wave streams its lam, u and w blocks into registers, two blocks
//    ahead of use;
//  * u_d * h_d stays in registers; the four directions are summed in
//    direction-bit order through an fp32 LDS plane and y is stored once.
//
// Backward (one workgroup = `cw` channels of one weight group, one wave per
// channel, directions one after another, waves in lock-step):
//  * horizontal directions first: each wave stages its x and dy planes in its
//    own LDS plane (one dword per pixel) and reads columns from there; their
//    dx terms collect in registers (this lane's row) and then seed the plane
//    as an fp32 dx accumulator for the vertical directions, which read x and
//    dy rows from global memory;
//  * per direction a reverse sweep computes the adjoint a_i (kept in
//    registers), then a forward sweep recomputes h_i and forms du, dlam
//    (stored once per 8-line block), dx, and the weight-gradient terms
//    a_i * h_{i-1}[j+k-1], which are summed over the workgroup's channels
//    through double-buffered LDS slots, one barrier per two steps; when a
//    group spans several workgroups the sums go to fp32 partials that a
//    second kernel adds in fixed order.
#include <algorithm>

#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;

constexpr int kYPitch = 68;                // fp32 LDS row pitch (16-byte rows, conflict-free b128)
constexpr int kPlanePitch = 64;            // dwords per row of a wave's LDS plane (XOR-swizzled)
constexpr int kPrefetch = 16;              // steps of per-step row loads in flight (backward)
constexpr int kLdsAhead = 3;               // steps of staged (x, dy) LDS reads in flight (backward)

// One tridiagonal step: h_i = w0 h_{i-1}[j-1] + w1 h_{i-1}[j] + w2 h_{i-1}[j+1] + inj.
__device__ __forceinline__ float tri_step(float h, float w0, float w1, float w2, float inj)
{
    float hn = fmaf(w1, h, inj);
    hn = fmaf(w0, from_left<64>(h), hn);
    hn = fmaf(w2, from_right<64>(h), hn);
    return hn;
}

// The same in three instructions, the shifts fused into the multiply-adds
// (same operations in the same order, so the same result).  The backward,
// whose time goes mostly to issuing instructions, uses this form.
__device__ __forceinline__ float tri_step_f(float h, float w0, float w1, float w2, float inj)
{
    float hn = fmaf(w1, h, inj);
    hn = fmac_left(hn, h, w0);
    hn = fmac_right(hn, h, w2);
    return hn;
}

// Transposed step: a_i = w1_{i+1}[j] a[j] + (w0_{i+1} a)[j+1] + (w2_{i+1} a)[j-1] + inj.
__device__ __forceinline__ float tri_step_t(float an, float w0, float w1, float w2, float inj)
{
    float a = fmaf(w1, an, inj);
    a += from_right<64>(w0 * an);
    a += from_left<64>(w2 * an);
    return a;
}

// bf16 x plane in LDS with an odd dword pitch: a row walk (one bf16 per lane)
// and a column walk (one row per lane) are both conflict-free.
template <int W>
struct XPlane {
    static constexpr int kPitchDw = (W / 2) | 1;        // dwords per row
    static constexpr int kPitchB = 4 * kPitchDw;        // bytes per row
};

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------

// One direction's scan over one channel plane.  D: direction index (0 T2B,
// 1 B2T, 2 L2R, 3 R2L).  lam, u: the channel's blocked line-major planes; w:
// the 3 tap planes; xs: the bf16 x plane in LDS.
template <int H, int W, int D, bool PM>
__device__ __forceinline__ void scan_fwd_dir(int j, rsrc_t lam, rsrc_t u, rsrc_t w,
                                             const uint8_t *xs, float (&yr)[64])
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int L = VERT ? H : W, P = VERT ? W : H;
    constexpr int NB = L / 8;                 // blocks of 8 lines
    constexpr uint32_t PL = 2 * H * W;        // bytes of one plane
    const Sel s = make_sel(j, P);
    const int jc = j < P ? j : P - 1;
    // frame block fb (steps 8fb..8fb+7) is storage block fb, or NB-1-fb when
    // the scan runs against the storage order
    uint4 rl[NB], ru[NB], r0[NB], r1[NB], r2[NB];
    // lam and u come from HBM once, two blocks ahead; the taps, shared by the
    // group's channels and mostly served by L2, one block ahead
#define FLOADLU(fb)                                                  \
    do {                                                             \
        const int sq_ = REV ? NB - 1 - (fb) : (fb);                  \
        rl[fb] = ld_piece<PM, VERT, true>(lam, jc, sq_, P, W);       \
        ru[fb] = ld_piece<PM, VERT, true>(u, jc, sq_, P, W);         \
    } while (0)
#define FLOADW(fb)                                                   \
    do {                                                             \
        const int sq_ = REV ? NB - 1 - (fb) : (fb);                  \
        r0[fb] = ld_piece<PM, VERT, false>(w, jc, sq_, P, W);        \
        r1[fb] = ld_piece<PM, VERT, false>(w, jc, sq_, P, W, PL);    \
        r2[fb] = ld_piece<PM, VERT, false>(w, jc, sq_, P, W, 2 * PL);\
    } while (0)
    FLOADLU(0);
    FLOADW(0);
    if (NB > 1)
        FLOADLU(1);
    float h = 0.f;
#pragma unroll
    for (int fb = 0; fb < NB; ++fb) {
        if (fb + 2 < NB)
            FLOADLU(fb + 2);
        if (fb + 1 < NB)
            FLOADW(fb + 1);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const int e = REV ? 7 - t : t;                      // element of the piece
            const float lv = elem(rl[fb], e, s.lo1, s.hi1);
            const float uv = elem(ru[fb], e);
            const int row = VERT ? (REV ? H - 1 - i : i) : jc;
            const int col = VERT ? jc : (REV ? W - 1 - i : i);
            const float xv = bf_lo(lds_u16(xs, row * XPlane<W>::kPitchB + 2 * col));
            const float inj = lv * xv;
            if (i == 0)
                h = inj;
            else
                h = tri_step(h, elem(r0[fb], e, s.lo0, s.hi0), elem(r1[fb], e, s.lo1, s.hi1),
                             elem(r2[fb], e, s.lo2, s.hi2), inj);
            yr[i] = mul_nc(uv, h);   // rounded product, added in the merge
        }
        step_fence();
    }
#undef FLOADLU
#undef FLOADW
}

template <int H, int W, bool PM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void fwd_med_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, bf16_t *__restrict__ y, int mask, int B, int C, int G,
    Magic divC, Magic divCpg)
{
    static_assert(H <= 64 && W <= 64 && H % 8 == 0 && W % 8 == 0, "shape");
    constexpr int HW = H * W;
    constexpr int XB = H * XPlane<W>::kPitchB;              // x plane bytes
    constexpr int YB = H * kYPitch * 4;                     // merge plane bytes
    constexpr int LB = XB > YB ? XB : YB;
    // the merge plane replaces the x plane once every scan has finished
    __shared__ float4 lds4[(LB + 15) / 16];
    uint8_t *xs = reinterpret_cast<uint8_t *>(lds4);
    float4 *Y4 = lds4;
    float *Y = reinterpret_cast<float *>(lds4);

    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int b = mdiv(blk, divC);
    const int c = blk - b * C;
    const int g = mdiv(c, divCpg);
    const bool mine = (mask >> d) & 1;
    const int s = __popc(mask & ((1 << d) - 1));
    const int64_t pc = ((int64_t)b * C + c) * HW;
    const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
    const int64_t pw = (((int64_t)s * B + b) * G + g) * 3 * HW;

    // x plane -> LDS (coalesced 16-byte pieces, scattered into padded rows)
    {
        const rsrc_t xr = make_rsrc(x + pc, 2 * HW);
        for (int t = threadIdx.x; t < HW / 8; t += 256) {
            const uint4 v = ld128(xr, 16u * t, 0);
            const int r = t / (W / 8), q = t - r * (W / 8);
            uint32_t *dst = reinterpret_cast<uint32_t *>(xs + r * XPlane<W>::kPitchB) + 4 * q;
            dst[0] = v.x;
            dst[1] = v.y;
            dst[2] = v.z;
            dst[3] = v.w;
        }
    }
    lds_barrier();

    float yr[64];
    if (mine) {
        const rsrc_t rl = make_rsrc(lam + pd, 2 * HW);
        const rsrc_t ru = make_rsrc(u + pd, 2 * HW);
        const rsrc_t rw = make_rsrc(w + pw, 6 * HW);
        if (d == 0)
            scan_fwd_dir<H, W, 0, PM>(lane, rl, ru, rw, xs, yr);
        else if (d == 1)
            scan_fwd_dir<H, W, 1, PM>(lane, rl, ru, rw, xs, yr);
        else if (d == 2)
            scan_fwd_dir<H, W, 2, PM>(lane, rl, ru, rw, xs, yr);
        else
            scan_fwd_dir<H, W, 3, PM>(lane, rl, ru, rw, xs, yr);
    }
    lds_barrier();   // the x plane becomes the merge plane

    // Sum the directions in bit order through LDS: the first present one
    // stores, the others add, one direction per phase.
    const int first = __ffs(mask) - 1;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (d == p && mine) {
            const bool st = p == first;
            if (p < 2) {
                if (lane < W) {
#pragma unroll
                    for (int i = 0; i < H; ++i) {
                        float *a = Y + (p == 1 ? H - 1 - i : i) * kYPitch + lane;
                        *a = st ? yr[i] : add_nc(*a, yr[i]);
                    }
                }
            } else if (lane < H) {
#pragma unroll
                for (int cm = 0; cm < W / 8; ++cm) {
                    float4 *a = Y4 + (lane * kYPitch + 8 * cm) / 4;
                    float v[8];
#pragma unroll
                    for (int t = 0; t < 8; ++t) {
                        const int col = 8 * cm + t;
                        v[t] = yr[p == 3 ? W - 1 - col : col];
                    }
                    float4 a0 = make_float4(v[0], v[1], v[2], v[3]);
                    float4 a1 = make_float4(v[4], v[5], v[6], v[7]);
                    if (!st) {
                        const float4 o0 = a[0], o1 = a[1];
                        a0 = make_float4(add_nc(o0.x, a0.x), add_nc(o0.y, a0.y),
                                         add_nc(o0.z, a0.z), add_nc(o0.w, a0.w));
                        a1 = make_float4(add_nc(o1.x, a1.x), add_nc(o1.y, a1.y),
                                         add_nc(o1.z, a1.z), add_nc(o1.w, a1.w));
                    }
                    a[0] = a0;
                    a[1] = a1;
                }
            }
        }
        lds_barrier();
    }

    const u32x4 yo = make_sdesc(y + pc, 2 * HW);
    for (int t = threadIdx.x; t < H * (W / 8); t += 256) {
        const int r = t / (W / 8);
        const int cm = t - r * (W / 8);
        const float4 a0 = Y4[(r * kYPitch + 8 * cm) / 4];
        const float4 a1 = Y4[(r * kYPitch + 8 * cm) / 4 + 1];
        st128_nt(yo, 16u * t, 0, make_uint4(pack2(a0.x, a0.y), pack2(a0.z, a0.w), pack2(a1.x, a1.y),
                                         pack2(a1.z, a1.w)));
    }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------

// A wave's LDS plane (x and dy staged for the horizontal directions, then the
// fp32 dx accumulator) has rows of 64 dwords with element (r, c) at
// r * 64 + (c ^ r): a row walk and a column walk are both free of bank
// conflicts, at no padding.
__device__ __forceinline__ int pidx(int r, int c) { return r * kPlanePitch + (c ^ r); }

// The weight gradient of step i is sum_c a_c,i[j] h_c,i-1[j+k-1] over the
// workgroup's channels.  Each wave writes its a_i and h_{i-1} to LDS
// slots[buf][st][q][j][v] (v: a or h; q: channel slot, absent channels stay
// zero; j: position), two buffers of kBatch steps, one barrier per batch.
// After the barrier the wave that owns step st of the batch (one per SIMD)
// reads the 2 x NS values of its position, forms the three products with
// the neighbours' h from adjacent lanes (DPP), sums them in channel order
// and stores the line while the next batch runs.
// NS channel slots per step: 8, or 4 where two 4-channel workgroups per CU
// keep more waves busy than one of up to 8 channels (the slot area shrinks
// with NS).
constexpr int kSlots = 8;                  // the most channels of a workgroup
constexpr int kBatch = 4;
constexpr int slot_floats(int ns) { return 2 * kBatch * 2 * ns * 64; }

// a and h of (buffer, step, channel slot q, position j) are adjacent, so a
// wave writes both with one 8-byte LDS store and a reducer reads them with one
// 8-byte load.
template <int NS>
__device__ __forceinline__ float2 *slot_pair(float *slots, int buf, int st, int q)
{
    return reinterpret_cast<float2 *>(slots + ((buf * kBatch + st) * NS + q) * 128);
}

struct BwdArgs {
    rsrc_t x, dy;          // channel planes (pixel-major)
    rsrc_t lam, u;         // direction planes (blocked line-major)
    rsrc_t w;              // the 3 tap planes of (direction, group)
    u32x4 dlam, du;        // direction planes (store descriptors)
    u32x4 dw;              // 3 tap planes: final bf16 dw or fp32 partial
    float *Xq;             // this wave's LDS plane (pidx layout)
    float *slots;          // dw term slots
    int wave, cw;          // this wave, waves of the workgroup
    bool partial;          // dw holds fp32 partials
    bool first;            // first direction adding into the dx plane: store
};

// One direction of the backward.  D: direction index.  IMM: the workgroup has
// fewer waves than steps in a batch, so the reduction is not deferred.
// Horizontal
// directions read x and dy from the staged plane `stg` and add their dx
// terms to dxr (this lane's row); vertical directions read x and dy rows from
// global memory and add dx into the LDS dx plane.  When both vertical
// directions run, the first (SH 1) leaves the column's dy and x packed two
// rows to a dword in vdy and vx (rows 2k, 2k+1 in the low, high halves), and
// the second (SH 2) takes them from there instead of reading the rows again
// (dy only with WV).
template <int H, int W, int D, bool IMM, bool PC, int NS, bool PM, bool WPM, bool WV = false,
          int SH = 0>
__device__ __forceinline__ void dir_bwd(const BwdArgs &A, int j, bool cvalid, const uint8_t *stg,
                                        float (&dxr)[64], bool dx_first, uint32_t (&vdy)[H / 2],
                                        uint32_t (&vx)[H / 2])
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    static_assert(SH == 0 || (SH == 1 && D == 0) || (SH == 2 && D == 1), "vertical pair only");
    constexpr bool KEEP = SH == 2;                      // dy comes from vdy
    constexpr bool KEEPX = KEEP && !WV;                 // and x from vx
    constexpr int L = VERT ? H : W, P = VERT ? W : H;
    constexpr int NB = L / 8;
    constexpr uint32_t PL2 = 2 * H * W;                 // bytes of one bf16 plane
    // lam and u: pixel-major, except horizontal ones whose copies were
    // re-laid out with the weights (WPM false)
    constexpr bool LPM = PM && (VERT || WPM);
    // w: blocked, or pixel-major where the call's weights are (WPM); WV:
    // with one channel per group a vertical direction reads them in place
    // (rows, as lambda and u; a copy would be as large as lambda)
    constexpr bool WPD = WPM || (WV && VERT);
    const Sel s = make_sel(cvalid ? j : 64, P);         // an idle wave computes zeros
    const bool act = cvalid && j < P;
    const int jj = j < P ? j : P - 1;
    auto wpiece = [&](int sq_, uint32_t off) -> uint4 {
        return ld_piece<WPD, VERT, false>(A.w, jj, sq_, P, W, off);
    };
    const uint32_t vr = 2u * (uint32_t)jj;              // this lane's bf16 of a pixel row
    auto sblk = [](int fb) { return REV ? NB - 1 - fb : fb; };   // storage block of frame block fb
    auto line_of = [](int i) { return REV ? L - 1 - i : i; };   // storage line of step i
    auto rowoff = [&](int i) -> uint32_t { return 2u * (uint32_t)(line_of(i) * W); };
    auto stg_at = [&](int i) { return lds_u32(stg, 4u * (uint32_t)pidx(jj, line_of(i))); };
    // the kept value of storage line l
    auto kept = [](const uint32_t *a, int l) { return (l & 1) ? bf_hi(a[l >> 1]) : bf_lo(a[l >> 1]); };

    // the forward sweep's pieces: its first two blocks are loaded during the
    // reverse sweep's last two, so that they arrive while it ends
    uint4 rl[NB], p0[NB], p1[NB], p2[NB];
    uint32_t rx[VERT ? L : 1];
#define FLOADB(fb)                                                   \
    do {                                                             \
        const int sq_ = sblk(fb);                                    \
        rl[fb] = ld_piece<LPM, VERT, true>(A.lam, jj, sq_, P, W);     \
        p0[fb] = wpiece(sq_, 0u);                                     \
        p1[fb] = wpiece(sq_, PL2);                                    \
        p2[fb] = wpiece(sq_, 2 * PL2);                                \
    } while (0)

    // --- reverse sweep: adjoint a_i -------------------------------------
    float ahist[L];
    // dy of the column packed by pairs: storage rows for the first vertical
    // direction (its steps are the rows), steps otherwise
    uint32_t (&pdy)[H / 2] = vdy;
    {
        uint4 ru[NB], q0[NB], q1[NB], q2[NB];
        uint32_t rd[VERT ? L : 1];
#define RLOAD(fb)                                                    \
    do {                                                             \
        const int sq_ = sblk(fb);                                    \
        ru[fb] = ld_piece<LPM, VERT, true>(A.u, jj, sq_, P, W);       \
        q0[fb] = wpiece(sq_, 0u);                                     \
        q1[fb] = wpiece(sq_, PL2);                                    \
        q2[fb] = wpiece(sq_, 2 * PL2);                                \
    } while (0)
        RLOAD(NB - 1);
        if (NB > 1)
            RLOAD(NB - 2);
        if (VERT && !KEEP) {
#pragma unroll
            for (int i = L - 1; i >= L - kPrefetch; --i)
                rd[VERT ? i : 0] = ld16(A.dy, vr, rowoff(i));
        }
        float an = 0.f;
        // horizontal directions: the staged (x, dy) dwords are read kLdsAhead
        // steps ahead so their LDS latency overlaps the arithmetic
        uint32_t xq[VERT ? 1 : L];
        if (!VERT) {
#pragma unroll
            for (int i = L - 1; i >= L - kLdsAhead; --i)
                xq[VERT ? 0 : i] = stg_at(i);
        }
#pragma unroll
        for (int fb = NB - 1; fb >= 0; --fb) {
            if (fb >= 2)
                RLOAD(fb - 2);
            else if (fb == 1 || NB == 1)
                FLOADB(0);
            else
                FLOADB(1);
#pragma unroll
            for (int t = 7; t >= 0; --t) {
                const int i = 8 * fb + t;
                if (VERT && !KEEP && i - kPrefetch >= 0)
                    rd[VERT ? i - kPrefetch : 0] = ld16(A.dy, vr, rowoff(i - kPrefetch));
                if (VERT && !KEEPX && i - kPrefetch < 0)
                    rx[VERT ? kPrefetch - 1 - i : 0] =
                        ld16(A.x, vr, rowoff(kPrefetch - 1 - i));
                float dyv;
                if (VERT) {
                    dyv = KEEP ? kept(pdy, line_of(i)) : bf_lo(rd[VERT ? i : 0]);
                } else {
                    if (i - kLdsAhead >= 0)
                        xq[VERT ? 0 : i - kLdsAhead] = stg_at(i - kLdsAhead);
                    dyv = bf_hi(xq[VERT ? 0 : i]);
                }
                const int e = REV ? 7 - t : t;
                const float inj = elem(ru[fb], e, s.lo1, s.hi1) * dyv;
                float a;
                if (i + 1 == L) {
                    a = inj;
                } else {
                    // taps of step i+1 (the next block's first line for t = 7)
                    const int fn = (i + 1) >> 3, tn = (i + 1) & 7;
                    const int en = REV ? 7 - tn : tn;
                    a = tri_step_t(an, elem(q0[fn], en, s.lo0, s.hi0),
                                   elem(q1[fn], en, s.lo1, s.hi1), elem(q2[fn], en, s.lo2, s.hi2),
                                   inj);
                }
                ahist[i] = a;
                an = a;
                if (VERT && !KEEP && (i & 1) == 0)
                    pdy[VERT ? i >> 1 : 0] =
                        __builtin_amdgcn_perm(rd[VERT ? i + 1 : 0], rd[VERT ? i : 0], 0x05040100u);
                step_fence();
            }
        }
#undef RLOAD
    }

    // --- forward sweep: states, local gradients, dw terms ---------------

    // Reduction roles: step st of a batch belongs to wave st (waves 0..3, one
    // per SIMD); with fewer than kBatch waves (IMM) each wave takes several
    // steps and reduces them right after the barrier.
    float pa[NS], ph[NS];
    auto read_step = [&](int buf, int st) {
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            const float2 v2 = slot_pair<NS>(A.slots, buf, st, q)[j];
            pa[q] = v2.x;
            ph[q] = v2.y;
        }
    };
    // step i's weight gradient: the three products summed in channel order
    auto reduce_step = [&](int i) {
        float d0 = 0.f, d1 = 0.f, d2 = 0.f;
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            d0 = fmac_left(d0, ph[q], pa[q]);
            d1 = fmaf(pa[q], ph[q], d1);
            d2 = fmac_right(d2, ph[q], pa[q]);
        }
        if (j < P) {
            const int l = line_of(i);
            if (A.partial) {
                // line-major fp32 partials: the wave writes whole lines, with
                // the default cache policy since dw_sum_kernel reads them back
                // right after this kernel (non-temporal stores: 6 us more here
                // and 4 us more there at 64 x 64)
                const uint32_t f = (uint32_t)(l * P + j);
                st32(A.dw, 4u * f, 0, __float_as_uint(d0));
                st32(A.dw, 4u * (f + H * W), 0, __float_as_uint(d1));
                st32(A.dw, 4u * (f + 2 * H * W), 0, __float_as_uint(d2));
            } else {
                const uint32_t el = 2u * (uint32_t)dir_offset(PM, VERT, l, j, L, P, W);
                st16(A.dw, el, 0, pack1(d0));
                st16(A.dw, el + PL2, 0, pack1(d1));
                st16(A.dw, el + 2 * PL2, 0, pack1(d2));
            }
        }
    };
    const bool reducer = A.wave < kBatch;

    float h = 0.f;
    // this block's du and dlam as bf16 pairs in storage element order; the
    // value of the first step of a pair waits in du0 / dl0
    uint32_t dup[4], dlp[4];
    float du0 = 0.f, dl0 = 0.f;
    // one channel per group (PC): the weight gradient is this wave's own
    // products, packed per block like du
    uint32_t dwp[3][4];
    float dw0[3] = {0.f, 0.f, 0.f};
    uint32_t xq[VERT ? 1 : L];
    if (!VERT) {
#pragma unroll
        for (int i = 0; i < kLdsAhead; ++i)
            xq[VERT ? 0 : i] = stg_at(i);
    }
    float dx_next = 0.f;     // vertical: dx plane value of this step's row, read a step ahead
    if (VERT && !A.first)
        dx_next = A.Xq[pidx(line_of(0), jj)];
#pragma unroll
    for (int fb = 0; fb < NB; ++fb) {
        if (fb + 2 < NB)
            FLOADB(fb + 2);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const int e = REV ? 7 - t : t;
            if (VERT && !KEEPX && i + kPrefetch < L)
                rx[VERT ? i + kPrefetch : 0] = ld16(A.x, vr, rowoff(i + kPrefetch));
            float xv, dyv;
            if (VERT) {
                xv = KEEPX ? kept(vx, line_of(i)) : bf_lo(rx[VERT ? i : 0]);
                dyv = KEEP ? kept(pdy, line_of(i))
                           : (i & 1) ? bf_hi(pdy[VERT ? i >> 1 : 0]) : bf_lo(pdy[VERT ? i >> 1 : 0]);
                if (SH == 1 && !WV && (i & 1))
                    vx[VERT ? i >> 1 : 0] =
                        __builtin_amdgcn_perm(rx[VERT ? i : 0], rx[VERT ? i - 1 : 0], 0x05040100u);
            } else {
                if (i + kLdsAhead < L)
                    xq[VERT ? 0 : i + kLdsAhead] = stg_at(i + kLdsAhead);
                const uint32_t xd = xq[VERT ? 0 : i];
                xv = bf_lo(xd);
                dyv = bf_hi(xd);
            }
            const float lv = elem(rl[fb], e, s.lo1, s.hi1);
            const float hp = h;
            if (i == 0)
                h = lv * xv;
            else
                h = tri_step_f(hp, elem(p0[fb], e, s.lo0, s.hi0), elem(p1[fb], e, s.lo1, s.hi1),
                             elem(p2[fb], e, s.lo2, s.hi2), lv * xv);
            const float a = ahist[i];
            const float duv = dyv * h, dlv = a * xv;
            if ((t & 1) == 0) {
                du0 = duv;
                dl0 = dlv;
            } else {
                // steps t-1, t hold elements e+1, e (reverse) or e-1, e
                dup[e >> 1] = REV ? pack2(duv, du0) : pack2(du0, duv);
                dlp[e >> 1] = REV ? pack2(dlv, dl0) : pack2(dl0, dlv);
            }
            if (VERT) {
                // this wave is the only writer of its dx plane: the row of the
                // next step is read one step ahead, added to and written back
                // (an LDS float atomic costs several times more here)
                float *xa = A.Xq + pidx(line_of(i), jj);
                const float prev = dx_next;
                if (!A.first && i + 1 < L)
                    dx_next = A.Xq[pidx(line_of(i + 1), jj)];
                if (act)
                    *xa = A.first ? a * lv : fmaf(a, lv, prev);
            } else {
                const int cc = line_of(i);
                dxr[cc] = dx_first ? a * lv : fmaf(a, lv, dxr[cc]);
            }
            if constexpr (PC) {
                // w_i couples line i-1 to line i (h_{-1} = 0 zeroes line 0)
                const float dv[3] = {a * from_left<64>(hp), a * hp, a * from_right<64>(hp)};
#pragma unroll
                for (int k = 0; k < 3; ++k) {
                    if ((t & 1) == 0)
                        dw0[k] = dv[k];
                    else
                        dwp[k][e >> 1] = REV ? pack2(dv[k], dw0[k]) : pack2(dw0[k], dv[k]);
                }
            } else {
                // finish the previous batch: its slot reads were issued after
                // the last barrier and overlapped a step of arithmetic
                if (!IMM && (i & 3) == 1 && i >= 5 && reducer)
                    reduce_step(i - 5 + A.wave);
                // w_i couples line i-1 to line i: a_i and h_{i-1} go to the
                // slots (h_{-1} = 0 makes line 0's gradient zero)
                const int buf = (i >> 2) & 1;
                slot_pair<NS>(A.slots, buf, i & 3, A.wave)[j] = make_float2(a, hp);
                if ((i & 3) == 3) {
                    lds_barrier();
                    if (IMM) {
                        for (int st = A.wave; st < kBatch; st += A.cw) {
                            read_step(buf, st);
                            reduce_step(i - 3 + st);
                        }
                    } else if (reducer) {
                        read_step(buf, A.wave);
                    }
                }
            }
            if (PM && !VERT && act) {
                // pixel-major horizontal outputs: (du, dlam) of this pixel
                // replace its staged (x, dy), which no later step of this
                // direction reads; the plane leaves by whole rows afterwards
                reinterpret_cast<uint32_t *>(A.Xq)[pidx(jj, line_of(i))] = pack2(duv, dlv);
            }
            if (t == 7 && act) {
                if (!PM || VERT) {
                    st_piece<PM, VERT, true>(A.du, jj, sblk(fb), P, W,
                                             make_uint4(dup[0], dup[1], dup[2], dup[3]));
                    st_piece<PM, VERT, true>(A.dlam, jj, sblk(fb), P, W,
                                             make_uint4(dlp[0], dlp[1], dlp[2], dlp[3]));
                }
                if constexpr (PC) {
#pragma unroll
                    for (int k = 0; k < 3; ++k)
                        st_piece<PM && (VERT || !WV), VERT, true>(A.dw, jj, sblk(fb), P, W,
                                                 make_uint4(dwp[k][0], dwp[k][1], dwp[k][2], dwp[k][3]),
                                                 k * PL2);
                }
            }
            step_fence();
        }
    }
    if (!PC && !IMM && reducer)
        reduce_step(L - 4 + A.wave);
#undef FLOADB
}

// Shape and frame of direction D, shared by both backward variants.
template <int H, int W, int D>
struct BwdDir {
    static constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    static constexpr int L = VERT ? H : W, P = VERT ? W : H;
    static constexpr int NB = L / 8;
    static constexpr uint32_t PL2 = 2 * H * W;          // bytes of one bf16 plane
    static_assert(L % 8 == 0, "whole blocks");

    __device__ static int sblk(int fb) { return REV ? NB - 1 - fb : fb; }   // storage block
    __device__ static int line_of(int i) { return REV ? L - 1 - i : i; }   // storage line of step i
    // the staged (x, dy) dword of step i at position jj
    __device__ static uint32_t stg_at(const uint8_t *stg, int jj, int i)
    {
        const int l = line_of(i);
        return lds_u32(stg, 4u * (uint32_t)(VERT ? pidx(l, jj) : pidx(jj, l)));
    }
};

// The weight-gradient sum of step i from the slot values read for it.
template <int H, int W, int D, int NS, bool PM>
__device__ __forceinline__ void dw_store(const BwdArgs &A, int j, int i, const float (&pa)[NS],
                                         const float (&ph)[NS])
{
    using F = BwdDir<H, W, D>;
    float d0 = 0.f, d1 = 0.f, d2 = 0.f;
#pragma unroll
    for (int q = 0; q < NS; ++q) {
        d0 = fmac_left(d0, ph[q], pa[q]);
        d1 = fmaf(pa[q], ph[q], d1);
        d2 = fmac_right(d2, ph[q], pa[q]);
    }
    if (j < F::P) {
        const int l = F::line_of(i);
        if (A.partial) {
            // line-major fp32 partials: the wave writes whole lines (default
            // cache policy, as in dir_bwd)
            const uint32_t f = (uint32_t)(l * F::P + j);
            st32(A.dw, 4u * f, 0, __float_as_uint(d0));
            st32(A.dw, 4u * (f + H * W), 0, __float_as_uint(d1));
            st32(A.dw, 4u * (f + 2 * H * W), 0, __float_as_uint(d2));
        } else {
            const uint32_t el = 2u * (uint32_t)dir_offset(PM, F::VERT, l, j, F::L, F::P, W);
            st16(A.dw, el, 0, pack1(d0));
            st16(A.dw, el + F::PL2, 0, pack1(d1));
            st16(A.dw, el + 2 * F::PL2, 0, pack1(d2));
        }
    }
}

template <int NS>
__device__ __forceinline__ void read_slots(const BwdArgs &A, int j, int buf, int st,
                                           float (&pa)[NS], float (&ph)[NS])
{
#pragma unroll
    for (int q = 0; q < NS; ++q) {
        const float2 v2 = slot_pair<NS>(A.slots, buf, st, q)[j];
        pa[q] = v2.x;
        ph[q] = v2.y;
    }
}

// The slot traffic of the n-th step (n = 0, 1, ... in the order a pass takes
// them; that step is step_of(n)) with its adjoint a and previous state hp.
// Step st of a batch belongs to wave st (waves 0..3, one per SIMD), which
// issues the batch's slot reads after the barrier and finishes the sum 1.5
// steps later; with fewer than kBatch waves (IMM) each wave takes several
// steps and sums them right after the barrier.
template <int H, int W, int D, bool IMM, int NS, bool PM, class StepOf>
__device__ __forceinline__ void slot_step(const BwdArgs &A, int j, int n, float a, float hp,
                                          float (&pa)[NS], float (&ph)[NS], StepOf step_of)
{
    const bool reducer = A.wave < kBatch;
    // finish the previous batch: its slot reads were issued after the last
    // barrier and overlapped a step of arithmetic
    if (!IMM && (n & 3) == 1 && n >= 5 && reducer)
        dw_store<H, W, D, NS, PM>(A, j, step_of(n - 5 + A.wave), pa, ph);
    const int buf = (n >> 2) & 1;
    slot_pair<NS>(A.slots, buf, n & 3, A.wave)[j] = make_float2(a, hp);
    if ((n & 3) == 3) {
        lds_barrier();
        if (IMM) {
            for (int st = A.wave; st < kBatch; st += A.cw) {
                read_slots<NS>(A, j, buf, st, pa, ph);
                dw_store<H, W, D, NS, PM>(A, j, step_of(n - 3 + st), pa, ph);
            }
        } else if (reducer) {
            read_slots<NS>(A, j, buf, A.wave, pa, ph);
        }
    }
}

template <int H, int W, int D, bool IMM, int NS, bool PM, class StepOf>
__device__ __forceinline__ void slot_finish(const BwdArgs &A, int j, const float (&pa)[NS],
                                            const float (&ph)[NS], StepOf step_of)
{
    if (!IMM && A.wave < kBatch)
        dw_store<H, W, D, NS, PM>(A, j, step_of(BwdDir<H, W, D>::L - 4 + A.wave), pa, ph);
}

// One horizontal direction of the backward without the adjoint history, for
// when dxa already holds the 64 dx row sums of the other horizontal
// direction and both would not fit in registers: a forward
// pass keeps h at the last step of every 8-step block; a reverse pass then
// takes the blocks last to first, recomputes the block's h from the previous
// checkpoint and runs the adjoint and every local gradient over the block in
// reverse.  The live scan state is 2 x 8 floats instead of L; the price is a
// second read of lam and w (the first one leaves them in L2) and one more h
// recurrence per step.
template <int H, int W, int D, bool IMM, bool PC, int NS, bool PM, bool WPM, bool WV = false>
__device__ __forceinline__ void dir_bwd_ck(const BwdArgs &A, int j, bool cvalid, const uint8_t *stg,
                                           float (&dxa)[64])
{
    using F = BwdDir<H, W, D>;
    constexpr bool REV = F::REV;
    constexpr int L = F::L, P = F::P, NB = F::NB;
    constexpr uint32_t PL2 = F::PL2;
    const Sel s = make_sel(cvalid ? j : 64, P);         // an idle wave computes zeros
    const bool act = cvalid && j < P;
    const int jj = j < P ? j : P - 1;
    constexpr bool VERT = F::VERT;
    constexpr bool LPM = PM && (VERT || WPM);           // as in dir_bwd

    // --- forward pass: h at the end of every block ------------------------
    float hck[NB];
    {
        uint4 rl[NB], p0[NB], p1[NB], p2[NB];
#define ALOAD(fb)                                                    \
    do {                                                             \
        const int sq_ = F::sblk(fb);                                 \
        rl[fb] = ld_piece<LPM, VERT, false>(A.lam, jj, sq_, P, W);    \
        p0[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W);      \
        p1[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W, PL2); \
        p2[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W, 2 * PL2); \
    } while (0)
        ALOAD(0);
        if (NB > 1)
            ALOAD(1);
        uint32_t xq[L];
#pragma unroll
        for (int i = 0; i < kLdsAhead; ++i)
            xq[i] = F::stg_at(stg, jj, i);
        float h = 0.f;
#pragma unroll
        for (int fb = 0; fb < NB; ++fb) {
            if (fb + 2 < NB)
                ALOAD(fb + 2);
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int i = 8 * fb + t;
                const int e = REV ? 7 - t : t;
                if (i + kLdsAhead < L)
                    xq[i + kLdsAhead] = F::stg_at(stg, jj, i + kLdsAhead);
                const float inj = elem(rl[fb], e, s.lo1, s.hi1) * bf_lo(xq[i]);
                h = i == 0 ? inj
                           : tri_step_f(h, elem(p0[fb], e, s.lo0, s.hi0), elem(p1[fb], e, s.lo1, s.hi1),
                                      elem(p2[fb], e, s.lo2, s.hi2), inj);
                if (t == 7)
                    hck[fb] = h;
                step_fence();
            }
        }
#undef ALOAD
    }

    // --- reverse pass by blocks -------------------------------------------
    float pa[NS], ph[NS];
    // the n-th step of this pass is step L-1-n
    auto step_of = [](int n) { return L - 1 - n; };
    uint4 rl[NB], ru[NB], p0[NB], p1[NB], p2[NB];
#define BLOAD(fb)                                                    \
    do {                                                             \
        const int sq_ = F::sblk(fb);                                 \
        rl[fb] = ld_piece<LPM, VERT, true>(A.lam, jj, sq_, P, W);     \
        ru[fb] = ld_piece<LPM, VERT, true>(A.u, jj, sq_, P, W);       \
        p0[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W);      \
        p1[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W, PL2); \
        p2[fb] = ld_piece<WPM, VERT, false>(A.w, jj, sq_, P, W, 2 * PL2); \
    } while (0)
    BLOAD(NB - 1);
    uint32_t xd[NB][8];        // staged (x, dy) of a block, read a block ahead
#pragma unroll
    for (int t = 0; t < 8; ++t)
        xd[NB - 1][t] = F::stg_at(stg, jj, 8 * (NB - 1) + t);
    float an = 0.f, wn0 = 0.f, wn1 = 0.f, wn2 = 0.f;   // a and taps of the step after
#pragma unroll
    for (int fb = NB - 1; fb >= 0; --fb) {
        // one block ahead: a block takes two recurrences per step here
        if (fb >= 1) {
            BLOAD(fb - 1);
#pragma unroll
            for (int t = 0; t < 8; ++t)
                xd[fb - 1][t] = F::stg_at(stg, jj, 8 * (fb - 1) + t);
        }
        // h over the block from the previous block's checkpoint
        const float h0 = fb > 0 ? hck[fb > 0 ? fb - 1 : 0] : 0.f;
        float hb[8];
        {
            float h = h0;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int i = 8 * fb + t;
                const int e = REV ? 7 - t : t;
                const float inj = elem(rl[fb], e, s.lo1, s.hi1) * bf_lo(xd[fb][t]);
                h = i == 0 ? inj
                           : tri_step_f(h, elem(p0[fb], e, s.lo0, s.hi0), elem(p1[fb], e, s.lo1, s.hi1),
                                      elem(p2[fb], e, s.lo2, s.hi2), inj);
                hb[t] = h;
                step_fence();
            }
        }
        // the adjoint extracts its operands again rather than keeping the
        // 32 widened values of the recompute alive
        launder(rl[fb]);
        launder(p0[fb]);
        launder(p1[fb]);
        launder(p2[fb]);
        // du and dlam of the block as bf16 pairs in storage element order;
        // the later step of a pair waits in du1 / dl1
        uint32_t dup[4], dlp[4];
        float du1 = 0.f, dl1 = 0.f;
        uint32_t dwp[3][4];
        float dw1[3] = {0.f, 0.f, 0.f};
#pragma unroll
        for (int t = 7; t >= 0; --t) {
            const int i = 8 * fb + t;
            const int e = REV ? 7 - t : t;
            const float xv = bf_lo(xd[fb][t]), dyv = bf_hi(xd[fb][t]);
            const float inj = elem(ru[fb], e, s.lo1, s.hi1) * dyv;
            const float a = i + 1 == L ? inj : tri_step_t(an, wn0, wn1, wn2, inj);
            an = a;
            wn0 = elem(p0[fb], e, s.lo0, s.hi0);
            wn1 = elem(p1[fb], e, s.lo1, s.hi1);
            wn2 = elem(p2[fb], e, s.lo2, s.hi2);
            const float lv = elem(rl[fb], e, s.lo1, s.hi1);
            const float hp = t > 0 ? hb[t > 0 ? t - 1 : 0] : h0;     // h_{i-1}
            const float duv = dyv * hb[t], dlv = a * xv;
            if (t & 1) {
                du1 = duv;
                dl1 = dlv;
            } else {
                // steps t, t+1 hold elements e, e+1 (forward) or e, e-1 (reverse)
                dup[e >> 1] = REV ? pack2(du1, duv) : pack2(duv, du1);
                dlp[e >> 1] = REV ? pack2(dl1, dlv) : pack2(dlv, dl1);
            }
            const int cc = F::line_of(i);
            dxa[cc] = fmaf(a, lv, dxa[cc]);
            if constexpr (PC) {
                const float dv[3] = {a * from_left<64>(hp), a * hp, a * from_right<64>(hp)};
#pragma unroll
                for (int k = 0; k < 3; ++k) {
                    if (t & 1)
                        dw1[k] = dv[k];
                    else
                        dwp[k][e >> 1] = REV ? pack2(dw1[k], dv[k]) : pack2(dv[k], dw1[k]);
                }
            } else {
                slot_step<H, W, D, IMM, NS, PM>(A, j, L - 1 - i, a, hp, pa, ph, step_of);
            }
            if (PM && act) {
                // pixel-major outputs in place of the staged (x, dy) (see dir_bwd)
                reinterpret_cast<uint32_t *>(A.Xq)[pidx(jj, F::line_of(i))] = pack2(duv, dlv);
            }
            if (t == 0 && act) {
                if (!PM) {
                    st_piece<PM, VERT, true>(A.du, jj, F::sblk(fb), P, W,
                                             make_uint4(dup[0], dup[1], dup[2], dup[3]));
                    st_piece<PM, VERT, true>(A.dlam, jj, F::sblk(fb), P, W,
                                             make_uint4(dlp[0], dlp[1], dlp[2], dlp[3]));
                }
                if constexpr (PC) {
#pragma unroll
                    for (int k = 0; k < 3; ++k)
                        st_piece<PM && (VERT || !WV), VERT, true>(A.dw, jj, F::sblk(fb), P, W,
                                                 make_uint4(dwp[k][0], dwp[k][1], dwp[k][2], dwp[k][3]),
                                                 k * F::PL2);
                }
            }
            step_fence();
        }
    }
    if constexpr (!PC)
        slot_finish<H, W, D, IMM, NS, PM>(A, j, pa, ph, step_of);
#undef BLOAD
}

// PC: one channel per weight group; a workgroup then takes cw consecutive
// channels (groups), each wave sums nothing with the others, and nchunk /
// divChunk count the workgroups per batch.
// WV: one channel per group, pixel-major, vertical weights read in place and
// horizontal ones from the blocked copies wh.
template <int H, int W, bool IMM, bool PC, int NS, bool PM, bool WPM, bool WV = false>
__global__ __launch_bounds__(512) void bwd_med_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, const bf16_t *__restrict__ dy, bf16_t *__restrict__ dx,
    bf16_t *__restrict__ dw, bf16_t *__restrict__ dlam, bf16_t *__restrict__ du,
    float *__restrict__ dwp, int mask, int B, int C, int G, int cw, int nchunk, Magic divChunk,
    Magic divG, const bf16_t *__restrict__ lamh, const bf16_t *__restrict__ uh,
    const bf16_t *__restrict__ wh, bf16_t *__restrict__ dwh, int blk0)
{
    static_assert(H <= 64 && W <= 64 && H % 8 == 0 && W % 8 == 0 && H == W, "shape");
    constexpr int HW = H * W;
    constexpr int XPLANE = H * kPlanePitch;                 // floats per wave plane
    extern __shared__ float4 smem4[];
    float *smem = reinterpret_cast<float *>(smem4);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = blk0 + xcd_remap(blockIdx.x, gridDim.x);   // this launch: blk0 ..
    int b, g, c, chunk;
    bool cvalid;
    if constexpr (PC) {
        b = mdiv(blk, divChunk);
        chunk = blk - b * nchunk;
        const int c0 = chunk * cw;
        cvalid = wave < min(cw, C - c0);
        c = c0 + (cvalid ? wave : 0);
        g = c;
    } else {
        const int bg = mdiv(blk, divChunk);
        chunk = blk - bg * nchunk;
        b = mdiv(bg, divG);
        g = bg - b * G;
        const int cpg = mdiv(C, divG);
        const int cfirst = chunk * cw;
        cvalid = wave < min(cw, cpg - cfirst);
        c = g * cpg + cfirst + (cvalid ? wave : 0);
    }
    const int D = __popc(mask);
    const int64_t pc = ((int64_t)b * C + c) * HW;

    BwdArgs A;
    A.x = make_rsrc(x + pc, 2 * HW);
    A.dy = make_rsrc(dy + pc, 2 * HW);
    A.Xq = smem + wave * XPLANE;
    A.slots = smem + cw * XPLANE;
    // slots of channels this workgroup does not have must read as zero
    if (!PC) {
        for (int t = threadIdx.x; t < slot_floats(NS); t += blockDim.x)
            A.slots[t] = 0.f;
    }
    lds_barrier();
    A.wave = wave;
    A.cw = cw;
    A.partial = !PC && nchunk > 1;

    // Horizontal directions read x and dy columns: stage both planes in this
    // wave's LDS dx plane (still unused), coalesced; their dx terms collect in
    // registers (this lane's row) and move into the dx plane afterwards.
    const bool horiz = (mask & 12) != 0;
    const uint8_t *stg = reinterpret_cast<const uint8_t *>(A.Xq);
    auto stage_xdy = [&]() {
        uint32_t *st = reinterpret_cast<uint32_t *>(A.Xq);
        constexpr int NP = HW / 8;                          // 16-byte pieces per plane
#pragma unroll
        for (int t = 0; t < (NP + 63) / 64; ++t) {
            const int p = t * 64 + lane;
            if (p < NP) {
                const uint4 vx = ld128(A.x, 16u * p, 0);
                const uint4 vd = ld128(A.dy, 16u * p, 0);
                const int pr = p / (W / 8), pq = p - pr * (W / 8);
                const uint32_t xs_[4] = {vx.x, vx.y, vx.z, vx.w};
                const uint32_t ds_[4] = {vd.x, vd.y, vd.z, vd.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    st[pidx(pr, 8 * pq + 2 * e)] = __builtin_amdgcn_perm(ds_[e], xs_[e], 0x05040100u);
                    st[pidx(pr, 8 * pq + 2 * e + 1)] =
                        __builtin_amdgcn_perm(ds_[e], xs_[e], 0x07060302u);
                }
            }
        }
        // the same wave reads what it wrote: LDS keeps its order
    };
    if (horiz)
        stage_xdy();
    // Pixel-major horizontal directions leave du and dlam in the plane, one
    // (du, dlam) pair per pixel: out by whole rows, lane t taking 8
    // consecutive columns of a row.
    auto flush_out = [&]() {
        if (!cvalid)
            return;
        constexpr int NP = HW / 8;
#pragma unroll
        for (int it = 0; it < (NP + 63) / 64; ++it) {
            const int t = it * 64 + lane;
            if (t < NP) {
                const int r = t / (W / 8), cm = t - r * (W / 8);
                uint32_t v[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    v[e] = reinterpret_cast<const uint32_t *>(A.Xq)[pidx(r, 8 * cm + e)];
                uint32_t du4[4], dl4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    du4[e] = __builtin_amdgcn_perm(v[2 * e + 1], v[2 * e], 0x05040100u);
                    dl4[e] = __builtin_amdgcn_perm(v[2 * e + 1], v[2 * e], 0x07060302u);
                }
                st128_nt(A.du, 16u * (uint32_t)t, 0, make_uint4(du4[0], du4[1], du4[2], du4[3]));
                st128_nt(A.dlam, 16u * (uint32_t)t, 0, make_uint4(dl4[0], dl4[1], dl4[2], dl4[3]));
            }
        }
    };

    // Per-direction descriptors.  An idle wave (no channel left in this
    // chunk) still joins every barrier; it reads channel `c` of the chunk,
    // computes zeros and stores nothing of its own.
    auto setup = [&](int d) {
        const int s = __popc(mask & ((1 << d) - 1));
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const int64_t unit = ((int64_t)s * B + b) * G + g;
        if (PM && !WPM && d >= 2) {
            // the re-laid-out copies hold the horizontal slots only
            const int64_t ph = (((int64_t)(s - __popc(mask & 3)) * B + b) * C + c) * HW;
            A.lam = make_rsrc(lamh + ph, 2 * HW);
            A.u = make_rsrc(uh + ph, 2 * HW);
        } else {
            A.lam = make_rsrc(lam + pd, 2 * HW);
            A.u = make_rsrc(u + pd, 2 * HW);
        }
        A.dlam = make_sdesc(dlam + pd, 2 * HW);
        A.du = make_sdesc(du + pd, 2 * HW);
        if (WV && d >= 2) {
            // one channel per group: blocked copies of the horizontal slots
            const int64_t uh_ = ((int64_t)(s - __popc(mask & 3)) * B + b) * G + g;
            A.w = make_rsrc(wh + uh_ * 3 * HW, 6 * HW);
        } else {
            A.w = make_rsrc(w + unit * 3 * HW, 6 * HW);
        }
        if (A.partial)
            A.dw = make_sdesc(dwp + ((int64_t)chunk * D * B * G + unit) * 3 * HW, 12 * HW);
        else if (WV && d >= 2)
            // horizontal weight gradients in the blocked order (whole 16-byte
            // lines), turned pixel-major by a transpose launch afterwards
            A.dw = make_sdesc(dwh + (((int64_t)(s - __popc(mask & 3)) * B + b) * G + g) * 3 * HW,
                              6 * HW);
        else
            A.dw = make_sdesc(dw + unit * 3 * HW, 6 * HW);
    };

    // horizontal directions first (x and dy staged), dx in registers
    float dxr[64];
    // the column's dy and x, from T2B to B2T (dy only where the vertical
    // weights are read in place as rows: no registers to spare for x there)
    uint32_t vdy[H / 2], vx[H / 2];
    A.first = false;
    if (mask & 4) {
        setup(2);
        dir_bwd<H, W, 2, IMM, PC, NS, PM, WPM, WV>(A, lane, cvalid, stg, dxr, true, vdy, vx);
        lds_barrier();   // slot buffers are reused by the next direction
        if (PM) {
            flush_out();
            if (mask & 8)
                stage_xdy();   // x and dy again for the other horizontal direction
        }
    }
    if (mask & 8) {
        setup(3);
        if ((mask & 4) && H >= 64)
            dir_bwd_ck<H, W, 3, IMM, PC, NS, PM, WPM, WV>(A, lane, cvalid, stg, dxr);
        else
            dir_bwd<H, W, 3, IMM, PC, NS, PM, WPM, WV>(A, lane, cvalid, stg, dxr, (mask & 4) == 0,
                                                      vdy, vx);
        lds_barrier();
        if (PM)
            flush_out();
    }
    if (horiz && lane < H) {
        // the horizontal dx terms (this lane's row) seed the dx plane that the
        // vertical directions add to
#pragma unroll
        for (int q = 0; q < W; ++q)
            A.Xq[pidx(lane, q)] = dxr[q];
    }
    if (mask & 1) {
        setup(0);
        A.first = !horiz;
        dir_bwd<H, W, 0, IMM, PC, NS, PM, WPM, WV, 1>(A, lane, cvalid, stg, dxr, false, vdy, vx);
        lds_barrier();
    }
    if (mask & 2) {
        setup(1);
        A.first = !horiz && (mask & 1) == 0;
        if (mask & 1)
            dir_bwd<H, W, 1, IMM, PC, NS, PM, WPM, WV, 2>(A, lane, cvalid, stg, dxr, false, vdy,
                                                          vx);
        else
            dir_bwd<H, W, 1, IMM, PC, NS, PM, WPM, WV>(A, lane, cvalid, stg, dxr, false, vdy, vx);
        lds_barrier();
    }

    // dx out of this wave's plane: lane t takes 8 consecutive columns of a
    // row, so each store instruction covers whole 128-byte lines (the LDS
    // reads of a lane hit 64 different banks across the wave)
    if (cvalid) {
        const u32x4 dxo = make_sdesc(dx + pc, 2 * HW);
        constexpr int NP = HW / 8;
#pragma unroll
        for (int it = 0; it < (NP + 63) / 64; ++it) {
            const int t = it * 64 + lane;
            if (t < NP) {
                const int r = t / (W / 8), cm = t - r * (W / 8);
                float a[8];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    a[e] = A.Xq[pidx(r, 8 * cm + e)];
                st128_nt(dxo, 16u * (uint32_t)t, 0,
                         make_uint4(pack2(a[0], a[1]), pack2(a[2], a[3]), pack2(a[4], a[5]),
                                    pack2(a[6], a[7])));
            }
        }
    }
}

// dw (bf16) = sum over chunks of the fp32 partials, in chunk order.
// Partials are line-major per (chunk, unit, tap): storage line l, position j
// at float l * S + j.
// Blocked dw: one thread makes the 8 outputs of one (unit, tap, 8-line
// block, position): eight reads per chunk and one 16-byte store, both
// contiguous across the wave.
template <int S>
__global__ __launch_bounds__(256) void dw_sum_kernel(const float *__restrict__ dwp,
                                                     uint4 *__restrict__ dw, int64_t nuk, int nchunk)
{
    constexpr int NQ = S / 8, HW = S * S;
    const int64_t n = nuk * NQ * S;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int j = (int)(o % S);
        const int64_t r = o / S;
        const int q = (int)(r % NQ);
        const int64_t uk = r / NQ;                      // unit * 3 + tap
        float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        for (int c = 0; c < nchunk; ++c) {
            const float *src = dwp + ((int64_t)c * nuk + uk) * HW + (int64_t)(8 * q) * S + j;
#pragma unroll
            for (int t = 0; t < 8; ++t)
                v[t] += src[t * S];
        }
        gst128(dw + (uk * HW + (int64_t)8 * S * q + 8 * j) / 8,
               make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7])));
    }
}

// The same into pixel-major dw, one workgroup per (unit, tap) plane.  A
// vertical direction's lines are image rows: each thread sums and stores 8
// consecutive pixels of a row.  A horizontal direction's lines are columns:
// the partials are read along their lines (coalesced), summed, turned around
// through LDS, and stored by rows.  vslots: bit s set when direction slot s
// is vertical; per_slot: units * 3 of one slot.  This launch takes, in every
// slot, the (unit, tap) planes r0 .. r0 + rn - 1 of the slot.
template <int S>
__global__ __launch_bounds__(256) void dw_sum_pm_kernel(const float *__restrict__ dwp,
                                                        uint4 *__restrict__ dw, int64_t nuk,
                                                        int nchunk, int vslots, int64_t per_slot,
                                                        int64_t r0, int64_t rn)
{
    constexpr int HW = S * S, NQ = S / 8;
    __shared__ float T[S][S + 1];
    const int64_t sl = blockIdx.x / rn;
    const int64_t uk = sl * per_slot + r0 + (blockIdx.x - sl * rn);
    const bool vert = (vslots >> (int)(uk / per_slot)) & 1;   // uniform over the workgroup
    uint4 *dst = dw + uk * (HW / 8);
    const float4 *src = reinterpret_cast<const float4 *>(dwp + uk * HW);
    const int64_t cstride = nuk * (HW / 4);                    // float4s between chunks
    for (int t = threadIdx.x; t < HW / 8; t += 256) {
        // 8 consecutive values of a line, summed over the chunks in chunk
        // order; four chunks' loads in flight at a time
        float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        int c = 0;
        for (; c + 4 <= nchunk; c += 4) {
            float4 a[4], b[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                a[k] = src[(c + k) * cstride + 2 * t];
                b[k] = src[(c + k) * cstride + 2 * t + 1];
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[0] += a[k].x, v[1] += a[k].y, v[2] += a[k].z, v[3] += a[k].w;
                v[4] += b[k].x, v[5] += b[k].y, v[6] += b[k].z, v[7] += b[k].w;
            }
        }
        for (; c < nchunk; ++c) {
            const float4 a = src[c * cstride + 2 * t], b = src[c * cstride + 2 * t + 1];
            v[0] += a.x, v[1] += a.y, v[2] += a.z, v[3] += a.w;
            v[4] += b.x, v[5] += b.y, v[6] += b.z, v[7] += b.w;
        }
        if (vert) {
            gst128(dst + t, make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]),
                                       pack2(v[6], v[7])));
        } else {
            const int l = t / NQ, pos = 8 * (t - l * NQ);        // line (column), first row
#pragma unroll
            for (int k = 0; k < 8; ++k)
                T[pos + k][l] = v[k];
        }
    }
    if (vert)
        return;
    __syncthreads();
    for (int t = threadIdx.x; t < HW / 8; t += 256) {
        const int r = t / NQ, cq = t - r * NQ;
        const float *row = &T[r][8 * cq];
        gst128(dst + t, make_uint4(pack2(row[0], row[1]), pack2(row[2], row[3]),
                                   pack2(row[4], row[5]), pack2(row[6], row[7])));
    }
}

template <int H, int W, bool PM>
hipError_t fwd_med_t(const Problem &p, hipStream_t st)
{
    if (p.ws->counting)
        return hipSuccess;
    hipLaunchKernelGGL((fwd_med_kernel<H, W, PM>), dim3((unsigned)(p.B * p.C)), dim3(256), 0, st,
                       (const bf16_t *)p.x, (const bf16_t *)p.w, (const bf16_t *)p.lam,
                       (const bf16_t *)p.u, (bf16_t *)p.y, p.mask, p.B, p.C, p.G,
                       make_magic((uint32_t)p.C), make_magic((uint32_t)(p.C / p.G)));
    return hipGetLastError();
}

// Workgroups blk0 .. blk0 + nblk - 1 (nblk < 0: all of them).
template <int H, int W, bool IMM, bool PC, int NS, bool PM, bool WPM, bool WV = false>
hipError_t bwd_med_launch(const Problem &p, hipStream_t st, int cw, int nchunk, size_t lds,
                          float *dwp, const void *lamh, const void *uh, const void *wh = nullptr,
                          void *dwh = nullptr, int blk0 = 0, int nblk = -1)
{
    hipError_t e = hipFuncSetAttribute((const void *)bwd_med_kernel<H, W, IMM, PC, NS, PM, WPM, WV>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    const unsigned grid = nblk >= 0 ? (unsigned)nblk
                                    : (unsigned)(PC ? p.B * nchunk : p.B * p.G * nchunk);
    hipLaunchKernelGGL((bwd_med_kernel<H, W, IMM, PC, NS, PM, WPM, WV>), dim3(grid),
                       dim3(64 * cw), lds, st, (const bf16_t *)p.x, (const bf16_t *)p.w,
                       (const bf16_t *)p.lam, (const bf16_t *)p.u, (const bf16_t *)p.dy,
                       (bf16_t *)p.dx, (bf16_t *)p.dw, (bf16_t *)p.dlam, (bf16_t *)p.du, dwp,
                       p.mask, p.B, p.C, p.G, cw, nchunk, make_magic((uint32_t)nchunk),
                       make_magic((uint32_t)p.G), (const bf16_t *)lamh, (const bf16_t *)uh,
                       (const bf16_t *)wh, (bf16_t *)dwh, blk0);
    return hipGetLastError();
}

// Registers the NS = 4 backward holds per lane (for the occupancy estimate of
// the slot-count choice); 0 if unknown.
template <int H, int W, bool PM, bool WPM>
int bwd_ns4_regs()
{
    hipFuncAttributes fa;
    if (hipFuncGetAttributes(&fa, (const void *)bwd_med_kernel<H, W, false, false, 4, PM, WPM>) !=
        hipSuccess)
        return 0;
    return fa.numRegs;
}

// WPM: the weights are pixel-major (else blocked, e.g. re-laid out by
// launch_w_to_blocked); the other per-direction tensors follow PM.
template <int H, int W, bool PM, bool WPM>
hipError_t bwd_med_t(const Problem &p, hipStream_t st, const void *lamh = nullptr,
                     const void *uh = nullptr, const void *wh = nullptr, void *dwh = nullptr)
{
    const int lds_max = kLdsBytes;
    const size_t per_ch = (size_t)H * kPlanePitch * 4;              // wave plane
    const int cpg = p.C / p.G;
    if (cpg == 1) {
        // one channel per group: workgroups of up to kSlots channels, no slots
        const int cw = p.C < kSlots ? p.C : kSlots;
        const int nct = (p.C + cw - 1) / cw;
        if ((size_t)cw * per_ch > (size_t)lds_max)
            return hipErrorInvalidConfiguration;
        if (p.ws->counting)
            return hipSuccess;
        if (PM && !WPM && wh != nullptr) {
            hipError_t e = bwd_med_launch<H, W, false, true, kSlots, PM, WPM, true>(
                p, st, cw, nct, (size_t)cw * per_ch, nullptr, lamh, uh, wh, dwh);
            const int nvd = __builtin_popcount(p.mask & 3), nhd = __builtin_popcount(p.mask & 12);
            // the horizontal dw planes, blocked [q][p] pieces -> pixel-major
            // [p][q]: the piece transpose of a plane of H/8 rows of 8 W
            // columns
            if (e == hipSuccess && nhd > 0)
                e = launch_planes_pieces(dwh,
                                  static_cast<bf16_t *>(p.dw) + (int64_t)nvd * p.B * p.G * 3 * H * W,
                                  0, (int64_t)nhd * p.B * p.G * 3, H / 8, 8 * W, st);
            return e;
        }
        return bwd_med_launch<H, W, false, true, kSlots, PM, WPM>(
            p, st, cw, nct, (size_t)cw * per_ch, nullptr, lamh, uh);
    }
    // A group's channels in nchunk workgroups of cw channels, NS slots per
    // step.  NS = 4 (at most 4 channels, a smaller slot area) is taken where
    // it puts more waves on a CU than NS = 8 for at most one more chunk, e.g.
    // 56 x 56 with 12 channels per group: two 4-wave workgroups per CU (8
    // waves, 2 per SIMD) instead of one of 6 waves.
    struct Plan {
        int nchunk = 0, cw = 0;
        size_t lds = 0;
    };
    auto plan = [&](int ns) {
        Plan q;
        const size_t sl = (size_t)slot_floats(ns) * 4;
        int cap = lds_max > (int)sl ? (int)(((size_t)lds_max - sl) / per_ch) : 0;
        cap = cap < ns ? cap : ns;
        if (cap >= 1) {
            q.nchunk = (cpg + cap - 1) / cap;
            q.cw = (cpg + q.nchunk - 1) / q.nchunk;
            q.lds = (size_t)q.cw * per_ch + sl;
        }
        return q;
    };
    const Plan p8 = plan(kSlots), p4 = plan(4);
    if (p8.nchunk < 1)
        return hipErrorInvalidConfiguration;
    bool use4 = false;
    if (p.slots == 4 || p.slots == 8) {
        use4 = p.slots == 4 && p4.nchunk >= 1 && p4.cw == 4;
    } else if (p4.nchunk >= 1 && p4.cw == 4 && p4.nchunk <= p8.nchunk + 1) {
        const int regs = bwd_ns4_regs<H, W, PM, WPM>();
        if (regs > 0) {
            const int per_simd = 512 / ((regs + 7) / 8 * 8);   // waves a SIMD holds
            auto waves = [&](const Plan &q) {
                const int by_lds = (int)((size_t)kLdsBytes / q.lds) * q.cw;
                return by_lds < 4 * per_simd ? by_lds : 4 * per_simd;
            };
            use4 = waves(p4) > waves(p8);
        }
    }
    const Plan &pl = use4 ? p4 : p8;
    const int nchunk = pl.nchunk, cw = pl.cw;
    const size_t lds = pl.lds;
    const int D = __builtin_popcount(p.mask);
    const int64_t ndw = (int64_t)D * p.B * p.G * 3 * H * W;

    float *dwp = nullptr;
    hipError_t e = hipSuccess;
    if (nchunk > 1) {
        e = p.ws->take((void **)&dwp, (size_t)nchunk * ndw * sizeof(float));
        if (e != hipSuccess)
            return e;
    }
    if (p.ws->counting)
        return hipSuccess;
    auto scan = [&](int blk0, int nblk) {
        if (use4)
            return bwd_med_launch<H, W, false, false, 4, PM, WPM>(p, st, cw, nchunk, lds, dwp, lamh,
                                                                  uh, nullptr, nullptr, blk0, nblk);
        return cw >= kBatch ? bwd_med_launch<H, W, false, false, kSlots, PM, WPM>(
                                  p, st, cw, nchunk, lds, dwp, lamh, uh, nullptr, nullptr, blk0, nblk)
                            : bwd_med_launch<H, W, true, false, kSlots, PM, WPM>(
                                  p, st, cw, nchunk, lds, dwp, lamh, uh, nullptr, nullptr, blk0, nblk);
    };
    const int64_t units = (int64_t)p.B * p.G;          // (b, g), nchunk workgroups each
    if (PM && nchunk > 1) {
        // Rounds of whole units, each exactly as many workgroups as the device
        // runs at once, the partial sum of a round right after its scan: the
        // round's partials (50 MB at 64 x 64) are then mostly still in the
        // Infinity Cache when the sum reads them (64 x 64, B = 8, C = 768,
        // G = 24: three rounds, backward 373 -> 363 us).  Only where the
        // rounds come out even: each boundary drains the device, and at
        // 56 x 56 (512 workgroups at once, units of 3) four uneven rounds
        // took the backward from 360 to 423 us.
        int vslots = 0;
        for (int d = 0, sl = 0; d < 4; ++d)
            if ((p.mask >> d) & 1) {
                if (d < 2)
                    vslots |= 1 << sl;
                ++sl;
            }
        int dev = 0, ncu = 0;
        int64_t ru = units;                              // units per round
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
            ncu > 0) {
            const int per_cu = std::max(1, std::min((int)((size_t)kLdsBytes / lds), 8 / cw));
            const int64_t fit = (int64_t)ncu * per_cu;
            if (fit % nchunk == 0 && units % (fit / nchunk) == 0)
                ru = fit / nchunk;
        }
        const int64_t nuk = (int64_t)D * units * 3;
        for (int64_t u0 = 0; u0 < units && e == hipSuccess; u0 += ru) {
            const int64_t nu = std::min(ru, units - u0);
            e = scan((int)(u0 * nchunk), (int)(nu * nchunk));
            if (e == hipSuccess) {
                hipLaunchKernelGGL((dw_sum_pm_kernel<H>), dim3((unsigned)(D * nu * 3)), dim3(256), 0,
                                   st, (const float *)dwp, (uint4 *)p.dw, nuk, nchunk, vslots,
                                   units * 3, u0 * 3, nu * 3);
                e = hipGetLastError();
            }
        }
        return e;
    }
    e = scan(0, -1);
    if (e == hipSuccess && nchunk > 1) {
        const int64_t nuk = (int64_t)D * p.B * p.G * 3;
        const int64_t n8 = ndw / 8;
        int64_t blocks = (n8 + 255) / 256;
        blocks = blocks < 16384 ? blocks : 16384;
        hipLaunchKernelGGL((dw_sum_kernel<H>), dim3((unsigned)blocks), dim3(256), 0, st,
                           (const float *)dwp, (uint4 *)p.dw, nuk, nchunk);
        e = hipGetLastError();
    }
    return e;
}

template <int H, int W>
hipError_t fwd_med_l(const Problem &p, hipStream_t st)
{
    if (p.layout != kPixelMajor)
        return fwd_med_t<H, W, false>(p, st);
    return launch_fwd_pm(p, st);
}

template <int H, int W>
hipError_t bwd_med_l(const Problem &p, hipStream_t st)
{
    if (p.layout != kPixelMajor)
        return bwd_med_t<H, W, false, false>(p, st);
    // the group's weights, and lambda and u of the horizontal directions,
    // re-laid out once into the blocked order of their direction
    // (workspace), read there as 16-byte pieces: a horizontal scan would read
    // each pixel-major piece from 64 rows
    // One channel per group (weights as large as lambda): only the
    // horizontal directions' weights are copied, vertical ones read in place.
    // The backward of a training pair finds these copies in the reserve its
    // forward wrote (take_reserve: the same pieces in the same order).
    const bool pc = p.C == p.G && !p.w_blocked;   // (formed weights are all blocked)
    const int nvd = __builtin_popcount(p.mask & 3), nhd = __builtin_popcount(p.mask & 12);
    const int64_t nw = (int64_t)(pc ? nhd : nvd + nhd) * p.B * p.G * 3 * H * W;
    const int64_t nh = (int64_t)nhd * p.B * p.C * H * W;
    void *wb = const_cast<void *>(p.w), *lamh = nullptr, *uh = nullptr;
    hipError_t e = hipSuccess;
    if (p.rs_read && p.rsp != nullptr) {
        if (p.rsp->w != nullptr)
            wb = p.rsp->w;
        lamh = p.rsp->lamh;
        uh = p.rsp->uh;
    } else {
        if (!p.w_blocked && nw > 0)
            e = p.ws->take(&wb, (size_t)nw * 2);
        if (e == hipSuccess && nh > 0)
            e = p.ws->take(&lamh, (size_t)nh * 2);
        if (e == hipSuccess && nh > 0)
            e = p.ws->take(&uh, (size_t)nh * 2);
    }
    void *dwh = nullptr;
    if (e == hipSuccess && pc && nw > 0)
        e = p.ws->take(&dwh, (size_t)nw * 2);
    if (e != hipSuccess)
        return e;
    if (!p.ws->counting && !(p.rs_read && p.rsp != nullptr)) {
        if (pc)
            e = nw > 0 ? launch_planes_to_blocked(
                             static_cast<const bf16_t *>(p.w) + (int64_t)nvd * p.B * p.G * 3 * H * W,
                             wb, (int)(nw / ((int64_t)H * W)), H, st)
                       : hipSuccess;
        else if (!p.w_blocked)
            e = launch_w_to_blocked(p, wb, st);
        if (e == hipSuccess && nh > 0)
            e = launch_horiz_to_blocked(p, lamh, uh, st);
        if (e != hipSuccess)
            return e;
    }
    if (pc)
        return bwd_med_t<H, W, true, false>(p, st, lamh, uh, wb, dwh);
    Problem q = p;
    q.w = wb;
    return bwd_med_t<H, W, true, false>(q, st, lamh, uh);
}

}  // namespace

// Entry points of one side (explicitly instantiated, one translation unit per
// side, so that the sides compile in parallel).
template <int S>
hipError_t med_fwd(const Problem &p, hipStream_t st)
{
    return fwd_med_l<S, S>(p, st);
}

template <int S>
hipError_t med_bwd(const Problem &p, hipStream_t st)
{
    return bwd_med_l<S, S>(p, st);
}

}  // namespace gspn
