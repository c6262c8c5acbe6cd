// Line scans for bf16 planes with both sides at most 16 (token grids such as
// 14 x 14), forward and backward.
//
// A workgroup takes up to 64 channels of one weight group, so that the
// group's weight-gradient sum stays in the workgroup; each wave holds four
// channels, one per 16-lane row, lane j of a row being line position j (DPP
// row shifts give the tridiagonal neighbours, Sec. 3, Eq. (gspn_recurrence)).
// A plane is 392 bytes at 14 x 14, too small for the per-lane streaming of
// the larger kernels, so every plane a direction needs (x and dy of the
// channels, their lam_d and u_d, the group's three taps) is copied into LDS
// with the widest coalesced accesses its alignment allows and read from
// there.
//  * forward: the directions run one after another; the planes of the next
//    direction are copied into a second LDS buffer by direct-to-LDS loads
//    while the current one computes; each lane keeps its channel's u_d * h_d
//    in registers (a column for vertical directions, a row for horizontal
//    ones); both are added through an fp32 LDS plane and y leaves with one
//    coalesced copy;
//  * backward: a reverse sweep (adjoint, kept in registers) and a forward
//    sweep (recomputed h) per direction; du and dlam overwrite the staged u
//    and lam in place and leave with one coalesced copy per plane; the
//    weight-gradient terms are summed over the wave's four channels with
//    lane-swap instructions and over the waves through LDS, once per
//    direction;
//    dx is merged like y.
#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;

constexpr int kMaxCh = 64;                 // channels per workgroup
constexpr int kLaneRow = 16;               // lanes of one channel slot
constexpr int kSlotW = 4;                  // channel slots per wave

__host__ __device__ constexpr int round8(int n) { return (n + 7) & ~7; }

__device__ __forceinline__ float bfv(const uint16_t *p, int i)
{
    return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
// A bf16 value of an LDS plane, or 0 where `on` is false.  The read itself
// is unconditional -- every caller's address lies inside the workgroup's
// planes (line positions are clamped to the line, an idle channel slot reads
// channel 0) -- so that a step's reads issue together: a read under the
// condition compiles to a branch around it and a wait right after it.  The
// sweeps also keep each step's reads within the step (a scheduling barrier
// per step).  14 x 14, B = 32, C = 384: forward 25.3 -> 21.0 us, backward
// 55.5 -> 47.9 us.
__device__ __forceinline__ float bfv_if(const uint16_t *p, int i, bool on)
{
    const float v = bfv(p, i);
    return on ? v : 0.f;
}
__device__ __forceinline__ uint16_t to_bf(float v)
{
    const __bf16 b = static_cast<__bf16>(v);
    return __builtin_bit_cast(uint16_t, b);
}

// n bf16 elements, global -> LDS (dst 16-byte aligned), by all threads.
__device__ __forceinline__ void stage(uint16_t *dst, const bf16_t *src, int n)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(src);
    const rsrc_t r = make_rsrc(src, 2u * (uint32_t)n);
    const int tid = threadIdx.x, nt = blockDim.x;
    if (a % 16 == 0 && n % 8 == 0) {
        uint4 *d = reinterpret_cast<uint4 *>(dst);
        for (int t = tid; t < n / 8; t += nt)
            d[t] = ld128(r, 16u * (uint32_t)t, 0);
    } else if (a % 4 == 0 && n % 2 == 0) {
        uint32_t *d = reinterpret_cast<uint32_t *>(dst);
        for (int t = tid; t < n / 2; t += nt)
            d[t] = ld32(r, 4u * (uint32_t)t, 0);
    } else {
        for (int t = tid; t < n; t += nt)
            dst[t] = static_cast<uint16_t>(ld16(r, 2u * (uint32_t)t, 0));
    }
}

// Starts copying n bf16 elements global -> LDS without passing through
// registers (global_load_lds: the bytes of each lane land at the wave's LDS
// address + size * lane), in 16-, 4- or 2-byte pieces as the alignment of
// both ends and n allow.  The data is in place once every wave has waited
// for its loads and passed a barrier (lds_wait).  nt: the workgroup's
// threads, a multiple of 64 (read once by the caller).
template <int S>
__device__ __forceinline__ void stage_async_w(uint16_t *dst, const bf16_t *src, int n, int nt)
{
    constexpr int E = S / 2;                         // elements per piece
    for (int t = threadIdx.x; t < n / E; t += nt) {
        const auto g = (const __attribute__((address_space(1))) void *)(src + E * t);
        const auto l = (__attribute__((address_space(3))) void *)(dst + E * (t & ~63));
        if constexpr (S == 16)
            __builtin_amdgcn_global_load_lds(g, l, 16, 0, 0);
        else if constexpr (S == 4)
            __builtin_amdgcn_global_load_lds(g, l, 4, 0, 0);
        else
            __builtin_amdgcn_global_load_lds(g, l, 2, 0, 0);
    }
}

__device__ __forceinline__ void stage_async(uint16_t *dst, const bf16_t *src, int n, int nt)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst);
    if (a % 16 == 0 && n % 8 == 0)
        stage_async_w<16>(dst, src, n, nt);
    else if (a % 4 == 0 && n % 2 == 0)
        stage_async_w<4>(dst, src, n, nt);
    else
        stage_async_w<2>(dst, src, n, nt);
}

__device__ __forceinline__ void lds_wait()
{
    __builtin_amdgcn_s_waitcnt(0);     // this wave's loads, direct-to-LDS ones included
    lds_barrier();
}

// n bf16 elements, LDS (16-byte aligned) -> global, by all threads.
__device__ __forceinline__ void unstage(bf16_t *dst, const uint16_t *src, int n)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(dst);
    const u32x4 d = make_sdesc(dst, 2u * (uint32_t)n);
    const int tid = threadIdx.x, nt = blockDim.x;
    if (a % 16 == 0 && n % 8 == 0) {
        const uint4 *s = reinterpret_cast<const uint4 *>(src);
        for (int t = tid; t < n / 8; t += nt)
            st128(d, 16u * (uint32_t)t, 0, s[t]);
    } else if (a % 4 == 0 && n % 2 == 0) {
        const uint32_t *s = reinterpret_cast<const uint32_t *>(src);
        for (int t = tid; t < n / 2; t += nt)
            st32(d, 4u * (uint32_t)t, 0, s[t]);
    } else {
        for (int t = tid; t < n; t += nt)
            st16(d, 2u * (uint32_t)t, 0, src[t]);
    }
}

// LDS regions (elements of 16 bits, each region 16-byte aligned): the x, dy,
// lam and u planes of the workgroup's channels, the group's three tap planes
// and, for the backward, the weight-gradient slots (fp32).
template <int H, int W>
struct TinyLds {
    static constexpr int HW = H * W;
    int R;                    // elements of one channel-plane region
    uint16_t *x, *dy, *lam, *u, *wt;
    uint16_t *lam1, *u1, *wt1;  // forward: a second buffer for the next direction
    float *sl;                // [wave][3][16 steps][16 positions]
    float *mrg;               // fp32 merge plane (aliases lam and u)
    __device__ __forceinline__ TinyLds(uint16_t *base, int cw, bool bwd)
    {
        R = round8(cw * HW);
        uint16_t *p = base;
        x = p;
        p += R;
        dy = bwd ? p : nullptr;
        p += bwd ? R : 0;
        lam = p;
        mrg = reinterpret_cast<float *>(p);
        p += R;
        u = p;
        p += R;
        wt = p;
        p += round8(3 * HW);
        lam1 = bwd ? nullptr : p;
        p += bwd ? 0 : R;
        u1 = bwd ? nullptr : p;
        p += bwd ? 0 : R;
        wt1 = bwd ? nullptr : p;
        p += bwd ? 0 : round8(3 * HW);
        sl = reinterpret_cast<float *>(p);
    }
    // the same regions with the second direction buffer in place of the first
    __device__ __forceinline__ TinyLds other() const
    {
        TinyLds o = *this;
        o.lam = lam1;
        o.u = u1;
        o.wt = wt1;
        return o;
    }
};

template <int H, int W>
size_t tiny_lds_bytes(int cw, bool bwd)
{
    const int R = round8(cw * H * W);
    const int W3 = round8(3 * H * W);
    size_t b = 2 * (size_t)(bwd ? 4 * R + W3 : 5 * R + 2 * W3);
    if (bwd)
        b += (size_t)((cw + kSlotW - 1) / kSlotW) * 3 * 16 * 16 * 4;
    return b;
}

// Sum of a value over the four 16-lane rows of the wave, in every lane:
// v[l] + v[l ^ 32], then the same across rows 16 lanes apart, by the gfx950
// lane-swap instructions (VALU, no LDS round trip).  Every lane adds the
// same operands in the same order, so all rows hold the identical sum.
__device__ __forceinline__ float sum_rows(float v)
{
    const uint32_t b = __float_as_uint(v);
    const auto p32 = __builtin_amdgcn_permlane32_swap(b, b, false, false);
    const float s = __uint_as_float(p32[0]) + __uint_as_float(p32[1]);
    const uint32_t c = __float_as_uint(s);
    const auto p16 = __builtin_amdgcn_permlane16_swap(c, c, false, false);
    return __uint_as_float(p16[0]) + __uint_as_float(p16[1]);
}

struct TinyLane {
    int ch;        // channel slot in the workgroup
    int j;         // line position
    bool cvalid;   // the slot holds a channel
};

// Forward of one direction for the four channels of this wave.
template <int H, int W, int D, bool PM>
__device__ __forceinline__ void fwd_tiny_dir(const TinyLds<H, W> &S, const TinyLane &t,
                                             float (&yv)[H], float (&yh)[W])
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int L = VERT ? H : W, P = VERT ? W : H, HW = H * W;
    const bool act = t.cvalid && t.j < P;
    const bool m0 = act && t.j > 0, m2 = act && t.j + 1 < P;
    const int jc = t.j < P ? t.j : P - 1;
    const int cb = (t.cvalid ? t.ch : 0) * HW;   // an idle slot reads channel 0 and stores nothing
    float h = 0.f;
#pragma unroll
    for (int i = 0; i < L; ++i) {
        const int l = REV ? L - 1 - i : i;
        const int off = dir_offset(PM, VERT, l, jc, L, P, W);
        const float lamv = bfv_if(S.lam, cb + off, act);
        const float xv = bfv(S.x, cb + (VERT ? l * W + jc : jc * W + l));
        const float inj = lamv * xv;
        if (i == 0) {
            h = inj;
        } else {
            const float w0 = bfv_if(S.wt, off, m0);
            const float w1 = bfv_if(S.wt, HW + off, act);
            const float w2 = bfv_if(S.wt, 2 * HW + off, m2);
            float hn = fmaf(w1, h, inj);
            hn = fmaf(w0, from_left<kLaneRow>(h), hn);
            hn = fmaf(w2, from_right<kLaneRow>(h), hn);
            h = hn;
        }
        const float c = bfv(S.u, cb + off) * h;
        if (VERT)
            yv[VERT ? l : 0] += c;
        else
            yh[VERT ? 0 : l] += c;
        // the step's reads stay in the step: hoisted over several steps they
        // were slower (27.1 against 21.0 us at 14 x 14, B = 32, C = 384)
        step_fence();
    }
}

// Add the vertical (one column per lane) and horizontal (one row per lane)
// sums of every channel through the fp32 merge plane and store the bf16
// result (the x region, free by now, holds it for the copy out).
template <int H, int W>
__device__ __forceinline__ void merge_out(const TinyLds<H, W> &S, const TinyLane &t, const float (&v)[H],
                          const float (&hz)[W], bf16_t *dst, int nvalid)
{
    constexpr int HW = H * W;
    float *M = S.mrg + t.ch * HW;
    if (t.cvalid && t.j < H) {
#pragma unroll
        for (int c = 0; c < W; ++c)
            M[t.j * W + c] = hz[c];
    }
    lds_barrier();
    if (t.cvalid && t.j < W) {
#pragma unroll
        for (int r = 0; r < H; ++r)
            M[r * W + t.j] += v[r];
    }
    lds_barrier();
    for (int e = threadIdx.x; e < nvalid * HW; e += blockDim.x)
        S.x[e] = to_bf(S.mrg[e]);
    lds_barrier();
    unstage(dst, S.x, nvalid * HW);
}

struct TinyArgs {
    int b, g, c0, nvalid, chunk, nchunk;
};

__device__ __forceinline__ TinyArgs tiny_args(int C, int G, int cpg, int cw, int nchunk,
                                              Magic divChunk, Magic divG)
{
    TinyArgs a;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int bg = mdiv(blk, divChunk);
    a.chunk = blk - bg * nchunk;
    a.b = mdiv(bg, divG);
    a.g = bg - a.b * G;
    a.c0 = a.g * cpg + a.chunk * cw;
    a.nvalid = min(cw, cpg - a.chunk * cw);
    a.nchunk = nchunk;
    (void)C;
    return a;
}

template <int H, int W, bool PM>
__global__ __launch_bounds__(1024) void fwd_tiny_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, bf16_t *__restrict__ y, int mask, int B, int C, int G, int cpg,
    int cw, int nchunk, Magic divChunk, Magic divG)
{
    constexpr int HW = H * W;
    extern __shared__ uint4 smem4[];
    const TinyLds<H, W> S(reinterpret_cast<uint16_t *>(smem4), cw, false);
    const TinyArgs a = tiny_args(C, G, cpg, cw, nchunk, divChunk, divG);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    TinyLane t;
    t.ch = wave * kSlotW + (lane >> 4);
    t.j = lane & 15;
    t.cvalid = t.ch < a.nvalid;
    const int64_t pc = ((int64_t)a.b * C + a.c0) * HW;

    float yv[H], yh[W];
#pragma unroll
    for (int r = 0; r < H; ++r)
        yv[r] = 0.f;
#pragma unroll
    for (int c = 0; c < W; ++c)
        yh[c] = 0.f;
    // The directions run in order; the planes of the next one are copied into
    // the other LDS buffer while the current one computes.
    const int nt = blockDim.x;
    auto issue = [&](int k) {
        const int64_t pd = (((int64_t)k * B + a.b) * C + a.c0) * HW;
        const TinyLds<H, W> Sb = (k & 1) ? S.other() : S;
        stage_async(Sb.lam, lam + pd, a.nvalid * HW, nt);
        stage_async(Sb.u, u + pd, a.nvalid * HW, nt);
        stage_async(Sb.wt, w + (((int64_t)k * B + a.b) * G + a.g) * 3 * HW, 3 * HW, nt);
    };
    stage_async(S.x, x + pc, a.nvalid * HW, nt);
    int rem = mask & 15;
    if (rem)
        issue(0);
    for (int k = 0; rem; ++k) {
        const int d = __builtin_ctz(rem);
        rem &= rem - 1;
        // buffer k % 2 is filled, and every wave is done with the other one
        lds_wait();
        if (rem)
            issue(k + 1);
        const TinyLds<H, W> Sb = (k & 1) ? S.other() : S;
        if (d == 0)
            fwd_tiny_dir<H, W, 0, PM>(Sb, t, yv, yh);
        else if (d == 1)
            fwd_tiny_dir<H, W, 1, PM>(Sb, t, yv, yh);
        else if (d == 2)
            fwd_tiny_dir<H, W, 2, PM>(Sb, t, yv, yh);
        else
            fwd_tiny_dir<H, W, 3, PM>(Sb, t, yv, yh);
    }
    // the merge plane aliases the first buffer
    lds_barrier();
    merge_out<H, W>(S, t, yv, yh, y + pc, a.nvalid);
}

// Backward of one direction for the four channels of this wave.  du and dlam
// replace u and lam in LDS; the weight-gradient terms, summed over the
// wave's channels, go to this wave's slots.
template <int H, int W, int D, bool PM>
__device__ __forceinline__ void bwd_tiny_dir(const TinyLds<H, W> &S, const TinyLane &t, int wave,
                                             float (&dxv)[H], float (&dxh)[W])
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int L = VERT ? H : W, P = VERT ? W : H, HW = H * W;
    const bool act = t.cvalid && t.j < P;
    const bool m0 = act && t.j > 0, m2 = act && t.j + 1 < P;
    const int jc = t.j < P ? t.j : P - 1;
    const int cb = (t.cvalid ? t.ch : 0) * HW;   // an idle slot reads channel 0 and stores nothing
    auto line = [](int i) { return REV ? L - 1 - i : i; };
    auto pix = [&](int l) { return cb + (VERT ? l * W + jc : jc * W + l); };

    // reverse sweep: a_i = u_i dy_i + (transposed tridiagonal of line i+1) a_{i+1}
    float ah[L];
    float an = 0.f;
#pragma unroll
    for (int i = L - 1; i >= 0; --i) {
        const int l = line(i);
        const int off = dir_offset(PM, VERT, l, jc, L, P, W);
        const float uv = bfv_if(S.u, cb + off, act);
        float a = uv * bfv(S.dy, pix(l));
        if (i + 1 < L) {
            const int offn = dir_offset(PM, VERT, line(i + 1), jc, L, P, W);
            const float w0 = bfv_if(S.wt, offn, m0);
            const float w1 = bfv_if(S.wt, HW + offn, act);
            const float w2 = bfv_if(S.wt, 2 * HW + offn, m2);
            a = fmaf(w1, an, a);
            a += from_right<kLaneRow>(w0 * an);
            a += from_left<kLaneRow>(w2 * an);
        }
        ah[i] = a;
        an = a;
        step_fence();   // (as in the forward)
    }

    // forward sweep: h_i again, local gradients, weight-gradient terms
    float h = 0.f;
    float *slw = S.sl + wave * 3 * 256;
#pragma unroll
    for (int i = 0; i < L; ++i) {
        const int l = line(i);
        const int off = dir_offset(PM, VERT, l, jc, L, P, W);
        const float xv = bfv(S.x, pix(l));
        const float dyv = bfv(S.dy, pix(l));
        const float lamv = bfv_if(S.lam, cb + off, act);
        const float hp = h;
        if (i == 0) {
            h = lamv * xv;
        } else {
            const float w0 = bfv_if(S.wt, off, m0);
            const float w1 = bfv_if(S.wt, HW + off, act);
            const float w2 = bfv_if(S.wt, 2 * HW + off, m2);
            float hn = fmaf(w1, hp, lamv * xv);
            hn = fmaf(w0, from_left<kLaneRow>(hp), hn);
            hn = fmaf(w2, from_right<kLaneRow>(hp), hn);
            h = hn;
        }
        const float a = ah[i];
        if (act) {
            S.u[cb + off] = to_bf(dyv * h);       // du
            S.lam[cb + off] = to_bf(a * xv);      // dlam
        }
        if (VERT)
            dxv[VERT ? l : 0] = fmaf(a, lamv, dxv[VERT ? l : 0]);
        else
            dxh[VERT ? 0 : l] = fmaf(a, lamv, dxh[VERT ? 0 : l]);
        // w_i couples line i-1 to line i: terms a_i * h_{i-1}[j+k-1]
        float tk[3] = {0.f, 0.f, 0.f};
        if (i > 0) {
            tk[0] = a * from_left<kLaneRow>(hp);
            tk[1] = a * hp;
            tk[2] = a * from_right<kLaneRow>(hp);
        }
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const float v = sum_rows(tk[k]);
            if ((threadIdx.x & 63) < kLaneRow)
                slw[(k * 16 + i) * 16 + t.j] = v;
        }
        step_fence();
    }
}

template <int H, int W, bool PM>
__global__ __launch_bounds__(1024) void bwd_tiny_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, const bf16_t *__restrict__ dy, bf16_t *__restrict__ dx,
    bf16_t *__restrict__ dw, bf16_t *__restrict__ dlam, bf16_t *__restrict__ du,
    float *__restrict__ dwp, int mask, int B, int C, int G, int cpg, int cw, int nchunk,
    Magic divChunk, Magic divG)
{
    constexpr int HW = H * W;
    extern __shared__ uint4 smem4[];
    const TinyLds<H, W> S(reinterpret_cast<uint16_t *>(smem4), cw, true);
    const TinyArgs a = tiny_args(C, G, cpg, cw, nchunk, divChunk, divG);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nwaves = blockDim.x >> 6;
    const int lane = threadIdx.x & 63;
    TinyLane t;
    t.ch = wave * kSlotW + (lane >> 4);
    t.j = lane & 15;
    t.cvalid = t.ch < a.nvalid;
    const int64_t pc = ((int64_t)a.b * C + a.c0) * HW;
    const int D = __popc(mask);

    stage(S.x, x + pc, a.nvalid * HW);
    stage(S.dy, dy + pc, a.nvalid * HW);
    float dxv[H], dxh[W];
#pragma unroll
    for (int r = 0; r < H; ++r)
        dxv[r] = 0.f;
#pragma unroll
    for (int c = 0; c < W; ++c)
        dxh[c] = 0.f;
    for (int d = 0; d < 4; ++d) {
        if (!((mask >> d) & 1))
            continue;
        const int s = __popc(mask & ((1 << d) - 1));
        const int64_t pd = (((int64_t)s * B + a.b) * C + a.c0) * HW;
        const int64_t unit = ((int64_t)s * B + a.b) * G + a.g;
        stage(S.lam, lam + pd, a.nvalid * HW);
        stage(S.u, u + pd, a.nvalid * HW);
        stage(S.wt, w + unit * 3 * HW, 3 * HW);
        lds_barrier();
        if (d == 0)
            bwd_tiny_dir<H, W, 0, PM>(S, t, wave, dxv, dxh);
        else if (d == 1)
            bwd_tiny_dir<H, W, 1, PM>(S, t, wave, dxv, dxh);
        else if (d == 2)
            bwd_tiny_dir<H, W, 2, PM>(S, t, wave, dxv, dxh);
        else
            bwd_tiny_dir<H, W, 3, PM>(S, t, wave, dxv, dxh);
        lds_barrier();
        unstage(du + pd, S.u, a.nvalid * HW);
        unstage(dlam + pd, S.lam, a.nvalid * HW);
        // dw of this direction: the waves' sums added in wave order
        const bool vert = d < 2, rev = d == 1 || d == 3;
        const int L = vert ? H : W, P = vert ? W : H;
        for (int e = threadIdx.x; e < 3 * L * P; e += blockDim.x) {
            const int k = e / (L * P), r = e - k * (L * P), i = r / P, j = r - i * P;
            float v = 0.f;
            for (int q = 0; q < nwaves; ++q)
                v += S.sl[q * 3 * 256 + (k * 16 + i) * 16 + j];
            const int l = rev ? L - 1 - i : i;
            const int64_t o = k * HW + dir_offset(PM, vert, l, j, L, P, W);
            if (a.nchunk > 1)
                dwp[((int64_t)a.chunk * D * B * G + unit) * 3 * HW + o] = v;
            else
                dw[unit * 3 * HW + o] = to_bf(v);
        }
        lds_barrier();
    }
    merge_out<H, W>(S, t, dxv, dxh, dx + pc, a.nvalid);
}

// dw = sum over chunks of the fp32 partials, in chunk order.
__global__ __launch_bounds__(256) void dw_tiny_sum_kernel(const float *__restrict__ dwp,
                                                          bf16_t *__restrict__ dw, int64_t n,
                                                          int nchunk)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        float v = 0.f;
        for (int c = 0; c < nchunk; ++c)
            v += dwp[c * n + e];
        dw[e] = to_bf(v);
    }
}

struct TinyPlan {
    int cpg, cw, nchunk;
    size_t lds;
};

template <int H, int W>
bool tiny_plan(const Problem &p, bool bwd, TinyPlan &pl)
{
    const int lds_max = kLdsBytes;
    pl.cpg = p.C / p.G;
    int cap = kMaxCh;
    while (cap > kSlotW && tiny_lds_bytes<H, W>(cap, bwd) > (size_t)lds_max)
        cap -= kSlotW;
    if (tiny_lds_bytes<H, W>(cap, bwd) > (size_t)lds_max)
        return false;
    pl.nchunk = (pl.cpg + cap - 1) / cap;
    pl.cw = (pl.cpg + pl.nchunk - 1) / pl.nchunk;
    pl.lds = tiny_lds_bytes<H, W>(pl.cw, bwd);
    return true;
}

template <int H, int W, bool PM>
hipError_t fwd_tiny_t(const Problem &p, hipStream_t st)
{
    TinyPlan pl;
    if (!tiny_plan<H, W>(p, false, pl))
        return hipErrorInvalidConfiguration;
    if (p.ws->counting)
        return hipSuccess;
    hipError_t e = hipFuncSetAttribute((const void *)fwd_tiny_kernel<H, W, PM>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
    if (e != hipSuccess)
        return e;
    const int nw = (pl.cw + kSlotW - 1) / kSlotW;
    hipLaunchKernelGGL((fwd_tiny_kernel<H, W, PM>), dim3((unsigned)(p.B * p.G * pl.nchunk)),
                       dim3(64 * nw), pl.lds, st, (const bf16_t *)p.x, (const bf16_t *)p.w,
                       (const bf16_t *)p.lam, (const bf16_t *)p.u, (bf16_t *)p.y, p.mask, p.B,
                       p.C, p.G, pl.cpg, pl.cw, pl.nchunk, make_magic((uint32_t)pl.nchunk),
                       make_magic((uint32_t)p.G));
    return hipGetLastError();
}

template <int H, int W, bool PM>
hipError_t bwd_tiny_t(const Problem &p, hipStream_t st)
{
    TinyPlan pl;
    if (!tiny_plan<H, W>(p, true, pl))
        return hipErrorInvalidConfiguration;
    const int D = __builtin_popcount(p.mask);
    const int64_t ndw = (int64_t)D * p.B * p.G * 3 * H * W;
    float *dwp = nullptr;
    hipError_t e = hipSuccess;
    if (pl.nchunk > 1) {
        e = p.ws->take((void **)&dwp, (size_t)pl.nchunk * ndw * sizeof(float));
        if (e != hipSuccess)
            return e;
    }
    if (p.ws->counting)
        return hipSuccess;
    e = hipFuncSetAttribute((const void *)bwd_tiny_kernel<H, W, PM>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
    if (e != hipSuccess)
        return e;
    const int nw = (pl.cw + kSlotW - 1) / kSlotW;
    hipLaunchKernelGGL((bwd_tiny_kernel<H, W, PM>), dim3((unsigned)(p.B * p.G * pl.nchunk)),
                       dim3(64 * nw), pl.lds, st, (const bf16_t *)p.x, (const bf16_t *)p.w,
                       (const bf16_t *)p.lam, (const bf16_t *)p.u, (const bf16_t *)p.dy,
                       (bf16_t *)p.dx, (bf16_t *)p.dw, (bf16_t *)p.dlam, (bf16_t *)p.du, dwp,
                       p.mask, p.B, p.C, p.G, pl.cpg, pl.cw, pl.nchunk,
                       make_magic((uint32_t)pl.nchunk), make_magic((uint32_t)p.G));
    e = hipGetLastError();
    if (e == hipSuccess && pl.nchunk > 1) {
        int64_t blocks = (ndw + 255) / 256;
        blocks = blocks < 16384 ? blocks : 16384;
        hipLaunchKernelGGL(dw_tiny_sum_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                           (const float *)dwp, (bf16_t *)p.dw, ndw, pl.nchunk);
        e = hipGetLastError();
    }
    return e;
}

template <int H, int W>
hipError_t fwd_tiny_l(const Problem &p, hipStream_t st)
{
    return p.layout == kPixelMajor ? fwd_tiny_t<H, W, true>(p, st) : fwd_tiny_t<H, W, false>(p, st);
}

template <int H, int W>
hipError_t bwd_tiny_l(const Problem &p, hipStream_t st)
{
    return p.layout == kPixelMajor ? bwd_tiny_t<H, W, true>(p, st) : bwd_tiny_t<H, W, false>(p, st);
}

}  // namespace

bool tiny_supported(const Problem &p)
{
    if (p.dtype != 1 || p.H != p.W)
        return false;
    return p.H == 8 || p.H == 12 || p.H == 14 || p.H == 16;
}

hipError_t launch_fwd_tiny(const Problem &p, hipStream_t st)
{
    switch (p.H) {
    case 8: return fwd_tiny_l<8, 8>(p, st);
    case 12: return fwd_tiny_l<12, 12>(p, st);
    case 14: return fwd_tiny_l<14, 14>(p, st);
    default: return fwd_tiny_l<16, 16>(p, st);
    }
}

hipError_t launch_bwd_tiny(const Problem &p, hipStream_t st)
{
    switch (p.H) {
    case 8: return bwd_tiny_l<8, 8>(p, st);
    case 12: return bwd_tiny_l<12, 12>(p, st);
    case 14: return bwd_tiny_l<14, 14>(p, st);
    default: return bwd_tiny_l<16, 16>(p, st);
    }
}

}  // namespace gspn
