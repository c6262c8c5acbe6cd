// Line scans for bf16 planes of a compile-time shape (H, W <= 64, multiples
// of 8), with per-direction tensors in line-major layout (every scanned line
// contiguous) and x, y, dx, dy pixel-major.
//
// Lane layout: one lane per position of a line (the perpendicular axis), one
// line per wave, h in a VGPR for the whole scan, DPP for the two neighbours of
// the tridiagonal step (Sec. 3, Eq. (gspn_recurrence)).  bf16 is widened with
// one v_perm_b32 whose per-lane selector also zeroes the taps that leave the
// grid, so ignored taps may hold any value.
//
// Every global access reads or writes whole 128-byte lines: on this GPU the
// cost of a load is set by the lines it touches, not by its bytes, so a
// per-lane 16-byte access that straddles 64 different lines runs at a sixth
// of the bandwidth of a coalesced one.
//
// Forward (one workgroup = one channel plane, one wave per direction):
//  * the x plane is loaded once, coalesced, into LDS and read from there by
//    all four directions (rows for vertical scans, columns for horizontal);
//  * each wave streams its lam, u and w lines in blocks of 8 lines with
//    16-byte coalesced loads (two blocks in flight in registers) and turns a
//    block around through a small per-wave LDS buffer, one bf16 per lane per
//    line;
//  * u_d * h_d stays in registers; the four directions are summed in
//    direction-bit order through an fp32 LDS plane and y is stored once.
//
// Backward (one workgroup = `cw` channels of one weight group, one wave per
// channel, directions one after another, waves in lock-step):
//  * horizontal directions first: each wave loads its x and dy planes
//    coalesced, turns them around through its own LDS dx plane (still free)
//    into registers holding its row, then scans;
//  * vertical directions read x and dy rows directly;
//  * per direction a reverse sweep computes the adjoint a_i (kept in
//    registers), then a forward sweep recomputes h_i and forms du, dlam, dx
//    (an fp32 LDS plane per channel) and the weight-gradient terms
//    a_i * h_{i-1}[j+k-1], summed over the workgroup's channels through LDS
//    once per step; when a group spans several workgroups the sums go to
//    fp32 partials that a second kernel adds in fixed order.
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

constexpr uint32_t kSelLo = 0x01000C0Cu;   // bf16 in bits [15:0]  -> fp32
constexpr uint32_t kSelHi = 0x03020C0Cu;   // bf16 in bits [31:16] -> fp32
constexpr uint32_t kSelZero = 0x0C0C0C0Cu; // -> +0.0f
constexpr int kYPitch = 68;                // fp32 LDS row pitch (16-byte rows, conflict-free b128)
constexpr int kDxPitch = 65;               // fp32 LDS row pitch for per-step dx (odd: column walks conflict-free)
constexpr int kPrefetch = 8;               // steps of per-step loads in flight (backward)

// Keep the software pipeline as written: nothing is scheduled across a step
// boundary, so each step's prefetch stays kPrefetch steps ahead of its use
// instead of every load of the unrolled scan being hoisted to the top.
__device__ __forceinline__ void step_fence() { __builtin_amdgcn_sched_barrier(0); }

// Workgroup barrier that orders LDS only.  __syncthreads() also orders global
// memory, which makes every wave drain its prefetched loads at each barrier.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Raw buffer access: a uniform descriptor per tensor plane (SGPRs), one
// per-lane byte offset (VGPR) and a uniform per-step offset (SGPR), so no
// 64-bit per-lane addresses are formed.
using rsrc_t = __amdgpu_buffer_rsrc_t;
constexpr int kRsrcWord3 = 0x00020000;   // gfx9 raw buffer: 32-bit data format, no swizzle

// The base address is passed through readfirstlane: every caller's pointer
// is wave-uniform, and saying so keeps the compiler from wrapping each buffer
// access in a loop over distinct descriptors.
__device__ __forceinline__ rsrc_t make_rsrc(const void *p, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
    void *q = reinterpret_cast<void *>((static_cast<uint64_t>(hi) << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(q, (short)0,
                                             (int)__builtin_amdgcn_readfirstlane(bytes),
                                             kRsrcWord3);
}
__device__ __forceinline__ uint32_t ld16(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
__device__ __forceinline__ uint4 ld128(rsrc_t r, uint32_t voff, uint32_t soff)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void st16(rsrc_t r, uint32_t voff, uint32_t soff, uint16_t v)
{
    __builtin_amdgcn_raw_buffer_store_b16(v, r, voff, soff, 0);
}
__device__ __forceinline__ void st32f(rsrc_t r, uint32_t voff, uint32_t soff, float v)
{
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, voff, soff, 0);
}
__device__ __forceinline__ void st128(rsrc_t r, uint32_t voff, uint32_t soff, uint4 v)
{
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    u4 t = {v.x, v.y, v.z, v.w};
    __builtin_amdgcn_raw_buffer_store_b128(t, r, voff, soff, 0);
}

__device__ __forceinline__ float widen(uint32_t v, uint32_t sel)
{
    return __uint_as_float(__builtin_amdgcn_perm(0u, v, sel));
}
__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

__device__ __forceinline__ uint32_t pack2(float lo, float hi)
{
    typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
    bf2 p;
    p.x = static_cast<__bf16>(lo);
    p.y = static_cast<__bf16>(hi);
    return __builtin_bit_cast(uint32_t, p);
}
__device__ __forceinline__ uint16_t pack1(float v)
{
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

template <int K>
__device__ __forceinline__ uint32_t comp(const uint4 &v)
{
    static_assert(K >= 0 && K < 4, "component");
    return K == 0 ? v.x : (K == 1 ? v.y : (K == 2 ? v.z : v.w));
}

// Element E (0..7) of a 16-byte chunk of 8 bf16, widened with the selector
// pair (lo, hi) of the lane.
template <int E>
__device__ __forceinline__ float elem(const uint4 &v, uint32_t sel_lo, uint32_t sel_hi)
{
    return widen(comp<E / 2>(v), (E & 1) ? sel_hi : sel_lo);
}
template <int E>
__device__ __forceinline__ float elem(const uint4 &v)
{
    return (E & 1) ? bf_hi(comp<E / 2>(v)) : bf_lo(comp<E / 2>(v));
}

// Workgroups go to the 8 XCDs round-robin by blockIdx.  Give each XCD a
// contiguous range of logical ids so that neighbouring channels -- which
// share a weight group's w -- run under one L2.
__device__ __forceinline__ int xcd_remap(int bid, int n)
{
    constexpr int X = 8;
    const int q = n / X, r = n % X;
    const int xcd = bid % X, k = bid / X;
    return xcd < r ? xcd * (q + 1) + k : r * (q + 1) + (xcd - r) * q + k;
}

struct Sel {
    uint32_t lo0, lo1, lo2, hi0, hi1, hi2;   // taps 0/1/2 (1 also gates lam, u)
};

__device__ __forceinline__ Sel make_sel(int j, int P)
{
    const bool act = j < P;
    const bool v0 = act && j > 0;
    const bool v2 = act && j + 1 < P;
    Sel s;
    s.lo0 = v0 ? kSelLo : kSelZero;
    s.hi0 = v0 ? kSelHi : kSelZero;
    s.lo1 = act ? kSelLo : kSelZero;
    s.hi1 = act ? kSelHi : kSelZero;
    s.lo2 = v2 ? kSelLo : kSelZero;
    s.hi2 = v2 ? kSelHi : kSelZero;
    return s;
}

// One tridiagonal step: h_i = w0 h_{i-1}[j-1] + w1 h_{i-1}[j] + w2 h_{i-1}[j+1] + inj.
__device__ __forceinline__ float tri_step(float h, float w0, float w1, float w2, float inj)
{
    float hn = fmaf(w1, h, inj);
    hn = fmaf(w0, from_left<64>(h), hn);
    hn = fmaf(w2, from_right<64>(h), hn);
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

__device__ __forceinline__ uint32_t lds_u16(const uint8_t *base, uint32_t byte_off)
{
    return *reinterpret_cast<const uint16_t *>(base + byte_off);
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------

// One direction's scan over one channel plane.  D: direction index (0 T2B,
// 1 B2T, 2 L2R, 3 R2L).  lam, u: line-major channel planes; w: the 3 tap
// planes; xs: the bf16 x plane in LDS; blk: this wave's block buffer
// (5 tensors x 8 lines x P bf16).
template <int H, int W, int D>
__device__ __forceinline__ void scan_fwd_dir(int j, rsrc_t lam, rsrc_t u, rsrc_t w,
                                             const uint8_t *xs, uint8_t *blk, float (&yr)[64])
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int L = VERT ? H : W, P = VERT ? W : H;
    constexpr int NB = L / 8;                 // blocks of 8 lines
    constexpr uint32_t TB = 16 * P;           // bytes of one tensor in one block
    constexpr uint32_t PL = 2 * H * W;        // bytes of one plane
    const Sel s = make_sel(j, P);
    const int jc = j < P ? j : P - 1;
    const bool ld = j < P;                    // lanes that load a 16-byte piece of a block
    const uint32_t vo = 16u * (uint32_t)(ld ? j : 0);
    // block b covers lines [8b', 8b'+8) with b' = b (forward) or NB-1-b (reverse)
    auto boff = [](int b) -> uint32_t { return TB * (uint32_t)(REV ? NB - 1 - b : b); };
    uint4 rl[NB], ru[NB], r0[NB], r1[NB], r2[NB];
#define FLOAD(b)                                                     \
    do {                                                             \
        const uint32_t so_ = boff(b);                                \
        rl[b] = ld128(lam, vo, so_);                                 \
        ru[b] = ld128(u, vo, so_);                                   \
        r0[b] = ld128(w, vo, so_);                                   \
        r1[b] = ld128(w, vo, so_ + PL);                              \
        r2[b] = ld128(w, vo, so_ + 2 * PL);                          \
    } while (0)
    FLOAD(0);
    if (NB > 1)
        FLOAD(1);
    float h = 0.f;
    uint4 *bw = reinterpret_cast<uint4 *>(blk) + j;   // this lane's 16-byte slot
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        // turn block b around: lane j wrote piece j of each tensor's 8 lines
        if (ld) {
            bw[0 * TB / 16] = rl[b];
            bw[1 * TB / 16] = ru[b];
            bw[2 * TB / 16] = r0[b];
            bw[3 * TB / 16] = r1[b];
            bw[4 * TB / 16] = r2[b];
        }
        if (b + 2 < NB)
            FLOAD(b + 2);
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * b + t;
            const int ln = REV ? 7 - t : t;                     // line within the block
            const uint32_t lo = 2u * (uint32_t)(ln * P + jc);   // this lane's bf16 in a tensor's block
            const float lv = widen(lds_u16(blk, lo), s.lo1);
            const float uv = bf_lo(lds_u16(blk, TB + lo));
            const int row = VERT ? (REV ? H - 1 - i : i) : jc;
            const int col = VERT ? jc : (REV ? W - 1 - i : i);
            const float xv = bf_lo(lds_u16(xs, row * XPlane<W>::kPitchB + 2 * col));
            const float inj = lv * xv;
            if (i == 0)
                h = inj;
            else
                h = tri_step(h, widen(lds_u16(blk, 2 * TB + lo), s.lo0),
                             widen(lds_u16(blk, 3 * TB + lo), s.lo1),
                             widen(lds_u16(blk, 4 * TB + lo), s.lo2), inj);
            yr[i] = uv * h;
        }
        step_fence();
    }
#undef FLOAD
}

template <int H, int W>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void fwd_med_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, bf16_t *__restrict__ y, int mask, int B, int C, int G)
{
    static_assert(H <= 64 && W <= 64 && H % 8 == 0 && W % 8 == 0, "shape");
    constexpr int HW = H * W;
    constexpr int XB = H * XPlane<W>::kPitchB;              // x plane bytes
    constexpr int PMAX = H > W ? H : W;
    constexpr int BLK = 5 * 16 * PMAX;                      // block buffer bytes per wave
    constexpr int YB = H * kYPitch * 4;                     // merge plane bytes
    static_assert(YB <= 4 * BLK, "merge plane reuses the block buffers");
    __shared__ float4 lds4[(XB + 4 * BLK + 15) / 16];
    uint8_t *lds = reinterpret_cast<uint8_t *>(lds4);
    uint8_t *xs = lds;
    uint8_t *blks = lds + (XB + 15) / 16 * 16;
    float4 *Y4 = reinterpret_cast<float4 *>(blks);           // after the scans
    float *Y = reinterpret_cast<float *>(Y4);

    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int b = blk / C;
    const int c = blk - b * C;
    const int g = c / (C / G);
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
        uint8_t *myblk = blks + d * BLK;
        if (d == 0)
            scan_fwd_dir<H, W, 0>(lane, rl, ru, rw, xs, myblk, yr);
        else if (d == 1)
            scan_fwd_dir<H, W, 1>(lane, rl, ru, rw, xs, myblk, yr);
        else if (d == 2)
            scan_fwd_dir<H, W, 2>(lane, rl, ru, rw, xs, myblk, yr);
        else
            scan_fwd_dir<H, W, 3>(lane, rl, ru, rw, xs, myblk, yr);
    }
    lds_barrier();   // block buffers become the merge plane

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
                        *a = st ? yr[i] : *a + yr[i];
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
                        a0 = make_float4(o0.x + a0.x, o0.y + a0.y, o0.z + a0.z, o0.w + a0.w);
                        a1 = make_float4(o1.x + a1.x, o1.y + a1.y, o1.z + a1.z, o1.w + a1.w);
                    }
                    a[0] = a0;
                    a[1] = a1;
                }
            }
        }
        lds_barrier();
    }

    const rsrc_t yo = make_rsrc(y + pc, 2 * HW);
    for (int t = threadIdx.x; t < H * (W / 8); t += 256) {
        const int r = t / (W / 8);
        const int cm = t - r * (W / 8);
        const float4 a0 = Y4[(r * kYPitch + 8 * cm) / 4];
        const float4 a1 = Y4[(r * kYPitch + 8 * cm) / 4 + 1];
        st128(yo, 16u * t, 0, make_uint4(pack2(a0.x, a0.y), pack2(a0.z, a0.w), pack2(a1.x, a1.y),
                                         pack2(a1.z, a1.w)));
    }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------

struct BwdArgs {
    rsrc_t x, dy;          // channel planes (pixel-major)
    rsrc_t lam, u;         // direction planes (line-major)
    rsrc_t w;              // the 3 tap planes of (direction, group)
    rsrc_t dlam, du;       // direction planes
    rsrc_t dw;             // 3 tap planes: final bf16 dw or fp32 partial
    float *Xq;             // this wave's dx plane in LDS, [H][kDxPitch]
    float *slots;          // [2][cw][3][64] per-step dw terms
    int wave, nwaves, nvalid, cw;
    bool partial;          // dw holds fp32 partials
    bool first;            // first direction processed: store dx, don't add
};

// Per-step dw terms live in LDS as slots[buf][k][q][j] (q = channel slot of
// the workgroup, 8 slots, absent channels zero): a wave writes one
// contiguous row per tap and a reducing lane reads its 8 slots, all
// conflict-free.
constexpr int kSlots = 8;   // channel slots per (tap, position)

__device__ __forceinline__ float *slot_ptr(float *slots, int buf, int k, int q)
{
    return slots + ((buf * 3 + k) * kSlots + q) * 64;
}

// While the horizontal directions run, a wave's LDS dx plane holds x and dy
// interleaved: one dword per pixel (x in bits [15:0], dy in [31:16]) at row
// pitch kDxPitch, so one conflict-free read per step returns both.
__device__ __forceinline__ uint32_t lds_u32(const uint8_t *base, uint32_t byte_off)
{
    return *reinterpret_cast<const uint32_t *>(base + byte_off);
}

// One direction of the backward.  D: direction index.  Horizontal directions
// read x and dy from the staged planes `stg` (x then dy, bf16, odd pitch) and
// add their dx terms to dxr (this lane's row); vertical directions read x
// and dy rows from global memory and add dx into the LDS dx plane.
template <int H, int W, int D>
__device__ __forceinline__ void dir_bwd(const BwdArgs &A, int j, bool cvalid, const uint8_t *stg,
                                        float (&dxr)[64], bool dx_first)
{
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int L = VERT ? H : W, P = VERT ? W : H;
    constexpr uint32_t PL2 = 2 * H * W;                  // bytes of one bf16 plane
    const Sel s = make_sel(cvalid ? j : 64, P);          // an idle wave computes zeros
    const bool act = cvalid && j < P;
    const int jj = j < P ? j : P - 1;
    const uint32_t vo = 2u * (uint32_t)jj;               // line-major lane offset (bf16)
    // line-major byte offset of line(i); pixel offset of a vertical row
    auto lnoff = [](int i) -> uint32_t { return 2u * (uint32_t)((REV ? L - 1 - i : i) * P); };
    auto col_of = [](int i) { return REV ? L - 1 - i : i; };   // storage row/col scanned at step i

    // --- reverse sweep: adjoint a_i -------------------------------------
    float ahist[L];
    uint32_t pdy[VERT ? L / 2 : 1];
    {
        uint32_t ru[L], rd[VERT ? L : 1], r0[L], r1[L], r2[L];
#define ALOAD(i)                                                     \
    do {                                                             \
        const uint32_t so_ = lnoff(i);                               \
        ru[i] = ld16(A.u, vo, so_);                                  \
        if (VERT)                                                    \
            rd[VERT ? (i) : 0] = ld16(A.dy, vo, so_);                \
        if ((i) + 1 < L) {                                           \
            const uint32_t sn_ = lnoff((i) + 1);                     \
            r0[i] = ld16(A.w, vo, sn_);                              \
            r1[i] = ld16(A.w, vo, sn_ + PL2);                        \
            r2[i] = ld16(A.w, vo, sn_ + 2 * PL2);                    \
        }                                                            \
    } while (0)
#pragma unroll
        for (int i = L - 1; i >= L - kPrefetch && i >= 0; --i)
            ALOAD(i);
        float an = 0.f;
        // horizontal directions: the staged (x, dy) dword of the next step is
        // read one step ahead so its LDS latency overlaps the arithmetic
        auto stg_at = [&](int i) { return lds_u32(stg, 4u * (uint32_t)(jj * kDxPitch + col_of(i))); };
        uint32_t xd_next = VERT ? 0u : stg_at(L - 1);
#pragma unroll
        for (int i = L - 1; i >= 0; --i) {
            if (i - kPrefetch >= 0)
                ALOAD(i - kPrefetch);
            float dyv;
            if (VERT) {
                dyv = bf_lo(rd[VERT ? i : 0]);
            } else {
                dyv = bf_hi(xd_next);
                if (i > 0)
                    xd_next = stg_at(i - 1);
            }
            const float inj = widen(ru[i], s.lo1) * dyv;
            float a;
            if (i + 1 == L)
                a = inj;
            else
                a = tri_step_t(an, widen(r0[i], s.lo0), widen(r1[i], s.lo1), widen(r2[i], s.lo2),
                               inj);
            ahist[i] = a;
            an = a;
            if (VERT && (i & 1) == 0)
                pdy[VERT ? i >> 1 : 0] =
                    __builtin_amdgcn_perm(rd[VERT ? i + 1 : 0], rd[VERT ? i : 0], 0x05040100u);
            step_fence();
        }
#undef ALOAD
    }

    // --- forward sweep: states, local gradients, dw terms ---------------
    uint32_t rx[VERT ? L : 1], rl[L], r0[L], r1[L], r2[L];
#define BLOAD(i)                                                     \
    do {                                                             \
        const uint32_t so_ = lnoff(i);                               \
        if (VERT)                                                    \
            rx[VERT ? (i) : 0] = ld16(A.x, vo, so_);                 \
        rl[i] = ld16(A.lam, vo, so_);                                \
        if ((i) > 0) {                                               \
            r0[i] = ld16(A.w, vo, so_);                              \
            r1[i] = ld16(A.w, vo, so_ + PL2);                        \
            r2[i] = ld16(A.w, vo, so_ + 2 * PL2);                    \
        }                                                            \
    } while (0)
#pragma unroll
    for (int i = 0; i < kPrefetch && i < L; ++i)
        BLOAD(i);
    // Reduction of the dw terms of line i over the workgroup's channels:
    // wave k (< 3) owns tap k.  Its eight slot reads are issued right after
    // the barrier and summed one step later, in channel order.  With fewer
    // than three waves the remaining taps are summed at once by wave 0.
    float pr[kSlots];
    auto store_dw = [&](int i, int k, float v) {
        const uint32_t so = lnoff(i);
        if (j < P) {
            if (A.partial)
                st32f(A.dw, 2u * vo, 2u * (so + k * PL2), v);
            else
                st16(A.dw, vo, so + k * PL2, pack1(v));
        }
    };
    auto issue_dw = [&](int i) {
        if (A.wave < 3) {
#pragma unroll
            for (int q = 0; q < kSlots; ++q)
                pr[q] = slot_ptr(A.slots, i & 1, A.wave, q)[j];
        }
        if (A.nwaves < 3 && A.wave == 0) {
            for (int k = A.nwaves; k < 3; ++k) {
                float sum = 0.f;
                for (int q = 0; q < kSlots; ++q)
                    sum += slot_ptr(A.slots, i & 1, k, q)[j];
                store_dw(i, k, sum);
            }
        }
    };
    auto flush_dw = [&](int i) {
        if (A.wave < 3) {
            float sum = 0.f;
#pragma unroll
            for (int q = 0; q < kSlots; ++q)
                sum += pr[q];
            store_dw(i, A.wave, sum);
        }
    };
    float h = 0.f;
    auto stg_at = [&](int i) { return lds_u32(stg, 4u * (uint32_t)(jj * kDxPitch + col_of(i))); };
    uint32_t xd_next = VERT ? 0u : stg_at(0);
#pragma unroll
    for (int i = 0; i < L; ++i) {
        if (i + kPrefetch < L)
            BLOAD(i + kPrefetch);
        float xv, dyv;
        if (VERT) {
            xv = bf_lo(rx[VERT ? i : 0]);
            dyv = (i & 1) ? bf_hi(pdy[VERT ? i >> 1 : 0]) : bf_lo(pdy[VERT ? i >> 1 : 0]);
        } else {
            const uint32_t xd = xd_next;
            if (i + 1 < L)
                xd_next = stg_at(i + 1);
            xv = bf_lo(xd);
            dyv = bf_hi(xd);
        }
        const float lv = widen(rl[i], s.lo1);
        const float hp = h;
        if (i == 0)
            h = lv * xv;
        else
            h = tri_step(hp, widen(r0[i], s.lo0), widen(r1[i], s.lo1), widen(r2[i], s.lo2),
                         lv * xv);
        const float a = ahist[i];
        const uint32_t so = lnoff(i);
        // dw terms of line i (zero on line 0; taps leaving the grid read zeros)
        float t0 = 0.f, t1 = 0.f, t2 = 0.f;
        if (i > 0) {
            t0 = a * from_left<64>(hp);
            t1 = a * hp;
            t2 = a * from_right<64>(hp);
        }
        if (act) {
            st16(A.du, vo, so, pack1(dyv * h));
            st16(A.dlam, vo, so, pack1(a * xv));
            if (VERT) {
                // this wave is the only writer of its dx plane: a returnless
                // LDS add keeps the order and does not wait
                float *xa = A.Xq + col_of(i) * kDxPitch + jj;
                if (A.first)
                    *xa = a * lv;
                else
                    __hip_atomic_fetch_add(xa, a * lv, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
            }
        }
        if (!VERT) {
            const int cc = col_of(i);
            dxr[cc] = dx_first ? a * lv : fmaf(a, lv, dxr[cc]);
        }
        // finish the reduction of line i-1 (its slot reads were issued after
        // the previous barrier and overlapped this step's arithmetic)
        if (i > 0)
            flush_dw(i - 1);
        slot_ptr(A.slots, i & 1, 0, A.wave)[j] = t0;
        slot_ptr(A.slots, i & 1, 1, A.wave)[j] = t1;
        slot_ptr(A.slots, i & 1, 2, A.wave)[j] = t2;
        lds_barrier();
        issue_dw(i);
        step_fence();
    }
    flush_dw(L - 1);
#undef BLOAD
}

template <int H, int W>
__global__ __launch_bounds__(512) void bwd_med_kernel(
    const bf16_t *__restrict__ x, const bf16_t *__restrict__ w, const bf16_t *__restrict__ lam,
    const bf16_t *__restrict__ u, const bf16_t *__restrict__ dy, bf16_t *__restrict__ dx,
    bf16_t *__restrict__ dw, bf16_t *__restrict__ dlam, bf16_t *__restrict__ du,
    float *__restrict__ dwp, int mask, int B, int C, int G, int cw, int nchunk)
{
    static_assert(H <= 64 && W <= 64 && H % 8 == 0 && W % 8 == 0 && H == W, "shape");
    constexpr int HW = H * W;
    constexpr int XPLANE = H * kDxPitch;                    // floats per dx plane
    extern __shared__ float4 smem4[];
    float *smem = reinterpret_cast<float *>(smem4);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int nwaves = blockDim.x >> 6;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int chunk = blk % nchunk;
    const int bg = blk / nchunk;
    const int g = bg % G;
    const int b = bg / G;
    const int cpg = C / G;
    const int cfirst = chunk * cw;
    const int nvalid = min(cw, cpg - cfirst);
    const bool cvalid = wave < nvalid;
    const int c = g * cpg + cfirst + (cvalid ? wave : 0);
    const int D = __popc(mask);
    const int64_t pc = ((int64_t)b * C + c) * HW;

    BwdArgs A;
    A.x = make_rsrc(x + pc, 2 * HW);
    A.dy = make_rsrc(dy + pc, 2 * HW);
    A.Xq = smem + wave * XPLANE;
    A.slots = smem + cw * XPLANE;
    // slots of channels this workgroup does not have must read as zero
    for (int t = threadIdx.x; t < 2 * 3 * 64 * kSlots; t += blockDim.x)
        A.slots[t] = 0.f;
    lds_barrier();
    A.wave = wave;
    A.nwaves = nwaves;
    A.nvalid = nvalid;
    A.cw = cw;
    A.partial = nchunk > 1;

    // Horizontal directions read x and dy columns: stage both planes in this
    // wave's LDS dx plane (still unused), coalesced; their dx terms collect in
    // registers (this lane's row) and move into the dx plane afterwards.
    const bool horiz = (mask & 12) != 0;
    const bool vert = (mask & 3) != 0;
    const uint8_t *stg = reinterpret_cast<const uint8_t *>(A.Xq);
    if (horiz) {
        uint32_t *st = reinterpret_cast<uint32_t *>(A.Xq);
        constexpr int NP = HW / 8;                          // 16-byte pieces per plane
#pragma unroll
        for (int t = 0; t < (NP + 63) / 64; ++t) {
            const int p = t * 64 + lane;
            if (p < NP) {
                const uint4 vx = ld128(A.x, 16u * p, 0);
                const uint4 vd = ld128(A.dy, 16u * p, 0);
                const int pr = p / (W / 8), pq = p - pr * (W / 8);
                uint32_t *dst = st + pr * kDxPitch + 8 * pq;
                const uint32_t xs_[4] = {vx.x, vx.y, vx.z, vx.w};
                const uint32_t ds_[4] = {vd.x, vd.y, vd.z, vd.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    dst[2 * e] = __builtin_amdgcn_perm(ds_[e], xs_[e], 0x05040100u);
                    dst[2 * e + 1] = __builtin_amdgcn_perm(ds_[e], xs_[e], 0x07060302u);
                }
            }
        }
        // the same wave reads what it wrote: LDS keeps its order
    }

    // Per-direction descriptors.  An idle wave (no channel left in this
    // chunk) still joins every barrier; it reads channel `c` of the chunk,
    // computes zeros and stores nothing of its own.
    auto setup = [&](int d) {
        const int s = __popc(mask & ((1 << d) - 1));
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const int64_t unit = ((int64_t)s * B + b) * G + g;
        A.lam = make_rsrc(lam + pd, 2 * HW);
        A.u = make_rsrc(u + pd, 2 * HW);
        A.dlam = make_rsrc(dlam + pd, 2 * HW);
        A.du = make_rsrc(du + pd, 2 * HW);
        A.w = make_rsrc(w + unit * 3 * HW, 6 * HW);
        if (A.partial)
            A.dw = make_rsrc(dwp + ((int64_t)chunk * D * B * G + unit) * 3 * HW, 12 * HW);
        else
            A.dw = make_rsrc(dw + unit * 3 * HW, 6 * HW);
    };

    // horizontal directions first (x and dy staged), dx in registers
    float dxr[64];
    A.first = false;
    if (mask & 4) {
        setup(2);
        dir_bwd<H, W, 2>(A, lane, cvalid, stg, dxr, true);
        lds_barrier();   // slot buffers are reused by the next direction
    }
    if (mask & 8) {
        setup(3);
        dir_bwd<H, W, 3>(A, lane, cvalid, stg, dxr, (mask & 4) == 0);
        lds_barrier();
    }
    if (horiz) {
        // the horizontal dx terms (this lane's row) seed the dx plane the
        // vertical directions add to, or go out directly
        if (vert) {
            if (lane < H) {
#pragma unroll
                for (int q = 0; q < W; ++q)
                    A.Xq[lane * kDxPitch + q] = dxr[q];
            }
        } else if (cvalid && lane < H) {
            const rsrc_t dxo = make_rsrc(dx + pc, 2 * HW);
#pragma unroll
            for (int q = 0; q < W / 8; ++q)
                st128(dxo, 2u * (uint32_t)(lane * W), 16u * q,
                      make_uint4(pack2(dxr[8 * q], dxr[8 * q + 1]),
                                 pack2(dxr[8 * q + 2], dxr[8 * q + 3]),
                                 pack2(dxr[8 * q + 4], dxr[8 * q + 5]),
                                 pack2(dxr[8 * q + 6], dxr[8 * q + 7])));
        }
    }
    if (mask & 1) {
        setup(0);
        A.first = !horiz;
        dir_bwd<H, W, 0>(A, lane, cvalid, stg, dxr, false);
        lds_barrier();
    }
    if (mask & 2) {
        setup(1);
        A.first = !horiz && (mask & 1) == 0;
        dir_bwd<H, W, 1>(A, lane, cvalid, stg, dxr, false);
        lds_barrier();
    }

    if (vert && cvalid && lane < H) {
        const float *Xr = A.Xq + lane * kDxPitch;
        const rsrc_t dxo = make_rsrc(dx + pc, 2 * HW);
        const uint32_t vo = 2u * (uint32_t)(lane * W);
#pragma unroll
        for (int q = 0; q < W / 8; ++q) {
            const float *a = Xr + 8 * q;
            st128(dxo, vo, 16u * q, make_uint4(pack2(a[0], a[1]), pack2(a[2], a[3]),
                                               pack2(a[4], a[5]), pack2(a[6], a[7])));
        }
    }
}

// dw = sum over chunks of the fp32 partials, in chunk order; 8 outputs per
// thread with 16-byte accesses (n is a multiple of 8 on this path).
__global__ __launch_bounds__(256) void dw_sum_kernel(const float4 *__restrict__ dwp,
                                                     uint4 *__restrict__ dw, int64_t n8, int nchunk)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n8;
         e += (int64_t)gridDim.x * blockDim.x) {
        float4 a = dwp[2 * e], b = dwp[2 * e + 1];
        for (int k = 1; k < nchunk; ++k) {
            const float4 p = dwp[(k * n8 + e) * 2], q = dwp[(k * n8 + e) * 2 + 1];
            a = make_float4(a.x + p.x, a.y + p.y, a.z + p.z, a.w + p.w);
            b = make_float4(b.x + q.x, b.y + q.y, b.z + q.z, b.w + q.w);
        }
        dw[e] = make_uint4(pack2(a.x, a.y), pack2(a.z, a.w), pack2(b.x, b.y), pack2(b.z, b.w));
    }
}

template <int H, int W>
hipError_t fwd_med_t(const Problem &p, hipStream_t st)
{
    hipLaunchKernelGGL((fwd_med_kernel<H, W>), dim3((unsigned)(p.B * p.C)), dim3(256), 0, st,
                       (const bf16_t *)p.x, (const bf16_t *)p.w, (const bf16_t *)p.lam,
                       (const bf16_t *)p.u, (bf16_t *)p.y, p.mask, p.B, p.C, p.G);
    return hipGetLastError();
}

template <int H, int W>
hipError_t bwd_med_t(const Problem &p, hipStream_t st)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    int lds_max = 0;
    e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess)
        return e;
    const size_t per_ch = (size_t)H * kDxPitch * 4;                 // dx plane
    const size_t slots = (size_t)2 * 3 * 64 * kSlots * 4;           // per-step dw terms
    const int cpg = p.C / p.G;
    int cap = lds_max > (int)slots ? (int)(((size_t)lds_max - slots) / per_ch) : 0;
    cap = cap < kSlots ? cap : kSlots;
    if (cap < 1)
        return hipErrorInvalidConfiguration;
    const int nchunk = (cpg + cap - 1) / cap;
    const int cw = (cpg + nchunk - 1) / nchunk;
    const size_t lds = (size_t)cw * per_ch + slots;
    const int D = __builtin_popcount(p.mask);
    const int64_t ndw = (int64_t)D * p.B * p.G * 3 * H * W;

    e = hipFuncSetAttribute((const void *)bwd_med_kernel<H, W>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    float *dwp = nullptr;
    if (nchunk > 1) {
        e = scratch_alloc((void **)&dwp, (size_t)nchunk * ndw * sizeof(float), st);
        if (e != hipSuccess)
            return e;
    }
    hipLaunchKernelGGL((bwd_med_kernel<H, W>), dim3((unsigned)(p.B * p.G * nchunk)),
                       dim3(64 * cw), lds, st, (const bf16_t *)p.x, (const bf16_t *)p.w,
                       (const bf16_t *)p.lam, (const bf16_t *)p.u, (const bf16_t *)p.dy,
                       (bf16_t *)p.dx, (bf16_t *)p.dw, (bf16_t *)p.dlam, (bf16_t *)p.du, dwp,
                       p.mask, p.B, p.C, p.G, cw, nchunk);
    e = hipGetLastError();
    if (e == hipSuccess && nchunk > 1) {
        const int64_t n8 = ndw / 8;
        int64_t blocks = (n8 + 255) / 256;
        blocks = blocks < 16384 ? blocks : 16384;
        hipLaunchKernelGGL(dw_sum_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                           (const float4 *)dwp, (uint4 *)p.dw, n8, nchunk);
        e = hipGetLastError();
    }
    if (dwp) {
        hipError_t e2 = scratch_free(dwp, st);
        if (e == hipSuccess)
            e = e2;
    }
    return e;
}

}  // namespace

bool med_supported(const Problem &p)
{
    return p.dtype == 1 && ((p.H == 64 && p.W == 64) || (p.H == 56 && p.W == 56));
}

hipError_t launch_fwd_med(const Problem &p, hipStream_t st)
{
    if (p.H == 64)
        return fwd_med_t<64, 64>(p, st);
    return fwd_med_t<56, 56>(p, st);
}

hipError_t launch_bwd_med(const Problem &p, hipStream_t st)
{
    if (p.H == 64)
        return bwd_med_t<64, 64>(p, st);
    return bwd_med_t<56, 56>(p, st);
}

}  // namespace gspn
