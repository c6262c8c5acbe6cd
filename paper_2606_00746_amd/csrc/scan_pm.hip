// Pixel-major per-direction tensors on the square bf16 planes of side 24 to
// 64 (multiples of 8): the forward, and the weight re-layout that both
// passes start from.
//
// A horizontal scan needs a column of every per-direction plane at each step,
// while a pixel-major plane holds rows: one line of the scan touches every
// 128-byte row of the plane.  On this GPU a load costs what the lines it
// touches cost, so the kernels move whole rows only and turn them around on
// chip:
//  * the weights, shared by the C/G channels of a group, are re-laid out once
//    per call into the blocked line-major order of their direction (one
//    workgroup per tap plane, rows staged in LDS) in the caller's workspace,
//    where the scans read them as 16-byte pieces of 8 steps;
//  * the forward stages the x plane and each direction's lambda plane in LDS
//    with coalesced direct-to-LDS loads (no registers), reads rows for
//    vertical scans and 16-byte column pieces for horizontal ones, keeps
//    each lane's states h in registers, and applies u afterwards, row by
//    row: each direction's h plane goes through an fp32 LDS plane and every
//    thread adds u_d * h_d for 8 pixels of a row, u_d loaded into registers
//    with coalesced 16-byte row pieces while the planes are staged (Sec. 3,
//    Eqs. (gspn_recurrence), (gspn_output)).
#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;

typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glb_void;

// Row pitch (bytes) of a staged bf16 plane of side S: whole 16-byte pieces,
// padded so that the pitch in dwords is 4 mod 8; 8 lanes reading 16 bytes of
// 8 consecutive rows then hit distinct banks.
template <int S>
struct PmPlane {
    static constexpr int kPitch = 2 * S + ((S / 2) % 8 == 4 ? 0 : 16);
    static constexpr int kSlots = kPitch / 16;          // 16-byte slots per row
    static constexpr int kBytes = S * kPitch;
    // fp32 merge plane: row pitch in floats, 4 mod 8
    static constexpr int kPitchF = S + ((S % 8) == 4 ? 0 : 4);
    static constexpr int kBytesF = S * kPitchF * 4;
};

// Starts the copy of one S x S bf16 plane (row-major, rows of 2S bytes) into
// LDS rows of PmPlane<S>::kPitch bytes, by the nw waves of the workgroup:
// wave-instruction k covers slots 64k .. 64k+63 (slot s = row s / kSlots,
// piece s % kSlots; padding slots are skipped).  The bytes land once the
// issuing wave has waited for its loads.
template <int S>
__device__ __forceinline__ void stage_plane(uint8_t *dst, const bf16_t *src, int wave, int nw,
                                            int lane)
{
    using Pl = PmPlane<S>;
    constexpr int NS = S * Pl::kSlots;
    constexpr int NI = (NS + 63) / 64;
    const uint8_t *g = reinterpret_cast<const uint8_t *>(src);
    for (int k = wave; k < NI; k += nw) {
        const int s = 64 * k + lane;
        const int row = s / Pl::kSlots, pc = s - row * Pl::kSlots;
        if (s < NS && pc < S / 8)
            __builtin_amdgcn_global_load_lds((glb_void *)(g + row * 2 * S + 16 * pc),
                                             (lds_void *)(dst + 1024 * k), 16, 0, 0);
    }
}

// ---------------------------------------------------------------------------
// weights: pixel-major -> blocked line-major, one workgroup per tap plane
// ---------------------------------------------------------------------------

// Plane pl of a stack of planes grouped per direction slot (slot pl /
// per_slot, whose direction is vertical when bit slot of vslots is set).  The plane's rows
// are staged in LDS; then each thread writes 16-byte pieces of the blocked
// layout (piece (q, p): lines 8q..8q+7 at position p, contiguous across the
// wave).
template <int S>
__global__ __launch_bounds__(256) void to_blocked_kernel(const bf16_t *__restrict__ w,
                                                         uint4 *__restrict__ out, int vslots,
                                                         int per_slot)
{
    using Pl = PmPlane<S>;
    __shared__ uint4 sm[Pl::kBytes / 16];
    uint8_t *pl = reinterpret_cast<uint8_t *>(sm);
    const int p0 = blockIdx.x;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    stage_plane<S>(pl, w + (int64_t)p0 * S * S, wave, 4, lane);
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
    const bool vert = (vslots >> (p0 / per_slot)) & 1;
    constexpr int NQ = S / 8;
    uint4 *dst = out + (int64_t)p0 * (S * S / 8);
    for (int t = threadIdx.x; t < NQ * S; t += 256) {
        const int q = t / S, p = t - q * S;               // piece (q, p) at 16 bytes * t
        uint4 v;
        if (vert) {
            // lines are rows: the 8 rows 8q.. of column p
            uint32_t e[8];
#pragma unroll
            for (int k = 0; k < 8; ++k)
                e[k] = lds_u16(pl, (8 * q + k) * Pl::kPitch + 2 * p);
            v = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                           e[6] | (e[7] << 16));
        } else {
            // lines are columns: 8 consecutive columns of row p
            v = *reinterpret_cast<const uint4 *>(pl + p * Pl::kPitch + 16 * q);
        }
        gst128(dst + t, v);
    }
}

// Logits -> normalized weights, pixel-major -> blocked, one workgroup per
// direction slot, batch and group (three tap planes): the logit planes are
// staged in LDS, each thread forms the weights of the 8 pixels of one
// output piece (q, p) from their three logits (Sec. 3,
// Eq. (row_stochastic_norm)) and writes the piece of every tap.  The line
// position p decides taps 0 and 2, as in the unfused normalization.
template <int S>
__global__ __launch_bounds__(256) void norm_to_blocked_kernel(const bf16_t *__restrict__ wt,
                                                              uint4 *__restrict__ out, int vslots,
                                                              int per_slot)
{
    using Pl = PmPlane<S>;
    __shared__ uint4 sm[3 * Pl::kBytes / 16];
    uint8_t *pl = reinterpret_cast<uint8_t *>(sm);
    const int set = blockIdx.x;                           // slot * per_slot + (b, g)
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < 3; ++k)
        stage_plane<S>(pl + k * Pl::kBytes, wt + ((int64_t)set * 3 + k) * S * S, wave, 4, lane);
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
    const bool vert = (vslots >> (set / per_slot)) & 1;
    constexpr int NQ = S / 8;
    uint4 *dst = out + (int64_t)set * 3 * (S * S / 8);
    for (int t = threadIdx.x; t < NQ * S; t += 256) {
        const int q = t / S, p = t - q * S;               // piece (q, p)
        float lg[3][8];
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const uint8_t *pk = pl + k * Pl::kBytes;
            if (vert) {
                // rows 8q.. of column p
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    lg[k][e] = __uint_as_float(lds_u16(pk, (8 * q + e) * Pl::kPitch + 2 * p) << 16);
            } else {
                // columns 8q.. of row p
                const uint4 v = *reinterpret_cast<const uint4 *>(pk + p * Pl::kPitch + 16 * q);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    lg[k][e] = elem(v, e);
            }
        }
        const bool on0 = p > 0, on2 = p + 1 < S;
        uint32_t pk3[3][4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            float w0[3], w1[3];
            const float t0[3] = {lg[0][e], lg[1][e], lg[2][e]};
            const float t1[3] = {lg[0][e + 1], lg[1][e + 1], lg[2][e + 1]};
            norm3(t0, on0, on2, w0);
            norm3(t1, on0, on2, w1);
#pragma unroll
            for (int k = 0; k < 3; ++k)
                pk3[k][e / 2] = pack2(w0[k], w1[k]);
        }
#pragma unroll
        for (int k = 0; k < 3; ++k)
            gst128(dst + k * (S * S / 8) + t,
                   make_uint4(pk3[k][0], pk3[k][1], pk3[k][2], pk3[k][3]));
    }
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------

// The scan of direction D over one channel plane: h of every step stays in
// hr (hr[i] = state of this lane's position after step i).  xs, ls: the
// staged x and lambda planes; w: the direction's blocked tap planes.
// WL: the taps too are staged pixel-major planes in LDS (wls, three planes
// of PmPlane<S>::kBytes), else blocked pieces of w in global memory.
template <int S, int D, bool WL>
__device__ __forceinline__ void pm_fwd_dir(int j, const uint8_t *xs, const uint8_t *ls, rsrc_t w,
                                           const uint8_t *wls, float (&hr)[S])
{
    using Pl = PmPlane<S>;
    constexpr bool VERT = D < 2, REV = D == 1 || D == 3;
    constexpr int NB = S / 8;
    constexpr uint32_t PL = 2 * S * S;                 // bytes of one tap plane
    const Sel s = make_sel(j, S);
    const int jc = j < S ? j : S - 1;
    uint4 r0[NB], r1[NB], r2[NB];
    auto wload = [&](int fb) {
        const int sq = REV ? NB - 1 - fb : fb;
        if (WL) {
            if (!VERT) {
                // this lane's row, the block's 8 columns, per tap
                const int o = jc * Pl::kPitch + 16 * sq;
                r0[fb] = *reinterpret_cast<const uint4 *>(wls + o);
                r1[fb] = *reinterpret_cast<const uint4 *>(wls + Pl::kBytes + o);
                r2[fb] = *reinterpret_cast<const uint4 *>(wls + 2 * Pl::kBytes + o);
            }
        } else {
            r0[fb] = ld_piece<false, VERT, false>(w, jc, sq, S, S);
            r1[fb] = ld_piece<false, VERT, false>(w, jc, sq, S, S, PL);
            r2[fb] = ld_piece<false, VERT, false>(w, jc, sq, S, S, 2 * PL);
        }
    };
    wload(0);
    if (NB > 1)
        wload(1);
    float h = 0.f;
#pragma unroll
    for (int fb = 0; fb < NB; ++fb) {
        if (fb + 2 < NB)
            wload(fb + 2);
        const int sq = REV ? NB - 1 - fb : fb;             // storage block
        uint4 xq, lq;
        if (!VERT) {
            // this lane's row, the block's 8 columns: one 16-byte piece each
            xq = *reinterpret_cast<const uint4 *>(xs + jc * Pl::kPitch + 16 * sq);
            lq = *reinterpret_cast<const uint4 *>(ls + jc * Pl::kPitch + 16 * sq);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int i = 8 * fb + t;
            const int e = REV ? 7 - t : t;                 // element of the block's piece
            float xv, lv;
            if (VERT) {
                const int row = 8 * sq + e;
                xv = bf_lo(lds_u16(xs, row * Pl::kPitch + 2 * jc));
                lv = widen(lds_u16(ls, row * Pl::kPitch + 2 * jc), s.lo1);
            } else {
                xv = elem(xq, e);
                lv = elem(lq, e, s.lo1, s.hi1);
            }
            const float inj = lv * xv;
            if (i == 0) {
                h = inj;
            } else {
                float w0, w1, w2;
                if (WL && VERT) {
                    const int o = (8 * sq + e) * Pl::kPitch + 2 * jc;
                    w0 = widen(lds_u16(wls, o), s.lo0);
                    w1 = widen(lds_u16(wls + Pl::kBytes, o), s.lo1);
                    w2 = widen(lds_u16(wls + 2 * Pl::kBytes, o), s.lo2);
                } else {
                    w0 = elem(r0[fb], e, s.lo0, s.hi0);
                    w1 = elem(r1[fb], e, s.lo1, s.hi1);
                    w2 = elem(r2[fb], e, s.lo2, s.hi2);
                }
                float hn = fmaf(w1, h, inj);
                hn = fmaf(w0, from_left<64>(h), hn);
                hn = fmaf(w2, from_right<64>(h), hn);
                h = hn;
            }
            hr[i] = h;
        }
        step_fence();
    }
}

// LDS of fwd_pm_kernel: x and the 4 lambda planes, with WL also the 12 tap
// planes; the fp32 merge plane reuses it afterwards.
template <int S>
constexpr size_t fwd_pm_lds(bool wl)
{
    using Pl = PmPlane<S>;
    const size_t stg = (size_t)(wl ? 17 : 5) * Pl::kBytes;
    return stg > (size_t)Pl::kBytesF ? stg : (size_t)Pl::kBytesF;
}

// One workgroup per (b, c), one wave per direction.  w: the blocked weights,
// or with WL (one channel per group, where a re-layout would copy as much as
// the lambda planes) the pixel-major weights, staged in LDS with the rest.
// lamh, uh (wh with WL): where a training forward leaves the blocked copies
// its backward reads, or null: lambda and u of the horizontal directions
// [nh][B][C][plane] (with WL their tap planes [nh][B][G][3][plane]), taken
// from the staged planes and the u pieces already in registers.
template <int S, bool WL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WL ? 1 : 3))) void
fwd_pm_kernel(const bf16_t *__restrict__ x, const bf16_t *__restrict__ wb,
              const bf16_t *__restrict__ lam, const bf16_t *__restrict__ u,
              bf16_t *__restrict__ y, int mask, int B, int C, int G, Magic divC, Magic divCpg,
              bf16_t *__restrict__ lamh, bf16_t *__restrict__ uh, bf16_t *__restrict__ wh)
{
    using Pl = PmPlane<S>;
    constexpr int HW = S * S;
    constexpr int NCH = HW / 8;                           // 8-pixel pieces of a plane
    constexpr int PER = (NCH + 255) / 256;                // pieces per thread
    extern __shared__ uint4 lds4[];
    uint8_t *base = reinterpret_cast<uint8_t *>(lds4);
    float *M = reinterpret_cast<float *>(lds4);           // merge plane, after the scans

    const int d = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
    const int lane = threadIdx.x & 63;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int b = mdiv(blk, divC);
    const int c = blk - b * C;
    const int g = mdiv(c, divCpg);
    const int64_t pc = ((int64_t)b * C + c) * HW;

    // x (plane 0) and every present direction's lambda (plane 1 + d)
    stage_plane<S>(base, x + pc, d, 4, lane);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        if ((mask >> k) & 1) {
            const int sk = __popc(mask & ((1 << k) - 1));
            stage_plane<S>(base + (1 + k) * Pl::kBytes,
                           lam + (((int64_t)sk * B + b) * C + c) * HW, d, 4, lane);
            if (WL) {
                // the three tap planes of direction k (planes 5 + 3k ..)
                const bf16_t *wk = wb + (((int64_t)sk * B + b) * G + g) * 3 * HW;
#pragma unroll
                for (int t = 0; t < 3; ++t)
                    stage_plane<S>(base + (5 + 3 * k + t) * Pl::kBytes, wk + t * HW, d, 4, lane);
            }
        }
    }
    // every direction's u, 8 pixels of a row per thread and piece, loaded
    // beside the staging: the merge below waits on no load
    uint4 uq[4][PER];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if ((mask >> p) & 1) {
            const int sp = __popc(mask & ((1 << p) - 1));
            const rsrc_t ur = make_rsrc(u + (((int64_t)sp * B + b) * C + c) * HW, 2 * HW);
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                const int t = threadIdx.x + 256 * k;
                uq[p][k] = t < NCH ? ld128_nt(ur, 16u * (uint32_t)t, 0) : make_uint4(0, 0, 0, 0);
            }
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();

    // the reserve of a training forward: piece (q, p) of a horizontal
    // direction's blocked plane is columns 8q .. 8q+7 of row p, which this
    // thread holds (u) or finds staged (lambda, taps) for its row pieces;
    // the 8 threads of one column block write whole 128-byte lines
    if (lamh != nullptr) {
        const int nvd = __popc(mask & 3);
#pragma unroll
        for (int p = 2; p < 4; ++p) {
            if (!((mask >> p) & 1))
                continue;
            const int sh = __popc(mask & ((1 << p) - 1)) - nvd;
            uint4 *lo = reinterpret_cast<uint4 *>(lamh + (((int64_t)sh * B + b) * C + c) * HW);
            uint4 *uo = reinterpret_cast<uint4 *>(uh + (((int64_t)sh * B + b) * C + c) * HW);
            uint4 *wo = reinterpret_cast<uint4 *>(WL ? wh + (((int64_t)sh * B + b) * G + g) * 3 * HW
                                                     : wh);
#pragma unroll
            for (int k = 0; k < PER; ++k) {
                const int t = threadIdx.x + 256 * k;
                if (t < NCH) {
                    const int r = t / (S / 8), cq = t - r * (S / 8);
                    const int o = cq * S + r, so = r * Pl::kPitch + 16 * cq;
                    gst128(lo + o, *reinterpret_cast<const uint4 *>(base + (1 + p) * Pl::kBytes + so));
                    gst128(uo + o, uq[p][k]);
                    if (WL) {
#pragma unroll
                        for (int tp = 0; tp < 3; ++tp)
                            gst128(wo + tp * NCH + o, *reinterpret_cast<const uint4 *>(
                                                          base + (5 + 3 * p + tp) * Pl::kBytes + so));
                    }
                }
            }
        }
    }

    const bool mine = (mask >> d) & 1;
    const int s = __popc(mask & ((1 << d) - 1));
    float hr[S];
    if (mine) {
        const int64_t pw = (((int64_t)s * B + b) * G + g) * 3 * HW;
        const rsrc_t rw = make_rsrc(wb + pw, 6 * HW);
        const uint8_t *ls = base + (1 + d) * Pl::kBytes;
        const uint8_t *wls = base + (5 + 3 * d) * Pl::kBytes;
        if (d == 0)
            pm_fwd_dir<S, 0, WL>(lane, base, ls, rw, wls, hr);
        else if (d == 1)
            pm_fwd_dir<S, 1, WL>(lane, base, ls, rw, wls, hr);
        else if (d == 2)
            pm_fwd_dir<S, 2, WL>(lane, base, ls, rw, wls, hr);
        else
            pm_fwd_dir<S, 3, WL>(lane, base, ls, rw, wls, hr);
    }
    lds_barrier();   // the staged planes become the merge plane

    // y = sum_d u_d * h_d, directions in bit order, 8 pixels of a row per
    // thread and piece
    float acc[PER][8];
#pragma unroll
    for (int k = 0; k < PER; ++k)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            acc[k][e] = 0.f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (!((mask >> p) & 1))
            continue;
        if (d == p && lane < S) {
            if (p < 2) {
                // column `lane`, row of step i
#pragma unroll
                for (int i = 0; i < S; ++i)
                    M[(p == 1 ? S - 1 - i : i) * Pl::kPitchF + lane] = hr[i];
            } else {
                // row `lane`, column of step i, 16-byte stores
                float4 *row = reinterpret_cast<float4 *>(M + lane * Pl::kPitchF);
#pragma unroll
                for (int q = 0; q < S / 4; ++q) {
                    float v4[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int col = 4 * q + e;
                        v4[e] = hr[p == 3 ? S - 1 - col : col];
                    }
                    row[q] = make_float4(v4[0], v4[1], v4[2], v4[3]);
                }
            }
        }
        lds_barrier();
#pragma unroll
        for (int k = 0; k < PER; ++k) {
            const int t = threadIdx.x + 256 * k;
            if (t < NCH) {
                const int r = t / (S / 8), cq = t - r * (S / 8);
                const float4 *src = reinterpret_cast<const float4 *>(M + r * Pl::kPitchF + 8 * cq);
                const float4 h0 = src[0], h1 = src[1];
                const float hv[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
                // u_d * h_d rounded, then added (as the blocked-layout
                // kernels do: both layouts give the same bits)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc[k][e] = add_nc(acc[k][e], mul_nc(elem(uq[p][k], e), hv[e]));
            }
        }
        lds_barrier();
    }
    const u32x4 yo = make_sdesc(y + pc, 2 * HW);
#pragma unroll
    for (int k = 0; k < PER; ++k) {
        const int t = threadIdx.x + 256 * k;
        if (t < NCH)
            st128_nt(yo, 16u * (uint32_t)t, 0,
                     make_uint4(pack2(acc[k][0], acc[k][1]), pack2(acc[k][2], acc[k][3]),
                                pack2(acc[k][4], acc[k][5]), pack2(acc[k][6], acc[k][7])));
    }
}

template <int S>
hipError_t w_to_blocked_t(const Problem &p, void *wb, hipStream_t st)
{
    int vslots = 0;
    for (int d = 0, sl = 0; d < 4; ++d)
        if ((p.mask >> d) & 1) {
            if (d < 2)
                vslots |= 1 << sl;
            ++sl;
        }
    const int per_slot = p.B * p.G * 3;
    const int planes = __builtin_popcount(p.mask) * per_slot;
    hipLaunchKernelGGL((to_blocked_kernel<S>), dim3((unsigned)planes), dim3(256), 0, st,
                       (const bf16_t *)p.w, (uint4 *)wb, vslots, per_slot);
    return hipGetLastError();
}

// lam and u of the horizontal directions (slots nv .. D-1, nv the vertical
// directions of the mask) into [D - nv][B][C][plane] blocked copies each.
template <int S>
hipError_t horiz_to_blocked_t(const Problem &p, void *lamh, void *uh, hipStream_t st)
{
    const int nv = __builtin_popcount(p.mask & 3), nh = __builtin_popcount(p.mask & 12);
    const int64_t skip = (int64_t)nv * p.B * p.C * S * S;
    const int planes = nh * p.B * p.C;
    if (planes == 0)
        return hipSuccess;
    hipLaunchKernelGGL((to_blocked_kernel<S>), dim3((unsigned)planes), dim3(256), 0, st,
                       (const bf16_t *)p.lam + skip, (uint4 *)lamh, 0, planes);
    hipLaunchKernelGGL((to_blocked_kernel<S>), dim3((unsigned)planes), dim3(256), 0, st,
                       (const bf16_t *)p.u + skip, (uint4 *)uh, 0, planes);
    return hipGetLastError();
}

template <int S>
hipError_t norm_blocked_t(const Problem &p, const void *wt, void *wb, hipStream_t st)
{
    int vslots = 0;
    for (int d = 0, sl = 0; d < 4; ++d)
        if ((p.mask >> d) & 1) {
            if (d < 2)
                vslots |= 1 << sl;
            ++sl;
        }
    const int per_slot = p.B * p.G;
    const int sets = __builtin_popcount(p.mask) * per_slot;
    hipLaunchKernelGGL((norm_to_blocked_kernel<S>), dim3((unsigned)sets), dim3(256), 0, st,
                       (const bf16_t *)wt, (uint4 *)wb, vslots, per_slot);
    return hipGetLastError();
}

template <int S, bool WL>
hipError_t fwd_pm_launch(const Problem &p, const void *w, hipStream_t st, const ReserveParts &r)
{
    const size_t lds = fwd_pm_lds<S>(WL);
    hipError_t e = hipFuncSetAttribute((const void *)fwd_pm_kernel<S, WL>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((fwd_pm_kernel<S, WL>), dim3((unsigned)(p.B * p.C)), dim3(256), lds, st,
                       (const bf16_t *)p.x, (const bf16_t *)w, (const bf16_t *)p.lam,
                       (const bf16_t *)p.u, (bf16_t *)p.y, p.mask, p.B, p.C, p.G,
                       make_magic((uint32_t)p.C), make_magic((uint32_t)(p.C / p.G)),
                       (bf16_t *)r.lamh, (bf16_t *)r.uh, (bf16_t *)r.w);
    return hipGetLastError();
}

template <int S>
hipError_t fwd_pm_t(const Problem &p, hipStream_t st)
{
    // a training forward leaves the blocked copies of its backward in the
    // reserve (parts taken by the entry point): the weights' re-layout
    // writes there, the kernel the rest
    ReserveParts r;
    hipError_t e = hipSuccess;
    if (p.rs_write && p.rsp != nullptr)
        r = *p.rsp;
    // one channel per group: the weights are staged with the channel's
    // other planes (no copy); else re-laid out once for the group's channels
    if (p.C == p.G && !p.w_blocked)
        return p.ws->counting ? hipSuccess : fwd_pm_launch<S, true>(p, p.w, st, r);
    const int64_t nw = (int64_t)__builtin_popcount(p.mask) * p.B * p.G * 3 * S * S;
    void *wb = const_cast<void *>(p.w);
    if (!p.w_blocked) {
        if (p.rs_write && p.rsp != nullptr)
            wb = r.w;
        else
            e = p.ws->take(&wb, (size_t)nw * 2);
    }
    if (e != hipSuccess || p.ws->counting)
        return e;
    if (!p.w_blocked)
        e = w_to_blocked_t<S>(p, wb, st);
    if (e != hipSuccess)
        return e;
    ReserveParts k = r;
    k.w = nullptr;                 // (the weights are written above)
    return fwd_pm_launch<S, false>(p, wb, st, k);
}

}  // namespace

hipError_t launch_w_to_blocked(const Problem &p, void *wb, hipStream_t st)
{
    switch (p.H) {
    case 64: return w_to_blocked_t<64>(p, wb, st);
    case 56: return w_to_blocked_t<56>(p, wb, st);
    case 48: return w_to_blocked_t<48>(p, wb, st);
    case 40: return w_to_blocked_t<40>(p, wb, st);
    case 32: return w_to_blocked_t<32>(p, wb, st);
    default: return w_to_blocked_t<24>(p, wb, st);
    }
}

hipError_t launch_planes_to_blocked(const void *src, void *dst, int n, int S, hipStream_t st)
{
    if (n == 0)
        return hipSuccess;
    switch (S) {
    case 64:
        hipLaunchKernelGGL((to_blocked_kernel<64>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    case 56:
        hipLaunchKernelGGL((to_blocked_kernel<56>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    case 48:
        hipLaunchKernelGGL((to_blocked_kernel<48>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    case 40:
        hipLaunchKernelGGL((to_blocked_kernel<40>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    case 32:
        hipLaunchKernelGGL((to_blocked_kernel<32>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    default:
        hipLaunchKernelGGL((to_blocked_kernel<24>), dim3((unsigned)n), dim3(256), 0, st,
                           (const bf16_t *)src, (uint4 *)dst, 0, n);
        break;
    }
    return hipGetLastError();
}

hipError_t launch_horiz_to_blocked(const Problem &p, void *lamh, void *uh, hipStream_t st)
{
    switch (p.H) {
    case 64: return horiz_to_blocked_t<64>(p, lamh, uh, st);
    case 56: return horiz_to_blocked_t<56>(p, lamh, uh, st);
    case 48: return horiz_to_blocked_t<48>(p, lamh, uh, st);
    case 40: return horiz_to_blocked_t<40>(p, lamh, uh, st);
    case 32: return horiz_to_blocked_t<32>(p, lamh, uh, st);
    default: return horiz_to_blocked_t<24>(p, lamh, uh, st);
    }
}

hipError_t launch_norm_blocked(const Problem &p, const void *wt, void *wb, hipStream_t st)
{
    switch (p.H) {
    case 64: return norm_blocked_t<64>(p, wt, wb, st);
    case 56: return norm_blocked_t<56>(p, wt, wb, st);
    case 48: return norm_blocked_t<48>(p, wt, wb, st);
    case 40: return norm_blocked_t<40>(p, wt, wb, st);
    case 32: return norm_blocked_t<32>(p, wt, wb, st);
    default: return norm_blocked_t<24>(p, wt, wb, st);
    }
}

hipError_t launch_fwd_pm(const Problem &p, hipStream_t st)
{
    switch (p.H) {
    case 64: return fwd_pm_t<64>(p, st);
    case 56: return fwd_pm_t<56>(p, st);
    case 48: return fwd_pm_t<48>(p, st);
    case 40: return fwd_pm_t<40>(p, st);
    case 32: return fwd_pm_t<32>(p, st);
    default: return fwd_pm_t<24>(p, st);
    }
}

}  // namespace gspn
