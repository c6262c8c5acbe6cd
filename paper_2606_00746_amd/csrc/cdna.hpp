// gfx950 building blocks shared by the libgspn kernels: raw buffer access
// with uniform descriptors, stores issued with their wait states, bf16
// widening with per-lane masks, LDS-only barriers and the XCD-aware
// workgroup order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gspn {
namespace cdna {

constexpr uint32_t kSelLo = 0x01000C0Cu;   // bf16 in bits [15:0]  -> fp32
constexpr uint32_t kSelHi = 0x03020C0Cu;   // bf16 in bits [31:16] -> fp32
constexpr uint32_t kSelZero = 0x0C0C0C0Cu; // -> +0.0f

// Keep the software pipeline as written: nothing is scheduled across a step
// boundary, so each step's prefetch stays ahead of its use instead of every
// load of the unrolled scan being hoisted to the top.
// Makes v opaque to the compiler, so values derived from it before this point
// are not reused after it (they are derived again).
__device__ __forceinline__ void launder(uint4 &v)
{
    asm volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

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
                                             (int)__builtin_amdgcn_readfirstlane(bytes), kRsrcWord3);
}
__device__ __forceinline__ uint32_t ld16(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t ld32(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}
__device__ __forceinline__ uint4 ld128(rsrc_t r, uint32_t voff, uint32_t soff)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
// Streams read exactly once (lam, u) are loaded non-temporal, so that the L2
// keeps what several waves or sweeps read again (x, dy and a group's w).
__device__ __forceinline__ uint4 ld128_nt(rsrc_t r, uint32_t voff, uint32_t soff)
{
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 2 /* nt */);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
// Stores go through inline assembly, each wide one together with the wait
// states after it.  A VALU write to a VGPR that a wide store still has to
// read (its data registers are read after issue, later still when it queues
// behind another store) corrupts the stored value in some lanes; this
// compiler inserts no wait states for that on gfx950, and its register
// allocator can place such a write (a copy) directly after the store, where
// no scheduling barrier reaches.  One asm block keeps the two together.
// Store targets use a raw buffer descriptor held in SGPRs as four words.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 make_sdesc(const void *p, uint32_t bytes)
{
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    u32x4 d;
    d.x = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
    d.y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32)) & 0xffffu;  // stride 0
    d.z = __builtin_amdgcn_readfirstlane(bytes);
    d.w = kRsrcWord3;
    return d;
}
// 2- and 4-byte stores go through the compiler's buffer-store builtins, so that
// it keeps the stored register intact until the store has read it (an asm
// store of 2 bytes lost its data to the next VALU write of that register) and
// counts the stores in its memory-counter waits.
__device__ __forceinline__ rsrc_t as_rsrc(const u32x4 &d)
{
    void *p = reinterpret_cast<void *>((static_cast<uint64_t>(d.y & 0xffffu) << 32) | d.x);
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)d.z, (int)d.w);
}
__device__ __forceinline__ void st16(const u32x4 &d, uint32_t voff, uint32_t soff, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b16((uint16_t)v, as_rsrc(d), voff, soff, 0);
}
__device__ __forceinline__ void st32(const u32x4 &d, uint32_t voff, uint32_t soff, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, as_rsrc(d), voff, soff, 0);
}
// Non-temporal dword store, for waves whose lanes cover whole lines.
__device__ __forceinline__ void st32_nt(const u32x4 &d, uint32_t voff, uint32_t soff, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, as_rsrc(d), voff, soff, 2 /* nt */);
}
__device__ __forceinline__ void st64(const u32x4 &d, uint32_t voff, uint32_t soff, uint32_t a,
                                     uint32_t b)
{
    const u32x2 t = {a, b};
    asm volatile("buffer_store_dwordx2 %0, %1, %2, %3 offen\n\ts_nop 7\n\ts_nop 7"
                 : : "v"(t), "v"(voff), "s"(d), "s"(soff) : "memory");
}
__device__ __forceinline__ void st64_nt(const u32x4 &d, uint32_t voff, uint32_t soff, uint32_t a,
                                        uint32_t b)
{
    const u32x2 t = {a, b};
    asm volatile("buffer_store_dwordx2 %0, %1, %2, %3 offen nt\n\ts_nop 7\n\ts_nop 7"
                 : : "v"(t), "v"(voff), "s"(d), "s"(soff) : "memory");
}
__device__ __forceinline__ void st128(const u32x4 &d, uint32_t voff, uint32_t soff, uint4 v)
{
    const u32x4 t = {v.x, v.y, v.z, v.w};
    asm volatile("buffer_store_dwordx4 %0, %1, %2, %3 offen\n\ts_nop 7\n\ts_nop 7"
                 : : "v"(t), "v"(voff), "s"(d), "s"(soff) : "memory");
}
// Non-temporal variant for stores whose wave covers whole 128-byte lines
// (partial-line non-temporal stores are not merged in the L2 and cost more
// write traffic than they save).
__device__ __forceinline__ void st128_nt(const u32x4 &d, uint32_t voff, uint32_t soff, uint4 v)
{
    const u32x4 t = {v.x, v.y, v.z, v.w};
    asm volatile("buffer_store_dwordx4 %0, %1, %2, %3 offen nt\n\ts_nop 7\n\ts_nop 7"
                 : : "v"(t), "v"(voff), "s"(d), "s"(soff) : "memory");
}
__device__ __forceinline__ void gst64(uint2 *p, uint32_t a, uint32_t b)
{
    const u32x2 t = {a, b};
    asm volatile("global_store_dwordx2 %0, %1, off\n\ts_nop 7\n\ts_nop 7" : : "v"(p), "v"(t)
                 : "memory");
}
__device__ __forceinline__ void gst128(uint4 *p, uint4 v)
{
    const u32x4 t = {v.x, v.y, v.z, v.w};
    asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 7\n\ts_nop 7" : : "v"(p), "v"(t)
                 : "memory");
}

// A lane's 16-byte piece of a per-direction plane: the values of storage
// lines 8q .. 8q+7 at line position j, in line order (two bf16 per dword,
// the lower line in the low half).  Blocked line-major planes hold it as one
// 16-byte piece; in a pixel-major plane it is 8 consecutive pixels of row j
// for a horizontal direction (one 16-byte access) and 8 pixels of column j,
// one per row, for a vertical one (eight 2-byte accesses, each a full row
// across the wave).  P: line length; W: image row length.
__device__ __forceinline__ uint32_t ld16_nt(rsrc_t r, uint32_t voff, uint32_t soff)
{
    return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 2 /* nt */);
}
// `base`: a byte offset added to the plane (e.g. to reach another tap plane).
template <bool PM, bool VERT, bool NT>
__device__ __forceinline__ uint4 ld_piece(rsrc_t r, int j, int q, int P, int W, uint32_t base = 0)
{
    if constexpr (!PM) {
        return NT ? ld128_nt(r, 16u * (uint32_t)j, base + 16u * (uint32_t)(P * q))
                  : ld128(r, 16u * (uint32_t)j, base + 16u * (uint32_t)(P * q));
    } else if constexpr (!VERT) {
        return NT ? ld128_nt(r, 2u * (uint32_t)(W * j), base + 16u * (uint32_t)q)
                  : ld128(r, 2u * (uint32_t)(W * j), base + 16u * (uint32_t)q);
    } else {
        uint32_t v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t so = base + 2u * (uint32_t)(W * (8 * q + t));
            v[t] = NT ? ld16_nt(r, 2u * (uint32_t)j, so) : ld16(r, 2u * (uint32_t)j, so);
        }
        return make_uint4(__builtin_amdgcn_perm(v[1], v[0], 0x05040100u),
                          __builtin_amdgcn_perm(v[3], v[2], 0x05040100u),
                          __builtin_amdgcn_perm(v[5], v[4], 0x05040100u),
                          __builtin_amdgcn_perm(v[7], v[6], 0x05040100u));
    }
}
// Stores a piece (see ld_piece).  Blocked planes: one full-line 16-byte
// store (non-temporal if NT); pixel-major horizontal: one 16-byte store into
// the row, default policy so that the L2 merges the row's pieces; pixel-major
// vertical: eight 2-byte stores, each a full row across the wave.
template <bool PM, bool VERT, bool NT>
__device__ __forceinline__ void st_piece(const u32x4 &d, int j, int q, int P, int W, uint4 v,
                                         uint32_t base = 0)
{
    if constexpr (!PM) {
        if (NT)
            st128_nt(d, 16u * (uint32_t)j, base + 16u * (uint32_t)(P * q), v);
        else
            st128(d, 16u * (uint32_t)j, base + 16u * (uint32_t)(P * q), v);
    } else if constexpr (!VERT) {
        st128(d, 2u * (uint32_t)(W * j), base + 16u * (uint32_t)q, v);
    } else {
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int t = 0; t < 8; ++t)
            st16(d, 2u * (uint32_t)j, base + 2u * (uint32_t)(W * (8 * q + t)),
                 (t & 1) ? (w4[t >> 1] >> 16) : w4[t >> 1]);
    }
}

// Product and sum that the compiler may not fuse into a multiply-add (the
// direction sums of the forwards round u_d * h_d, then add, in every layout).
__device__ __forceinline__ float mul_nc(float a, float b)
{
#pragma clang fp contract(off)
    return a * b;
}
__device__ __forceinline__ float add_nc(float a, float b)
{
#pragma clang fp contract(off)
    return a + b;
}

__device__ __forceinline__ float widen(uint32_t v, uint32_t sel)
{
    return __uint_as_float(__builtin_amdgcn_perm(0u, v, sel));
}
__device__ __forceinline__ float bf_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// acc + w * v[lane-1] and acc + w * v[lane+1] over the whole wave (the lanes
// without a neighbour read 0), each one v_fmac_f32 with a DPP wave shift of
// its first operand: the compiler keeps the shift as a separate v_mov for a
// fused multiply-add.  The s_nop provides the two wait states a DPP read
// needs after a VALU write of its source, which the compiler does not track
// inside inline assembly.
__device__ __forceinline__ float fmac_left(float acc, float v, float w)
{
    asm("s_nop 1\n\tv_fmac_f32_dpp %0, %1, %2 wave_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
        : "+v"(acc)
        : "v"(v), "v"(w));
    return acc;
}

__device__ __forceinline__ float fmac_right(float acc, float v, float w)
{
    asm("s_nop 1\n\tv_fmac_f32_dpp %0, %1, %2 wave_shl:1 row_mask:0xf bank_mask:0xf bound_ctrl:1"
        : "+v"(acc)
        : "v"(v), "v"(w));
    return acc;
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> bf16 (RNE) in one v_cvt_pk_bf16_f32, lo in the low half.
__device__ __forceinline__ uint32_t pack2(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// One fp32 -> bf16 (RNE) in the low half, for 16-bit stores (the high half
// holds bf16 zero and is not meant to be read).
__device__ __forceinline__ uint32_t pack1(float v) { return pack2(v, 0.f); }

// Component k (0..3) of a 16-byte piece; k is a constant once unrolled.
__device__ __forceinline__ uint32_t part(const uint4 &v, int k)
{
    return k == 0 ? v.x : (k == 1 ? v.y : (k == 2 ? v.z : v.w));
}

// Element e (0..7) of a lane's 8-line piece (the lane's position on lines
// 8q..8q+7 of a block), widened with the selector pair of the lane, or
// unmasked.
__device__ __forceinline__ float elem(const uint4 &v, int e, uint32_t sel_lo, uint32_t sel_hi)
{
    return widen(part(v, e >> 1), (e & 1) ? sel_hi : sel_lo);
}
__device__ __forceinline__ float elem(const uint4 &v, int e)
{
    const uint32_t d = part(v, e >> 1);
    return (e & 1) ? bf_hi(d) : bf_lo(d);
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

__device__ __forceinline__ uint32_t lds_u16(const uint8_t *base, uint32_t byte_off)
{
    return *reinterpret_cast<const uint16_t *>(base + byte_off);
}
__device__ __forceinline__ uint32_t lds_u32(const uint8_t *base, uint32_t byte_off)
{
    return *reinterpret_cast<const uint32_t *>(base + byte_off);
}

}  // namespace cdna
}  // namespace gspn
