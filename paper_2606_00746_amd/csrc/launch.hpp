// Host-side kernel launchers of libgspn (internal; not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gspn {

// Device memory a call may use beyond its inputs and outputs, handed in by
// the caller.  take() returns 256-byte aligned pieces in order; nothing is
// ever returned to it within a call.  In counting mode nothing is launched:
// the launchers only add up what they would take (the workspace-size query
// runs the same code as the call).
struct Workspace {
    char *base = nullptr;
    size_t size = 0;
    size_t used = 0;
    bool counting = false;
    // hipErrorOutOfMemory when the caller's workspace is too small (the
    // library never allocates, so this is the only source of that code)
    hipError_t take(void **p, size_t bytes)
    {
        const size_t off = (used + 255) & ~(size_t)255;
        used = off + bytes;
        *p = nullptr;
        if (counting)
            return hipSuccess;
        if (used > size)
            return hipErrorOutOfMemory;
        *p = base + off;
        return hipSuccess;
    }
};

// Layout of the per-direction tensors (lam, u, w and their gradients).
enum Layout { kBlocked = 0, kPixelMajor = 1 };

// The blocked copies a training pair keeps in its reserve (take_reserve):
// the weights (all directions, or with one channel per group only the
// horizontal directions' ones), and lambda and u of the horizontal
// directions.  Null where a piece has no element.
struct ReserveParts {
    void *w = nullptr, *lamh = nullptr, *uh = nullptr;
};

struct Problem {
    const void *x, *w, *lam, *u, *dy;
    void *y, *dx, *dw, *dlam, *du;
    int mask, B, C, G, H, W, dtype;
    int layout;
    Workspace *ws;
    // channel slots per step of the register-streamed backward: 0 the
    // planner's choice, 4 or 8 that plan where the shape can take it
    int slots = 0;
    // w is already in the blocked order of its direction although the call
    // is pixel-major (weights the library formed itself, launch_norm_blocked)
    bool w_blocked = false;
    // Reserve of a training pair (pixel-major register-streamed shapes): the
    // forward writes into it the blocked copies that the backward of the same
    // inputs would otherwise make (rs_write), the backward reads them from
    // it (rs_read).  The entry point takes the parts once (take_reserve, the
    // same order for both calls, so that their offsets agree; counting mode
    // sizes it) and hands them over in rsp.
    Workspace *rs = nullptr;
    bool rs_write = false, rs_read = false;
    const ReserveParts *rsp = nullptr;
};

// Takes the reserve's parts from p.rs.  Weights the library forms itself
// (w_blocked) are kept for every direction.
inline hipError_t take_reserve(const Problem &p, ReserveParts *r)
{
    const int64_t HW = (int64_t)p.H * p.W;
    const int nvd = __builtin_popcount(p.mask & 3), nhd = __builtin_popcount(p.mask & 12);
    const bool pc = p.C == p.G && !p.w_blocked;
    const int64_t nw = (int64_t)(pc ? nhd : nvd + nhd) * p.B * p.G * 3 * HW;
    const int64_t nh = (int64_t)nhd * p.B * p.C * HW;
    hipError_t e = hipSuccess;
    if (nw > 0)
        e = p.rs->take(&r->w, (size_t)nw * 2);
    if (e == hipSuccess && nh > 0)
        e = p.rs->take(&r->lamh, (size_t)nh * 2);
    if (e == hipSuccess && nh > 0)
        e = p.rs->take(&r->uh, (size_t)nh * 2);
    return e;
}

// Planes whose sides are both <= kSmallSide run on the register-resident path.
constexpr int kSmallSide = 64;

// LDS a workgroup may use on gfx950 (the only target of this library).
constexpr int kLdsBytes = 160 * 1024;

hipError_t launch_fwd_small(const Problem &p, hipStream_t s);
hipError_t launch_bwd_small(const Problem &p, hipStream_t s);
bool tiny_supported(const Problem &p);
hipError_t launch_fwd_tiny(const Problem &p, hipStream_t s);
hipError_t launch_bwd_tiny(const Problem &p, hipStream_t s);
// Weights from logits (dw == nullptr) or the logits' gradient from dw, for
// every direction of p (Sec. 3, Eq. (row_stochastic_norm)); wt, dw, out in
// p's storage type and weight layout.
hipError_t launch_norm(const Problem &p, const void *wt, const void *dw, void *out, hipStream_t s);
bool med_supported(const Problem &p);
hipError_t launch_fwd_med(const Problem &p, hipStream_t s);
hipError_t launch_bwd_med(const Problem &p, hipStream_t s);
// one side of the register-streamed path (instantiated per side)
template <int S>
hipError_t med_fwd(const Problem &p, hipStream_t s);
template <int S>
hipError_t med_bwd(const Problem &p, hipStream_t s);
bool wide_supported(const Problem &p);
// Pixel-major problems of the register-streamed shapes: the weights are
// re-laid out into the blocked order (launch_w_to_blocked, workspace of
// |w| bytes) when a group has at least kReblockCpg channels, so that the
// copy costs at most a quarter of the lambda traffic; then the forward is
// launch_fwd_pm.
constexpr int kReblockCpg = 1;
inline bool pm_weights_reblocked(const Problem &p)
{
    return p.layout == kPixelMajor && p.C / p.G >= kReblockCpg;
}
hipError_t launch_w_to_blocked(const Problem &p, void *wb, hipStream_t s);
// nv vertical planes, then nh horizontal ones, of H x W (multiples of 8,
// W <= 256, or any H with W = 8 * (H's pieces) as a 16-byte piece transpose)
// pixel-major -> blocked line-major (scan_wide.hip, pieces_kernel).
hipError_t launch_planes_pieces(const void *src, void *dst, int64_t nv, int64_t nh, int H, int W,
                                hipStream_t s);
// n planes of a horizontal direction (square side S of the register-streamed
// shapes) into the blocked order of that direction.
hipError_t launch_planes_to_blocked(const void *src, void *dst, int n, int S, hipStream_t s);
// lam and u of the horizontal directions into blocked copies [nh][B][C][plane].
hipError_t launch_horiz_to_blocked(const Problem &p, void *lamh, void *uh, hipStream_t s);
hipError_t launch_fwd_pm(const Problem &p, hipStream_t s);
// Pixel-major logits -> normalized weights in the blocked order (|w| bytes
// at wb), for the register-streamed shapes: the normalization of
// launch_norm and the re-layout of launch_w_to_blocked in one pass.
hipError_t launch_norm_blocked(const Problem &p, const void *wt, void *wb, hipStream_t s);
hipError_t launch_fwd_wide(const Problem &p, hipStream_t s);
hipError_t launch_fwd_general(const Problem &p, hipStream_t s);
hipError_t launch_bwd_general(const Problem &p, hipStream_t s);

// 1x1 convolutions of the latent sublayer (bf16, fp32 accumulation):
// y[b] = a x[b] with a [M][K], x [B][K][H*W], y [B][M][H*W]; and the
// parameter product that writes u, lambda and normalized w of every
// direction in the scan's blocked layout from x_c [B][Cc][H*W].
// launch_project may read x on a different grid Hi x Wi sharing the top-left
// corner (pixels outside it read as 0); launch_latent_params may write planes
// of a grid padded beyond the image Hv x Wv, whose edges decide the taps
// (0: the same grid).
hipError_t launch_project(const void *a, const void *x, void *y, int B, int M, int K, int H, int W,
                          hipStream_t s, int Hi = 0, int Wi = 0);
hipError_t launch_latent_params(const void *xc, const void *lu, const void *ll, const void *lw,
                                void *u, void *lam, void *w, int mask, int B, int Cc, int H, int W,
                                hipStream_t s, int Hv = 0, int Wv = 0);


}  // namespace gspn
