// Host-side kernel launchers of libgspn (internal; not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gspn {

struct Problem {
    const void *x, *w, *lam, *u, *dy;
    void *y, *dx, *dw, *dlam, *du;
    int mask, B, C, G, H, W, dtype;
};

// Planes whose sides are both <= kSmallSide run on the register-resident path.
constexpr int kSmallSide = 64;

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
bool wide_supported(const Problem &p);
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

// Stream-ordered scratch from the device's default pool.
hipError_t scratch_alloc(void **ptr, size_t bytes, hipStream_t s);
hipError_t scratch_free(void *ptr, hipStream_t s);

}  // namespace gspn
