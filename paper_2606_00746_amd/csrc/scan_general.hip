// Line scans for planes with a side above 64 (up to GSPN_MAX_SIDE).
//
// A workgroup runs one line scan; each thread owns positions j, j + NT, ...
// of the line and the previous line's states are read from a triple-buffered
// LDS line (one barrier per step).  The per-direction results go through
// fp32 scratch and small merge kernels that sum them in direction order.
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ int nth_dir(int mask, int s)
{
    for (int d = 0; d < 4; ++d) {
        if (mask & (1 << d)) {
            if (s == 0)
                return d;
            --s;
        }
    }
    return 0;
}

// ys[s][b][c][H][W] = u_d * h_d for the s-th direction of the mask.
template <typename S>
__global__ __launch_bounds__(kThreads) void fwd_general_kernel(
    const S *__restrict__ x, const S *__restrict__ w, const S *__restrict__ lam,
    const S *__restrict__ u, float *__restrict__ ys, int mask, int B, int C, int G, int H, int W,
    int pm)
{
    extern __shared__ float hb[];  // [3][P]
    int idx = blockIdx.x;
    const int c = idx % C;
    idx /= C;
    const int b = idx % B;
    const int s = idx / B;
    const int d = nth_dir(mask, s);
    const int g = c / (C / G);
    const int L = scan_len(d, H, W);
    const int P = line_len(d, H, W);
    const int HW = H * W;
    const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
    const S *xp = x + ((int64_t)b * C + c) * HW;
    const S *lp = lam + pd;
    const S *up = u + pd;
    float *yp = ys + pd;
    const S *wp = w + (((int64_t)s * B + b) * G + g) * 3 * HW;

    for (int i = 0; i < L; ++i) {
        float *cur = hb + (i % 3) * P;
        const float *prev = hb + ((i + 2) % 3) * P;
        for (int j = threadIdx.x; j < P; j += blockDim.x) {
            const Frame f = make_frame(d, j, H, W, W, pm != 0);
            const int e = f.e0 + i * f.es;   // pixel (x, y slots)
            const int q = f.lm(i);           // per-direction planes (lam, u, w)
            float v = load_f(lp + q) * load_f(xp + e);
            if (i > 0) {
                v = fmaf(load_f(wp + HW + q), prev[j], v);
                if (j > 0)
                    v = fmaf(load_f(wp + q), prev[j - 1], v);
                if (j + 1 < P)
                    v = fmaf(load_f(wp + 2 * HW + q), prev[j + 1], v);
            }
            cur[j] = v;
            yp[e] = load_f(up + q) * v;
        }
        __syncthreads();
    }
}

// out[e] = sum over the D slots of in[s * n + e], in slot order.
template <typename S>
__global__ __launch_bounds__(256) void sum_slots_kernel(const float *__restrict__ in,
                                                        S *__restrict__ out, int64_t n, int D)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        float sum = 0.f;
        for (int s = 0; s < D; ++s)
            sum += in[s * n + e];
        store_f(out + e, sum);
    }
}

// One workgroup per (direction slot, batch, group); the group's channels run
// one after another, so the group's weight gradient (fp32, dws) has a single
// writer.  hs holds the line states of the current channel.
template <typename S>
__global__ __launch_bounds__(kThreads) void bwd_general_kernel(
    const S *__restrict__ x, const S *__restrict__ w, const S *__restrict__ lam,
    const S *__restrict__ u, const S *__restrict__ dy, float *__restrict__ dxs,
    float *__restrict__ dws, S *__restrict__ dlam, S *__restrict__ du,
    float *__restrict__ hs_all, int mask, int B, int C, int G, int H, int W, int pm)
{
    extern __shared__ float ab[];  // [3][P] adjoint lines
    int idx = blockIdx.x;
    const int g = idx % G;
    idx /= G;
    const int b = idx % B;
    const int s = idx / B;
    const int d = nth_dir(mask, s);
    const int L = scan_len(d, H, W);
    const int P = line_len(d, H, W);
    const int HW = H * W;
    const int cpg = C / G;
    const int64_t unit = ((int64_t)s * B + b) * G + g;
    const S *wp = w + unit * 3 * HW;
    float *dwp = dws + unit * 3 * HW;
    float *hs = hs_all + unit * HW;   // [L][P]

    for (int cl = 0; cl < cpg; ++cl) {
        const int c = g * cpg + cl;
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const S *xp = x + ((int64_t)b * C + c) * HW;
        const S *dyp = dy + ((int64_t)b * C + c) * HW;
        const S *lp = lam + pd;
        const S *up = u + pd;

        for (int i = 0; i < L; ++i) {
            for (int j = threadIdx.x; j < P; j += blockDim.x) {
                const Frame f = make_frame(d, j, H, W, W, pm != 0);
                const int e = f.e0 + i * f.es;
                const int q = f.lm(i);
                float v = load_f(lp + q) * load_f(xp + e);
                if (i > 0) {
                    const float *prev = hs + (i - 1) * P;
                    v = fmaf(load_f(wp + HW + q), prev[j], v);
                    if (j > 0)
                        v = fmaf(load_f(wp + q), prev[j - 1], v);
                    if (j + 1 < P)
                        v = fmaf(load_f(wp + 2 * HW + q), prev[j + 1], v);
                }
                hs[i * P + j] = v;
            }
            __syncthreads();
        }

        for (int i = L - 1; i >= 0; --i) {
            float *cur = ab + (i % 3) * P;
            const float *next = ab + ((i + 1) % 3) * P;
            for (int j = threadIdx.x; j < P; j += blockDim.x) {
                const Frame f = make_frame(d, j, H, W, W, pm != 0);
                const int e = f.e0 + i * f.es;   // pixel (x, dy, dx slots)
                const int q = f.lm(i);           // per-direction planes (lam, u, w, dlam, du, dw)
                const float dyv = load_f(dyp + e);
                float a = load_f(up + q) * dyv;
                if (i + 1 < L) {
                    a = fmaf(load_f(wp + HW + f.lm(i + 1)), next[j], a);
                    if (j + 1 < P)   // target j+1 on line i+1 reads j through its tap 0
                        a = fmaf(load_f(wp + f.lm_at(i + 1, j + 1)), next[j + 1], a);
                    if (j > 0)       // target j-1 on line i+1 reads j through its tap 2
                        a = fmaf(load_f(wp + 2 * HW + f.lm_at(i + 1, j - 1)), next[j - 1], a);
                }
                cur[j] = a;
                const float hv = hs[i * P + j];
                store_f(du + pd + q, dyv * hv);
                store_f(dlam + pd + q, a * load_f(xp + e));
                dxs[pd + e] = a * load_f(lp + q);
                for (int k = 0; k < 3; ++k) {
                    const int jj = j + k - 1;
                    const bool valid = i > 0 && jj >= 0 && jj < P;
                    const float t = valid ? a * hs[(i - 1) * P + jj] : 0.f;
                    float *dst = dwp + k * HW + q;
                    *dst = (cl == 0) ? t : *dst + t;
                }
            }
            __syncthreads();
        }
    }
}

template <typename S>
__global__ __launch_bounds__(256) void cast_kernel(const float *__restrict__ in, S *__restrict__ out,
                                                   int64_t n)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x)
        store_f(out + e, in[e]);
}

unsigned grid_for(int64_t n)
{
    int64_t blocks = (n + 255) / 256;
    return (unsigned)(blocks < 16384 ? blocks : 16384);
}

template <typename S>
hipError_t fwd_general_t(const Problem &p, hipStream_t st)
{
    const int D = __builtin_popcount(p.mask);
    const int64_t n = (int64_t)p.B * p.C * p.H * p.W;
    const int maxp = p.H > p.W ? p.H : p.W;
    float *ys = nullptr;
    hipError_t e = p.ws->take((void **)&ys, (size_t)D * n * sizeof(float));
    if (e != hipSuccess || p.ws->counting)
        return e;
    hipLaunchKernelGGL((fwd_general_kernel<S>), dim3((unsigned)(D * p.B * p.C)), dim3(kThreads),
                       3 * maxp * sizeof(float), st, (const S *)p.x, (const S *)p.w,
                       (const S *)p.lam, (const S *)p.u, ys, p.mask, p.B, p.C, p.G, p.H, p.W,
                       p.layout);
    e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL((sum_slots_kernel<S>), dim3(grid_for(n)), dim3(256), 0, st,
                           (const float *)ys, (S *)p.y, n, D);
        e = hipGetLastError();
    }
    return e;
}

template <typename S>
hipError_t bwd_general_t(const Problem &p, hipStream_t st)
{
    const int D = __builtin_popcount(p.mask);
    const int64_t n = (int64_t)p.B * p.C * p.H * p.W;
    const int64_t HW = (int64_t)p.H * p.W;
    const int64_t units = (int64_t)D * p.B * p.G;
    const int maxp = p.H > p.W ? p.H : p.W;
    // dx terms per direction, the groups' fp32 weight gradients, line states
    float *dxs = nullptr;
    const int64_t nf = D * n + units * 3 * HW + units * HW;
    hipError_t e = p.ws->take((void **)&dxs, (size_t)nf * sizeof(float));
    if (e != hipSuccess || p.ws->counting)
        return e;
    float *dws = dxs + D * n, *hs = dws + units * 3 * HW;
    hipLaunchKernelGGL((bwd_general_kernel<S>), dim3((unsigned)units), dim3(kThreads),
                       3 * maxp * sizeof(float), st, (const S *)p.x, (const S *)p.w,
                       (const S *)p.lam, (const S *)p.u, (const S *)p.dy, dxs, dws,
                       (S *)p.dlam, (S *)p.du, hs, p.mask, p.B, p.C, p.G, p.H, p.W, p.layout);
    e = hipGetLastError();
    if (e == hipSuccess) {
        hipLaunchKernelGGL((sum_slots_kernel<S>), dim3(grid_for(n)), dim3(256), 0, st,
                           (const float *)dxs, (S *)p.dx, n, D);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL((cast_kernel<S>), dim3(grid_for(units * 3 * HW)), dim3(256), 0, st,
                           (const float *)dws, (S *)p.dw, units * 3 * HW);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace

hipError_t launch_fwd_general(const Problem &p, hipStream_t st)
{
    return p.dtype == 0 ? fwd_general_t<float>(p, st) : fwd_general_t<bf16_t>(p, st);
}

hipError_t launch_bwd_general(const Problem &p, hipStream_t st)
{
    return p.dtype == 0 ? bwd_general_t<float>(p, st) : bwd_general_t<bf16_t>(p, st);
}

}  // namespace gspn
