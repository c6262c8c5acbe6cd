// Register-resident line scans for planes with H, W <= 64.
//
// One lane owns one position of a line (the perpendicular axis); a line of P
// positions occupies T lanes (T = 16, 32 or 64, T >= P) and a wave holds
// 64 / T lines, i.e. 64 / T channels.  The hidden state h stays in a VGPR for
// the whole scan; the tridiagonal step reads the two neighbours of the
// previous line with DPP lane shifts (Sec. 3, Eq. (gspn_recurrence)).
//
// Forward: a workgroup is 4 waves, one per scan direction, over the same
// 64 / T channels.  Each wave keeps its direction's contributions u_d * h_d in
// registers and the four are summed in direction-bit order through an fp32
// LDS plane, so y is stored once, in the storage type.
//
// Backward: a workgroup is up to 8 waves over `cw` channels of one weight
// group.  Every wave runs the directions one after another: a forward sweep
// that keeps the line states h_0..h_{L-1} in registers, then the reverse
// adjoint sweep.  dx accumulates in an fp32 LDS plane per channel; the weight
// gradient of each step is reduced over the workgroup's channels through LDS
// (all waves step in lock-step, one barrier per step) and written either as
// the final dw or, when a group spans several workgroups, as an fp32 partial
// that a second kernel sums in fixed order.
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

template <int T, typename S>
__global__ __launch_bounds__(256) void fwd_small_kernel(
    const S *__restrict__ x, const S *__restrict__ w, const S *__restrict__ lam,
    const S *__restrict__ u, S *__restrict__ y, int mask, int B, int C, int G, int H, int W,
    int pm)
{
    constexpr int NL = 64 / T;        // lines (channels) per wave
    constexpr int PITCH = T + 1;      // odd LDS row pitch: column walks are conflict-free
    __shared__ float acc[NL * T * PITCH];

    const int d = threadIdx.x >> 6;   // this wave's direction index
    const int lane = threadIdx.x & 63;
    const int line = lane / T;
    const int j = lane % T;
    const int nblk = (C + NL - 1) / NL;
    const int b = blockIdx.x / nblk;
    const int c0 = (blockIdx.x % nblk) * NL;
    const int c = c0 + line;
    const bool cvalid = c < C;
    const int cc = cvalid ? c : C - 1;
    const int g = cc / (C / G);
    const int bit = 1 << d;
    const bool mine = (mask & bit) != 0;
    const int HW = H * W;
    const int P = line_len(d, H, W);
    const bool active = cvalid && j < P;
    const int jc = active ? j : 0;

    float yr[T];
    if (mine) {
        const Frame f = make_frame(d, jc, H, W, W, pm != 0);
        const int s = dir_slot(mask, bit);
        const S *xp = x + ((int64_t)b * C + cc) * HW;
        const int64_t pd = (((int64_t)s * B + b) * C + cc) * HW;
        const S *lp = lam + pd;
        const S *up = u + pd;
        const S *wp = w + (((int64_t)s * B + b) * G + g) * 3 * HW;
        const bool m0 = active && j > 0;
        const bool m2 = active && j + 1 < P;
        float h = 0.f;
        // Steps past the line's end (T > L) repeat its last step's reads and
        // leave results that the merge never reads: no branch per step, so
        // the compiler can issue the loads of later steps early.
#pragma unroll
        for (int i = 0; i < T; ++i) {
            const int ic = i < f.L ? i : f.L - 1;
            const int e = f.e0 + ic * f.es;      // pixel (x)
            const int q = f.lm(ic);              // per-direction planes (lam, u, w)
            float inj = load_f(lp + q) * load_f(xp + e);
            inj = active ? inj : 0.f;
            float hn = inj;
            if (i > 0) {
                float w0 = load_f(wp + q);
                float w1 = load_f(wp + HW + q);
                float w2 = load_f(wp + 2 * HW + q);
                w0 = m0 ? w0 : 0.f;
                w1 = active ? w1 : 0.f;
                w2 = m2 ? w2 : 0.f;
                const float hl = from_left<T>(h);
                const float hr = from_right<T>(h);
                hn = fmaf(w1, h, hn);
                hn = fmaf(w0, hl, hn);
                hn = fmaf(w2, hr, hn);
            }
            h = hn;
            yr[i] = load_f(up + q) * h;
        }
    }

    // Merge the directions in bit order: the first one present stores, the
    // others add.  One direction per phase, so every sum has a fixed order.
    float *a = acc + line * T * PITCH;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        if (d == p && mine && active) {
            const Frame fl = make_frame(d, jc, H, W, PITCH);
            const bool first = (mask & ((1 << p) - 1)) == 0;
#pragma unroll
            for (int i = 0; i < T; ++i) {
                if (i < fl.L) {
                    const int e = fl.e0 + i * fl.es;
                    a[e] = first ? yr[i] : a[e] + yr[i];
                }
            }
        }
        __syncthreads();
    }

    const int nch = min(NL, C - c0);
    S *yb = y + ((int64_t)b * C + c0) * HW;
    for (int t = threadIdx.x; t < nch * HW; t += blockDim.x) {
        const int l = t / HW;
        const int rc = t - l * HW;
        const int r = rc / W;
        const int col = rc - r * W;
        store_f(yb + t, acc[(l * T + r) * PITCH + col]);
    }
}

template <int T, typename S>
__global__ __launch_bounds__(512) void bwd_small_kernel(
    const S *__restrict__ x, const S *__restrict__ w, const S *__restrict__ lam,
    const S *__restrict__ u, const S *__restrict__ dy, S *__restrict__ dx,
    S *__restrict__ dw, S *__restrict__ dlam, S *__restrict__ du, float *__restrict__ dwp,
    int mask, int B, int C, int G, int H, int W, int cw, int nchunk, int pm)
{
    constexpr int NL = 64 / T;
    extern __shared__ float smem[];
    const int pitch = W | 1;                  // odd pitch: column walks are conflict-free
    const int plane = H * pitch;
    float *X = smem;                          // [cw][H][pitch]   dx accumulators
    float *slots = smem + cw * plane;         // [2][cw][3][T]    per-step dw terms

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int line = lane / T;
    const int j = lane % T;
    const int cpg = C / G;
    const int chunk = blockIdx.x % nchunk;
    const int bg = blockIdx.x / nchunk;
    const int g = bg % G;
    const int b = bg / G;
    const int cfirst = chunk * cw;            // first channel of this chunk, within the group
    const int nvalid = min(cw, cpg - cfirst);
    const int q = wave * NL + line;           // channel slot inside the workgroup
    const bool cvalid = q < nvalid;
    const int c = g * cpg + cfirst + (cvalid ? q : 0);
    const int HW = H * W;
    const int D = __popc(mask);
    const int dfirst = __ffs(mask) - 1;
    float *Xq = X + q * plane;
    const S *xp = x + ((int64_t)b * C + c) * HW;
    const S *dyp = dy + ((int64_t)b * C + c) * HW;

    for (int d = 0; d < 4; ++d) {
        const int bit = 1 << d;
        if (!(mask & bit))
            continue;
        const int s = dir_slot(mask, bit);
        const int L = scan_len(d, H, W);
        const int P = line_len(d, H, W);
        const bool active = cvalid && j < P;
        const int jc = active ? j : 0;
        const Frame f = make_frame(d, jc, H, W, W, pm != 0);
        const Frame fl = make_frame(d, jc, H, W, pitch);
        const int64_t pd = (((int64_t)s * B + b) * C + c) * HW;
        const S *lp = lam + pd;
        const S *up = u + pd;
        S *dlp = dlam + pd;
        S *dup = du + pd;
        const S *wp = w + (((int64_t)s * B + b) * G + g) * 3 * HW;
        const bool m0 = active && j > 0;
        const bool m2 = active && j + 1 < P;

        // Forward sweep: line states of this direction, kept in registers.
        float hist[T];
        float h = 0.f;
#pragma unroll
        for (int i = 0; i < T; ++i) {
            if (i < L) {
                const int e = f.e0 + i * f.es;   // pixel (x)
                const int q = f.lm(i);           // per-direction planes (lam, u, w)
                float inj = load_f(lp + q) * load_f(xp + e);
                inj = active ? inj : 0.f;
                float hn = inj;
                if (i > 0) {
                    float w0 = load_f(wp + q);
                    float w1 = load_f(wp + HW + q);
                    float w2 = load_f(wp + 2 * HW + q);
                    w0 = m0 ? w0 : 0.f;
                    w1 = active ? w1 : 0.f;
                    w2 = m2 ? w2 : 0.f;
                    const float hl = from_left<T>(h);
                    const float hr = from_right<T>(h);
                    hn = fmaf(w1, h, hn);
                    hn = fmaf(w0, hl, hn);
                    hn = fmaf(w2, hr, hn);
                }
                h = hn;
                hist[i] = h;
            }
        }

        // Reverse sweep: adjoint a_i from a_{i+1} through the transposed
        // tridiagonal step (the neighbours' taps of line i+1).
        float an = 0.f;
#pragma unroll
        for (int i = T - 1; i >= 0; --i) {
            if (i < L) {
                const int e = f.e0 + i * f.es;   // pixel (x, dy)
                const int qd = f.lm(i);          // per-direction planes (lam, u, w, dlam, du)
                const float dyv = load_f(dyp + e);
                float a = load_f(up + qd) * dyv;
                if (i + 1 < L) {
                    const int qn = f.lm(i + 1);
                    float w0 = load_f(wp + qn);
                    float w1 = load_f(wp + HW + qn);
                    float w2 = load_f(wp + 2 * HW + qn);
                    w0 = m0 ? w0 : 0.f;
                    w1 = active ? w1 : 0.f;
                    w2 = m2 ? w2 : 0.f;
                    // target j+1 reads this position through its tap 0,
                    // target j-1 through its tap 2.
                    const float q0 = from_right<T>(w0 * an);
                    const float q2 = from_left<T>(w2 * an);
                    a = fmaf(w1, an, a);
                    a += q0;
                    a += q2;
                }
                a = active ? a : 0.f;
                const float xv = load_f(xp + e);
                const float lv = load_f(lp + qd);
                if (active) {
                    store_f(dup + qd, dyv * hist[i]);
                    store_f(dlp + qd, a * xv);
                    const int ae = fl.e0 + i * fl.es;
                    Xq[ae] = (d == dfirst) ? a * lv : Xq[ae] + a * lv;
                }
                // weight-gradient terms of line i (zero on line 0 and on
                // taps that leave the grid)
                float t0 = 0.f, t1 = 0.f, t2 = 0.f;
                if (i > 0) {
                    const float hp = hist[i - 1];
                    const float hl = from_left<T>(hp);
                    const float hr = from_right<T>(hp);
                    t0 = m0 ? a * hl : 0.f;
                    t1 = active ? a * hp : 0.f;
                    t2 = m2 ? a * hr : 0.f;
                }
                float *sl = slots + ((i & 1) * cw + q) * 3 * T;
                sl[j] = t0;
                sl[T + j] = t1;
                sl[2 * T + j] = t2;
                __syncthreads();
                for (int t = threadIdx.x; t < 3 * P; t += blockDim.x) {
                    const int k = t / P;
                    const int jj = t - k * P;
                    const float *src = slots + (i & 1) * cw * 3 * T + k * T + jj;
                    float sum = 0.f;
                    for (int qq = 0; qq < nvalid; ++qq)
                        sum += src[qq * 3 * T];
                    const Frame ft = make_frame(d, jj, H, W, W, pm != 0);
                    const int et = k * HW + ft.lm(i);
                    const int64_t unit = ((int64_t)s * B + b) * G + g;
                    if (nchunk == 1)
                        store_f(dw + unit * 3 * HW + et, sum);
                    else
                        dwp[((int64_t)chunk * D * B * G + unit) * 3 * HW + et] = sum;
                }
                an = a;
            }
        }
        __syncthreads();   // slot buffers are reused by the next direction
    }

    // dx of this wave's channels
    const int nmine = max(0, min(NL, nvalid - wave * NL));
    S *dxb = dx + ((int64_t)b * C + g * cpg + cfirst + wave * NL) * HW;
    const float *Xw = X + wave * NL * plane;
    for (int t = lane; t < nmine * HW; t += 64) {
        const int l = t / HW;
        const int rc = t - l * HW;
        const int r = rc / W;
        const int col = rc - r * W;
        store_f(dxb + t, Xw[l * plane + r * pitch + col]);
    }
}

// dw = sum over chunks of the fp32 partials, in chunk order.
template <typename S>
__global__ __launch_bounds__(256) void dw_reduce_kernel(const float *__restrict__ dwp,
                                                        S *__restrict__ dw, int64_t n, int nchunk)
{
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
         e += (int64_t)gridDim.x * blockDim.x) {
        float sum = 0.f;
        for (int k = 0; k < nchunk; ++k)
            sum += dwp[k * n + e];
        store_f(dw + e, sum);
    }
}

template <int T, typename S>
hipError_t fwd_small_t(const Problem &p, hipStream_t st)
{
    if (p.ws->counting)
        return hipSuccess;
    constexpr int NL = 64 / T;
    const int nblk = (p.C + NL - 1) / NL;
    const dim3 grid((unsigned)(p.B * nblk));
    hipLaunchKernelGGL((fwd_small_kernel<T, S>), grid, dim3(256), 0, st,
                       (const S *)p.x, (const S *)p.w, (const S *)p.lam, (const S *)p.u, (S *)p.y,
                       p.mask, p.B, p.C, p.G, p.H, p.W, p.layout);
    return hipGetLastError();
}

template <int T, typename S>
hipError_t bwd_small_t(const Problem &p, hipStream_t st)
{
    constexpr int NL = 64 / T;
    hipError_t e = hipSuccess;
    const int lds_max = kLdsBytes;
    const int pitch = p.W | 1;
    const size_t per_ch = (size_t)p.H * pitch * 4 + 2 * 3 * T * 4;
    const int cpg = p.C / p.G;
    int cap = (int)((size_t)lds_max / per_ch);
    cap = cap < 8 * NL ? cap : 8 * NL;
    cap = cap / NL * NL;
    if (cap < NL)
        return hipErrorInvalidConfiguration;
    const int nchunk = (cpg + cap - 1) / cap;
    int cw = (cpg + nchunk - 1) / nchunk;
    cw = (cw + NL - 1) / NL * NL;
    const int nwaves = cw / NL;
    const size_t lds = (size_t)cw * per_ch;
    const int D = __builtin_popcount(p.mask);
    const int64_t ndw = (int64_t)D * p.B * p.G * 3 * p.H * p.W;

    float *dwp = nullptr;
    if (nchunk > 1) {
        e = p.ws->take((void **)&dwp, (size_t)nchunk * ndw * sizeof(float));
        if (e != hipSuccess)
            return e;
    }
    if (p.ws->counting)
        return hipSuccess;
    e = hipFuncSetAttribute((const void *)bwd_small_kernel<T, S>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess)
        return e;
    const dim3 grid((unsigned)(p.B * p.G * nchunk));
    hipLaunchKernelGGL((bwd_small_kernel<T, S>), grid, dim3(64 * nwaves), lds, st,
                       (const S *)p.x, (const S *)p.w, (const S *)p.lam, (const S *)p.u,
                       (const S *)p.dy, (S *)p.dx, (S *)p.dw, (S *)p.dlam, (S *)p.du, dwp,
                       p.mask, p.B, p.C, p.G, p.H, p.W, cw, nchunk, p.layout);
    e = hipGetLastError();
    if (e == hipSuccess && nchunk > 1) {
        int64_t blocks = (ndw + 255) / 256;
        blocks = blocks < 8192 ? blocks : 8192;
        hipLaunchKernelGGL((dw_reduce_kernel<S>), dim3((unsigned)blocks), dim3(256), 0, st,
                           (const float *)dwp, (S *)p.dw, ndw, nchunk);
        e = hipGetLastError();
    }
    return e;
}

template <int T>
hipError_t fwd_small_dt(const Problem &p, hipStream_t st)
{
    return p.dtype == 0 ? fwd_small_t<T, float>(p, st) : fwd_small_t<T, bf16_t>(p, st);
}

template <int T>
hipError_t bwd_small_dt(const Problem &p, hipStream_t st)
{
    return p.dtype == 0 ? bwd_small_t<T, float>(p, st) : bwd_small_t<T, bf16_t>(p, st);
}

int lanes_per_line(int H, int W)
{
    const int m = H > W ? H : W;
    return m <= 16 ? 16 : (m <= 32 ? 32 : 64);
}

}  // namespace

hipError_t launch_fwd_small(const Problem &p, hipStream_t st)
{
    switch (lanes_per_line(p.H, p.W)) {
    case 16: return fwd_small_dt<16>(p, st);
    case 32: return fwd_small_dt<32>(p, st);
    default: return fwd_small_dt<64>(p, st);
    }
}

hipError_t launch_bwd_small(const Problem &p, hipStream_t st)
{
    switch (lanes_per_line(p.H, p.W)) {
    case 16: return bwd_small_dt<16>(p, st);
    case 32: return bwd_small_dt<32>(p, st);
    default: return bwd_small_dt<64>(p, st);
    }
}

}  // namespace gspn
