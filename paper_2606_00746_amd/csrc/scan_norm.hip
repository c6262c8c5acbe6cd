// Tridiagonal weights from their logits, Sec. 3, Eq. (row_stochastic_norm),
// and the gradient with respect to the logits.
//
// For every pixel of a direction's tap planes:
//   s_k = sigmoid(wt_k) for the taps k whose neighbour lies on the grid
//         (0 for the others), S = max(s_0 + s_1 + s_2, kNormEps),
//   w_k = s_k / S,
//   dwt_m = s_m (1 - s_m) (dw_m - sum_k w_k dw_k) / S   (the sum term drops
//         where the clamp holds S at kNormEps).
// A group's weights serve all C/G of its channels, so they are formed once
// here rather than in every channel's scan.
//
// Blocked line-major planes: one 16-byte piece of a full 8-line block holds
// the 8 consecutive lines of one line position, which decides the validity
// of taps 0 and 2; a last, partial block is taken element by element.
// Pixel-major planes: 8 consecutive pixels of an image row at a time.
#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;


__device__ __forceinline__ void load8(const float *p, float (&v)[8])
{
    const float4 a = *reinterpret_cast<const float4 *>(p);
    const float4 b = *reinterpret_cast<const float4 *>(p + 4);
    v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w, v[4] = b.x, v[5] = b.y, v[6] = b.z, v[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t *p, float (&v)[8])
{
    const uint4 a = *reinterpret_cast<const uint4 *>(p);
    const uint32_t q[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        v[2 * e] = __uint_as_float(q[e] << 16);
        v[2 * e + 1] = __uint_as_float(q[e] & 0xffff0000u);
    }
}
__device__ __forceinline__ void store8(float *p, const float (&v)[8])
{
    *reinterpret_cast<float4 *>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4 *>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void store8(bf16_t *p, const float (&v)[8])
{
    gst128(reinterpret_cast<uint4 *>(p),
           make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7])));
}

// Every direction of the mask in one launch: for direction slot s, the B*G
// tap-plane triples of HW elements, lines of P positions, L lines.
// dw == nullptr: write the weights; else the logits' gradient.  vec: the
// planes start on 16-byte boundaries, so full blocks go by 8-element pieces.
template <typename T>
__global__ __launch_bounds__(256) void norm_kernel(const T *__restrict__ wt, const T *__restrict__ dw,
                                                   T *__restrict__ out, int mask, int64_t sets, int H,
                                                   int W, bool vec)
{
    const int HW = H * W;
    // units (pieces, then single elements) per tap-plane triple of each slot
    int64_t cum[5];
    int Ls[4], Ps[4];
    int nd = 0;
    cum[0] = 0;
    for (int d = 0; d < 4; ++d) {
        if (!((mask >> d) & 1))
            continue;
        const int L = d < 2 ? H : W, P = d < 2 ? W : H;
        const int nfull = vec ? L / 8 : 0;
        Ls[nd] = L;
        Ps[nd] = P;
        cum[nd + 1] = cum[nd] + sets * ((int64_t)nfull * P + (int64_t)(L - 8 * nfull) * P);
        ++nd;
    }
    const int64_t n = cum[nd];
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n;
         o += (int64_t)gridDim.x * blockDim.x) {
        int sl = 0;
        while (sl + 1 < nd && o >= cum[sl + 1])
            ++sl;
        const int L = Ls[sl], P = Ps[sl];
        const int nfull = vec ? L / 8 : 0;
        const int64_t pieces = (int64_t)nfull * P;
        const int64_t per = pieces + (int64_t)(L - 8 * nfull) * P;
        const int64_t oo = o - cum[sl];
        const int64_t set = (int64_t)sl * sets + oo / per;
        const int64_t r = oo % per;
        const T *src = wt + set * 3 * HW;
        const T *gsrc = dw ? dw + set * 3 * HW : nullptr;
        T *dst = out + set * 3 * HW;
        if (r < pieces) {
            const int p = (int)(r % P);
            const int64_t e = 8 * r;                    // 8 lines of position p
            const bool on0 = p > 0, on2 = p + 1 < P;
            float t[3][8], v[3][8];
#pragma unroll
            for (int k = 0; k < 3; ++k)
                load8(src + k * HW + e, t[k]);
            if (gsrc) {
                float g[3][8];
#pragma unroll
                for (int k = 0; k < 3; ++k)
                    load8(gsrc + k * HW + e, g[k]);
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float tq[3] = {t[0][q], t[1][q], t[2][q]};
                    const float gq[3] = {g[0][q], g[1][q], g[2][q]};
                    float d[3];
                    norm3_bwd(tq, gq, on0, on2, d);
                    v[0][q] = d[0], v[1][q] = d[1], v[2][q] = d[2];
                }
            } else {
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float tq[3] = {t[0][q], t[1][q], t[2][q]};
                    float wq[3];
                    norm3(tq, on0, on2, wq);
                    v[0][q] = wq[0], v[1][q] = wq[1], v[2][q] = wq[2];
                }
            }
#pragma unroll
            for (int k = 0; k < 3; ++k)
                store8(dst + k * HW + e, v[k]);
        } else {
            // element by element: block q of nl lines, position p
            const int64_t e = 8 * pieces + (r - pieces);
            const int q = (int)(e / (8 * P));
            const int rem = (int)(e - (int64_t)q * 8 * P);
            const int nl = L - 8 * q < 8 ? L - 8 * q : 8;
            const int p = rem / nl;
            const bool on0 = p > 0, on2 = p + 1 < P;
            const float tq[3] = {load_f(src + e), load_f(src + HW + e), load_f(src + 2 * HW + e)};
            float v[3];
            if (gsrc) {
                const float gq[3] = {load_f(gsrc + e), load_f(gsrc + HW + e), load_f(gsrc + 2 * HW + e)};
                norm3_bwd(tq, gq, on0, on2, v);
            } else {
                norm3(tq, on0, on2, v);
            }
#pragma unroll
            for (int k = 0; k < 3; ++k)
                store_f(dst + k * HW + e, v[k]);
        }
    }
}

// Pixel-major tap planes ([3][H][W] per set): a thread takes 8 consecutive
// pixels of an image row when rows are whole 16-byte pieces (vec), else one
// pixel.  The line position deciding taps 0 and 2 is the column for vertical
// directions and the row for horizontal ones.
template <typename T>
__global__ __launch_bounds__(256) void norm_pm_kernel(const T *__restrict__ wt,
                                                      const T *__restrict__ dw, T *__restrict__ out,
                                                      int mask, int64_t sets, int H, int W, bool vec)
{
    const int HW = H * W;
    const int E = vec ? 8 : 1;                      // pixels per thread
    const int per = HW / E;                         // units per tap-plane triple
    int dirs[4];
    int nd = 0;
    for (int d = 0; d < 4; ++d)
        if ((mask >> d) & 1)
            dirs[nd++] = d;
    const int64_t n = (int64_t)nd * sets * per;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n;
         o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t set = o / per;                // slot * sets + (b, g)
        const int r = (int)(o - set * per);
        const int d = dirs[set / sets];
        const int64_t e = (int64_t)r * E;           // first pixel
        const int row = (int)(e / W), col0 = (int)(e - (int64_t)row * W);
        const T *src = wt + set * 3 * HW;
        const T *gsrc = dw ? dw + set * 3 * HW : nullptr;
        T *dst = out + set * 3 * HW;
        if (vec) {
            float t[3][8], v[3][8];
#pragma unroll
            for (int k = 0; k < 3; ++k)
                load8(src + k * HW + e, t[k]);
            float g[3][8];
            if (gsrc) {
#pragma unroll
                for (int k = 0; k < 3; ++k)
                    load8(gsrc + k * HW + e, g[k]);
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int pos = d < 2 ? col0 + q : row;
                const int len = d < 2 ? W : H;
                const bool on0 = pos > 0, on2 = pos + 1 < len;
                const float tq[3] = {t[0][q], t[1][q], t[2][q]};
                float r3[3];
                if (gsrc) {
                    const float gq[3] = {g[0][q], g[1][q], g[2][q]};
                    norm3_bwd(tq, gq, on0, on2, r3);
                } else {
                    norm3(tq, on0, on2, r3);
                }
                v[0][q] = r3[0], v[1][q] = r3[1], v[2][q] = r3[2];
            }
#pragma unroll
            for (int k = 0; k < 3; ++k)
                store8(dst + k * HW + e, v[k]);
        } else {
            const int pos = d < 2 ? col0 : row;
            const int len = d < 2 ? W : H;
            const bool on0 = pos > 0, on2 = pos + 1 < len;
            const float tq[3] = {load_f(src + e), load_f(src + HW + e), load_f(src + 2 * HW + e)};
            float v[3];
            if (gsrc) {
                const float gq[3] = {load_f(gsrc + e), load_f(gsrc + HW + e),
                                     load_f(gsrc + 2 * HW + e)};
                norm3_bwd(tq, gq, on0, on2, v);
            } else {
                norm3(tq, on0, on2, v);
            }
#pragma unroll
            for (int k = 0; k < 3; ++k)
                store_f(dst + k * HW + e, v[k]);
        }
    }
}

template <typename T>
hipError_t launch_norm_t(const Problem &p, const void *wt, const void *dw, void *out, hipStream_t st)
{
    if (p.layout == kPixelMajor) {
        const int64_t HW = (int64_t)p.H * p.W;
        const int64_t sets = (int64_t)p.B * p.G;
        const bool vec = p.W % 8 == 0;
        const int64_t n = (int64_t)__builtin_popcount(p.mask) * sets * (vec ? HW / 8 : HW);
        int64_t blocks = (n + 255) / 256;
        blocks = blocks < 16384 ? blocks : 16384;
        hipLaunchKernelGGL((norm_pm_kernel<T>), dim3((unsigned)blocks), dim3(256), 0, st,
                           static_cast<const T *>(wt), static_cast<const T *>(dw),
                           static_cast<T *>(out), p.mask, sets, p.H, p.W, vec);
        return hipGetLastError();
    }
    const int64_t HW = (int64_t)p.H * p.W;
    const int64_t sets = (int64_t)p.B * p.G;            // tap-plane triples per direction
    const bool vec = HW % 8 == 0;
    const int64_t per = vec ? HW / 8 + 8 : HW;           // units per triple, at most
    const int64_t n = (int64_t)__builtin_popcount(p.mask) * sets * per;
    int64_t blocks = (n + 255) / 256;
    blocks = blocks < 16384 ? blocks : 16384;
    hipLaunchKernelGGL((norm_kernel<T>), dim3((unsigned)blocks), dim3(256), 0, st,
                       static_cast<const T *>(wt), static_cast<const T *>(dw), static_cast<T *>(out),
                       p.mask, sets, p.H, p.W, vec);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_norm(const Problem &p, const void *wt, const void *dw, void *out, hipStream_t st)
{
    return p.dtype == 0 ? launch_norm_t<float>(p, wt, dw, out, st)
                        : launch_norm_t<bf16_t>(p, wt, dw, out, st);
}

}  // namespace gspn
