// The per-pixel (1x1) convolutions of the latent-space propagation sublayer
// (Sec. 5, Eqs. (latent_down), (latent_params), (latent_up)) on the matrix
// cores.  Each is a product per batch image, out[b] = A x[b]: A is an M x K
// weight matrix and x[b] a K x HW channel-major feature map, both bf16;
// products accumulate in fp32 and the result is rounded to bf16 once.
//
// Workgroup: 4 waves and an output tile of 64 rows x 128 pixels.  Wave v
// owns pixels 32v .. 32v+31 of the tile and both 32-row halves, as two
// v_mfma_f32_32x32x16_bf16 accumulators (16 fp32 registers each).  K runs
// in stages of 64: a stage's 64 x 128 block of x and 64 x 64 block of A go to
// LDS, and each wave then takes 4 steps of 16 along K.  Operand layout of the
// instruction: lane l holds row (or column) l % 32 and the 8 consecutive
// K-values from 8 (l / 32); the result's register r of lane l is row
// 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
//
// The x block is kept as [k][pixel]; a B fragment takes 8 rows of one pixel
// column.  Lanes 32..63 read the 8 rows after those of lanes 0..31, which
// with a 256-byte row pitch would fall in the same LDS banks; rows whose
// bit 3 is set therefore keep their two 64-byte halves swapped.
//
// Tiles and outputs:
//  * plain product (P_down, P_up): 128 consecutive pixels; the tile goes
//    through LDS once more so that every store writes 128 contiguous bytes;
//  * the parameter product (L_u, L_lambda, L_w of all directions stacked):
//    8 image rows x 16 columns, so that the stores of one tile fill whole
//    8-line runs of the scan's blocked line-major planes.  Its rows are
//    u (d, c), then lambda (d, c), then for every (d, c) the three tap
//    logits of w and one zero row: a lane's 4 consecutive result rows are
//    the three logits of one pixel, normalized in registers (Sec. 3,
//    Eq. (row_stochastic_norm)) before they are stored.
#include "cdna.hpp"
#include "device.hpp"
#include "launch.hpp"

namespace gspn {

namespace {

using namespace cdna;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kMT = 64;     // output rows of a workgroup
constexpr int kNT = 128;    // pixels of a workgroup
constexpr int kKS = 64;     // K of one LDS stage
constexpr int kAP = 72;     // pitch of the A block in LDS, in bf16 (16-byte aligned rows)
constexpr float kNormEps = 1e-30f;

enum class Mode { Plain, Params };

struct ProjArgs {
    const bf16_t *a;                 // plain: A [M][K]
    const bf16_t *lu, *ll, *lw;      // params: L_u [D][Cc][Cc], L_lambda [D][Cc][Cc], L_w [D][Cc][3][Cc]
    const bf16_t *x;                 // [B][K][HW]
    bf16_t *y;                       // plain: [B][M][HW]
    bf16_t *u, *lam, *w;             // params: [D][B][Cc][plane], [D][B][Cc][plane], [D][B][Cc][3][plane]
    int B, M, K, H, W, HW;
    int ntiles, mtiles, tiles_w;     // pixel tiles, row tiles, params: tiles across a row
    int Cc, DCc;                     // params: latent channels, D * Cc
    int dirs[4];                     // params: direction index of each stacked slot
    Magic div_m, div_n, div_cc, div_tw;
};

__device__ __forceinline__ float sigmoid(float t) { return 1.f / (1.f + __expf(-t)); }

__device__ __forceinline__ uint16_t bf16_bits(float v)
{
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// Pixel of tile position j (0 .. 127): image row and column, or -1 if off
// the image.
template <Mode MODE>
__device__ __forceinline__ int tile_pixel(const ProjArgs &A, int nt, int j, int &row, int &col)
{
    if (MODE == Mode::Plain) {
        const int n = nt * kNT + j;
        row = col = 0;
        return n < A.HW ? n : -1;
    } else {
        const int rb = mdiv(nt, A.div_tw), cb = nt - rb * A.tiles_w;
        row = 8 * rb + (j >> 4);
        col = 16 * cb + (j & 15);
        return (row < A.H && col < A.W) ? row * A.W + col : -1;
    }
}

// Source row m of the stacked weight matrix, nullptr for a zero row.
template <Mode MODE>
__device__ __forceinline__ const bf16_t *a_row(const ProjArgs &A, int m)
{
    if (MODE == Mode::Plain)
        return m < A.M ? A.a + (int64_t)m * A.K : nullptr;
    if (m < A.DCc)
        return A.lu + (int64_t)m * A.K;
    if (m < 2 * A.DCc)
        return A.ll + (int64_t)(m - A.DCc) * A.K;
    if (m < A.M) {
        const int q = m - 2 * A.DCc, tap = q & 3;
        return tap == 3 ? nullptr : A.lw + ((int64_t)(q >> 2) * 3 + tap) * A.K;
    }
    return nullptr;
}

// Blocked line-major offset of pixel (row, col) in a plane of direction d.
__device__ __forceinline__ int plane_offset(int d, int row, int col, int H, int W)
{
    return d < 2 ? lm_offset(row, col, H, W) : lm_offset(col, row, W, H);
}

template <Mode MODE>
__global__ __launch_bounds__(256) void proj_kernel(ProjArgs A)
{
    __shared__ __attribute__((aligned(16))) uint16_t xs[kKS * kNT];
    __shared__ __attribute__((aligned(16))) uint16_t as[kMT * kAP];

    const int t = threadIdx.x;
    const int v = __builtin_amdgcn_readfirstlane(t >> 6);
    const int l = t & 63, h = l >> 5, l32 = l & 31;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    // the row tiles of one pixel tile are neighbours: they run under one L2
    const int rest = mdiv(blk, A.div_m);
    const int mt = blk - rest * A.mtiles;
    const int b = mdiv(rest, A.div_n);
    const int nt = rest - b * A.ntiles;
    const int m0 = mt * kMT;

    // this thread's staging pixel (the same in every stage)
    const int js = t & (kNT - 1), ks0 = t >> 7;
    int srow, scol;
    const int spix = tile_pixel<MODE>(A, nt, js, srow, scol);
    const bf16_t *xb = A.x + (int64_t)b * A.K * A.HW;

    f32x16_t acc[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[rt][r] = 0.f;

    for (int kc = 0; kc < A.K; kc += kKS) {
        __syncthreads();   // the previous stage's fragments are read
        // x block: rows kc + 2 i + ks0, this thread's pixel column
        uint16_t xv[kKS / 2];
#pragma unroll
        for (int i = 0; i < kKS / 2; ++i) {
            const int k = kc + 2 * i + ks0;
            xv[i] = (spix >= 0 && k < A.K) ? xb[(int64_t)k * A.HW + spix] : (uint16_t)0;
        }
        // A block: 64 rows x 8 pieces of 8 K-values
        uint4 av[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int p = t + 256 * i, r = p >> 3, kq = kc + 8 * (p & 7);
            const bf16_t *src = a_row<MODE>(A, m0 + r);
            av[i] = (src != nullptr && kq < A.K) ? *reinterpret_cast<const uint4 *>(src + kq)
                                                  : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < kKS / 2; ++i) {
            const int kr = 2 * i + ks0;
            xs[kr * kNT + (js ^ ((kr & 8) << 2))] = xv[i];
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int p = t + 256 * i;
            *reinterpret_cast<uint4 *>(&as[(p >> 3) * kAP + 8 * (p & 7)]) = av[i];
        }
        __syncthreads();
#pragma unroll
        for (int s = 0; s < kKS / 16; ++s) {
            bf16x8_t bf;
            const uint16_t *xr = xs + (16 * s + 8 * h) * kNT + ((32 * v + l32) ^ (h << 5));
#pragma unroll
            for (int i = 0; i < 8; ++i)
                bf[i] = __builtin_bit_cast(__bf16, xr[i * kNT]);
#pragma unroll
            for (int rt = 0; rt < 2; ++rt) {
                const bf16x8_t af =
                    *reinterpret_cast<const bf16x8_t *>(&as[(32 * rt + l32) * kAP + 16 * s + 8 * h]);
                acc[rt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf, acc[rt], 0, 0, 0);
            }
        }
    }

    const int jc = 32 * v + l32;   // this lane's result column (tile pixel)
    if (MODE == Mode::Plain) {
        __syncthreads();           // every wave is done with the x block
        uint16_t *os = xs;         // [64][128] bf16 result tile
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                os[(32 * rt + 8 * (r >> 2) + 4 * h + (r & 3)) * kNT + jc] = bf16_bits(acc[rt][r]);
        __syncthreads();
        if (spix >= 0) {
            bf16_t *yb = A.y + (int64_t)b * A.M * A.HW + spix;
#pragma unroll 4
            for (int i = 0; i < kMT / 2; ++i) {
                const int r = 2 * i + ks0;
                if (m0 + r < A.M)
                    yb[(int64_t)(m0 + r) * A.HW] = os[r * kNT + js];
            }
        }
    } else {
        int row, col;
        if (tile_pixel<MODE>(A, nt, jc, row, col) < 0)
            return;
        const int64_t HW = A.HW;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int m = m0 + 32 * rt + 8 * g + 4 * h;   // a multiple of 4
                const float v0 = acc[rt][4 * g], v1 = acc[rt][4 * g + 1];
                const float v2 = acc[rt][4 * g + 2], v3 = acc[rt][4 * g + 3];
                if (m < 2 * A.DCc) {
                    // four channels c .. c+3 of one direction: u, or lambda
                    const bool is_u = m < A.DCc;
                    const int q = is_u ? m : m - A.DCc;
                    const int s = mdiv(q, A.div_cc), c = q - s * A.Cc;
                    const int d = A.dirs[s];
                    bf16_t *dst = (is_u ? A.u : A.lam) + ((int64_t)s * A.B + b) * A.Cc * HW +
                                  (int64_t)c * HW + plane_offset(d, row, col, A.H, A.W);
                    dst[0] = bf16_bits(v0);
                    dst[HW] = bf16_bits(v1);
                    dst[2 * HW] = bf16_bits(v2);
                    dst[3 * HW] = bf16_bits(v3);
                } else if (m < A.M) {
                    // the three tap logits of channel c, direction slot s
                    const int dc = (m - 2 * A.DCc) >> 2;
                    const int s = mdiv(dc, A.div_cc), c = dc - s * A.Cc;
                    const int d = A.dirs[s];
                    const int p = d < 2 ? col : row, P = d < 2 ? A.W : A.H;
                    const float s0 = p > 0 ? sigmoid(v0) : 0.f;
                    const float s1 = sigmoid(v1);
                    const float s2 = p < P - 1 ? sigmoid(v2) : 0.f;
                    const float inv = 1.f / fmaxf((s0 + s1) + s2, kNormEps);
                    bf16_t *dst = A.w + (((int64_t)s * A.B + b) * A.Cc + c) * 3 * HW +
                                  plane_offset(d, row, col, A.H, A.W);
                    dst[0] = bf16_bits(s0 * inv);
                    dst[HW] = bf16_bits(s1 * inv);
                    dst[2 * HW] = bf16_bits(s2 * inv);
                }
            }
        }
    }
}

template <Mode MODE>
hipError_t launch_proj(ProjArgs &A, hipStream_t st)
{
    A.mtiles = (A.M + kMT - 1) / kMT;
    A.div_m = make_magic((uint32_t)A.mtiles);
    A.div_n = make_magic((uint32_t)A.ntiles);
    const int64_t nblk = (int64_t)A.B * A.ntiles * A.mtiles;
    if (nblk > 0x7fffffff)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(proj_kernel<MODE>, dim3((unsigned)nblk), dim3(256), 0, st, A);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_project(const void *a, const void *x, void *y, int B, int M, int K, int H, int W,
                          hipStream_t st)
{
    ProjArgs A{};
    A.a = static_cast<const bf16_t *>(a);
    A.x = static_cast<const bf16_t *>(x);
    A.y = static_cast<bf16_t *>(y);
    A.B = B, A.M = M, A.K = K, A.H = H, A.W = W, A.HW = H * W;
    A.ntiles = (A.HW + kNT - 1) / kNT;
    return launch_proj<Mode::Plain>(A, st);
}

hipError_t launch_latent_params(const void *xc, const void *lu, const void *ll, const void *lw,
                                void *u, void *lam, void *w, int mask, int B, int Cc, int H, int W,
                                hipStream_t st)
{
    ProjArgs A{};
    A.lu = static_cast<const bf16_t *>(lu);
    A.ll = static_cast<const bf16_t *>(ll);
    A.lw = static_cast<const bf16_t *>(lw);
    A.x = static_cast<const bf16_t *>(xc);
    A.u = static_cast<bf16_t *>(u);
    A.lam = static_cast<bf16_t *>(lam);
    A.w = static_cast<bf16_t *>(w);
    int D = 0;
    for (int d = 0; d < 4; ++d)
        if ((mask >> d) & 1)
            A.dirs[D++] = d;
    A.B = B, A.K = Cc, A.H = H, A.W = W, A.HW = H * W;
    A.Cc = Cc, A.DCc = D * Cc, A.M = 6 * D * Cc;
    A.tiles_w = (W + 15) / 16;
    A.ntiles = ((H + 7) / 8) * A.tiles_w;
    A.div_cc = make_magic((uint32_t)Cc);
    A.div_tw = make_magic((uint32_t)A.tiles_w);
    return launch_proj<Mode::Params>(A, st);
}

}  // namespace gspn
