// The per-pixel (1x1) convolutions of the latent-space propagation sublayer
// (Sec. 5, Eqs. (latent_down), (latent_params), (latent_up)) on the matrix
// cores.  Each is a product per batch image, out[b] = A x[b]: A is an M x K
// weight matrix and x[b] a K x HW channel-major feature map, both bf16;
// products accumulate in fp32 and the result is rounded to bf16 once.
//
// Operand layout of v_mfma_f32_32x32x16_bf16: lane l holds row (or column)
// l % 32 and the 8 consecutive K-values from 8 (l / 32); the result's
// register r of lane l is row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32.
//
// A workgroup (4 waves) owns a tile of 128 pixels of one image; its block of
// x (64 K-rows x 128 pixels) is staged in LDS as [k][pixel].  A B fragment
// takes 8 rows of one pixel column; lanes 32..63 read the 8 rows after those
// of lanes 0..31, which with a 256-byte row pitch would fall in the same LDS
// banks, so rows whose bit 3 is set keep their two 64-byte halves swapped.
// Two kernels:
//  * proj_rows_kernel, K <= 64 (P_up, the parameter product): x is staged
//    once, every wave keeps the B fragments of all 128 pixels in registers
//    and the waves take the 32-row tiles of A in turn, 4 accumulators each;
//    a row tile's A rows are loaded while the tile before it is multiplied,
//    ahead of that tile's stores;
//  * proj_stage_kernel, K > 64 (P_down): a workgroup owns 64 rows x 128
//    pixels, wave v pixels 32v .. 32v+31 of both 32-row halves; K runs in
//    stages of 64 staged in LDS, the next stage's loads in flight while the
//    current one is multiplied.
//
// Tiles and outputs:
//  * plain product (P_down, P_up): 128 consecutive pixels;
//  * the parameter product (L_u, L_lambda, L_w of all directions stacked):
//    8 image rows x 16 columns, so that the stores of one tile fill whole
//    8-line runs of the scan's blocked line-major planes.  Its rows are
//    u (d, c), then lambda (d, c), then for every (d, c) the three tap
//    logits of w and one zero row: a lane's 4 consecutive result rows are
//    the three logits of one pixel, normalized in registers (Sec. 3,
//    Eq. (row_stochastic_norm)) before they are stored.
#include <algorithm>

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
// Plain products with K > 64 stage each K-row of a tile as whole 16-byte
// pieces: the tile's 128 pixels start at byte delta (0 .. 14) of the row's
// first piece, since a row of a map with an odd pixel count is only 2-byte
// aligned.  17 pieces a row; each 8-row octet sits 64 bytes after the end
// of the one before, so that a fragment's two 8-row halves fall in
// different LDS banks.
constexpr int kPieces = 2 * kNT / 16 + 1;
constexpr int kRawRow = 16 * kPieces;                // bytes of a staged row
constexpr int kRawBytes = kKS * kRawRow + 64 * (kKS / 8 - 1);
constexpr int kRawLoads = (kKS * kPieces + 255) / 256;   // pieces per thread and stage

enum class Mode { Plain, Params };

struct ProjArgs {
    const bf16_t *a;                 // plain: A [M][K]
    const bf16_t *lu, *ll, *lw;      // params: L_u [D][Cc][Cc], L_lambda [D][Cc][Cc], L_w [D][Cc][3][Cc]
    const bf16_t *x;                 // [B][K][HW]
    bf16_t *y;                       // plain: [B][M][HW]
    bf16_t *u, *lam, *w;             // params: [D][B][Cc][plane], [D][B][Cc][plane], [D][B][Cc][3][plane]
    int B, M, K, H, W, HW;           // output grid (params: the planes' grid)
    int HWi;                         // pixels of one input channel
    int Hi, Wi;                      // plain with remap: the input grid
    int Hv, Wv;                      // params: the grid whose edges decide which taps exist
    bool remap;                      // plain: input and output grids differ
    int ntiles, mtiles, tiles_w;     // pixel tiles, row tiles, params: tiles across a row
    int Cc, DCc;                     // params: latent channels, D * Cc
    int dirs[4];                     // params: direction index of each stacked slot
    int vslots;                      // params: bit s set when slot s is a vertical direction
    Magic div_m, div_n, div_cc, div_tw, div_w, div_wi;
};

__device__ __forceinline__ float sigmoid(float t) { return 1.f / (1.f + __expf(-t)); }

// 2-byte buffer store the compiler sees, so that it keeps the stored
// register intact until the store has read it.
__device__ __forceinline__ void bst16(rsrc_t r, uint32_t voff, uint32_t soff, uint16_t v)
{
    __builtin_amdgcn_raw_buffer_store_b16(v, r, voff, soff, 0);
}

// A byte offset beyond the range of every store descriptor of these kernels
// (each covers one image's maps or less, which the entry points keep under
// 2 GiB): the buffer's range check discards the store.  Stores of padding
// pixels and absent rows go there instead of under a branch, which would
// split the code and make the compiler wait for every earlier store before
// the next tile's products.
constexpr uint32_t kDrop = 0x80000000u;

__device__ __forceinline__ uint16_t bf16_bits(float v)
{
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(v));
}

// Pixel of tile position j (0 .. 127) in the output grid, or -1 if off it;
// `ipix` is the same pixel in the input map (-1: not there, reads as 0).
// Plain products may map between grids of different sizes that share their
// top-left corner (a grid padded at the bottom and right and the unpadded
// one); `row`, `col` are the output pixel's coordinates for the parameter
// product.
template <Mode MODE>
__device__ __forceinline__ int tile_pixel(const ProjArgs &A, int nt, int j, int &row, int &col,
                                          int &ipix)
{
    if (MODE == Mode::Plain) {
        const int n = nt * kNT + j;
        row = col = 0;
        if (n >= A.HW) {
            ipix = -1;
            return -1;
        }
        ipix = n;
        if (A.remap) {
            const int r = mdiv(n, A.div_w), c = n - r * A.W;
            ipix = (r < A.Hi && c < A.Wi) ? r * A.Wi + c : -1;
        }
        return n;
    } else {
        const int rb = mdiv(nt, A.div_tw), cb = nt - rb * A.tiles_w;
        row = 8 * rb + (j >> 4);
        col = 16 * cb + (j & 15);
        ipix = (row < A.H && col < A.W) ? row * A.W + col : -1;
        return ipix;
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

// Stores of the parameter product for result rows m .. m+3 (m a multiple of
// 4) at pixel (row, col) of image b.
__device__ __forceinline__ void store_params(const ProjArgs &A, int b, int m, int row, int col,
                                             float v0, float v1, float v2, float v3)
{
    const int64_t HW = A.HW;
    if (m < 2 * A.DCc) {
        // four channels c .. c+3 of one direction: u, or lambda
        const bool is_u = m < A.DCc;
        const int q = is_u ? m : m - A.DCc;
        const int s = mdiv(q, A.div_cc), c = q - s * A.Cc;
        bf16_t *dst = (is_u ? A.u : A.lam) + ((int64_t)s * A.B + b) * A.Cc * HW +
                      (int64_t)c * HW + plane_offset(A.dirs[s], row, col, A.H, A.W);
        dst[0] = bf16_bits(v0);
        dst[HW] = bf16_bits(v1);
        dst[2 * HW] = bf16_bits(v2);
        dst[3 * HW] = bf16_bits(v3);
    } else if (m < A.M) {
        // the three tap logits of channel c, direction slot s
        const int dc = (m - 2 * A.DCc) >> 2;
        const int s = mdiv(dc, A.div_cc), c = dc - s * A.Cc;
        const int d = A.dirs[s];
        const int p = d < 2 ? col : row, P = d < 2 ? A.Wv : A.Hv;
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

// The 64 x 128 block of x from K-row kc on: rows kc + 2 i + (t / 128), this
// thread's pixel column; 0 past K and off the image.
__device__ __forceinline__ void load_x_block(rsrc_t xr, int K, int HW, int kc, int ks0, int spix,
                                             uint32_t (&xv)[kKS / 2])
{
#pragma unroll
    for (int i = 0; i < kKS / 2; ++i) {
        const int k = kc + 2 * i + ks0;
        xv[i] = (spix >= 0 && k < K) ? ld16(xr, 2u * (uint32_t)(k * HW + spix), 0) : 0u;
    }
}

__device__ __forceinline__ void store_x_block(uint16_t *xs, int js, int ks0,
                                              const uint32_t (&xv)[kKS / 2])
{
#pragma unroll
    for (int i = 0; i < kKS / 2; ++i) {
        const int kr = 2 * i + ks0;
        xs[kr * kNT + (js ^ ((kr & 8) << 2))] = (uint16_t)xv[i];
    }
}

// B fragment of K-step s (16 rows from 16 s) for tile pixel column jc from
// rows staged as 16-byte pieces: row r's pixels start at byte
// (dbase + r * dstep) mod 16 of its first piece.
__device__ __forceinline__ bf16x8_t b_fragment_raw(const uint16_t *xs, int s, int h, int jc,
                                                   uint32_t dbase, uint32_t dstep)
{
    bf16x8_t bf;
    const uint8_t *xr = reinterpret_cast<const uint8_t *>(xs) + (16 * s + 8 * h) * kRawRow +
                        64 * (2 * s + h) + 2 * jc;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const uint32_t d = (dbase + (uint32_t)(16 * s + 8 * h + i) * dstep) & 15u;
        bf[i] = *reinterpret_cast<const __bf16 *>(xr + i * kRawRow + d);
    }
    return bf;
}

// B fragment of K-step s (16 rows from 16 s) for tile pixel column jc.
__device__ __forceinline__ bf16x8_t b_fragment(const uint16_t *xs, int s, int h, int jc)
{
    bf16x8_t bf;
    const uint16_t *xr = xs + (16 * s + 8 * h) * kNT + (jc ^ (h << 5));
#pragma unroll
    for (int i = 0; i < 8; ++i)
        bf[i] = __builtin_bit_cast(__bf16, xr[i * kNT]);
    return bf;
}

template <Mode MODE>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void proj_rows_kernel(
    ProjArgs A)
{
    __shared__ __attribute__((aligned(16))) uint16_t xs[kKS * kNT];

    const int t = threadIdx.x;
    const int v = __builtin_amdgcn_readfirstlane(t >> 6);
    const int l = t & 63, h = l >> 5, l32 = l & 31;
    const int blk = xcd_remap(blockIdx.x, gridDim.x);
    const int b = mdiv(blk, A.div_n);
    const int nt = blk - b * A.ntiles;

    {
        const int js = t & (kNT - 1), ks0 = t >> 7;
        int r_, c_, spix;
        tile_pixel<MODE>(A, nt, js, r_, c_, spix);
        const rsrc_t xr = make_rsrc(A.x + (int64_t)b * A.K * A.HWi, (uint32_t)(2 * A.K * A.HWi));
        uint32_t xv[kKS / 2];
        load_x_block(xr, A.K, A.HWi, 0, ks0, spix, xv);
        store_x_block(xs, js, ks0, xv);
    }
    __syncthreads();

    const int nsteps = (A.K + 15) >> 4;   // K-steps of 16 holding data
    const int RT = (A.M + 31) >> 5;
    // parameter product with Cc a multiple of 32: the 32 rows of a row tile
    // are 32 channels of u or lambda, or 8 channels x 4 taps of w, of one
    // direction slot, so a row's plane offset is a scalar.  The waves then
    // take the row tiles of vertical directions in a first pass and those of
    // horizontal ones in a second, each with the tile's pixels ordered along
    // the pass's blocked layout (8 lines of one position, resp. 8 positions
    // of one line, adjacent), so that the 32 lanes of a store write 64
    // contiguous bytes.
    const bool fast = MODE == Mode::Params && A.Cc % 32 == 0;
    rsrc_t yd = make_rsrc(A.y, 0);
    if (MODE == Mode::Plain)
        yd = make_rsrc(A.y + (int64_t)b * A.M * A.HW, (uint32_t)(2 * A.M * A.HW));
#pragma unroll 1
    for (int pass = 0; pass < (fast ? 2 : 1); ++pass) {
    // this pass's pixel of lane column 32 ct + l32 and its B fragments
    bf16x8_t bfr[4][kKS / 16];
    int prow[4], pcol[4], ppix[4];
    uint32_t po[4];
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
        const int jp = 32 * ct + l32;
        int js = jp;                      // the pixel's column in the staged block
        if (fast) {
            const int rl = pass == 0 ? (jp & 7) : ((jp >> 3) & 7);
            const int cl = pass == 0 ? (jp >> 3) : 8 * (jp >> 6) + (jp & 7);
            js = rl * 16 + cl;
        }
#pragma unroll
        for (int s = 0; s < kKS / 16; ++s)
            if (s < nsteps)
                bfr[ct][s] = b_fragment(xs, s, h, js);
        int ip_;
        ppix[ct] = tile_pixel<MODE>(A, nt, js, prow[ct], pcol[ct], ip_);
        po[ct] = 0;
        if (fast && ppix[ct] >= 0)
            po[ct] = 2u * (uint32_t)(pass == 0 ? lm_offset(prow[ct], pcol[ct], A.H, A.W)
                                                : lm_offset(pcol[ct], prow[ct], A.W, A.H));
    }
    // the row tiles this wave takes in this pass
    auto in_pass = [&](int rt) {
        if (!fast)
            return true;
        const int m0 = 32 * rt;
        const bool w_ = m0 >= 2 * A.DCc;
        const int q0 = w_ ? (m0 - 2 * A.DCc) >> 2 : (m0 < A.DCc ? m0 : m0 - A.DCc);
        const int sl = mdiv(q0, A.div_cc);
        return (((A.vslots >> sl) & 1) != 0) == (pass == 0);
    };
    auto next_tile = [&](int rt) {
        while (rt < RT && !in_pass(rt))
            rt += 4;
        return rt;
    };
    auto load_a = [&](int rt, bf16x8_t (&af)[kKS / 16]) {
        const bf16_t *src = a_row<MODE>(A, 32 * rt + l32);
#pragma unroll
        for (int s = 0; s < kKS / 16; ++s) {
            const int k = 16 * s + 8 * h;
            if (s < nsteps)
                af[s] = (src != nullptr && k < A.K) ? *reinterpret_cast<const bf16x8_t *>(src + k)
                                                    : bf16x8_t{};
        }
    };
    // One row tile: the product with af, then the next row tile's A rows
    // into an, then the stores.  The loop below alternates the two fragment
    // sets (no run-time index into them, which would go through scratch).
    auto tile = [&](int rt, int rn, const bf16x8_t (&af)[kKS / 16], bf16x8_t (&an)[kKS / 16]) {
        bool is_w = false, vert = true;
        rsrc_t dd = make_rsrc(A.u, 0);
        if (fast) {
            const int m0 = 32 * rt;
            is_w = m0 >= 2 * A.DCc;
            const int q0 = is_w ? (m0 - 2 * A.DCc) >> 2 : (m0 < A.DCc ? m0 : m0 - A.DCc);
            const int sl = mdiv(q0, A.div_cc), c0 = q0 - sl * A.Cc;
            vert = (A.vslots >> sl) & 1;
            const int64_t HW = A.HW;
            const bf16_t *base =
                is_w ? A.w + (((int64_t)sl * A.B + b) * A.Cc + c0) * 3 * HW
                     : (m0 < A.DCc ? A.u : A.lam) + (((int64_t)sl * A.B + b) * A.Cc + c0) * HW;
            dd = make_rsrc(base, (uint32_t)(2 * (is_w ? 24 : 32) * HW));
        }

        f32x16_t acc[4];
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                acc[ct][r] = 0.f;
#pragma unroll
        for (int s = 0; s < kKS / 16; ++s)
            if (s < nsteps)
#pragma unroll
                for (int ct = 0; ct < 4; ++ct)
                    acc[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s], bfr[ct][s], acc[ct],
                                                                      0, 0, 0);
        // the next tile's A rows, issued before this tile's stores: a later
        // wait for them then does not wait for the stores as well
        if (rn < RT)
            load_a(rn, an);
#pragma unroll
        for (int ct = 0; ct < 4; ++ct) {
            const bool pv = ppix[ct] >= 0;     // a pixel of the image (not padding)
            if (MODE == Mode::Plain) {
                // the lane's part of the offset in a register, the row's in soffset
                const uint32_t vo = 2u * (uint32_t)(ppix[ct] + 4 * h * A.HW);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int m = 32 * rt + 8 * (r >> 2) + (r & 3);
                    bst16(yd, pv && m + 4 * h < A.M ? vo : kDrop, 2u * (uint32_t)(m * A.HW),
                          bf16_bits(acc[ct][r]));
                }
            } else if (!fast) {
                if (!pv)
                    continue;
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    store_params(A, b, 32 * rt + 8 * g + 4 * h, prow[ct], pcol[ct],
                                 acc[ct][4 * g], acc[ct][4 * g + 1], acc[ct][4 * g + 2],
                                 acc[ct][4 * g + 3]);
            } else {
                // row 8 g + 4 h + e of the tile: plane 8 g + e (scalar) plus
                // 4 h (u, lambda) or channel 2 g + h, tap e: plane 6 g + e plus 3 h (w)
                const uint32_t vo =
                    pv ? po[ct] + 2u * (uint32_t)((is_w ? 3 : 4) * h * A.HW) : kDrop;
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    float o[4] = {acc[ct][4 * g], acc[ct][4 * g + 1], acc[ct][4 * g + 2],
                                  acc[ct][4 * g + 3]};
                    if (is_w) {
                        const int p = vert ? pcol[ct] : prow[ct], P = vert ? A.Wv : A.Hv;
                        // the sigmoids and the sum's reciprocal with the
                        // hardware reciprocal (1 ulp): this kernel is bound
                        // by the instructions it issues per stored value,
                        // and an IEEE division takes about ten
                        const float s0 = p > 0 ? __builtin_amdgcn_rcpf(1.f + __expf(-o[0])) : 0.f;
                        const float s1 = __builtin_amdgcn_rcpf(1.f + __expf(-o[1]));
                        const float s2 =
                            p < P - 1 ? __builtin_amdgcn_rcpf(1.f + __expf(-o[2])) : 0.f;
                        const float inv = __builtin_amdgcn_rcpf(fmaxf((s0 + s1) + s2, kNormEps));
                        o[0] = s0 * inv, o[1] = s1 * inv, o[2] = s2 * inv;
                    }
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        if (is_w && e == 3)
                            continue;
                        const int plane = is_w ? 6 * g + e : 8 * g + e;
                        bst16(dd, vo, 2u * (uint32_t)(plane * A.HW), bf16_bits(o[e]));
                    }
                }
            }
        }
    };
    bf16x8_t af0[kKS / 16], af1[kKS / 16];
    int rt = next_tile(v);
    if (rt < RT)
        load_a(rt, af0);
#pragma unroll 1
    while (rt < RT) {
        int rn = next_tile(rt + 4);
        tile(rt, rn, af0, af1);
        rt = rn;
        if (rt >= RT)
            break;
        rn = next_tile(rt + 4);
        tile(rt, rn, af1, af0);
        rt = rn;
    }
    }
}

template <Mode MODE>
__global__ __launch_bounds__(256) void proj_stage_kernel(ProjArgs A)
{
    // plain products: tiles of 128 consecutive input pixels, K-rows staged
    // as whole 16-byte pieces (the parameter product keeps 2-byte loads)
    constexpr bool RAW = MODE == Mode::Plain;
    __shared__ __attribute__((aligned(16))) uint16_t xs[RAW ? kRawBytes / 2 : kKS * kNT];
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

    // this thread's staging pixel and A pieces (the same in every stage)
    const int js = t & (kNT - 1), ks0 = t >> 7;
    int srow, scol, spix;
    int sopix;
    if constexpr (RAW) {
        // input pixel n of the tile -> output pixel (grids share their
        // top-left corner; -1: not on the output grid)
        const int n = nt * kNT + js;
        sopix = n < A.HWi ? n : -1;
        if (A.remap && sopix >= 0) {
            const int r = mdiv(n, A.div_wi), c = n - r * A.Wi;
            sopix = (r < A.H && c < A.W) ? r * A.W + c : -1;
        }
        spix = 0;
    } else {
        sopix = tile_pixel<MODE>(A, nt, js, srow, scol, spix);
    }
    const bf16_t *ximg = A.x + (int64_t)b * A.K * A.HWi;
    // RAW: the image's pieces counted from its base rounded down to 16 bytes
    const uint32_t d0 = RAW ? (uint32_t)(reinterpret_cast<uintptr_t>(ximg) & 15u) : 0u;
    const rsrc_t xr = make_rsrc(reinterpret_cast<const uint8_t *>(ximg) - d0,
                                (d0 + (uint32_t)(2 * A.K * A.HWi) + 15u) & ~15u);
    const uint32_t p0b = d0 + 2u * (uint32_t)(nt * kNT);          // byte of the tile's pixel 0, row 0
    const uint32_t rowb = 2u * (uint32_t)A.HWi;                     // bytes per K-row
    const bf16_t *asrc[2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
        asrc[i] = a_row<MODE>(A, m0 + ((t + 256 * i) >> 3));

    auto load_a = [&](int kc, uint4 (&av)[2]) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int kq = kc + 8 * ((t + 256 * i) & 7);
            av[i] = (asrc[i] != nullptr && kq < A.K)
                        ? *reinterpret_cast<const uint4 *>(asrc[i] + kq)
                        : make_uint4(0, 0, 0, 0);
        }
    };
    // RAW: piece q = t + 256 i of a stage is piece q % 17 of K-row q / 17;
    // a piece holds only bytes of its own 16-byte block, which lies in one
    // page with the row byte it was taken for, so no read leaves the map's
    // pages (pieces past the image read as 0, past the tile they are unused)
    auto load_raw = [&](int kc, uint4 (&rv)[kRawLoads]) {
#pragma unroll
        for (int i = 0; i < kRawLoads; ++i) {
            const int q = t + 256 * i;
            const int kr = q / kPieces, pc = q - kr * kPieces;
            const int k = kc + kr;
            rv[i] = (q < kKS * kPieces && k < A.K)
                        ? ld128(xr, ((p0b + (uint32_t)k * rowb) & ~15u) + 16u * (uint32_t)pc, 0)
                        : make_uint4(0, 0, 0, 0);
        }
    };
    auto store_raw = [&](const uint4 (&rv)[kRawLoads]) {
#pragma unroll
        for (int i = 0; i < kRawLoads; ++i) {
            const int q = t + 256 * i;
            const int kr = q / kPieces, pc = q - kr * kPieces;
            if (q < kKS * kPieces)
                *reinterpret_cast<uint4 *>(reinterpret_cast<uint8_t *>(xs) + kr * kRawRow +
                                           64 * (kr >> 3) + 16 * pc) = rv[i];
        }
    };

    f32x16_t acc[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            acc[rt][r] = 0.f;

    uint32_t xv[RAW ? 1 : kKS / 2];
    uint4 rv[RAW ? kRawLoads : 1];
    uint4 av[2];
    if constexpr (RAW)
        load_raw(0, rv);
    else
        load_x_block(xr, A.K, A.HWi, 0, ks0, spix, xv);
    load_a(0, av);
    const uint32_t dstep = rowb & 15u;
    for (int kc = 0; kc < A.K; kc += kKS) {
        __syncthreads();   // the previous stage's fragments are read
        if constexpr (RAW)
            store_raw(rv);
        else
            store_x_block(xs, js, ks0, xv);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int p = t + 256 * i;
            *reinterpret_cast<uint4 *>(&as[(p >> 3) * kAP + 8 * (p & 7)]) = av[i];
        }
        __syncthreads();
        if (kc + kKS < A.K) {   // the next stage's loads overlap this stage's products
            if constexpr (RAW)
                load_raw(kc + kKS, rv);
            else
                load_x_block(xr, A.K, A.HWi, kc + kKS, ks0, spix, xv);
            load_a(kc + kKS, av);
        }
        const uint32_t dbase = (p0b + (uint32_t)kc * rowb) & 15u;
#pragma unroll
        for (int s = 0; s < kKS / 16; ++s) {
            const bf16x8_t bf = RAW ? b_fragment_raw(xs, s, h, 32 * v + l32, dbase, dstep)
                                    : b_fragment(xs, s, h, 32 * v + l32);
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
        if (sopix >= 0) {
            bf16_t *yb = A.y + (int64_t)b * A.M * A.HW + sopix;
#pragma unroll 4
            for (int i = 0; i < kMT / 2; ++i) {
                const int r = 2 * i + ks0;
                if (m0 + r < A.M)
                    yb[(int64_t)(m0 + r) * A.HW] = os[r * kNT + js];
            }
        }
    } else {
        int row, col, ip_;
        if (tile_pixel<MODE>(A, nt, jc, row, col, ip_) < 0)
            return;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt)
#pragma unroll
            for (int g = 0; g < 4; ++g)
                store_params(A, b, m0 + 32 * rt + 8 * g + 4 * h, row, col, acc[rt][4 * g],
                             acc[rt][4 * g + 1], acc[rt][4 * g + 2], acc[rt][4 * g + 3]);
    }
}

// Output pixels (r, c) with r >= Hi or c >= Wi of every plane of an H x W
// output grid: 0.  blockIdx.x is the plane; the blocks along y stride over
// its margin pixels.
__global__ __launch_bounds__(256) void zero_margin_kernel(bf16_t *y, int H, int W, int Hi, int Wi)
{
    const int hi = min(H, Hi), wi = min(W, Wi);
    const int per = H * W - hi * wi;          // margin pixels of a plane
    const int side = hi * (W - wi);           // right of the rows that have input
    bf16_t *plane = y + (int64_t)blockIdx.x * H * W;
    for (int q = blockIdx.y * blockDim.x + threadIdx.x; q < per; q += gridDim.y * blockDim.x) {
        int r, c;
        if (q < side) {
            r = q / (W - wi);
            c = wi + (q - r * (W - wi));
        } else {
            r = hi + (q - side) / W;
            c = (q - side) - (r - hi) * W;
        }
        plane[r * W + c] = 0;
    }
}

template <Mode MODE>
hipError_t launch_proj(ProjArgs &A, hipStream_t st)
{
    if (A.K <= kKS) {
        A.div_n = make_magic((uint32_t)A.ntiles);
        const int64_t nblk = (int64_t)A.B * A.ntiles;
        hipLaunchKernelGGL(proj_rows_kernel<MODE>, dim3((unsigned)nblk), dim3(256), 0, st, A);
    } else {
        if (MODE == Mode::Plain) {
            // the stage kernel tiles the input pixels; output pixels with no
            // input pixel (the margin of a larger output grid) are zeroed
            A.ntiles = (A.HWi + kNT - 1) / kNT;
            if (A.H > A.Hi || A.W > A.Wi) {
                const int per = A.H * A.W - std::min(A.H, A.Hi) * std::min(A.W, A.Wi);
                hipLaunchKernelGGL(zero_margin_kernel,
                                   dim3((unsigned)(A.B * A.M), (unsigned)std::min((per + 255) / 256, 256)),
                                   dim3(256), 0, st, A.y, A.H, A.W, A.Hi, A.Wi);
            }
        }
        A.div_n = make_magic((uint32_t)A.ntiles);
        A.mtiles = (A.M + kMT - 1) / kMT;
        A.div_m = make_magic((uint32_t)A.mtiles);
        const int64_t nblk = (int64_t)A.B * A.ntiles * A.mtiles;
        hipLaunchKernelGGL(proj_stage_kernel<MODE>, dim3((unsigned)nblk), dim3(256), 0, st, A);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_project(const void *a, const void *x, void *y, int B, int M, int K, int H, int W,
                          hipStream_t st, int Hi, int Wi)
{
    ProjArgs A{};
    A.a = static_cast<const bf16_t *>(a);
    A.x = static_cast<const bf16_t *>(x);
    A.y = static_cast<bf16_t *>(y);
    A.B = B, A.M = M, A.K = K, A.H = H, A.W = W, A.HW = H * W;
    A.Hi = Hi > 0 ? Hi : H, A.Wi = Wi > 0 ? Wi : W, A.HWi = A.Hi * A.Wi;
    A.remap = A.Hi != H || A.Wi != W;
    A.div_w = make_magic((uint32_t)W);
    A.div_wi = make_magic((uint32_t)A.Wi);
    A.ntiles = (A.HW + kNT - 1) / kNT;
    return launch_proj<Mode::Plain>(A, st);
}

hipError_t launch_latent_params(const void *xc, const void *lu, const void *ll, const void *lw,
                                void *u, void *lam, void *w, int mask, int B, int Cc, int H, int W,
                                hipStream_t st, int Hv, int Wv)
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
        {
            if (d < 2)
                A.vslots |= 1 << D;      // slot D scans vertically
            A.dirs[D++] = d;
        }
    A.B = B, A.K = Cc, A.H = H, A.W = W, A.HW = H * W, A.HWi = A.HW;
    A.Hv = Hv > 0 ? Hv : H, A.Wv = Wv > 0 ? Wv : W;
    A.Cc = Cc, A.DCc = D * Cc, A.M = 6 * D * Cc;
    A.tiles_w = (W + 15) / 16;
    A.ntiles = ((H + 7) / 8) * A.tiles_w;
    A.div_cc = make_magic((uint32_t)Cc);
    A.div_tw = make_magic((uint32_t)A.tiles_w);
    return launch_proj<Mode::Params>(A, st);
}

}  // namespace gspn
