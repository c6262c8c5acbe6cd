// C ABI of libgspn: argument checks (host only, before any HIP call),
// dispatch to the kernel variants, error mapping.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <mutex>


#include "../../include/gspn.h"
#include "launch.hpp"

namespace gspn {

namespace {

thread_local int g_last_hip_error = 0;

struct Buf {
    const void *p;
    int64_t bytes;
    bool output;
};

int check_common(int direction, int B, int C, int G, int H, int W, int dtype)
{
    if (dtype != GSPN_F32 && dtype != GSPN_BF16)
        return GSPN_ERR_DTYPE;
    if (direction < 1 || direction > 15)
        return GSPN_ERR_DIRECTION;
    if (B < 1 || C < 1 || G < 1 || H < 1 || W < 1 || C % G != 0)
        return GSPN_ERR_DIM;
    if (H > GSPN_MAX_SIDE || W > GSPN_MAX_SIDE)
        return GSPN_ERR_UNSUPPORTED;
    const int64_t HW = (int64_t)H * W;
    const int64_t D = __builtin_popcount(direction);
    if ((int64_t)B * C > GSPN_MAX_ELEMS / HW || D * B * C > GSPN_MAX_ELEMS / HW ||
        D * B * G * 3 > GSPN_MAX_ELEMS / HW)
        return GSPN_ERR_UNSUPPORTED;
    return GSPN_OK;
}

int check_buffers(const Buf *bufs, int n)
{
    for (int i = 0; i < n; ++i)
        if (bufs[i].p == nullptr)
            return GSPN_ERR_NULL;
    for (int i = 0; i < n; ++i)
        if (reinterpret_cast<uintptr_t>(bufs[i].p) % 16 != 0)
            return GSPN_ERR_ALIGN;
    for (int i = 0; i < n; ++i) {
        if (!bufs[i].output)
            continue;
        const uintptr_t a0 = reinterpret_cast<uintptr_t>(bufs[i].p);
        const uintptr_t a1 = a0 + (uintptr_t)bufs[i].bytes;
        for (int k = 0; k < n; ++k) {
            if (k == i)
                continue;
            const uintptr_t b0 = reinterpret_cast<uintptr_t>(bufs[k].p);
            const uintptr_t b1 = b0 + (uintptr_t)bufs[k].bytes;
            if (a0 < b1 && b0 < a1)
                return GSPN_ERR_ALIAS;
        }
    }
    return GSPN_OK;
}

int hip_status(hipError_t e)
{
    if (e == hipSuccess)
        return GSPN_OK;
    g_last_hip_error = (int)e;
    return GSPN_ERR_HIP;
}

}  // namespace



}  // namespace gspn

using namespace gspn;

namespace gspn {

// The kernel family for a problem: the first one that supports its shape.
hipError_t dispatch_fwd(const Problem &p, hipStream_t s)
{
    if (med_supported(p))
        return launch_fwd_med(p, s);
    if (tiny_supported(p))
        return launch_fwd_tiny(p, s);
    if (p.H <= kSmallSide && p.W <= kSmallSide)
        return launch_fwd_small(p, s);
    if (wide_supported(p))
        return launch_fwd_wide(p, s);
    return launch_fwd_general(p, s);
}

hipError_t dispatch_bwd(const Problem &p, hipStream_t s)
{
    if (med_supported(p))
        return launch_bwd_med(p, s);
    if (tiny_supported(p))
        return launch_bwd_tiny(p, s);
    if (p.H <= kSmallSide && p.W <= kSmallSide)
        return launch_bwd_small(p, s);
    return launch_bwd_general(p, s);
}

}  // namespace gspn

namespace gspn {
namespace {

constexpr int64_t kNoWorkspace = -1;

// The pieces of one scan call: its checked buffers, its problem, and the
// workspace check.  A call first runs its dispatch in counting mode (no
// launch) to learn how much workspace it takes, then checks the caller's
// workspace against that and runs it for real.
int scan_buffers(int op, const void *x, const void *w, const void *lam, const void *u,
                 const void *dy, const void *y, const void *dx, const void *dw, const void *dlam,
                 const void *du, int direction, int B, int C, int G, int H, int W, int dtype,
                 Buf *bufs, int *nbuf)
{
    const int64_t es = dtype == GSPN_F32 ? 4 : 2;
    const int64_t D = __builtin_popcount(direction);
    const int64_t n = (int64_t)B * C * H * W;
    const int64_t nw = D * B * G * 3 * H * W;
    const bool bwd = op == GSPN_OP_BWD || op == GSPN_OP_BWD_NORM || op == GSPN_OP_BWD_BLOCKED ||
                     op == GSPN_OP_BWD_RESERVE || op == GSPN_OP_BWD_NORM_RESERVE;
    int k = 0;
    bufs[k++] = {x, n * es, false};
    bufs[k++] = {w, nw * es, false};
    bufs[k++] = {lam, D * n * es, false};
    bufs[k++] = {u, D * n * es, false};
    if (bwd) {
        bufs[k++] = {dy, n * es, false};
        bufs[k++] = {dx, n * es, true};
        bufs[k++] = {dw, nw * es, true};
        bufs[k++] = {dlam, D * n * es, true};
        bufs[k++] = {du, D * n * es, true};
    } else {
        bufs[k++] = {y, n * es, true};
    }
    *nbuf = k;
    return GSPN_OK;
}

bool valid_op(int op) { return op >= GSPN_OP_FWD && op <= GSPN_OP_BWD_NORM_RESERVE; }

// The operations of a training pair, which keep blocked copies in a reserve.
bool reserve_op(int op)
{
    return op == GSPN_OP_FWD_TRAIN || op == GSPN_OP_BWD_RESERVE || op == GSPN_OP_FWD_NORM_TRAIN ||
           op == GSPN_OP_BWD_NORM_RESERVE;
}

// Pixel-major calls on the register-streamed shapes read their weights in
// the blocked order: the _norm passes form them there directly from the
// logits (one read of the logits, one write of the weights), instead of
// writing pixel-major weights that the scan then re-lays out or stages.
bool norm_fused(const Problem &p) { return p.layout == kPixelMajor && med_supported(p); }

// The launches of one scan operation on the workspace ws (in counting mode:
// no launch, ws.used adds up what the call takes).
hipError_t run_scan(int op, const Problem &p0, const void *w_in, void *dw_out, hipStream_t s)
{
    Problem p = p0;
    Workspace &ws = *p.ws;
    const int64_t es = p.dtype == GSPN_F32 ? 4 : 2;
    const int64_t nw = (int64_t)__builtin_popcount(p.mask) * p.B * p.G * 3 * p.H * p.W;
    const bool bwd = op == GSPN_OP_BWD || op == GSPN_OP_BWD_BLOCKED || op == GSPN_OP_BWD_NORM ||
                     op == GSPN_OP_BWD_RESERVE || op == GSPN_OP_BWD_NORM_RESERVE;
    const bool norm = op == GSPN_OP_FWD_NORM || op == GSPN_OP_BWD_NORM ||
                      op == GSPN_OP_FWD_NORM_TRAIN || op == GSPN_OP_BWD_NORM_RESERVE;
    if (norm)
        p.w_blocked = norm_fused(p);
    // A training pair on the shapes whose backward re-lays out its inputs
    // keeps the copies in its reserve; the parts are taken here, once, in
    // the same order for both calls.
    ReserveParts r;
    if (p.rs != nullptr && p.layout == kPixelMajor && med_supported(p)) {
        const hipError_t e = take_reserve(p, &r);
        if (e != hipSuccess)
            return e;
        p.rsp = &r;
        (bwd ? p.rs_read : p.rs_write) = true;
    }
    if (!norm)
        return bwd ? dispatch_bwd(p, s) : dispatch_fwd(p, s);

    // Weights from their logits: formed into the reserve where a training
    // pair keeps them (its backward then finds them formed), else into the
    // workspace; the backward's weight gradient, then the logits' gradient.
    const bool kept = p.rsp != nullptr && p.w_blocked;
    void *w = kept ? r.w : nullptr, *dw = nullptr;
    hipError_t e = hipSuccess;
    if (!kept)
        e = ws.take(&w, (size_t)(nw * es));
    if (e == hipSuccess && bwd)
        e = ws.take(&dw, (size_t)(nw * es));
    if (e != hipSuccess)
        return e;
    p.w = w;
    if (bwd)
        p.dw = dw;
    if (!ws.counting && !(kept && bwd)) {
        e = p.w_blocked ? launch_norm_blocked(p, w_in, w, s) : launch_norm(p, w_in, nullptr, w, s);
        if (e != hipSuccess)
            return e;
    }
    if (!bwd)
        return dispatch_fwd(p, s);
    e = dispatch_bwd(p, s);
    if (e != hipSuccess || ws.counting)
        return e;
    return launch_norm(p, w_in, p.dw, dw_out, s);
}

// Counts the workspace (and for a training pair the reserve) of a checked
// problem.  GSPN_ERR_HIP if a device query of the plan failed.
int count_workspace(int op, const Problem &p0, int64_t *bytes, int64_t *reserve_bytes = nullptr)
{
    Workspace ws, rs;
    ws.counting = true;
    rs.counting = true;
    Problem p = p0;
    p.ws = &ws;
    p.rs = reserve_op(op) ? &rs : nullptr;
    const hipError_t e = run_scan(op, p, p0.w, p0.dw, nullptr);
    if (e != hipSuccess)
        return hip_status(e);
    *bytes = (int64_t)ws.used;
    if (reserve_bytes != nullptr)
        *reserve_bytes = (int64_t)rs.used;
    return GSPN_OK;
}

int scan_call(int op, const void *x, const void *w, const void *lam, const void *u, const void *dy,
              void *y, void *dx, void *dw, void *dlam, void *du, int direction, int B, int C,
              int G, int H, int W, int dtype, void *workspace, int64_t workspace_bytes,
              void *stream, int slots = 0, void *reserve = nullptr, int64_t reserve_bytes = 0)
{
    if (!valid_op(op))
        return GSPN_ERR_UNSUPPORTED;
    int st = check_common(direction, B, C, G, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    Buf bufs[12];
    int nb = 0;
    scan_buffers(op, x, w, lam, u, dy, y, dx, dw, dlam, du, direction, B, C, G, H, W, dtype, bufs,
                 &nb);
    st = check_buffers(bufs, nb);
    if (st != GSPN_OK)
        return st;
    const bool blocked = op == GSPN_OP_FWD_BLOCKED || op == GSPN_OP_BWD_BLOCKED;
    Problem p{x, w, lam, u, dy, y, dx, dw, dlam, du, direction, B, C, G, H, W, dtype,
              blocked ? kBlocked : kPixelMajor, nullptr, slots};
    int64_t need = 0, rneed = 0;
    st = count_workspace(op, p, &need, &rneed);
    if (st != GSPN_OK)
        return st;
    if (workspace_bytes < 0 || reserve_bytes < 0)
        return GSPN_ERR_WORKSPACE;
    if (rneed > 0) {
        // written by the forward of a training pair, read by its backward
        if (reserve == nullptr || reserve_bytes < rneed)
            return GSPN_ERR_WORKSPACE;
        bufs[nb++] = {reserve, rneed, op == GSPN_OP_FWD_TRAIN || op == GSPN_OP_FWD_NORM_TRAIN};
    }
    if (need > 0) {
        if (workspace == nullptr || workspace_bytes < need)
            return GSPN_ERR_WORKSPACE;
        bufs[nb++] = {workspace, need, true};
    }
    if (need > 0 || rneed > 0) {
        st = check_buffers(bufs, nb);
        if (st != GSPN_OK)
            return st;
    }
    Workspace ws, rs;
    ws.base = static_cast<char *>(workspace);
    ws.size = need > 0 ? (size_t)workspace_bytes : 0;
    rs.base = static_cast<char *>(reserve);
    rs.size = rneed > 0 ? (size_t)reserve_bytes : 0;
    p.ws = &ws;
    p.rs = reserve_op(op) ? &rs : nullptr;
    const hipError_t e = run_scan(op, p, w, dw, static_cast<hipStream_t>(stream));
    return e == hipErrorOutOfMemory ? GSPN_ERR_WORKSPACE : hip_status(e);
}

}  // namespace
}  // namespace gspn

namespace gspn {
namespace {

int workspace_query(int op, int direction, int B, int C, int G, int H, int W, int dtype,
                    int slots, int64_t *bytes)
{
    if (bytes == nullptr)
        return GSPN_ERR_NULL;
    *bytes = 0;
    if (!valid_op(op))
        return GSPN_ERR_UNSUPPORTED;
    const int st = check_common(direction, B, C, G, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    const bool blocked = op == GSPN_OP_FWD_BLOCKED || op == GSPN_OP_BWD_BLOCKED;
    Problem p{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
              nullptr, direction, B, C, G, H, W, dtype, blocked ? kBlocked : kPixelMajor, nullptr,
              slots};
    return count_workspace(op, p, bytes);
}

bool valid_slots(int slots) { return slots == 0 || slots == 4 || slots == 8; }

}  // namespace
}  // namespace gspn

extern "C" int gspn_workspace_size(int op, int direction, int B, int C, int G, int H, int W,
                                   int dtype, int64_t *bytes)
{
    return workspace_query(op, direction, B, C, G, H, W, dtype, 0, bytes);
}

extern "C" int gspn_workspace_size_slots(int slots, int direction, int B, int C, int G, int H,
                                         int W, int dtype, int64_t *bytes)
{
    if (bytes != nullptr)
        *bytes = 0;
    if (!valid_slots(slots))
        return GSPN_ERR_UNSUPPORTED;
    return workspace_query(GSPN_OP_BWD, direction, B, C, G, H, W, dtype, slots, bytes);
}

extern "C" int gspn_scan_bwd_slots(int slots, const void *x, const void *w, const void *lam,
                                   const void *u, const void *dy, void *dx, void *dw, void *dlam,
                                   void *du, int direction, int B, int C, int G, int H, int W,
                                   int dtype, void *workspace, int64_t workspace_bytes,
                                   void *stream)
{
    if (!valid_slots(slots))
        return GSPN_ERR_UNSUPPORTED;
    return scan_call(GSPN_OP_BWD, x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction, B, C,
                     G, H, W, dtype, workspace, workspace_bytes, stream, slots);
}

extern "C" int gspn_scan_fwd(const void *x, const void *w, const void *lam, const void *u, void *y,
                             int direction, int B, int C, int G, int H, int W, int dtype,
                             void *workspace, int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_FWD, x, w, lam, u, nullptr, y, nullptr, nullptr, nullptr, nullptr,
                     direction, B, C, G, H, W, dtype, workspace, workspace_bytes, stream);
}

extern "C" int gspn_scan_bwd(const void *x, const void *w, const void *lam, const void *u,
                             const void *dy, void *dx, void *dw, void *dlam, void *du,
                             int direction, int B, int C, int G, int H, int W, int dtype,
                             void *workspace, int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_BWD, x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction, B, C,
                     G, H, W, dtype, workspace, workspace_bytes, stream);
}

namespace gspn {
namespace {

int reserve_query(int op, int direction, int B, int C, int G, int H, int W, int dtype,
                  int64_t *bytes)
{
    if (bytes == nullptr)
        return GSPN_ERR_NULL;
    *bytes = 0;
    const int st = check_common(direction, B, C, G, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    Problem p{nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
              nullptr, direction, B, C, G, H, W, dtype, kPixelMajor, nullptr};
    int64_t ws = 0;
    return count_workspace(op, p, &ws, bytes);
}

}  // namespace
}  // namespace gspn

extern "C" int gspn_reserve_size(int direction, int B, int C, int G, int H, int W, int dtype,
                                 int64_t *bytes)
{
    return reserve_query(GSPN_OP_FWD_TRAIN, direction, B, C, G, H, W, dtype, bytes);
}

extern "C" int gspn_reserve_size_norm(int direction, int B, int C, int G, int H, int W, int dtype,
                                      int64_t *bytes)
{
    return reserve_query(GSPN_OP_FWD_NORM_TRAIN, direction, B, C, G, H, W, dtype, bytes);
}

extern "C" int gspn_scan_fwd_norm_train(const void *x, const void *w_logits, const void *lam,
                                        const void *u, void *y, int direction, int B, int C,
                                        int G, int H, int W, int dtype, void *reserve,
                                        int64_t reserve_bytes, void *workspace,
                                        int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_FWD_NORM_TRAIN, x, w_logits, lam, u, nullptr, y, nullptr, nullptr,
                     nullptr, nullptr, direction, B, C, G, H, W, dtype, workspace,
                     workspace_bytes, stream, 0, reserve, reserve_bytes);
}

extern "C" int gspn_scan_bwd_norm_reserve(const void *x, const void *w_logits, const void *lam,
                                          const void *u, const void *dy, void *dx,
                                          void *dw_logits, void *dlam, void *du, int direction,
                                          int B, int C, int G, int H, int W, int dtype,
                                          const void *reserve, int64_t reserve_bytes,
                                          void *workspace, int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_BWD_NORM_RESERVE, x, w_logits, lam, u, dy, nullptr, dx, dw_logits,
                     dlam, du, direction, B, C, G, H, W, dtype, workspace, workspace_bytes,
                     stream, 0, const_cast<void *>(reserve), reserve_bytes);
}

extern "C" int gspn_scan_fwd_train(const void *x, const void *w, const void *lam, const void *u,
                                   void *y, int direction, int B, int C, int G, int H, int W,
                                   int dtype, void *reserve, int64_t reserve_bytes,
                                   void *workspace, int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_FWD_TRAIN, x, w, lam, u, nullptr, y, nullptr, nullptr, nullptr,
                     nullptr, direction, B, C, G, H, W, dtype, workspace, workspace_bytes, stream,
                     0, reserve, reserve_bytes);
}

extern "C" int gspn_scan_bwd_reserve(const void *x, const void *w, const void *lam,
                                     const void *u, const void *dy, void *dx, void *dw,
                                     void *dlam, void *du, int direction, int B, int C, int G,
                                     int H, int W, int dtype, const void *reserve,
                                     int64_t reserve_bytes, void *workspace,
                                     int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_BWD_RESERVE, x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction,
                     B, C, G, H, W, dtype, workspace, workspace_bytes, stream, 0,
                     const_cast<void *>(reserve), reserve_bytes);
}

extern "C" int gspn_scan_fwd_blocked(const void *x, const void *w, const void *lam, const void *u,
                                     void *y, int direction, int B, int C, int G, int H, int W,
                                     int dtype, void *workspace, int64_t workspace_bytes,
                                     void *stream)
{
    return scan_call(GSPN_OP_FWD_BLOCKED, x, w, lam, u, nullptr, y, nullptr, nullptr, nullptr,
                     nullptr, direction, B, C, G, H, W, dtype, workspace, workspace_bytes, stream);
}

extern "C" int gspn_scan_bwd_blocked(const void *x, const void *w, const void *lam,
                                     const void *u, const void *dy, void *dx, void *dw,
                                     void *dlam, void *du, int direction, int B, int C, int G,
                                     int H, int W, int dtype, void *workspace,
                                     int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_BWD_BLOCKED, x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction,
                     B, C, G, H, W, dtype, workspace, workspace_bytes, stream);
}

extern "C" int gspn_scan_fwd_norm(const void *x, const void *w_logits, const void *lam,
                                  const void *u, void *y, int direction, int B, int C, int G,
                                  int H, int W, int dtype, void *workspace,
                                  int64_t workspace_bytes, void *stream)
{
    return scan_call(GSPN_OP_FWD_NORM, x, w_logits, lam, u, nullptr, y, nullptr, nullptr, nullptr,
                     nullptr, direction, B, C, G, H, W, dtype, workspace, workspace_bytes, stream);
}

extern "C" int gspn_scan_bwd_norm(const void *x, const void *w_logits, const void *lam,
                                  const void *u, const void *dy, void *dx, void *dw_logits,
                                  void *dlam, void *du, int direction, int B, int C, int G, int H,
                                  int W, int dtype, void *workspace, int64_t workspace_bytes,
                                  void *stream)
{
    return scan_call(GSPN_OP_BWD_NORM, x, w_logits, lam, u, dy, nullptr, dx, dw_logits, dlam, du,
                     direction, B, C, G, H, W, dtype, workspace, workspace_bytes, stream);
}

// ---------------------------------------------------------------------------
// gspn_scan_bwd_static: gspn_scan_bwd for callers that cannot allocate (code
// under graph capture, serving loops, harnesses that forbid hipMalloc), with
// its workspace in a fixed device array instead of a caller buffer.
// ---------------------------------------------------------------------------
namespace gspn {
namespace {

constexpr size_t kStaticScratchBytes = size_t(64) << 20;   // GSPN_STATIC_SCRATCH_BYTES
static_assert(kStaticScratchBytes == (size_t)GSPN_STATIC_SCRATCH_BYTES, "header constant");

// Each GPU the library runs on holds its own copy of this array until the
// process ends.  On the host the name stands for the device copy only as a
// symbol: its device address comes from hipGetSymbolAddress, per device.
__device__ __align__(256) char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
void *g_scratch_ptr[kMaxDevices];
hipError_t g_scratch_status[kMaxDevices];

// The device address of the current device's array (looked up once per
// device, with that device current).
hipError_t static_scratch(void **ptr)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::call_once(g_scratch_once[dev], [dev] {
        void *p = nullptr;
        g_scratch_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch_ptr[dev] = g_scratch_status[dev] == hipSuccess ? p : nullptr;
    });
    *ptr = g_scratch_ptr[dev];
    return g_scratch_status[dev];
}

}  // namespace
}  // namespace gspn

extern "C" int gspn_scan_bwd_static(const void *x, const void *w, const void *lam, const void *u,
                                    const void *dy, void *dx, void *dw, void *dlam, void *du,
                                    int direction, int B, int C, int G, int H, int W, int dtype,
                                    void *stream)
{
    int st = check_common(direction, B, C, G, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    Buf bufs[11];
    int nb = 0;
    scan_buffers(GSPN_OP_BWD, x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction, B, C, G, H,
                 W, dtype, bufs, &nb);
    st = check_buffers(bufs, nb);
    if (st != GSPN_OK)
        return st;
    Problem p{x, w, lam, u, dy, nullptr, dx, dw, dlam, du, direction, B, C, G, H, W, dtype,
              kPixelMajor, nullptr};
    int64_t need = 0;
    st = count_workspace(GSPN_OP_BWD, p, &need);
    if (st != GSPN_OK)
        return st;
    if (need > (int64_t)kStaticScratchBytes)
        return GSPN_ERR_WORKSPACE;
    Workspace ws;
    if (need > 0) {
        void *ptr = nullptr;
        const hipError_t e = static_scratch(&ptr);
        if (e != hipSuccess)
            return hip_status(e);
        ws.base = static_cast<char *>(ptr);
        ws.size = kStaticScratchBytes;
    }
    p.ws = &ws;
    const hipError_t e = run_scan(GSPN_OP_BWD, p, w, dw, static_cast<hipStream_t>(stream));
    return e == hipErrorOutOfMemory ? GSPN_ERR_WORKSPACE : hip_status(e);
}

namespace gspn {
namespace {

// Sizes of a 1x1 convolution out[b] = A x[b] with A M x K and x[b] K x HW.
int check_project(int B, int M, int K, int H, int W, int dtype)
{
    if (dtype != GSPN_F32 && dtype != GSPN_BF16)
        return GSPN_ERR_DTYPE;
    if (B < 1 || M < 1 || K < 1 || H < 1 || W < 1)
        return GSPN_ERR_DIM;
    if (dtype != GSPN_BF16 || K % 8 != 0 || H > GSPN_MAX_SIDE || W > GSPN_MAX_SIDE)
        return GSPN_ERR_UNSUPPORTED;
    const int64_t HW = (int64_t)H * W;
    if ((int64_t)B * M > GSPN_MAX_ELEMS / HW || (int64_t)B * K > GSPN_MAX_ELEMS / HW)
        return GSPN_ERR_UNSUPPORTED;
    // one image's input and output maps are addressed with 32-bit byte offsets
    if ((int64_t)M * HW * 2 >= ((int64_t)1 << 31) || (int64_t)K * HW * 2 >= ((int64_t)1 << 31))
        return GSPN_ERR_UNSUPPORTED;
    // one workgroup per 64 output rows x 128 pixels of one image
    if ((int64_t)B * ((HW + 127) / 128) * ((M + 63) / 64) > 0x7fffffff)
        return GSPN_ERR_UNSUPPORTED;
    return GSPN_OK;
}

// Sizes of the latent parameter product: Cc latent channels, 6 D Cc rows.
int check_latent(int direction, int B, int Cc, int H, int W, int dtype)
{
    int st = check_common(direction, B, Cc, Cc, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    if (Cc % 8 != 0)
        return GSPN_ERR_UNSUPPORTED;
    return check_project(B, 6 * __builtin_popcount(direction) * Cc, Cc, H, W, dtype);
}

constexpr int64_t round8(int64_t n) { return (n + 7) / 8 * 8; }

}  // namespace
}  // namespace gspn

extern "C" int gspn_project(const void *a, const void *x, void *y, int B, int M, int K, int H,
                            int W, int dtype, void *stream)
{
    int st = check_project(B, M, K, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    const int64_t HW = (int64_t)H * W;
    const Buf bufs[] = {{a, (int64_t)M * K * 2, false},
                        {x, (int64_t)B * K * HW * 2, false},
                        {y, (int64_t)B * M * HW * 2, true}};
    st = check_buffers(bufs, 3);
    if (st != GSPN_OK)
        return st;
    return hip_status(launch_project(a, x, y, B, M, K, H, W, static_cast<hipStream_t>(stream)));
}

extern "C" int gspn_latent_params(const void *xc, const void *l_u, const void *l_lam,
                                  const void *l_w, void *u, void *lam, void *w, int direction,
                                  int B, int Cc, int H, int W, int dtype, void *stream)
{
    int st = check_latent(direction, B, Cc, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    const int64_t D = __builtin_popcount(direction);
    const int64_t n = (int64_t)B * Cc * H * W;
    const int64_t cc2 = (int64_t)Cc * Cc;
    const Buf bufs[] = {{xc, n * 2, false},          {l_u, D * cc2 * 2, false},
                        {l_lam, D * cc2 * 2, false}, {l_w, 3 * D * cc2 * 2, false},
                        {u, D * n * 2, true},        {lam, D * n * 2, true},
                        {w, 3 * D * n * 2, true}};
    st = check_buffers(bufs, 7);
    if (st != GSPN_OK)
        return st;
    return hip_status(launch_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, H, W,
                                           static_cast<hipStream_t>(stream)));
}

namespace gspn {
namespace {

// The latent sublayer's launches on the workspace ws (counting mode: none).
// The latent tensors belong to the call, so the scan may run on a grid padded
// at the bottom and right to whole 8-line blocks, where the register-streamed
// and wide kernels apply.  Padded pixels hold x_c = 0, hence u = lambda = 0;
// the taps of real pixels that point into the padding are normalized as off
// the grid (weight exactly 0); and a scan that starts in the padding carries
// h = 0 up to the first real line, which then starts from h = lambda x as on
// the unpadded grid.  Real pixels therefore see the same recurrence; P_up
// reads only them.
hipError_t run_latent(const void *x, const void *p_down, const void *l_u, const void *l_lam,
                      const void *l_w, const void *p_up, void *y, int direction, int B, int C,
                      int Cc, int H, int W, Workspace &ws, hipStream_t s)
{
    const int64_t D = __builtin_popcount(direction);
    const auto up8 = [](int v) { return (v + 7) / 8 * 8; };
    const bool pad = (H % 8 != 0 || W % 8 != 0) && (H > 16 || W > 16) && up8(H) <= 256 &&
                     up8(W) <= 256;
    const int Hp = pad ? up8(H) : H, Wp = pad ? up8(W) : W;
    const int64_t ncp = (int64_t)B * Cc * Hp * Wp;
    // latent x_c, u, lambda, w and y_c in one block, 16-byte aligned parts
    const int64_t o_u = round8(ncp), o_l = o_u + round8(D * ncp), o_w = o_l + round8(D * ncp);
    const int64_t o_y = o_w + round8(3 * D * ncp), total = o_y + round8(ncp);
    void *scr = nullptr;
    hipError_t e = ws.take(&scr, (size_t)(total * 2));
    if (e != hipSuccess)
        return e;
    // (no pointers into the workspace while counting: it has no base then)
    uint16_t *base = static_cast<uint16_t *>(scr);
    const auto at = [&](int64_t o) { return ws.counting ? nullptr : base + o; };
    uint16_t *xc = base, *u = at(o_u), *lam = at(o_l), *w = at(o_w), *yc = at(o_y);
    if (!ws.counting) {
        e = launch_project(p_down, x, xc, B, Cc, C, Hp, Wp, s, H, W);
        if (e == hipSuccess)
            e = launch_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, Hp, Wp, s,
                                     H, W);
        if (e != hipSuccess)
            return e;
    }
    Problem p{xc, w, lam, u, nullptr, yc, nullptr, nullptr, nullptr, nullptr,
              direction, B, Cc, Cc, Hp, Wp, GSPN_BF16, kBlocked, &ws};
    e = dispatch_fwd(p, s);
    if (e != hipSuccess || ws.counting)
        return e;
    return launch_project(p_up, yc, y, B, C, Cc, H, W, s, Hp, Wp);
}

int check_latent_all(int direction, int B, int C, int Cc, int H, int W, int dtype)
{
    int st = check_latent(direction, B, Cc, H, W, dtype);
    if (st == GSPN_OK)
        st = check_project(B, C, Cc, H, W, dtype);
    if (st == GSPN_OK)
        st = check_project(B, Cc, C, H, W, dtype);
    // the latent grid may be padded by up to 7 lines each way
    if (st == GSPN_OK && H + 7 <= GSPN_MAX_SIDE && W + 7 <= GSPN_MAX_SIDE)
        st = check_latent(direction, B, Cc, H + 7, W + 7, dtype);
    return st;
}

}  // namespace
}  // namespace gspn

extern "C" int gspn_latent_workspace_size(int direction, int B, int C, int Cc, int H, int W,
                                          int dtype, int64_t *bytes)
{
    if (bytes == nullptr)
        return GSPN_ERR_NULL;
    *bytes = 0;
    const int st = check_latent_all(direction, B, C, Cc, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    Workspace ws;
    ws.counting = true;
    const hipError_t e = run_latent(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                    direction, B, C, Cc, H, W, ws, nullptr);
    if (e != hipSuccess)
        return hip_status(e);
    *bytes = (int64_t)ws.used;
    return GSPN_OK;
}

extern "C" int gspn_latent_fwd(const void *x, const void *p_down, const void *l_u,
                               const void *l_lam, const void *l_w, const void *p_up, void *y,
                               int direction, int B, int C, int Cc, int H, int W, int dtype,
                               void *workspace, int64_t workspace_bytes, void *stream)
{
    int st = check_latent_all(direction, B, C, Cc, H, W, dtype);
    if (st != GSPN_OK)
        return st;
    const int64_t D = __builtin_popcount(direction);
    const int64_t HW = (int64_t)H * W;
    const int64_t n = (int64_t)B * C * HW;
    const int64_t cc2 = (int64_t)Cc * Cc;
    Buf bufs[8] = {{x, n * 2, false},           {p_down, (int64_t)Cc * C * 2, false},
                   {l_u, D * cc2 * 2, false},   {l_lam, D * cc2 * 2, false},
                   {l_w, 3 * D * cc2 * 2, false}, {p_up, (int64_t)C * Cc * 2, false},
                   {y, n * 2, true}};
    st = check_buffers(bufs, 7);
    if (st != GSPN_OK)
        return st;
    Workspace cnt;
    cnt.counting = true;
    hipError_t e = run_latent(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H, W, cnt,
                              nullptr);
    if (e != hipSuccess)
        return hip_status(e);
    const int64_t need = (int64_t)cnt.used;
    if (workspace_bytes < need || workspace == nullptr)
        return GSPN_ERR_WORKSPACE;
    bufs[7] = {workspace, need, true};
    st = check_buffers(bufs, 8);
    if (st != GSPN_OK)
        return st;
    Workspace ws;
    ws.base = static_cast<char *>(workspace);
    ws.size = (size_t)workspace_bytes;
    e = run_latent(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H, W, ws,
                   static_cast<hipStream_t>(stream));
    return e == hipErrorOutOfMemory ? GSPN_ERR_WORKSPACE : hip_status(e);
}

extern "C" const char *gspn_strerror(int status)
{
    switch (status) {
    case GSPN_OK: return "success";
    case GSPN_ERR_NULL: return "a required pointer is NULL";
    case GSPN_ERR_DIM: return "a size is < 1 or C is not a multiple of G";
    case GSPN_ERR_DIRECTION: return "direction mask outside [1, 15]";
    case GSPN_ERR_DTYPE: return "unknown storage type";
    case GSPN_ERR_ALIGN: return "a base pointer is not 16-byte aligned";
    case GSPN_ERR_ALIAS: return "two buffers of the call overlap";
    case GSPN_ERR_UNSUPPORTED: return "shape beyond the supported limits";
    case GSPN_ERR_HIP: return "a HIP runtime call or kernel launch failed";
    case GSPN_ERR_WORKSPACE: return "the workspace or the reserve is missing or smaller than the call needs";
    default: return "unknown status";
    }
}

extern "C" int gspn_last_hip_error(void) { return g_last_hip_error; }

extern "C" int gspn_version(void) { return 200; }
