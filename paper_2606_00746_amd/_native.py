"""ctypes binding of libgspn (argument marshalling only).

The raw functions keep the C names and signatures of ``include/gspn.h``.
The torch front end (``scan_fwd``, ``scan_bwd``, ...) takes device tensors,
checks their sizes, dtypes and devices, derives the sizes from the shapes,
asks the library how much workspace the call needs and hands it a torch
buffer of that size, and raises :class:`GspnError` on a non-zero status.
Every step of the scan runs in the library's HIP kernels; there is no other
code path, and loading fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgspn.so")

T2B, B2T, L2R, R2L, ALL = 1, 2, 4, 8, 15
F32, BF16 = 0, 1
(OK, ERR_NULL, ERR_DIM, ERR_DIRECTION, ERR_DTYPE, ERR_ALIGN, ERR_ALIAS, ERR_UNSUPPORTED, ERR_HIP,
 ERR_WORKSPACE) = (0, -1, -2, -3, -4, -5, -6, -7, -8, -9)
(OP_FWD, OP_BWD, OP_FWD_NORM, OP_BWD_NORM, OP_FWD_BLOCKED, OP_BWD_BLOCKED, OP_FWD_TRAIN,
 OP_BWD_RESERVE, OP_FWD_NORM_TRAIN, OP_BWD_NORM_RESERVE) = range(10)
MAX_SIDE = 4096

# layouts of the per-direction tensors
PIXEL, BLOCKED = "pixel", "blocked"

EXPORTED = ("gspn_workspace_size", "gspn_scan_fwd", "gspn_scan_bwd", "gspn_scan_fwd_blocked",
            "gspn_scan_bwd_blocked", "gspn_scan_fwd_norm", "gspn_scan_bwd_norm",
            "gspn_scan_bwd_static", "gspn_workspace_size_slots", "gspn_scan_bwd_slots",
            "gspn_reserve_size", "gspn_scan_fwd_train", "gspn_scan_bwd_reserve",
            "gspn_reserve_size_norm", "gspn_scan_fwd_norm_train", "gspn_scan_bwd_norm_reserve",
            "gspn_project",
            "gspn_latent_params", "gspn_latent_workspace_size", "gspn_latent_fwd",
            "gspn_strerror", "gspn_last_hip_error", "gspn_version")

_lib = None


class GspnError(RuntimeError):
    def __init__(self, status: int, hip_error: int = 0):
        msg = f"libgspn status {status}: {gspn_strerror(status)}"
        if status == ERR_HIP:
            msg += f" (hipError_t {hip_error})"
        super().__init__(msg)
        self.status = status
        self.hip_error = hip_error


def load() -> ctypes.CDLL:
    """Load libgspn.so (built in place by ``paper_2606_00746_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2606_00746_amd.build` "
                "(there is no fallback implementation)")
        lib = ctypes.CDLL(LIB_PATH)
        vp, i, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        pi64 = ctypes.POINTER(ctypes.c_int64)
        scan8 = [i] * 7                     # direction, B, C, G, H, W, dtype
        ws = [vp, i64, vp]                  # workspace, workspace_bytes, stream
        lib.gspn_workspace_size.argtypes = [i] + scan8 + [pi64]
        for name in ("gspn_scan_fwd", "gspn_scan_fwd_blocked", "gspn_scan_fwd_norm"):
            getattr(lib, name).argtypes = [vp] * 5 + scan8 + ws
        for name in ("gspn_scan_bwd", "gspn_scan_bwd_blocked", "gspn_scan_bwd_norm"):
            getattr(lib, name).argtypes = [vp] * 9 + scan8 + ws
        lib.gspn_scan_bwd_static.argtypes = [vp] * 9 + scan8 + [vp]
        lib.gspn_workspace_size_slots.argtypes = [i] + scan8 + [pi64]
        lib.gspn_scan_bwd_slots.argtypes = [i] + [vp] * 9 + scan8 + ws
        for name in ("gspn_reserve_size", "gspn_reserve_size_norm"):
            getattr(lib, name).argtypes = scan8 + [pi64]
        for name in ("gspn_scan_fwd_train", "gspn_scan_fwd_norm_train"):
            getattr(lib, name).argtypes = [vp] * 5 + scan8 + [vp, i64] + ws
        for name in ("gspn_scan_bwd_reserve", "gspn_scan_bwd_norm_reserve"):
            getattr(lib, name).argtypes = [vp] * 9 + scan8 + [vp, i64] + ws
        lib.gspn_project.argtypes = [vp, vp, vp, i, i, i, i, i, i, vp]
        lib.gspn_latent_params.argtypes = [vp] * 7 + [i] * 6 + [vp]
        lib.gspn_latent_workspace_size.argtypes = [i] * 7 + [pi64]
        lib.gspn_latent_fwd.argtypes = [vp] * 7 + [i] * 7 + ws
        for name in EXPORTED:
            getattr(lib, name).restype = i
        lib.gspn_strerror.argtypes = [i]
        lib.gspn_strerror.restype = ctypes.c_char_p
        lib.gspn_last_hip_error.argtypes = []
        lib.gspn_version.argtypes = []
        _lib = lib
    return _lib


# ---------------------------------------------------------------------------
# raw C entry points (pointers as ints, sizes as ints)
# ---------------------------------------------------------------------------

def gspn_workspace_size(op, direction, B, C, G, H, W, dtype):
    """(status, bytes) of gspn_workspace_size."""
    n = ctypes.c_int64(0)
    st = load().gspn_workspace_size(op, direction, B, C, G, H, W, dtype, ctypes.byref(n))
    return st, n.value


def gspn_scan_fwd(x, w, lam, u, y, direction, B, C, G, H, W, dtype, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_fwd(x, w, lam, u, y, direction, B, C, G, H, W, dtype, ws, ws_bytes,
                                stream)


def gspn_scan_bwd(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W, dtype, ws,
                  ws_bytes, stream) -> int:
    return load().gspn_scan_bwd(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W,
                                dtype, ws, ws_bytes, stream)


def gspn_scan_fwd_blocked(x, w, lam, u, y, direction, B, C, G, H, W, dtype, ws, ws_bytes,
                          stream) -> int:
    return load().gspn_scan_fwd_blocked(x, w, lam, u, y, direction, B, C, G, H, W, dtype, ws,
                                        ws_bytes, stream)


def gspn_scan_bwd_blocked(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W, dtype, ws,
                          ws_bytes, stream) -> int:
    return load().gspn_scan_bwd_blocked(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H,
                                        W, dtype, ws, ws_bytes, stream)


def gspn_scan_fwd_norm(x, w_logits, lam, u, y, direction, B, C, G, H, W, dtype, ws, ws_bytes,
                       stream) -> int:
    return load().gspn_scan_fwd_norm(x, w_logits, lam, u, y, direction, B, C, G, H, W, dtype, ws,
                                     ws_bytes, stream)


def gspn_scan_bwd_norm(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du, direction, B, C, G, H,
                       W, dtype, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_bwd_norm(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du, direction,
                                     B, C, G, H, W, dtype, ws, ws_bytes, stream)


def gspn_scan_bwd_static(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W, dtype,
                         stream) -> int:
    return load().gspn_scan_bwd_static(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H,
                                       W, dtype, stream)


def gspn_reserve_size(direction, B, C, G, H, W, dtype):
    """(status, bytes) of gspn_reserve_size."""
    n = ctypes.c_int64(0)
    st = load().gspn_reserve_size(direction, B, C, G, H, W, dtype, ctypes.byref(n))
    return st, n.value


def gspn_scan_fwd_train(x, w, lam, u, y, direction, B, C, G, H, W, dtype, rs, rs_bytes, ws,
                        ws_bytes, stream) -> int:
    return load().gspn_scan_fwd_train(x, w, lam, u, y, direction, B, C, G, H, W, dtype, rs,
                                      rs_bytes, ws, ws_bytes, stream)


def gspn_scan_bwd_reserve(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W, dtype,
                          rs, rs_bytes, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_bwd_reserve(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G,
                                        H, W, dtype, rs, rs_bytes, ws, ws_bytes, stream)


def gspn_reserve_size_norm(direction, B, C, G, H, W, dtype):
    """(status, bytes) of gspn_reserve_size_norm."""
    n = ctypes.c_int64(0)
    st = load().gspn_reserve_size_norm(direction, B, C, G, H, W, dtype, ctypes.byref(n))
    return st, n.value


def gspn_scan_fwd_norm_train(x, w_logits, lam, u, y, direction, B, C, G, H, W, dtype, rs,
                             rs_bytes, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_fwd_norm_train(x, w_logits, lam, u, y, direction, B, C, G, H, W,
                                           dtype, rs, rs_bytes, ws, ws_bytes, stream)


def gspn_scan_bwd_norm_reserve(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du, direction, B,
                               C, G, H, W, dtype, rs, rs_bytes, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_bwd_norm_reserve(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du,
                                             direction, B, C, G, H, W, dtype, rs, rs_bytes, ws,
                                             ws_bytes, stream)


def gspn_workspace_size_slots(slots, direction, B, C, G, H, W, dtype):
    """(status, bytes) of gspn_workspace_size_slots."""
    n = ctypes.c_int64(0)
    st = load().gspn_workspace_size_slots(slots, direction, B, C, G, H, W, dtype, ctypes.byref(n))
    return st, n.value


def gspn_scan_bwd_slots(slots, x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W,
                        dtype, ws, ws_bytes, stream) -> int:
    return load().gspn_scan_bwd_slots(slots, x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C,
                                      G, H, W, dtype, ws, ws_bytes, stream)


STATIC_SCRATCH_BYTES = 64 << 20


def gspn_project(a, x, y, B, M, K, H, W, dtype, stream) -> int:
    return load().gspn_project(a, x, y, B, M, K, H, W, dtype, stream)


def gspn_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, H, W, dtype,
                       stream) -> int:
    return load().gspn_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, H, W,
                                     dtype, stream)


def gspn_latent_workspace_size(direction, B, C, Cc, H, W, dtype):
    """(status, bytes) of gspn_latent_workspace_size."""
    n = ctypes.c_int64(0)
    st = load().gspn_latent_workspace_size(direction, B, C, Cc, H, W, dtype, ctypes.byref(n))
    return st, n.value


def gspn_latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H, W, dtype, ws,
                    ws_bytes, stream) -> int:
    return load().gspn_latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H,
                                  W, dtype, ws, ws_bytes, stream)


def gspn_strerror(status: int) -> str:
    return load().gspn_strerror(status).decode()


def gspn_last_hip_error() -> int:
    return load().gspn_last_hip_error()


def gspn_version() -> int:
    return load().gspn_version()


# ---------------------------------------------------------------------------
# torch-tensor front end (sizes from shapes, current stream)
# ---------------------------------------------------------------------------

def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}; use float32 or bfloat16")


def _stream_handle(t, stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream(t.device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check_raise(status):
    if status != OK:
        raise GspnError(status, gspn_last_hip_error() if status == ERR_HIP else 0)


def _ndirs(direction: int) -> int:
    return bin(direction & 15).count("1")


def _check_tensors(ref, named):
    """Every tensor of `named` ({name: (tensor, numel)}) must sit on ref's GPU,
    share its dtype, be contiguous and hold exactly numel elements."""
    if not ref.is_contiguous():
        raise ValueError("x must be contiguous")
    for name, (t, numel) in named.items():
        if t.numel() != numel:
            raise ValueError(f"{name} must hold {numel} elements, not {t.numel()}")
        if t.dtype != ref.dtype:
            raise ValueError(f"{name} must have dtype {ref.dtype}, not {t.dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    if not ref.is_cuda:
        raise ValueError("tensors must be on a GPU")
    for name, (t, _) in named.items():
        if not t.is_cuda or t.device != ref.device:
            raise ValueError(f"{name} must be on {ref.device}")


def _sizes(x, w, direction):
    """(B, C, G, H, W) from x [B,C,H,W] and w [D,B,G,3,...]."""
    if x.dim() != 4 or w.dim() < 3:
        raise ValueError("x must be [B,C,H,W] and w [D,B,G,3,...]")
    B, C, H, W = x.shape
    return B, C, w.shape[2], H, W


def workspace_size(op, x, w, direction) -> int:
    """Bytes of workspace operation `op` (OP_*) takes for these tensors."""
    B, C, G, H, W = _sizes(x, w, direction)
    st, n = gspn_workspace_size(op, direction, B, C, G, H, W, _dtype_code(x))
    _check_raise(st)
    return n


def _workspace(op, direction, B, C, G, H, W, dtype, device, given=None, slots=0):
    """The device buffer operation `op` works in: `given` (a uint8 tensor on
    the same device) when it is large enough, else a new one (None if the
    call needs none)."""
    import torch
    st, n = (gspn_workspace_size_slots(slots, direction, B, C, G, H, W, dtype) if slots
             else gspn_workspace_size(op, direction, B, C, G, H, W, dtype))
    _check_raise(st)
    if n == 0:
        return None, 0
    if given is not None:
        if given.device != device or given.dtype != torch.uint8 or not given.is_contiguous():
            raise ValueError("workspace must be a contiguous uint8 tensor on the inputs' device")
        if given.numel() >= n:
            return given, given.numel()
    return torch.empty(n, dtype=torch.uint8, device=device), n


def _scan(op, x, w, lam, u, direction, outs, dy=None, stream=None, workspace=None, slots=0,
          reserve=None):
    B, C, G, H, W = _sizes(x, w, direction)
    D = _ndirs(direction)
    n, nd, nw = B * C * H * W, D * B * C * H * W, D * B * G * 3 * H * W
    named = {"w": (w, nw), "lam": (lam, nd), "u": (u, nd)}
    bwd = dy is not None
    if bwd:
        dx, dw, dlam, du = outs
        named.update(dy=(dy, n), dx=(dx, n), dw=(dw, nw), dlam=(dlam, nd), du=(du, nd))
    else:
        named.update(y=(outs[0], n))
    _check_tensors(x, named)
    if reserve is not None:
        import torch
        if (reserve.dtype != torch.uint8 or not reserve.is_contiguous() or not reserve.is_cuda
                or reserve.device != x.device):
            raise ValueError("reserve must be a contiguous uint8 tensor on the inputs' device")
    dt = _dtype_code(x)
    ws, nbytes = _workspace(op, direction, B, C, G, H, W, dt, x.device, workspace, slots)
    ptrs = [t.data_ptr() for t in (x, w, lam, u)]
    if bwd:
        ptrs += [t.data_ptr() for t in (dy, dx, dw, dlam, du)]
    else:
        ptrs.append(outs[0].data_ptr())
    fn = {OP_FWD: gspn_scan_fwd, OP_BWD: gspn_scan_bwd, OP_FWD_BLOCKED: gspn_scan_fwd_blocked,
          OP_BWD_BLOCKED: gspn_scan_bwd_blocked, OP_FWD_NORM: gspn_scan_fwd_norm,
          OP_BWD_NORM: gspn_scan_bwd_norm, OP_FWD_TRAIN: gspn_scan_fwd_train,
          OP_BWD_RESERVE: gspn_scan_bwd_reserve, OP_FWD_NORM_TRAIN: gspn_scan_fwd_norm_train,
          OP_BWD_NORM_RESERVE: gspn_scan_bwd_norm_reserve}[op]
    if slots:
        fn = lambda *a: gspn_scan_bwd_slots(slots, *a)          # noqa: E731
    if op in (OP_FWD_TRAIN, OP_BWD_RESERVE, OP_FWD_NORM_TRAIN, OP_BWD_NORM_RESERVE):
        rp, rn = (reserve.data_ptr(), reserve.numel()) if reserve is not None else (None, 0)
        fn0 = fn
        fn = lambda *a: fn0(*a[:-3], rp, rn, *a[-3:])            # noqa: E731
    status = fn(*ptrs, direction, B, C, G, H, W, dt, ws.data_ptr() if ws is not None else None,
                nbytes, _stream_handle(x, stream))
    _check_raise(status)


def _check_layout(layout):
    if layout not in (PIXEL, BLOCKED):
        raise ValueError(f"layout must be {PIXEL!r} or {BLOCKED!r}")


def scan_fwd(x, w, lam, u, direction: int = ALL, y=None, stream=None, layout: str = PIXEL,
             workspace=None):
    """y = sum_d u_d * h_d for device tensors (see include/gspn.h).

    x [B,C,H,W]; lam, u [D,B,C,H,W] and w [D,B,G,3,H,W] pixel-major, or, with
    layout="blocked", in the blocked line-major layout of the _blocked entry
    points (each plane H*W elements long).  `workspace`: an optional uint8
    device tensor the call may use (a new one is taken when it is missing or
    too small)."""
    import torch
    _check_layout(layout)
    if y is None:
        y = torch.empty_like(x)
    _scan(OP_FWD if layout == PIXEL else OP_FWD_BLOCKED, x, w, lam, u, direction, (y,),
          stream=stream, workspace=workspace)
    return y


def scan_bwd(x, w, lam, u, dy, direction: int = ALL, out=None, stream=None, layout: str = PIXEL,
             workspace=None, slots: int = 0):
    """Gradients (dx, dw, dlam, du) of <y, dy> for device tensors, in the
    layout of the inputs.  `slots` (4 or 8, pixel-major only) forces that
    plan of the register-streamed backward (gspn_scan_bwd_slots); 0 leaves
    the choice to the library."""
    import torch
    _check_layout(layout)
    if slots and layout != PIXEL:
        raise ValueError("slots applies to the pixel-major backward only")
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w), torch.empty_like(lam),
               torch.empty_like(u))
    _scan(OP_BWD if layout == PIXEL else OP_BWD_BLOCKED, x, w, lam, u, direction, out, dy=dy,
          stream=stream, workspace=workspace, slots=slots)
    return out


def reserve_size(x, w, direction, norm: bool = False) -> int:
    """Bytes of the reserve of the training pair for these tensors (norm: the
    pair of the _norm entry points, w holding the logits)."""
    B, C, G, H, W = _sizes(x, w, direction)
    st, n = (gspn_reserve_size_norm if norm else gspn_reserve_size)(direction, B, C, G, H, W,
                                                                     _dtype_code(x))
    _check_raise(st)
    return n


def _train_fwd(op, x, w, lam, u, direction, y, reserve, stream, workspace):
    import torch
    if y is None:
        y = torch.empty_like(x)
    n = reserve_size(x, w, direction, norm=op == OP_FWD_NORM_TRAIN)
    if n == 0:
        reserve = None
    elif reserve is None:
        reserve = torch.empty(n, dtype=torch.uint8, device=x.device)
    elif reserve.numel() < n:
        raise ValueError(f"reserve of {reserve.numel()} bytes, smaller than the {n} bytes "
                         "reserve_size gives for these tensors")
    _scan(op, x, w, lam, u, direction, (y,), stream=stream, workspace=workspace,
          reserve=reserve)
    return y, reserve


def scan_fwd_train(x, w, lam, u, direction: int = ALL, y=None, reserve=None, stream=None,
                   workspace=None):
    """scan_fwd (pixel-major) that also fills the reserve its backward,
    scan_bwd_reserve, reads.  Returns (y, reserve); `reserve`: a uint8 device
    tensor of at least reserve_size bytes, or None for a new one (None is
    returned where the shape needs no reserve)."""
    return _train_fwd(OP_FWD_TRAIN, x, w, lam, u, direction, y, reserve, stream, workspace)


def scan_fwd_norm_train(x, w_logits, lam, u, direction: int = ALL, y=None, reserve=None,
                        stream=None, workspace=None):
    """scan_fwd_norm that also fills the reserve scan_bwd_norm_reserve reads
    (the formed weights among it).  Returns (y, reserve) as scan_fwd_train."""
    return _train_fwd(OP_FWD_NORM_TRAIN, x, w_logits, lam, u, direction, y, reserve, stream,
                      workspace)


def scan_bwd_norm_reserve(x, w_logits, lam, u, dy, reserve, direction: int = ALL, out=None,
                          stream=None, workspace=None):
    """scan_bwd_norm reading the reserve that scan_fwd_norm_train wrote for
    the same x, logits, lam, u; returns (dx, dw_logits, dlam, du)."""
    import torch
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w_logits), torch.empty_like(lam),
               torch.empty_like(u))
    _scan(OP_BWD_NORM_RESERVE, x, w_logits, lam, u, direction, out, dy=dy, stream=stream,
          workspace=workspace, reserve=reserve)
    return out


def scan_bwd_reserve(x, w, lam, u, dy, reserve, direction: int = ALL, out=None, stream=None,
                     workspace=None):
    """scan_bwd (pixel-major) reading the reserve that scan_fwd_train wrote
    for the same x, w, lam, u."""
    import torch
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w), torch.empty_like(lam),
               torch.empty_like(u))
    _scan(OP_BWD_RESERVE, x, w, lam, u, direction, out, dy=dy, stream=stream,
          workspace=workspace, reserve=reserve)
    return out


def scan_fwd_norm(x, w_logits, lam, u, direction: int = ALL, y=None, stream=None,
                  workspace=None):
    """As :func:`scan_fwd`, with the weights given by their logits
    (Sec. 3, Eq. (row_stochastic_norm)); pixel-major."""
    import torch
    if y is None:
        y = torch.empty_like(x)
    _scan(OP_FWD_NORM, x, w_logits, lam, u, direction, (y,), stream=stream, workspace=workspace)
    return y


def scan_bwd_norm(x, w_logits, lam, u, dy, direction: int = ALL, out=None, stream=None,
                  workspace=None):
    """Gradients (dx, dw_logits, dlam, du) of <y, dy>, the weights given by
    their logits; pixel-major."""
    import torch
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w_logits), torch.empty_like(lam),
               torch.empty_like(u))
    _scan(OP_BWD_NORM, x, w_logits, lam, u, direction, out, dy=dy, stream=stream,
          workspace=workspace)
    return out


def project(a, x, y=None, stream=None):
    """1x1 convolution y[b] = a @ x[b]: a [M, K], x [B, K, H, W] -> y [B, M, H, W] (bf16)."""
    import torch
    if a.dim() != 2 or x.dim() != 4 or a.shape[1] != x.shape[1]:
        raise ValueError("a must be [M, K] and x [B, K, H, W]")
    M, K = a.shape
    B, _, H, W = x.shape
    if y is None:
        y = torch.empty((B, M, H, W), dtype=x.dtype, device=x.device)
    _check_tensors(x, {"a": (a, M * K), "y": (y, B * M * H * W)})
    status = gspn_project(a.data_ptr(), x.data_ptr(), y.data_ptr(), B, M, K, H, W, _dtype_code(x),
                          _stream_handle(x, stream))
    _check_raise(status)
    return y


def _latent_weights(l_u, l_lam, l_w, direction):
    D = _ndirs(direction)
    Cc = l_u.shape[-1]
    if (tuple(l_u.shape) != (D, Cc, Cc) or tuple(l_lam.shape) != (D, Cc, Cc)
            or tuple(l_w.shape) != (D, Cc, 3, Cc)):
        raise ValueError("l_u, l_lam must be [D, Cc, Cc] and l_w [D, Cc, 3, Cc]")
    return D, Cc


def latent_params(xc, l_u, l_lam, l_w, direction: int = ALL, out=None, stream=None):
    """u, lam and normalized w of every direction from the latent map xc [B, Cc, H, W]
    (Sec. 5, Eq. (latent_params); Sec. 3, Eq. (row_stochastic_norm)), in the
    scan's blocked line-major layout: u, lam [D, B, Cc, H*W], w [D, B, Cc, 3, H*W]."""
    import torch
    D, Cc = _latent_weights(l_u, l_lam, l_w, direction)
    B, _, H, W = xc.shape
    if out is None:
        kw = dict(dtype=xc.dtype, device=xc.device)
        out = (torch.empty((D, B, Cc, H * W), **kw), torch.empty((D, B, Cc, H * W), **kw),
               torch.empty((D, B, Cc, 3, H * W), **kw))
    u, lam, w = out
    n = B * Cc * H * W
    _check_tensors(xc, {"l_u": (l_u, D * Cc * Cc), "l_lam": (l_lam, D * Cc * Cc),
                        "l_w": (l_w, 3 * D * Cc * Cc), "u": (u, D * n), "lam": (lam, D * n),
                        "w": (w, 3 * D * n)})
    status = gspn_latent_params(*[t.data_ptr() for t in (xc, l_u, l_lam, l_w, u, lam, w)],
                                direction, B, Cc, H, W, _dtype_code(xc), _stream_handle(xc, stream))
    _check_raise(status)
    return u, lam, w


def latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, direction: int = ALL, y=None, stream=None):
    """The latent-space propagation sublayer (Sec. 5): y = P_up(Prop_2D(P_down x))
    with the propagation parameters predicted from the latent map.
    x [B, C, H, W], p_down [Cc, C], l_u, l_lam [D, Cc, Cc], l_w [D, Cc, 3, Cc],
    p_up [C, Cc] -> y [B, C, H, W] (bf16)."""
    import torch
    D, Cc = _latent_weights(l_u, l_lam, l_w, direction)
    B, C, H, W = x.shape
    if tuple(p_down.shape) != (Cc, C) or tuple(p_up.shape) != (C, Cc):
        raise ValueError("p_down must be [Cc, C] and p_up [C, Cc]")
    if y is None:
        y = torch.empty_like(x)
    _check_tensors(x, {"p_down": (p_down, Cc * C), "l_u": (l_u, D * Cc * Cc),
                       "l_lam": (l_lam, D * Cc * Cc), "l_w": (l_w, 3 * D * Cc * Cc),
                       "p_up": (p_up, C * Cc), "y": (y, B * C * H * W)})
    dt = _dtype_code(x)
    st, nbytes = gspn_latent_workspace_size(direction, B, C, Cc, H, W, dt)
    _check_raise(st)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    status = gspn_latent_fwd(*[t.data_ptr() for t in (x, p_down, l_u, l_lam, l_w, p_up, y)],
                             direction, B, C, Cc, H, W, dt,
                             ws.data_ptr() if ws is not None else None, nbytes,
                             _stream_handle(x, stream))
    _check_raise(status)
    return y
