"""ctypes binding of libgspn (argument marshalling only).

The raw functions keep the C names and signatures of ``include/gspn.h``.
``scan_fwd`` / ``scan_bwd`` take torch tensors, derive the sizes from their
shapes, and raise :class:`GspnError` on a non-zero status.  Every step of the
scan runs in the library's HIP kernels; there is no other code path, and
loading fails loudly when the library is missing.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgspn.so")

T2B, B2T, L2R, R2L, ALL = 1, 2, 4, 8, 15
F32, BF16 = 0, 1
OK, ERR_NULL, ERR_DIM, ERR_DIRECTION, ERR_DTYPE, ERR_ALIGN, ERR_ALIAS, ERR_UNSUPPORTED, ERR_HIP = (
    0, -1, -2, -3, -4, -5, -6, -7, -8)
MAX_SIDE = 4096

EXPORTED = ("gspn_scan_fwd", "gspn_scan_bwd", "gspn_scan_fwd_norm", "gspn_scan_bwd_norm",
            "gspn_project", "gspn_latent_params", "gspn_latent_fwd",
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
        vp, i = ctypes.c_void_p, ctypes.c_int
        lib.gspn_scan_fwd.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
        lib.gspn_scan_fwd.restype = i
        lib.gspn_scan_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
        lib.gspn_scan_bwd.restype = i
        lib.gspn_scan_fwd_norm.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
        lib.gspn_scan_fwd_norm.restype = i
        lib.gspn_scan_bwd_norm.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i,
                                           vp]
        lib.gspn_scan_bwd_norm.restype = i
        lib.gspn_project.argtypes = [vp, vp, vp, i, i, i, i, i, i, vp]
        lib.gspn_project.restype = i
        lib.gspn_latent_params.argtypes = [vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp]
        lib.gspn_latent_params.restype = i
        lib.gspn_latent_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, vp]
        lib.gspn_latent_fwd.restype = i
        lib.gspn_strerror.argtypes = [i]
        lib.gspn_strerror.restype = ctypes.c_char_p
        lib.gspn_last_hip_error.argtypes = []
        lib.gspn_last_hip_error.restype = i
        lib.gspn_version.argtypes = []
        lib.gspn_version.restype = i
        _lib = lib
    return _lib


# ---------------------------------------------------------------------------
# raw C entry points (pointers as ints, sizes as ints)
# ---------------------------------------------------------------------------

def gspn_scan_fwd(x, w, lam, u, y, direction, B, C, G, H, W, dtype, stream) -> int:
    return load().gspn_scan_fwd(x, w, lam, u, y, direction, B, C, G, H, W, dtype, stream)


def gspn_scan_bwd(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W, dtype,
                  stream) -> int:
    return load().gspn_scan_bwd(x, w, lam, u, dy, dx, dw, dlam, du, direction, B, C, G, H, W,
                                dtype, stream)


def gspn_scan_fwd_norm(x, w_logits, lam, u, y, direction, B, C, G, H, W, dtype, stream) -> int:
    return load().gspn_scan_fwd_norm(x, w_logits, lam, u, y, direction, B, C, G, H, W, dtype,
                                     stream)


def gspn_scan_bwd_norm(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du, direction, B, C, G, H,
                       W, dtype, stream) -> int:
    return load().gspn_scan_bwd_norm(x, w_logits, lam, u, dy, dx, dw_logits, dlam, du, direction,
                                     B, C, G, H, W, dtype, stream)


def gspn_project(a, x, y, B, M, K, H, W, dtype, stream) -> int:
    return load().gspn_project(a, x, y, B, M, K, H, W, dtype, stream)


def gspn_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, H, W, dtype,
                       stream) -> int:
    return load().gspn_latent_params(xc, l_u, l_lam, l_w, u, lam, w, direction, B, Cc, H, W,
                                     dtype, stream)


def gspn_latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H, W, dtype,
                    stream) -> int:
    return load().gspn_latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, y, direction, B, C, Cc, H,
                                  W, dtype, stream)


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


def _sizes(x, w, lam, u, direction):
    """(B, C, G, H, W) from x [B,C,H,W] and w [D,B,G,3,...] (line-major planes)."""
    if x.dim() != 4 or w.dim() < 3:
        raise ValueError("x must be [B,C,H,W] and w [D,B,G,3,plane]")
    B, C, H, W = x.shape
    G = w.shape[2]
    D = bin(direction & 15).count("1")
    if w.numel() != D * B * G * 3 * H * W:
        raise ValueError("w must hold D*B*G*3*H*W elements")
    if lam.numel() != D * B * C * H * W or u.numel() != D * B * C * H * W:
        raise ValueError("lam and u must hold D*B*C*H*W elements")
    return B, C, G, H, W


def _ptrs(*ts):
    for t in ts:
        if not t.is_contiguous():
            raise ValueError("all tensors must be contiguous")
    return [t.data_ptr() for t in ts]


def scan_fwd(x, w, lam, u, direction: int = ALL, y=None, stream=None):
    """y = sum_d u_d * h_d for device tensors (see include/gspn.h).

    x is pixel-major [B,C,H,W]; lam, u and w are line-major per direction
    (horizontal-direction planes transposed), e.g. from :func:`to_line_major`.
    """
    import torch
    B, C, G, H, W = _sizes(x, w, lam, u, direction)
    if y is None:
        y = torch.empty_like(x)
    status = gspn_scan_fwd(*_ptrs(x, w, lam, u, y), direction, B, C, G, H, W, _dtype_code(x),
                           _stream_handle(x, stream))
    _check_raise(status)
    return y


def scan_bwd(x, w, lam, u, dy, direction: int = ALL, out=None, stream=None):
    """Gradients (dx, dw, dlam, du) of <y, dy> for device tensors."""
    import torch
    B, C, G, H, W = _sizes(x, w, lam, u, direction)
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w), torch.empty_like(lam),
               torch.empty_like(u))
    dx, dw, dlam, du = out
    status = gspn_scan_bwd(*_ptrs(x, w, lam, u, dy, dx, dw, dlam, du), direction, B, C, G, H, W,
                           _dtype_code(x), _stream_handle(x, stream))
    _check_raise(status)
    return dx, dw, dlam, du


def scan_fwd_norm(x, w_logits, lam, u, direction: int = ALL, y=None, stream=None):
    """As :func:`scan_fwd`, with the weights given by their logits
    (Sec. 3, Eq. (row_stochastic_norm))."""
    import torch
    B, C, G, H, W = _sizes(x, w_logits, lam, u, direction)
    if y is None:
        y = torch.empty_like(x)
    status = gspn_scan_fwd_norm(*_ptrs(x, w_logits, lam, u, y), direction, B, C, G, H, W,
                                _dtype_code(x), _stream_handle(x, stream))
    _check_raise(status)
    return y


def scan_bwd_norm(x, w_logits, lam, u, dy, direction: int = ALL, out=None, stream=None):
    """Gradients (dx, dw_logits, dlam, du) of <y, dy>, the weights given by
    their logits."""
    import torch
    B, C, G, H, W = _sizes(x, w_logits, lam, u, direction)
    if out is None:
        out = (torch.empty_like(x), torch.empty_like(w_logits), torch.empty_like(lam),
               torch.empty_like(u))
    dx, dwl, dlam, du = out
    status = gspn_scan_bwd_norm(*_ptrs(x, w_logits, lam, u, dy, dx, dwl, dlam, du), direction, B,
                                C, G, H, W, _dtype_code(x), _stream_handle(x, stream))
    _check_raise(status)
    return dx, dwl, dlam, du


def project(a, x, y=None, stream=None):
    """1x1 convolution y[b] = a @ x[b]: a [M, K], x [B, K, H, W] -> y [B, M, H, W] (bf16)."""
    import torch
    if a.dim() != 2 or x.dim() != 4 or a.shape[1] != x.shape[1]:
        raise ValueError("a must be [M, K] and x [B, K, H, W]")
    M, K = a.shape
    B, _, H, W = x.shape
    if y is None:
        y = torch.empty((B, M, H, W), dtype=x.dtype, device=x.device)
    status = gspn_project(*_ptrs(a, x, y), B, M, K, H, W, _dtype_code(x),
                          _stream_handle(x, stream))
    _check_raise(status)
    return y


def _latent_weights(l_u, l_lam, l_w, direction):
    D = bin(direction & 15).count("1")
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
    status = gspn_latent_params(*_ptrs(xc, l_u, l_lam, l_w, u, lam, w), direction, B, Cc, H, W,
                                _dtype_code(xc), _stream_handle(xc, stream))
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
    status = gspn_latent_fwd(*_ptrs(x, p_down, l_u, l_lam, l_w, p_up, y), direction, B, C, Cc, H,
                             W, _dtype_code(x), _stream_handle(x, stream))
    _check_raise(status)
    return y


LINE_BLOCK = 8   # lines per block of the line-major layout


def _block_lines(plane):
    """[..., L, P] -> [..., L*P]: lines in blocks of 8, positions adjacent inside a block."""
    import torch
    L, P = plane.shape[-2:]
    lead = plane.shape[:-2]
    if L % LINE_BLOCK == 0:
        blk = plane.reshape(*lead, L // LINE_BLOCK, LINE_BLOCK, P)
        return blk.transpose(-1, -2).contiguous().reshape(*lead, L * P)
    parts = [plane[..., q:q + LINE_BLOCK, :].transpose(-1, -2).reshape(*lead, -1)
             for q in range(0, L, LINE_BLOCK)]
    return torch.cat(parts, dim=-1)


def _unblock_lines(flat, L, P):
    import torch
    lead = flat.shape[:-1]
    if L % LINE_BLOCK == 0:
        blk = flat.reshape(*lead, L // LINE_BLOCK, P, LINE_BLOCK)
        return blk.transpose(-1, -2).contiguous().reshape(*lead, L, P)
    parts, off = [], 0
    for q in range(0, L, LINE_BLOCK):
        n = min(LINE_BLOCK, L - q)
        parts.append(flat[..., off:off + n * P].reshape(*lead, P, n).transpose(-1, -2))
        off += n * P
    return torch.cat(parts, dim=-2)


def to_line_major(t, direction: int):
    """Pixel-major per-direction tensor [D, ..., H, W] -> blocked line-major [D, ..., H*W].

    The lines a direction scans are storage rows (vertical directions) or
    storage columns (horizontal ones).  Each plane stores its lines in blocks
    of 8 consecutive lines; inside a block the values of one line position
    are adjacent: line l, position p sits at 8*P*(l//8) + n*p + l%8 with
    n = min(8, L - 8*(l//8)).  A producer can also write this layout directly.
    """
    import torch
    bits = [b for b in (T2B, B2T, L2R, R2L) if direction & b]
    out = []
    for s, b in enumerate(bits):
        p = t[s] if b in (T2B, B2T) else t[s].transpose(-1, -2)
        out.append(_block_lines(p))
    return torch.stack(out)


def from_line_major(t, direction: int, H: int, W: int):
    """Inverse of :func:`to_line_major`."""
    import torch
    bits = [b for b in (T2B, B2T, L2R, R2L) if direction & b]
    out = []
    for s, b in enumerate(bits):
        if b in (T2B, B2T):
            out.append(_unblock_lines(t[s], H, W))
        else:
            out.append(_unblock_lines(t[s], W, H).transpose(-1, -2))
    return torch.stack(out).contiguous()
