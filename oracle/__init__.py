"""CPU oracle for the GSPN line scan -- TEST INFRASTRUCTURE ONLY.

Python front end (ctypes + numpy, float64) of ``gspn_oracle.c``.  Only the
tests, the smoke check and the benchmark's CPU-baseline leg use it; the GPU
library never imports it and shares no code with it.

Follows Sec. 3, Eqs. (gspn_recurrence), (gspn_output) and (row_stochastic_norm)
(the scan, and the weights from their logits) and Sec. 4.2, Eq. (2dsp) of the
paper; the readings taken where the paper is
silent are listed in ``gspn_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing; build it with python -m oracle.build")
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.oracle_scan_fwd.argtypes = [P, P, P, P, P, I, I, I, I, I, I]
        lib.oracle_scan_fwd.restype = None
        lib.oracle_scan_bwd.argtypes = [P, P, P, P, P, P, P, P, P, I, I, I, I, I, I]
        lib.oracle_scan_bwd.restype = None
        lib.oracle_norm_w.argtypes = [P, P, I, I, I, I, I]
        lib.oracle_norm_w.restype = None
        lib.oracle_norm_w_bwd.argtypes = [P, P, P, I, I, I, I, I]
        lib.oracle_norm_w_bwd.restype = None
        _lib = lib
    return _lib


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ndirs(dirs):
    return bin(dirs & 15).count("1")


def _check(x, w, lam, u, dirs, G):
    B, C, H, W = x.shape
    D = _ndirs(dirs)
    if not 1 <= dirs <= 15:
        raise ValueError("direction mask must be in [1, 15]")
    if C % G:
        raise ValueError("C must be a multiple of G")
    if w.shape != (D, B, G, 3, H, W):
        raise ValueError(f"w shape {w.shape} != {(D, B, G, 3, H, W)}")
    if lam.shape != (D, B, C, H, W) or u.shape != (D, B, C, H, W):
        raise ValueError("lam/u shape mismatch")
    return B, C, H, W


def scan_fwd(x, w, lam, u, dirs: int) -> np.ndarray:
    """y [B,C,H,W] = sum_d u_d * h_d, in float64."""
    x, w, lam, u = map(_f64, (x, w, lam, u))
    G = w.shape[2]
    B, C, H, W = _check(x, w, lam, u, dirs, G)
    y = np.empty((B, C, H, W), dtype=np.float64)
    _load().oracle_scan_fwd(x.ctypes.data, w.ctypes.data, lam.ctypes.data, u.ctypes.data,
                            y.ctypes.data, dirs, B, C, G, H, W)
    return y


def scan_bwd(x, w, lam, u, dy, dirs: int) -> dict:
    """Gradients {dx, dw, dlam, du} of <y, dy>, in float64."""
    x, w, lam, u, dy = map(_f64, (x, w, lam, u, dy))
    G = w.shape[2]
    B, C, H, W = _check(x, w, lam, u, dirs, G)
    if dy.shape != x.shape:
        raise ValueError("dy shape mismatch")
    dx = np.empty_like(x)
    dw = np.empty_like(w)
    dlam = np.empty_like(lam)
    du = np.empty_like(u)
    _load().oracle_scan_bwd(x.ctypes.data, w.ctypes.data, lam.ctypes.data, u.ctypes.data,
                            dy.ctypes.data, dx.ctypes.data, dw.ctypes.data, dlam.ctypes.data,
                            du.ctypes.data, dirs, B, C, G, H, W)
    return {"dx": dx, "dw": dw, "dlam": dlam, "du": du}


def _check_w(wt, dirs):
    if not 1 <= dirs <= 15:
        raise ValueError("direction mask must be in [1, 15]")
    if wt.ndim != 6 or wt.shape[0] != _ndirs(dirs) or wt.shape[3] != 3:
        raise ValueError(f"weight shape {wt.shape} is not [D, B, G, 3, H, W]")
    return wt.shape[1], wt.shape[2], wt.shape[4], wt.shape[5]


def normalize_w(wt, dirs: int) -> np.ndarray:
    """Row-stochastic tridiagonal weights from their logits (Sec. 3,
    Eq. (row_stochastic_norm)), float64, layout [D, B, G, 3, H, W]."""
    wt = _f64(wt)
    B, G, H, W = _check_w(wt, dirs)
    w = np.empty_like(wt)
    _load().oracle_norm_w(wt.ctypes.data, w.ctypes.data, dirs, B, G, H, W)
    return w


def normalize_w_bwd(wt, dw, dirs: int) -> np.ndarray:
    """Gradient with respect to the logits, given the gradient dw of the
    normalized weights, float64."""
    wt, dw = _f64(wt), _f64(dw)
    B, G, H, W = _check_w(wt, dirs)
    if dw.shape != wt.shape:
        raise ValueError("dw shape mismatch")
    dwt = np.empty_like(wt)
    _load().oracle_norm_w_bwd(wt.ctypes.data, dw.ctypes.data, dwt.ctypes.data, dirs, B, G, H, W)
    return dwt


def slice_group(inputs: dict, b: int, g: int, G: int) -> dict:
    """Inputs of one (batch b, weight group g) unit as a B=1, G=1 problem.

    Every output of that unit depends only on these slices, so the oracle can
    check sampled units of a full-size workload one at a time.
    """
    x = inputs["x"]
    C = x.shape[1]
    cpg = C // G
    cs = slice(g * cpg, (g + 1) * cpg)
    out = {
        "x": x[b:b + 1, cs],
        "w": inputs["w"][:, b:b + 1, g:g + 1],
        "lam": inputs["lam"][:, b:b + 1, cs],
        "u": inputs["u"][:, b:b + 1, cs],
    }
    if "dy" in inputs:
        out["dy"] = inputs["dy"][b:b + 1, cs]
    return out


# ---------------------------------------------------------------------------
# Latent-space propagation sublayer (Sec. 5, Eqs. (latent_down),
# (latent_params), (latent_recurrence), (latent_up)).
#
# Readings: the per-pixel projections are linear maps without bias and u,
# lambda take no activation (the paper names neither); every direction of the
# mask has its own L_u, L_lambda, L_w; w is normalized from its logits as in
# Eq. (row_stochastic_norm); the scan runs with one weight group per latent
# channel.  With ``storage="bf16"`` the stage results that a bf16
# implementation keeps in memory (x_c, u, lambda, w, y_c) are rounded to
# bf16 between the stages and the logits are not; the arithmetic itself is
# float64 throughout.
# ---------------------------------------------------------------------------

def round_bf16(a) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even), as float64."""
    a = _f64(a)
    m, e = np.frexp(a)                       # a = m * 2**e, 0.5 <= |m| < 1
    return np.ldexp(np.round(np.ldexp(m, 8)), e - 8)


def project(a, x) -> np.ndarray:
    """Per-pixel projection (1x1 convolution) y[b] = a @ x[b]: a [M, K],
    x [B, K, H, W] -> [B, M, H, W], float64."""
    a, x = _f64(a), _f64(x)
    B, K, H, W = x.shape
    if a.ndim != 2 or a.shape[1] != K:
        raise ValueError("a must be [M, K] with K = x.shape[1]")
    return np.matmul(a, x.reshape(B, K, H * W)).reshape(B, a.shape[0], H, W)


def latent_params(xc, l_u, l_lam, l_w, dirs: int, storage: str = "f64") -> dict:
    """u, lambda [D, B, Cc, H, W] and normalized w [D, B, Cc, 3, H, W] from the
    latent map xc [B, Cc, H, W] (Eq. (latent_params), then
    Eq. (row_stochastic_norm) on the tap logits)."""
    xc = _f64(xc)
    D = _ndirs(dirs)
    B, Cc, H, W = xc.shape
    l_u, l_lam, l_w = _f64(l_u), _f64(l_lam), _f64(l_w)
    if l_u.shape != (D, Cc, Cc) or l_lam.shape != (D, Cc, Cc) or l_w.shape != (D, Cc, 3, Cc):
        raise ValueError("l_u, l_lam must be [D, Cc, Cc] and l_w [D, Cc, 3, Cc]")
    u = np.stack([project(l_u[s], xc) for s in range(D)])
    lam = np.stack([project(l_lam[s], xc) for s in range(D)])
    wt = np.stack([project(l_w[s].reshape(3 * Cc, Cc), xc).reshape(B, Cc, 3, H, W)
                   for s in range(D)])
    w = normalize_w(wt, dirs)
    if storage == "bf16":
        u, lam, w = round_bf16(u), round_bf16(lam), round_bf16(w)
    return {"u": u, "lam": lam, "w": w, "wt": wt}


def latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, dirs: int, storage: str = "f64") -> np.ndarray:
    """The sublayer y = P_up(Prop_2D(P_down x)), float64 [B, C, H, W]."""
    rnd = round_bf16 if storage == "bf16" else (lambda a: a)
    xc = rnd(project(p_down, x))
    prm = latent_params(xc, l_u, l_lam, l_w, dirs, storage)
    yc = rnd(scan_fwd(xc, prm["w"], prm["lam"], prm["u"], dirs))
    return project(p_up, yc)
