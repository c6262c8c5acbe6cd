"""Seeded synthetic workloads for the GSPN line scan.

Shared by the tests, the benchmark and the smoke check.  Nothing here computes
any part of the scan: it only describes workload shapes and draws the numbers
(see ``gen.c`` for the counter-based generator).  Both the CPU oracle and the
GPU library read the arrays returned by :func:`make_inputs`.

Direction bits follow the library's convention: 1 = top-to-bottom,
2 = bottom-to-top, 4 = left-to-right, 8 = right-to-left.  Per-direction
tensors are stacked along a leading axis in increasing bit order.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgspn_inputs.so")

T2B, B2T, L2R, R2L = 1, 2, 4, 8
ALL_DIRS = 15
DIR_BITS = (T2B, B2T, L2R, R2L)

# tensor ids of the counter-based streams
_TID_X, _TID_LOGIT, _TID_LAM, _TID_U, _TID_DY, _TID_RAW_LOGIT = 0, 1, 2, 3, 4, 5
_TID_LATENT = 6   # slots: 0 x, 1 P_down, 2 L_u, 3 L_lambda, 4 L_w, 5 P_up


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, storage dtype and value recipe."""
    name: str
    B: int
    C: int
    G: int
    H: int
    W: int
    dtype: str            # "f32" or "bf16" storage; arithmetic is fp32 on the GPU
    dirs: int             # direction bitmask
    backward: bool        # whether the workload includes the backward pass
    gate: str             # "normal": lambda, u ~ N(0,1); "sigmoid": sigmoid(N(0,1))
    logit_sigma: float    # std-dev of the neighbour logits
    seed: int

    @property
    def ndirs(self) -> int:
        return bin(self.dirs).count("1")

    @property
    def pixels_channels(self) -> int:
        return self.B * self.C * self.H * self.W

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


# The five workloads: a tiny fp32 case the oracle checks in full, three ViT /
# hierarchical-encoder stages and one extreme-resolution inference case; then
# the 64x64 stage with one weight group per channel (the paper's original,
# ungrouped recurrence).
WORKLOADS = [
    Workload("tiny-16x16-c8-f32", 1, 8, 1, 16, 16, "f32", T2B, False, "normal", 1.0, 0),
    Workload("vit-s-14x14-b32-c384", 32, 384, 12, 14, 14, "bf16", ALL_DIRS, True, "sigmoid", 1.0, 1),
    Workload("hier-56x56-b64-c96", 64, 96, 8, 56, 56, "bf16", ALL_DIRS, True, "sigmoid", 1.0, 2),
    Workload("hires-64x64-b8-c768", 8, 768, 24, 64, 64, "bf16", ALL_DIRS, True, "sigmoid", 1.0, 3),
    Workload("xres-256x256-b1-c1024", 1, 1024, 32, 256, 256, "bf16", ALL_DIRS, False, "sigmoid", 2.0, 4),
    Workload("hires-64x64-b8-c768-g768", 8, 768, 768, 64, 64, "bf16", ALL_DIRS, True, "sigmoid", 1.0,
             5),
]


def workload(name_or_index) -> Workload:
    if isinstance(name_or_index, int):
        return WORKLOADS[name_or_index]
    for w in WORKLOADS:
        if w.name == name_or_index:
            return w
    raise KeyError(name_or_index)


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(
                f"{_LIB_PATH} is missing; build it with python -m gspn_inputs.build")
        lib = ctypes.CDLL(_LIB_PATH)
        lib.gspn_gen_normal.argtypes = [
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int,
            ctypes.c_int, ctypes.c_double, ctypes.c_double, ctypes.c_int, ctypes.c_int]
        lib.gspn_gen_normal.restype = None
        lib.gspn_gen_taps.argtypes = [
            ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_int, ctypes.c_uint64, ctypes.c_int, ctypes.c_int, ctypes.c_double,
            ctypes.c_int]
        lib.gspn_gen_taps.restype = None
        _lib = lib
    return _lib


def _normal(shape, seed, tid, slot, mean, sigma, transform, bf16):
    out = np.empty(shape, dtype=np.float32)
    _load().gspn_gen_normal(out.ctypes.data, out.size, seed, tid, slot, mean, sigma,
                            transform, int(bf16))
    return out


def make_inputs(wl: Workload, with_dy: bool | None = None) -> dict:
    """Draw every input of ``wl`` as float32 arrays.

    When ``wl.dtype == "bf16"`` every value is already bf16-representable, so
    :func:`to_bf16_bits` is exact.  Returns x [B,C,H,W], w [D,B,G,3,H,W],
    lam and u [D,B,C,H,W] and, for backward workloads, dy [B,C,H,W].
    """
    bf16 = wl.dtype == "bf16"
    B, C, G, H, W = wl.B, wl.C, wl.G, wl.H, wl.W
    D = wl.ndirs
    gate = 1 if wl.gate == "sigmoid" else 0
    x = _normal((B, C, H, W), wl.seed, _TID_X, 0, 0.0, 1.0, 0, bf16)
    w = np.empty((D, B, G, 3, H, W), dtype=np.float32)
    lam = np.empty((D, B, C, H, W), dtype=np.float32)
    u = np.empty((D, B, C, H, W), dtype=np.float32)
    s = 0
    for bit in DIR_BITS:
        if not wl.dirs & bit:
            continue
        vertical = 1 if bit in (T2B, B2T) else 0
        _load().gspn_gen_taps(w[s].ctypes.data, B, G, H, W, vertical, wl.seed,
                              _TID_LOGIT, bit, wl.logit_sigma, int(bf16))
        lam[s] = _normal((B, C, H, W), wl.seed, _TID_LAM, bit, 0.0, 1.0, gate, bf16)
        u[s] = _normal((B, C, H, W), wl.seed, _TID_U, bit, 0.0, 1.0, gate, bf16)
        s += 1
    out = {"x": x, "w": w, "lam": lam, "u": u}
    if with_dy is None:
        with_dy = wl.backward
    if with_dy:
        out["dy"] = _normal((B, C, H, W), wl.seed, _TID_DY, 0, 0.0, 1.0, 0, bf16)
    return out


def make_logits(wl: Workload) -> np.ndarray:
    """Raw tap logits [D,B,G,3,H,W] ~ N(0, logit_sigma^2) for the entry points
    that take the weights as logits (bf16-representable for bf16 workloads).
    Every tap gets a value, including those the operator ignores."""
    bf16 = wl.dtype == "bf16"
    D, B, G, H, W = wl.ndirs, wl.B, wl.G, wl.H, wl.W
    out = np.empty((D, B, G, 3, H, W), dtype=np.float32)
    s = 0
    for bit in DIR_BITS:
        if wl.dirs & bit:
            out[s] = _normal((B, G, 3, H, W), wl.seed, _TID_RAW_LOGIT, bit, 0.0, wl.logit_sigma, 0,
                             bf16)
            s += 1
    return out


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Exact view of bf16-representable float32 values as bf16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    if np.any(bits & 0xFFFF):
        raise ValueError("values are not bf16-representable")
    return (bits >> 16).astype(np.uint16)


def from_bf16_bits(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 values (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), as float32."""
    bits = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    bits = ((bits + 0x7FFF + lsb) & 0xFFFF0000).astype(np.uint32)
    return bits.view(np.float32)


def direction_bits(dirs: int) -> list:
    """Direction bits of a mask in slot order."""
    return [bit for bit in DIR_BITS if dirs & bit]


LINE_BLOCK = 8   # lines per block of the line-major layout


def block_lines(plane: np.ndarray) -> np.ndarray:
    """[..., L, P] (line l, position p) -> blocked line-major [..., L*P].

    Lines are grouped in blocks of 8 consecutive lines (the last block holds
    L mod 8 lines when L is not a multiple of 8); inside a block the values
    of one position are adjacent, so (l, p) sits at
    8*P*(l // 8) + n*p + l % 8 with n = min(8, L - 8*(l // 8)).
    """
    plane = np.asarray(plane)
    L, P = plane.shape[-2:]
    lead = plane.shape[:-2]
    if L % LINE_BLOCK == 0:
        blk = plane.reshape(lead + (L // LINE_BLOCK, LINE_BLOCK, P))
        return np.ascontiguousarray(np.swapaxes(blk, -1, -2)).reshape(lead + (L * P,))
    parts = [np.swapaxes(plane[..., q:q + LINE_BLOCK, :], -1, -2).reshape(lead + (-1,))
             for q in range(0, L, LINE_BLOCK)]
    return np.concatenate(parts, axis=-1)


def unblock_lines(flat: np.ndarray, L: int, P: int) -> np.ndarray:
    """Inverse of :func:`block_lines`: [..., L*P] -> [..., L, P]."""
    flat = np.asarray(flat)
    lead = flat.shape[:-1]
    if L % LINE_BLOCK == 0:
        blk = flat.reshape(lead + (L // LINE_BLOCK, P, LINE_BLOCK))
        return np.ascontiguousarray(np.swapaxes(blk, -1, -2)).reshape(lead + (L, P))
    parts, off = [], 0
    for q in range(0, L, LINE_BLOCK):
        n = min(LINE_BLOCK, L - q)
        parts.append(np.swapaxes(flat[..., off:off + n * P].reshape(lead + (P, n)), -1, -2))
        off += n * P
    return np.concatenate(parts, axis=-2)


def to_line_major(a: np.ndarray, dirs: int) -> np.ndarray:
    """Pixel-major per-direction tensor [D, ..., H, W] -> blocked line-major [D, ..., H*W].

    The lines a direction scans are storage rows for vertical directions and
    storage columns for horizontal ones; each plane is stored as those lines
    in 8-line blocks (:func:`block_lines`).  This is the library's layout for
    lam, u, w and their gradients.
    """
    a = np.asarray(a)
    H, W = a.shape[-2:]
    out = np.empty(a.shape[:-2] + (H * W,), dtype=a.dtype)
    for s, bit in enumerate(direction_bits(dirs)):
        plane = a[s] if bit in (T2B, B2T) else np.swapaxes(a[s], -1, -2)
        out[s] = block_lines(plane)
    return out


def from_line_major(a: np.ndarray, dirs: int, H: int, W: int) -> np.ndarray:
    """Inverse of :func:`to_line_major`: [D, ..., H*W] -> [D, ..., H, W]."""
    a = np.asarray(a)
    out = np.empty(a.shape[:-1] + (H, W), dtype=a.dtype)
    for s, bit in enumerate(direction_bits(dirs)):
        if bit in (T2B, B2T):
            out[s] = unblock_lines(a[s], H, W)
        else:
            out[s] = np.swapaxes(unblock_lines(a[s], W, H), -1, -2)
    return out


PER_DIRECTION = ("lam", "u", "w", "dlam", "du", "dw")


def inputs_line_major(inputs: dict, dirs: int) -> dict:
    """Copy of a pixel-major input dict with the per-direction tensors line-major."""
    return {k: (to_line_major(v, dirs) if k in PER_DIRECTION else v) for k, v in inputs.items()}


@dataclass(frozen=True)
class LatentWorkload:
    """A latent-space propagation sublayer (C-GSPN, Sec. 5): feature map
    [B, C, H, W] projected to Cc latent channels, scanned, projected back."""
    name: str
    B: int
    C: int
    Cc: int
    H: int
    W: int
    dirs: int
    seed: int

    @property
    def ndirs(self) -> int:
        return bin(self.dirs & 15).count("1")

    def with_(self, **kw) -> "LatentWorkload":
        return replace(self, **kw)


# Token grids of a ViT with 14-pixel patches at 518, 1036, 1554, 2058 and
# 2590 pixels (the sublayer latencies of Sec. 6 are quoted at these), width
# 1152 compressed to 64 latent channels, batch 32.
LATENT_WORKLOADS = tuple(
    LatentWorkload(f"cgspn-{n}x{n}-b32-c1152-cc64", 32, 1152, 64, n, n, ALL_DIRS, 21 + i)
    for i, n in enumerate((37, 74, 111, 147, 185)))


def latent_workload(name_or_index) -> LatentWorkload:
    if isinstance(name_or_index, int):
        return LATENT_WORKLOADS[name_or_index]
    for w in LATENT_WORKLOADS:
        if w.name == name_or_index:
            return w
    raise KeyError(name_or_index)


def make_latent_inputs(lw: LatentWorkload) -> dict:
    """bf16-representable float32 inputs of the sublayer: x ~ N(0, 1); every
    projection ~ N(0, 1/fan_in) (P_down: 1/C, the others 1/Cc), so that the
    latent map, u, lambda and the tap logits are of unit scale."""
    B, C, Cc, H, W, D = lw.B, lw.C, lw.Cc, lw.H, lw.W, lw.ndirs
    g = lambda shape, slot, sig: _normal(shape, lw.seed, _TID_LATENT, slot, 0.0, sig, 0, True)
    return {"x": g((B, C, H, W), 0, 1.0),
            "p_down": g((Cc, C), 1, C ** -0.5),
            "l_u": g((D, Cc, Cc), 2, Cc ** -0.5),
            "l_lam": g((D, Cc, Cc), 3, Cc ** -0.5),
            "l_w": g((D, Cc, 3, Cc), 4, Cc ** -0.5),
            "p_up": g((C, Cc), 5, Cc ** -0.5)}
