"""Helpers for the GPU parity tests: device upload/download and error metrics."""
import numpy as np

import gspn_inputs as gi


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need an MI355X; run them with -m gpu on a GPU host")
    return torch


def to_device(a: np.ndarray, dtype: str):
    torch = require_gpu()
    if dtype == "bf16":
        bits = gi.to_bf16_bits(a)
        return torch.from_numpy(bits.view(np.int16)).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def to_host(t) -> np.ndarray:
    torch = require_gpu()
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return gi.from_bf16_bits(bits).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def upload(inputs: dict, dtype: str, dirs: int, layout: str = "pixel") -> dict:
    """Device copies of pixel-major inputs; with layout="blocked" the
    per-direction tensors go in the blocked line-major layout."""
    if layout == "blocked":
        inputs = gi.inputs_line_major(inputs, dirs)
    return {k: to_device(v, dtype) for k, v in inputs.items()}


def normwise_err(a: np.ndarray, r: np.ndarray) -> float:
    """max_i |a_i - r_i| / max_i |r_i| (0 when both are all-zero)."""
    den = float(np.abs(r).max()) if r.size else 0.0
    num = float(np.abs(a - r).max()) if r.size else 0.0
    if den == 0.0:
        return num
    return num / den


def elementwise_err(a: np.ndarray, r: np.ndarray) -> float:
    """Diagnostic: max_i |a_i - r_i| / (|r_i| + 1e-3 max|r|)."""
    if r.size == 0:
        return 0.0
    scale = float(np.abs(r).max())
    if scale == 0.0:
        return float(np.abs(a - r).max())
    return float((np.abs(a - r) / (np.abs(r) + 1e-3 * scale)).max())


def report(tag: str, key: str, a: np.ndarray, r: np.ndarray) -> float:
    """Prints the normwise and element-wise errors of one output; returns the
    normwise one."""
    err = normwise_err(a, r)
    print(f"[err] {tag} {key}: normwise {err:.3e} elementwise {elementwise_err(a, r):.3e}",
          flush=True)
    return err


def tolerance(dtype: str) -> float:
    # fp32 storage: 1e-5; bf16 storage with fp32 accumulation: 2e-2
    return 1e-5 if dtype == "f32" else 2e-2


def ignored_taps(mask: int, H: int, W: int) -> np.ndarray:
    """[D, 3, H, W] boolean: taps that leave the grid or sit on the first scanned line."""
    out = []
    for bit in gi.DIR_BITS:
        if not mask & bit:
            continue
        m = np.zeros((3, H, W), dtype=bool)
        rows = np.arange(H)[:, None]
        cols = np.arange(W)[None, :]
        vertical = bit in (gi.T2B, gi.B2T)
        for k in range(3):
            if vertical:
                m[k] = ~((cols + k - 1 >= 0) & (cols + k - 1 < W)) | np.zeros((H, 1), bool)
            else:
                m[k] = ~((rows + k - 1 >= 0) & (rows + k - 1 < H)) | np.zeros((1, W), bool)
        if bit == gi.T2B:
            m[:, 0, :] = True
        elif bit == gi.B2T:
            m[:, H - 1, :] = True
        elif bit == gi.L2R:
            m[:, :, 0] = True
        else:
            m[:, :, W - 1] = True
        out.append(m)
    return np.stack(out)


def ulp_bf16(v: np.ndarray) -> np.ndarray:
    """Spacing of bf16 numbers at |v| (8 significant bits), taken at the
    smallest normal number for |v| below it."""
    a = np.maximum(np.abs(v), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 7)


def check_half_ulp(tag, got, ref, mag, K):
    """Asserts |got - ref| <= 0.5 ulp_bf16(max(|ref|, |got|)) + 2^-24 K mag
    element by element: one rounding to nearest of a value that fp32
    arithmetic got within 2^-24 K mag of the exact ref (mag: the element's
    sum of absolute terms).  Prints the worst ratio to the bound."""
    bound = 0.5 * ulp_bf16(np.maximum(np.abs(ref), np.abs(got))) + 2.0 ** -24 * K * mag
    excess = np.abs(got - ref) / bound
    worst = float(excess.max()) if excess.size else 0.0
    print(f"[err] {tag}: max |got-ref| / bound {worst:.3f} "
          f"(elements over half an ulp of r: "
          f"{float(np.mean(np.abs(got - ref) > 0.5 * ulp_bf16(ref) * (1 + 1e-9))):.2e})",
          flush=True)
    assert worst <= 1.0, f"{tag}: {int((excess > 1).sum())} of {excess.size} elements over bound"
