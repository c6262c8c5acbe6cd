"""The C ABI: the library loads, exports what include/gspn.h declares, and
rejects every invalid argument on the host, before any HIP call (so these
tests run without a GPU)."""
import os
import re

import pytest

import paper_2606_00746_amd as g
from paper_2606_00746_amd import _native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "gspn.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(gspn_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    lib = g.load()
    names = header_functions()
    assert set(names) == set(_native.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n
    assert g.gspn_version() >= 100


def test_header_constants_match_binding():
    text = open(os.path.join(ROOT, "include", "gspn.h")).read()
    consts = dict(re.findall(r"#define (GSPN_\w+) \(?(-?\d+)\)?\s", text))
    assert int(consts["GSPN_T2B"]) == g.T2B and int(consts["GSPN_R2L"]) == g.R2L
    assert int(consts["GSPN_BF16"]) == g.BF16
    assert int(consts["GSPN_ERR_HIP"]) == _native.ERR_HIP
    assert int(consts["GSPN_ERR_UNSUPPORTED"]) == _native.ERR_UNSUPPORTED
    assert int(consts["GSPN_MAX_SIDE"]) == _native.MAX_SIDE


def test_strerror_is_total():
    for s in range(-10, 2):
        assert isinstance(g.gspn_strerror(s), str) and g.gspn_strerror(s)


# Fake, never dereferenced device addresses: 1 MiB apart, 16-byte aligned.
BASE = 0x7F0000000000
def P(i, off=0):
    return BASE + i * (1 << 20) + off


def fwd(**kw):
    a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), y=P(4), direction=15, B=1, C=4, G=2, H=8, W=8,
             dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_scan_fwd(a["x"], a["w"], a["lam"], a["u"], a["y"], a["direction"], a["B"],
                           a["C"], a["G"], a["H"], a["W"], a["dtype"], a["stream"])


def bwd(**kw):
    a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), dy=P(4), dx=P(5), dw=P(6), dlam=P(7), du=P(8),
             direction=15, B=1, C=4, G=2, H=8, W=8, dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_scan_bwd(a["x"], a["w"], a["lam"], a["u"], a["dy"], a["dx"], a["dw"], a["dlam"],
                           a["du"], a["direction"], a["B"], a["C"], a["G"], a["H"], a["W"],
                           a["dtype"], a["stream"])


def fwd_norm(**kw):
    a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), y=P(4), direction=15, B=1, C=4, G=2, H=8, W=8,
             dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_scan_fwd_norm(a["x"], a["w"], a["lam"], a["u"], a["y"], a["direction"], a["B"],
                                a["C"], a["G"], a["H"], a["W"], a["dtype"], a["stream"])


def bwd_norm(**kw):
    a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), dy=P(4), dx=P(5), dw=P(6), dlam=P(7), du=P(8),
             direction=15, B=1, C=4, G=2, H=8, W=8, dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_scan_bwd_norm(a["x"], a["w"], a["lam"], a["u"], a["dy"], a["dx"], a["dw"],
                                a["dlam"], a["du"], a["direction"], a["B"], a["C"], a["G"],
                                a["H"], a["W"], a["dtype"], a["stream"])


@pytest.mark.parametrize("call", [fwd, bwd, fwd_norm, bwd_norm])
def test_invalid_arguments(call):
    ptrs = ["x", "w", "lam", "u", "y"] if call in (fwd, fwd_norm) else \
        ["x", "w", "lam", "u", "dy", "dx", "dw", "dlam", "du"]
    for name in ptrs:
        assert call(**{name: None}) == _native.ERR_NULL, name
        assert call(**{name: P(ptrs.index(name), 8)}) == _native.ERR_ALIGN, name
    for bad in (0, 16, -1, 31):
        assert call(direction=bad) == _native.ERR_DIRECTION
    for bad in (2, -1, 7):
        assert call(dtype=bad) == _native.ERR_DTYPE
    for dim in ("B", "C", "G", "H", "W"):
        assert call(**{dim: 0}) == _native.ERR_DIM, dim
        assert call(**{dim: -3}) == _native.ERR_DIM, dim
    assert call(C=6, G=4) == _native.ERR_DIM
    assert call(H=4097) == _native.ERR_UNSUPPORTED
    assert call(W=5000) == _native.ERR_UNSUPPORTED
    assert call(B=1 << 20, C=1 << 10, G=1, H=4096, W=4096) == _native.ERR_UNSUPPORTED


def test_overlapping_buffers_rejected():
    # output equal to an input
    assert fwd(y=P(0)) == _native.ERR_ALIAS
    # output range overlapping an input range (x spans 1*4*8*8*2 = 512 bytes)
    assert fwd(y=P(0, 256)) == _native.ERR_ALIAS
    # two outputs overlapping each other
    assert bwd(dlam=P(8)) == _native.ERR_ALIAS
    assert bwd(dx=P(4)) == _native.ERR_ALIAS


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_native, "_lib", None)
    monkeypatch.setattr(_native, "LIB_PATH", str(tmp_path / "libgspn.so"))
    with pytest.raises(RuntimeError, match="missing"):
        _native.load()


@pytest.mark.parametrize("H,W", [(5, 6), (16, 24), (13, 20)])
def test_torch_layout_helpers_match_numpy(H, W):
    import numpy as np
    import torch
    import gspn_inputs as gi
    a = np.random.default_rng(0).standard_normal((4, 2, 4, H, W)).astype(np.float32)
    for dirs in (15, 7, 12, 1):
        d = bin(dirs).count("1")
        t = torch.from_numpy(a[:d].copy())
        lm = g.to_line_major(t, dirs)
        np.testing.assert_array_equal(lm.numpy(), gi.to_line_major(a[:d], dirs))
        np.testing.assert_array_equal(g.from_line_major(lm, dirs, H, W).numpy(), a[:d])


def project(**kw):
    a = dict(a=P(0), x=P(1), y=P(2), B=1, M=64, K=64, H=8, W=8, dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_project(a["a"], a["x"], a["y"], a["B"], a["M"], a["K"], a["H"], a["W"],
                          a["dtype"], a["stream"])


def latent_params(**kw):
    a = dict(xc=P(0), l_u=P(1), l_lam=P(2), l_w=P(3), u=P(4), lam=P(5), w=P(6), direction=15,
             B=1, Cc=16, H=8, W=8, dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_latent_params(a["xc"], a["l_u"], a["l_lam"], a["l_w"], a["u"], a["lam"],
                                a["w"], a["direction"], a["B"], a["Cc"], a["H"], a["W"],
                                a["dtype"], a["stream"])


def latent_fwd(**kw):
    a = dict(x=P(0), p_down=P(1), l_u=P(2), l_lam=P(3), l_w=P(4), p_up=P(5), y=P(6),
             direction=15, B=1, C=32, Cc=16, H=8, W=8, dtype=g.BF16, stream=None)
    a.update(kw)
    return g.gspn_latent_fwd(a["x"], a["p_down"], a["l_u"], a["l_lam"], a["l_w"], a["p_up"],
                             a["y"], a["direction"], a["B"], a["C"], a["Cc"], a["H"], a["W"],
                             a["dtype"], a["stream"])


@pytest.mark.parametrize("call,ptrs,dims", [
    (project, ["a", "x", "y"], ["B", "M", "K", "H", "W"]),
    (latent_params, ["xc", "l_u", "l_lam", "l_w", "u", "lam", "w"], ["B", "Cc", "H", "W"]),
    (latent_fwd, ["x", "p_down", "l_u", "l_lam", "l_w", "p_up", "y"], ["B", "C", "Cc", "H", "W"]),
])
def test_latent_invalid_arguments(call, ptrs, dims):
    for name in ptrs:
        assert call(**{name: None}) == _native.ERR_NULL, name
        assert call(**{name: P(ptrs.index(name), 8)}) == _native.ERR_ALIGN, name
    for dim in dims:
        assert call(**{dim: 0}) == _native.ERR_DIM, dim
    assert call(dtype=7) == _native.ERR_DTYPE
    assert call(dtype=g.F32) == _native.ERR_UNSUPPORTED     # bf16 only
    assert call(H=4097) == _native.ERR_UNSUPPORTED
    if call is not project:
        for bad in (0, 16):
            assert call(direction=bad) == _native.ERR_DIRECTION
        assert call(Cc=12) == _native.ERR_UNSUPPORTED       # latent channels: multiple of 8
    else:
        assert call(K=12) == _native.ERR_UNSUPPORTED        # K: multiple of 8
    if call is latent_fwd:
        assert call(C=36) == _native.ERR_UNSUPPORTED
    # an output over an input
    assert call(**{ptrs[-1]: P(0)}) == _native.ERR_ALIAS
