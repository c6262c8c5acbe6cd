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


def _fwd_call(fn):
    def call(**kw):
        a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), y=P(4), direction=15, B=1, C=4, G=2, H=8,
                 W=8, dtype=g.BF16, ws=None, ws_bytes=0, stream=None)
        a.update(kw)
        return fn(a["x"], a["w"], a["lam"], a["u"], a["y"], a["direction"], a["B"], a["C"],
                  a["G"], a["H"], a["W"], a["dtype"], a["ws"], a["ws_bytes"], a["stream"])
    call.fwd = True
    return call


def _bwd_call(fn):
    def call(**kw):
        a = dict(x=P(0), w=P(1), lam=P(2), u=P(3), dy=P(4), dx=P(5), dw=P(6), dlam=P(7),
                 du=P(8), direction=15, B=1, C=4, G=2, H=8, W=8, dtype=g.BF16, ws=None,
                 ws_bytes=0, stream=None)
        a.update(kw)
        return fn(a["x"], a["w"], a["lam"], a["u"], a["dy"], a["dx"], a["dw"], a["dlam"],
                  a["du"], a["direction"], a["B"], a["C"], a["G"], a["H"], a["W"], a["dtype"],
                  a["ws"], a["ws_bytes"], a["stream"])
    call.fwd = False
    return call


fwd = _fwd_call(g.gspn_scan_fwd)
bwd = _bwd_call(g.gspn_scan_bwd)
fwd_blocked = _fwd_call(g.gspn_scan_fwd_blocked)
bwd_blocked = _bwd_call(g.gspn_scan_bwd_blocked)
fwd_norm = _fwd_call(g.gspn_scan_fwd_norm)
bwd_norm = _bwd_call(g.gspn_scan_bwd_norm)


@pytest.mark.parametrize("call", [fwd, bwd, fwd_blocked, bwd_blocked, fwd_norm, bwd_norm],
                         ids=["fwd", "bwd", "fwd_blocked", "bwd_blocked", "fwd_norm", "bwd_norm"])
def test_invalid_arguments(call):
    ptrs = ["x", "w", "lam", "u", "y"] if call.fwd else \
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


def test_workspace_size_query():
    # planes of 8 x 8 run on the LDS-staged kernels: no workspace, no device query
    for op in range(6):
        st, n = g.gspn_workspace_size(op, 15, 1, 4, 2, 8, 8, g.BF16)
        assert st == _native.OK and n == (0 if op not in (g.OP_FWD_NORM, g.OP_BWD_NORM) else n)
    # the _norm passes keep the normalized weights (and their gradient) there:
    # D * B * G * 3 * H * W elements, 256-byte aligned
    st, n = g.gspn_workspace_size(g.OP_FWD_NORM, 15, 1, 4, 2, 8, 8, g.BF16)
    assert st == _native.OK and n == 4 * 2 * 3 * 64 * 2
    st, n = g.gspn_workspace_size(g.OP_BWD_NORM, 15, 1, 4, 2, 8, 8, g.BF16)
    assert st == _native.OK and n == 2 * 4 * 2 * 3 * 64 * 2
    # the general planes (a side above 64) go through fp32 direction slots
    st, n = g.gspn_workspace_size(g.OP_FWD, 5, 1, 3, 1, 70, 100, g.F32)
    assert st == _native.OK and n == 2 * 3 * 70 * 100 * 4
    st, n = g.gspn_workspace_size(g.OP_BWD, 5, 1, 4, 2, 70, 100, g.BF16)
    D, HW = 2, 7000
    assert st == _native.OK and n == (D * 4 * HW + D * 2 * 3 * HW + D * 2 * HW) * 4
    # the same checks as the calls
    assert g.gspn_workspace_size(g.OP_FWD, 0, 1, 4, 2, 8, 8, g.BF16)[0] == _native.ERR_DIRECTION
    assert g.gspn_workspace_size(g.OP_FWD, 15, 1, 6, 4, 8, 8, g.BF16)[0] == _native.ERR_DIM
    for bad in (10, -1):
        assert g.gspn_workspace_size(bad, 15, 1, 4, 2, 8, 8, g.BF16)[0] == _native.ERR_UNSUPPORTED


# one shape per kernel family and storage type (tiny, register-resident small,
# register-streamed med, wide, general; bf16 and fp32)
FAMILY_SHAPES = [(1, 1, "bf16"), (5, 7, "bf16"), (8, 8, "bf16"), (14, 14, "bf16"),
                 (40, 24, "bf16"), (40, 24, "f32"), (64, 64, "bf16"), (56, 56, "bf16"),
                 (72, 136, "bf16"), (256, 256, "bf16"), (70, 100, "bf16"), (3, 130, "f32")]


@pytest.mark.parametrize("H,W,dt", FAMILY_SHAPES)
def test_workspace_query_launches_nothing(H, W, dt):
    """The size query runs the call's own dispatch in counting mode; a kernel
    launched there would fail on this GPU-less host (and, on a GPU, run on
    null pointers).  Every family, both layouts, every operation and a
    single-group, a grouped and a per-channel-weight case must come back OK."""
    dtype = g.BF16 if dt == "bf16" else g.F32
    for C, G in ((4, 1), (64, 2), (8, 8)):
        for op in range(10):
            for dirs in (15, 1, 6):
                st, n = g.gspn_workspace_size(op, dirs, 2, C, G, H, W, dtype)
                assert st == _native.OK and n >= 0, (H, W, dt, C, G, op, dirs, st)
    st, n = g.gspn_latent_workspace_size(15, 1, 32, 16, H, W, g.BF16)
    assert st in (_native.OK, _native.ERR_UNSUPPORTED), (H, W, st)


def test_workspace_checked_before_any_launch():
    # a shape that needs workspace (general planes): missing, too small,
    # misaligned or overlapping workspace is rejected on the host
    kw = dict(direction=5, B=1, C=4, G=2, H=70, W=100)
    st, need = g.gspn_workspace_size(g.OP_BWD, 5, 1, 4, 2, 70, 100, g.BF16)
    assert st == _native.OK and need > 0
    far = lambda i: BASE + (1 << 32) + i * (1 << 26)     # noqa: E731  (room for big buffers)
    big = dict(x=far(0), w=far(1), lam=far(2), u=far(3), dy=far(4), dx=far(5), dw=far(6),
               dlam=far(7), du=far(8))
    assert bwd(**kw, **big) == _native.ERR_WORKSPACE
    assert bwd(**kw, **big, ws=far(9), ws_bytes=need - 1) == _native.ERR_WORKSPACE
    assert bwd(**kw, **big, ws=far(9), ws_bytes=-1) == _native.ERR_WORKSPACE
    assert bwd(**kw, **big, ws=far(9) + 8, ws_bytes=need) == _native.ERR_ALIGN
    assert bwd(**kw, **big, ws=far(0), ws_bytes=need) == _native.ERR_ALIAS
    assert bwd(**kw, **big, ws=far(5), ws_bytes=need) == _native.ERR_ALIAS


def test_static_backward_checks_and_limit():
    """gspn_scan_bwd_static takes the checks of gspn_scan_bwd and refuses, on
    the host and before any device call, a problem whose workspace exceeds its
    fixed array."""
    call = lambda **kw: _bwd_call(lambda *a: g.gspn_scan_bwd_static(*a[:16], a[18]))(**kw)  # noqa
    for name in ("x", "w", "lam", "u", "dy", "dx", "dw", "dlam", "du"):
        assert call(**{name: None}) == _native.ERR_NULL, name
    assert call(direction=0) == _native.ERR_DIRECTION
    assert call(C=6, G=4) == _native.ERR_DIM
    assert call(dx=P(4)) == _native.ERR_ALIAS
    kw = dict(direction=15, B=16, C=64, G=2, H=70, W=100)
    st, need = g.gspn_workspace_size(g.OP_BWD, 15, 16, 64, 2, 70, 100, g.BF16)
    assert st == _native.OK and need > _native.STATIC_SCRATCH_BYTES
    far = lambda i: BASE + (1 << 36) + i * (1 << 32)     # noqa: E731
    big = dict(x=far(0), w=far(1), lam=far(2), u=far(3), dy=far(4), dx=far(5), dw=far(6),
               dlam=far(7), du=far(8))
    assert call(**kw, **big) == _native.ERR_WORKSPACE


def test_front_end_rejects_mismatched_tensors():
    import torch
    x = torch.zeros(1, 4, 8, 8, dtype=torch.bfloat16)
    lam = torch.zeros(4, 1, 4, 8, 8, dtype=torch.bfloat16)
    w = torch.zeros(4, 1, 2, 3, 8, 8, dtype=torch.bfloat16)
    dy = torch.zeros_like(x)
    with pytest.raises(ValueError, match="lam must hold"):
        g.scan_fwd(x, w, lam[:2], lam, 15)
    with pytest.raises(ValueError, match="w must hold"):
        g.scan_fwd(x, torch.zeros(4, 1, 2, 3, 8, 4, dtype=torch.bfloat16), lam, lam, 15)
    with pytest.raises(ValueError, match="dtype"):
        g.scan_fwd(x, w, lam.float(), lam, 15)
    with pytest.raises(ValueError, match="y must hold"):
        g.scan_fwd(x, w, lam, lam, 15, y=x[:, :2])
    with pytest.raises(ValueError, match="dy must hold"):
        g.scan_bwd(x, w, lam, lam, dy[:, :2], 15)
    with pytest.raises(ValueError, match="du must hold"):
        g.scan_bwd(x, w, lam, lam, dy, 15, out=(x, w, lam, lam[:3]))
    with pytest.raises(ValueError, match="contiguous"):
        g.scan_fwd(x, w, lam, lam.transpose(-1, -2), 15)
    with pytest.raises(ValueError, match="GPU"):
        g.scan_fwd(x, w, lam, lam, 15)


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
             direction=15, B=1, C=32, Cc=16, H=8, W=8, dtype=g.BF16, ws=P(7), ws_bytes=1 << 20,
             stream=None)
    a.update(kw)
    return g.gspn_latent_fwd(a["x"], a["p_down"], a["l_u"], a["l_lam"], a["l_w"], a["p_up"],
                             a["y"], a["direction"], a["B"], a["C"], a["Cc"], a["H"], a["W"],
                             a["dtype"], a["ws"], a["ws_bytes"], a["stream"])


def test_latent_workspace():
    st, n = g.gspn_latent_workspace_size(15, 1, 32, 16, 8, 8, g.BF16)
    # x_c, u, lambda, w (3 taps) and y_c: (2 + 5 D) latent maps of bf16
    assert st == _native.OK and n == (2 + 5 * 4) * 16 * 64 * 2
    assert latent_fwd(ws=None) == _native.ERR_WORKSPACE
    assert latent_fwd(ws_bytes=n - 2) == _native.ERR_WORKSPACE
    assert latent_fwd(ws=P(0)) == _native.ERR_ALIAS


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


def test_slot_plan_workspace():
    """The forced 4-slot plan of the register-streamed backward takes 4 channels
    per workgroup: a 32-channel group of 64 x 64 planes needs 8 fp32 partials
    of dw instead of the 4 that 8-slot workgroups (8 channels, as many as fit
    in LDS) need."""
    args = (15, 1, 64, 2, 64, 64, g.BF16)
    st8, n8 = g.gspn_workspace_size_slots(8, *args)
    st4, n4 = g.gspn_workspace_size_slots(4, *args)
    st0, n0 = g.gspn_workspace_size_slots(0, *args)
    assert st8 == st4 == st0 == _native.OK
    assert n0 == g.gspn_workspace_size(g.OP_BWD, *args)[1]
    ndw = 4 * 1 * 2 * 3 * 64 * 64                      # D B G 3 H W
    assert n4 - n8 == (8 - 4) * ndw * 4
    # per-channel weights (one channel per group) take no plan: same need
    args1 = (15, 1, 16, 16, 64, 64, g.BF16)
    assert g.gspn_workspace_size_slots(4, *args1) == g.gspn_workspace_size_slots(8, *args1)
    for bad in (1, 2, 16, -4):
        assert g.gspn_workspace_size_slots(bad, *args)[0] == _native.ERR_UNSUPPORTED
        assert g.gspn_scan_bwd_slots(bad, *[P(i) for i in range(9)], *args, None, 0,
                                     None) == _native.ERR_UNSUPPORTED
    assert g.gspn_scan_bwd_slots(4, *[P(i) for i in range(8)], None, *args, None, 0,
                                 None) == _native.ERR_NULL


def test_training_pair_reserve():
    """gspn_reserve_size: the blocked weights (horizontal directions only
    with one channel per group) plus lambda and u of the horizontal
    directions, 256-byte aligned, on the register-streamed shapes; 0
    elsewhere.  The reserve is checked on the host like a workspace."""
    def size(dirs, B, C, G, H, W, dt=g.BF16):
        st, n = g.gspn_reserve_size(dirs, B, C, G, H, W, dt)
        assert st == _native.OK
        return n
    HW = 64 * 64
    assert size(15, 1, 64, 2, 64, 64) == 4 * 2 * 3 * HW * 2 + 2 * (2 * 64 * HW * 2)
    assert size(15, 1, 16, 16, 64, 64) == 2 * 16 * 3 * HW * 2 + 2 * (2 * 16 * HW * 2)
    assert size(3, 1, 64, 2, 64, 64) == 2 * 2 * 3 * HW * 2            # vertical only
    assert size(3, 1, 16, 16, 64, 64) == 0                             # read in place
    for shape in ((14, 14), (8, 8), (70, 100), (256, 256), (64, 48)):
        assert size(15, 2, 8, 2, *shape) == 0, shape
    assert size(15, 1, 64, 2, 64, 64, g.F32) == 0
    assert g.gspn_reserve_size(0, 1, 4, 2, 64, 64, g.BF16)[0] == _native.ERR_DIRECTION
    assert g.gspn_reserve_size(15, 1, 6, 4, 64, 64, g.BF16)[0] == _native.ERR_DIM
    # the training pair's own workspace: none for the forward (its copies go
    # to the reserve), the partials only for the backward
    args = (15, 1, 64, 2, 64, 64, g.BF16)
    assert g.gspn_workspace_size(g.OP_FWD_TRAIN, *args) == (_native.OK, 0)
    st, nb = g.gspn_workspace_size(g.OP_BWD_RESERVE, *args)
    st0, nb0 = g.gspn_workspace_size(g.OP_BWD, *args)
    assert st == st0 == _native.OK and nb0 - nb == size(*args)
    # checks: a missing, small, misaligned or overlapping reserve is refused
    need = size(*args)
    far = lambda i: BASE + (1 << 33) + i * (1 << 26)     # noqa: E731
    fwd_ptrs = [far(i) for i in range(5)]
    bwd_ptrs = [far(i) for i in range(9)]
    def fwd(rs, n):
        return g.gspn_scan_fwd_train(*fwd_ptrs, *args, rs, n, None, 0, None)
    def bwd(rs, n, ws=None, nws=0):
        return g.gspn_scan_bwd_reserve(*bwd_ptrs, *args, rs, n, ws, nws, None)
    assert fwd(None, 0) == _native.ERR_WORKSPACE
    assert fwd(far(10), need - 1) == _native.ERR_WORKSPACE
    assert fwd(far(10), -1) == _native.ERR_WORKSPACE
    assert fwd(far(10) + 8, need) == _native.ERR_ALIGN
    assert fwd(far(0), need) == _native.ERR_ALIAS          # over an input
    assert fwd(far(4), need) == _native.ERR_ALIAS          # over the output
    assert bwd(None, 0, far(11), nb) == _native.ERR_WORKSPACE
    assert bwd(far(10), need, None, 0) == _native.ERR_WORKSPACE
    assert bwd(far(5), need, far(11), nb) == _native.ERR_ALIAS     # over an output
    assert bwd(far(10), need, far(10), nb) == _native.ERR_ALIAS    # over the workspace
    assert g.gspn_scan_fwd_train(None, *fwd_ptrs[1:], *args, far(10), need, None, 0,
                                 None) == _native.ERR_NULL


def test_norm_training_pair_reserve():
    """The _norm pair keeps the weights it forms for every direction (also
    with one channel per group, where the plain pair copies only the
    horizontal ones) plus the horizontal lambda and u; its forward takes no
    workspace, its backward only the weight gradient and the partials."""
    def size(dirs, B, C, G, H, W):
        st, n = g.gspn_reserve_size_norm(dirs, B, C, G, H, W, g.BF16)
        assert st == _native.OK
        return n
    HW = 64 * 64
    assert size(15, 1, 64, 2, 64, 64) == g.gspn_reserve_size(15, 1, 64, 2, 64, 64, g.BF16)[1]
    assert size(15, 1, 16, 16, 64, 64) == 4 * 16 * 3 * HW * 2 + 2 * (2 * 16 * HW * 2)
    assert size(3, 1, 16, 16, 64, 64) == 2 * 16 * 3 * HW * 2
    assert size(15, 2, 8, 2, 14, 14) == 0
    args = (15, 1, 64, 2, 64, 64, g.BF16)
    assert g.gspn_workspace_size(g.OP_FWD_NORM_TRAIN, *args) == (_native.OK, 0)
    st, nb = g.gspn_workspace_size(g.OP_BWD_NORM_RESERVE, *args)
    st0, nb0 = g.gspn_workspace_size(g.OP_BWD_NORM, *args)
    assert st == st0 == _native.OK and nb0 - nb == size(*args[:6])
    far = lambda i: BASE + (1 << 34) + i * (1 << 26)     # noqa: E731
    need = size(*args[:6])
    assert g.gspn_scan_fwd_norm_train(*[far(i) for i in range(5)], *args, None, 0, None, 0,
                                      None) == _native.ERR_WORKSPACE
    assert g.gspn_scan_bwd_norm_reserve(*[far(i) for i in range(9)], *args, far(10), need - 1,
                                        far(11), nb, None) == _native.ERR_WORKSPACE
    assert g.gspn_scan_bwd_norm_reserve(*[far(i) for i in range(9)], *args, far(6), need,
                                        far(11), nb, None) == _native.ERR_ALIAS
