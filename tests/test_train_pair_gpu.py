"""The training pair (gspn_scan_fwd_train, gspn_scan_bwd_reserve) against the
plain pair (gspn_scan_fwd, gspn_scan_bwd): the same results bit for bit, the
backward reading the forward's blocked copies from the reserve only (its own
workspace is fresh and filled with 0xFF bytes, NaN as bf16 or fp32, so that
nothing the forward left there can be used).  Register-streamed shapes with
grouped and per-channel weights and every kind of direction subset, shapes
that need no reserve, the full-size 64x64 workloads, a reserve reused for
other inputs, and one case against the oracle directly."""
import pytest

import gspn_inputs as gi
import oracle
import paper_2606_00746_amd as gspn
from gpu_util import report, require_gpu, to_host, tolerance, upload

pytestmark = pytest.mark.gpu


def case(name, B, C, G, H, W, dirs=15, dtype="bf16", seed=11):
    return gi.Workload(name, B, C, G, H, W, dtype, dirs, True, "sigmoid", 1.0, seed)


CASES = [
    case("64-grouped", 1, 64, 2, 64, 64),
    case("64-G=C", 1, 16, 16, 64, 64),
    case("56-grouped", 2, 24, 2, 56, 56),
    case("24-grouped", 2, 16, 4, 24, 24),
    case("40-vertical-only", 1, 16, 2, 40, 40, dirs=3),
    case("48-horizontal-only", 1, 16, 2, 48, 48, dirs=12),
    case("32-T2B+L2R", 1, 16, 4, 32, 32, dirs=5),
    case("64-G=C-R2L", 1, 8, 8, 64, 64, dirs=8),
    case("56-G=C-B2T+R2L", 1, 8, 8, 56, 56, dirs=10),
    case("48-G=C-vertical-only", 1, 8, 8, 48, 48, dirs=3),   # nothing to keep: reserve 0
]
NO_RESERVE = [
    case("14x14", 2, 24, 3, 14, 14),
    case("70x100", 1, 4, 2, 70, 100, dirs=5),
    case("64x64-f32", 1, 4, 2, 64, 64, dtype="f32"),
]


def expected_reserve(wl):
    """Bytes of the reserve: the blocked weights (all directions; with one
    channel per group the horizontal directions' only), then lambda and u of
    the horizontal directions, each 256-byte aligned."""
    HW = wl.H * wl.W
    nv = bin(wl.dirs & 3).count("1")
    nh = bin(wl.dirs & 12).count("1")
    nw = (nh if wl.C == wl.G else nv + nh) * wl.B * wl.G * 3 * HW * 2
    parts = [nw] + ([nh * wl.B * wl.C * HW * 2] * 2 if nh else [])
    total = 0
    for p in parts:
        if p:
            total = (total + 255) // 256 * 256 + p
    return total


def same_bits(a, b):
    import torch
    dt = torch.int32 if a.element_size() == 4 else torch.int16
    return torch.equal(a.contiguous().view(dt), b.contiguous().view(dt))


def run_pairs(t, wl, torch, reserve=None):
    y0 = gspn.scan_fwd(t["x"], t["w"], t["lam"], t["u"], wl.dirs)
    g0 = gspn.scan_bwd(t["x"], t["w"], t["lam"], t["u"], t["dy"], wl.dirs)
    y1, rs = gspn.scan_fwd_train(t["x"], t["w"], t["lam"], t["u"], wl.dirs, reserve=reserve)
    n = gspn.workspace_size(gspn.OP_BWD_RESERVE, t["x"], t["w"], wl.dirs)
    ws = torch.full((max(n, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    g1 = gspn.scan_bwd_reserve(t["x"], t["w"], t["lam"], t["u"], t["dy"], rs, wl.dirs,
                               workspace=ws)
    torch.cuda.synchronize()
    return (y0, *g0), (y1, *g1), rs


def check_same(wl, plain, train):
    for name, a, b in zip(("y", "dx", "dw", "dlam", "du"), plain, train):
        assert same_bits(a, b), f"{wl.name}: {name} differs from the plain pair"


@pytest.mark.parametrize("wl", CASES + NO_RESERVE, ids=lambda w: w.name)
def test_pair_matches_plain(wl):
    torch = require_gpu()
    print(f"[case] train pair {wl.name} B={wl.B} C={wl.C} G={wl.G} {wl.H}x{wl.W} "
          f"dirs={wl.dirs} {wl.dtype}", flush=True)
    inputs = gi.make_inputs(wl, with_dy=True)
    t = upload(inputs, wl.dtype, wl.dirs)
    n = gspn.reserve_size(t["x"], t["w"], wl.dirs)
    want = expected_reserve(wl) if wl in CASES else 0
    assert n == want, (wl.name, n, want)
    plain, train, rs = run_pairs(t, wl, torch)
    assert (rs is None) == (n == 0)
    check_same(wl, plain, train)


def test_reserve_reused_for_other_inputs():
    """A reserve written for one set of inputs and then for another serves
    the second backward exactly (nothing of the first stays in use)."""
    torch = require_gpu()
    wl = CASES[0]
    print(f"[case] train pair reuse {wl.name}", flush=True)
    t1 = upload(gi.make_inputs(wl, with_dy=True), wl.dtype, wl.dirs)
    _, _, rs = run_pairs(t1, wl, torch)
    wl2 = wl.with_(seed=wl.seed + 1)
    t2 = upload(gi.make_inputs(wl2, with_dy=True), wl2.dtype, wl2.dirs)
    plain, train, rs2 = run_pairs(t2, wl2, torch, reserve=rs)
    assert rs2.data_ptr() == rs.data_ptr()
    check_same(wl2, plain, train)


def test_pair_against_oracle():
    torch = require_gpu()
    wl = CASES[1].with_(name="64-G=C-oracle", C=4, G=4)
    print(f"[case] train pair oracle {wl.name}", flush=True)
    inputs = gi.make_inputs(wl, with_dy=True)
    t = upload(inputs, wl.dtype, wl.dirs)
    y, rs = gspn.scan_fwd_train(t["x"], t["w"], t["lam"], t["u"], wl.dirs)
    g = gspn.scan_bwd_reserve(t["x"], t["w"], t["lam"], t["u"], t["dy"], rs, wl.dirs)
    torch.cuda.synchronize()
    tol = tolerance(wl.dtype)
    ref_y = oracle.scan_fwd(inputs["x"], inputs["w"], inputs["lam"], inputs["u"], wl.dirs)
    assert report(wl.name, "y", to_host(y), ref_y) <= tol
    ref = oracle.scan_bwd(inputs["x"], inputs["w"], inputs["lam"], inputs["u"], inputs["dy"],
                          wl.dirs)
    for k, v in zip(("dx", "dw", "dlam", "du"), g):
        assert report(wl.name, k, to_host(v), ref[k]) <= tol, k


@pytest.mark.parametrize("idx", [3, 5], ids=["hires-64x64-b8-c768", "g768"])
def test_pair_full_size(idx):
    """The benchmark's 64 x 64 workloads at full size, in the launch
    configuration the benchmark times: bit for bit the plain pair."""
    torch = require_gpu()
    wl = gi.workload(idx)
    print(f"[case] train pair full size {wl.name}", flush=True)
    t = upload(gi.make_inputs(wl, with_dy=True), wl.dtype, wl.dirs)
    plain, train, rs = run_pairs(t, wl, torch)
    assert rs.numel() == expected_reserve(wl)
    check_same(wl, plain, train)
    del plain, train, rs, t
    torch.cuda.empty_cache()


def test_front_end_checks_the_reserve():
    """A reserve on another device, of another dtype or not contiguous is
    refused by the binding before any call; a short one by the library."""
    torch = require_gpu()
    wl = CASES[0].with_(C=4, G=2)
    print(f"[case] train pair reserve checks {wl.name}", flush=True)
    t = upload(gi.make_inputs(wl, with_dy=True), wl.dtype, wl.dirs)
    y, rs = gspn.scan_fwd_train(t["x"], t["w"], t["lam"], t["u"], wl.dirs)
    args = (t["x"], t["w"], t["lam"], t["u"], t["dy"])
    for bad in (rs.cpu(), rs.view(torch.int8), rs.view(-1, 2)[:, 0]):
        with pytest.raises(ValueError, match="reserve"):
            gspn.scan_bwd_reserve(*args, bad, wl.dirs)
    with pytest.raises(gspn.GspnError, match="workspace"):
        gspn.scan_bwd_reserve(*args, rs[: rs.numel() - 1], wl.dirs)
    with pytest.raises(gspn.GspnError, match="workspace"):
        gspn.scan_bwd_reserve(*args, None, wl.dirs)
    # a caller's reserve that is too small is refused, not replaced
    with pytest.raises(ValueError, match="reserve"):
        gspn.scan_fwd_train(t["x"], t["w"], t["lam"], t["u"], wl.dirs, reserve=rs[:-1])
    torch.cuda.synchronize()


NORM_CASES = [CASES[0], CASES[1], CASES[2], CASES[4], CASES[7],
              case("24-G=C-dirs5", 2, 5, 5, 24, 24, dirs=5), NO_RESERVE[0]]


def run_norm_pairs(t, wt, wl, torch):
    y0 = gspn.scan_fwd_norm(t["x"], wt, t["lam"], t["u"], wl.dirs)
    g0 = gspn.scan_bwd_norm(t["x"], wt, t["lam"], t["u"], t["dy"], wl.dirs)
    y1, rs = gspn.scan_fwd_norm_train(t["x"], wt, t["lam"], t["u"], wl.dirs)
    n = gspn.workspace_size(gspn.OP_BWD_NORM_RESERVE, t["x"], wt, wl.dirs)
    ws = torch.full((max(n, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    g1 = gspn.scan_bwd_norm_reserve(t["x"], wt, t["lam"], t["u"], t["dy"], rs, wl.dirs,
                                    workspace=ws)
    torch.cuda.synchronize()
    return (y0, *g0), (y1, *g1), rs


@pytest.mark.parametrize("wl", NORM_CASES, ids=lambda w: w.name)
def test_norm_pair_matches_plain(wl):
    """The _norm training pair (weights given as logits, the formed weights
    kept in the reserve) against gspn_scan_fwd_norm / gspn_scan_bwd_norm, bit
    for bit, including the logits' gradient."""
    torch = require_gpu()
    print(f"[case] norm train pair {wl.name} B={wl.B} C={wl.C} G={wl.G} {wl.H}x{wl.W} "
          f"dirs={wl.dirs}", flush=True)
    t = upload(gi.make_inputs(wl, with_dy=True), wl.dtype, wl.dirs)
    wt = upload({"w": gi.make_logits(wl)}, wl.dtype, wl.dirs)["w"]
    plain, train, rs = run_norm_pairs(t, wt, wl, torch)
    n = gspn.reserve_size(t["x"], wt, wl.dirs, norm=True)
    assert (rs is None) == (n == 0)
    check_same(wl, plain, train)


@pytest.mark.parametrize("idx", [3, 5], ids=["hires-64x64-b8-c768", "g768"])
def test_norm_pair_full_size(idx):
    torch = require_gpu()
    wl = gi.workload(idx)
    print(f"[case] norm train pair full size {wl.name}", flush=True)
    t = upload(gi.make_inputs(wl, with_dy=True), wl.dtype, wl.dirs)
    wt = upload({"w": gi.make_logits(wl)}, wl.dtype, wl.dirs)["w"]
    plain, train, rs = run_norm_pairs(t, wt, wl, torch)
    check_same(wl, plain, train)
    del plain, train, rs, t, wt
    torch.cuda.empty_cache()
