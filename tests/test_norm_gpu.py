"""GPU parity of the entry points that take the weights as logits
(Sec. 3, Eq. (row_stochastic_norm)) against the fp64 oracle: the oracle
normalizes the same logits, runs the scan, and takes the logits' gradient
from the gradient of the normalized weights.

The library stores the normalized weights, and their gradient on the way
back, in the storage type; with bf16 that adds one rounding of w and of dw to
what the oracle computes, which the bf16 tolerance covers.
"""
import numpy as np
import pytest

import gspn_inputs as gi
import oracle
import paper_2606_00746_amd as gspn
from gpu_util import ignored_taps, report, require_gpu, to_device, to_host, tolerance, upload

pytestmark = pytest.mark.gpu


def case(name, B, C, G, H, W, dirs=15, dtype="bf16", backward=True, sigma=1.0, seed=7):
    gate = "sigmoid" if dtype == "bf16" else "normal"
    return gi.Workload(name, B, C, G, H, W, dtype, dirs, backward, gate, sigma, seed)


CASES = [
    case("med64", 1, 64, 2, 64, 64),
    case("med56-dirs6", 2, 24, 2, 56, 56, dirs=6),
    # one channel per group: weights formed in the blocked order for both
    # passes (the plain calls read vertical ones in place instead)
    case("med64-G=C", 1, 16, 16, 64, 64),
    case("med56-G=C-dirs6", 2, 12, 12, 56, 56, dirs=6, sigma=2.0),
    # ... at every side of the register-streamed kernels
    case("med48-G=C-dirs9", 1, 8, 8, 48, 48, dirs=9),
    case("med40-G=C", 1, 8, 8, 40, 40),
    case("med32-G=C-dirs12", 2, 6, 6, 32, 32, dirs=12, sigma=2.0),
    case("med24-G=C-dirs3", 2, 8, 8, 24, 24, dirs=3),
    case("tiny14", 2, 24, 2, 14, 14),
    case("tiny16-R2L", 1, 8, 1, 16, 16, dirs=8, sigma=2.0),
    case("small-f32-40x24", 2, 6, 3, 40, 24, dtype="f32"),
    case("small-33x20-dirs5", 1, 6, 3, 33, 20, dirs=5),
    case("general-70x100", 1, 4, 2, 70, 100),
    case("wide-72x136-fwd", 1, 4, 2, 72, 136, backward=False),
]


def run(wl, inputs, wt):
    torch = require_gpu()
    print(f"[case] norm {wl.name} B={wl.B} C={wl.C} G={wl.G} {wl.H}x{wl.W} dirs={wl.dirs}",
          flush=True)
    t = upload(inputs, wl.dtype, wl.dirs)
    wtd = to_device(wt, wl.dtype)
    out = {"y": gspn.scan_fwd_norm(t["x"], wtd, t["lam"], t["u"], wl.dirs)}
    if wl.backward:
        dx, dwt, dlam, du = gspn.scan_bwd_norm(t["x"], wtd, t["lam"], t["u"], t["dy"], wl.dirs)
        out.update(dx=dx, dwt=dwt, dlam=dlam, du=du)
    torch.cuda.synchronize()
    return {k: to_host(v) for k, v in out.items()}


@pytest.mark.parametrize("wl", CASES, ids=lambda w: w.name)
def test_norm_parity_against_oracle(wl):
    inputs = gi.make_inputs(wl, with_dy=wl.backward)
    wt = gi.make_logits(wl)
    got = run(wl, inputs, wt)
    tol = tolerance(wl.dtype)
    w = oracle.normalize_w(wt, wl.dirs)
    ref_y = oracle.scan_fwd(inputs["x"], w, inputs["lam"], inputs["u"], wl.dirs)
    err = report(wl.name, "y", got["y"], ref_y)
    assert err <= tol, f"y err {err:.3g}"
    if wl.backward:
        ref = oracle.scan_bwd(inputs["x"], w, inputs["lam"], inputs["u"], inputs["dy"], wl.dirs)
        ref["dwt"] = oracle.normalize_w_bwd(wt, ref["dw"], wl.dirs)
        for k in ("dx", "dwt", "dlam", "du"):
            err = report(wl.name, k, got[k], ref[k])
            assert err <= tol, f"{k} err {err:.3g}"
        # taps off the grid get exactly zero (those on the first line carry
        # the normalization's share of their row, as in the oracle)
        off = np.zeros_like(got["dwt"], dtype=bool)
        ign = ignored_taps(wl.dirs, wl.H, wl.W)
        for s in range(wl.ndirs):
            for k in (0, 2):
                off[s, :, :, k] = ign[s, k] & ~_first_line(wl, s)
        assert np.all(got["dwt"][off] == 0.0)


def _first_line(wl, s):
    bit = [b for b in gi.DIR_BITS if wl.dirs & b][s]
    m = np.zeros((wl.H, wl.W), dtype=bool)
    if bit == gi.T2B:
        m[0] = True
    elif bit == gi.B2T:
        m[-1] = True
    elif bit == gi.L2R:
        m[:, 0] = True
    else:
        m[:, -1] = True
    return m


@pytest.mark.parametrize("wl", [case("nan-med64", 1, 8, 1, 64, 64), case("nan-tiny14", 1, 8, 2, 14, 14)],
                         ids=lambda w: w.name)
def test_norm_logits_off_the_grid_may_hold_nan(wl):
    inputs = gi.make_inputs(wl, with_dy=True)
    wt = gi.make_logits(wl)
    clean = run(wl, inputs, wt)
    dirty = wt.copy()
    ign = ignored_taps(wl.dirs, wl.H, wl.W)
    for s in range(wl.ndirs):
        for k in (0, 2):
            off = ign[s, k] & ~_first_line(wl, s)
            dirty[s, :, :, k][:, :, off] = np.nan
    got = run(wl, inputs, dirty)
    for k in clean:
        assert np.array_equal(got[k], clean[k]), k
