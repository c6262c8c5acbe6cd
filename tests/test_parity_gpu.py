"""GPU parity: libgspn (through the C ABI) against the fp64 CPU oracle.

Both sides read the same seeded inputs.  Tolerances (normwise max error per
output tensor): 1e-5 for fp32 storage, 2e-2 for bf16 storage with fp32
accumulation.  Taps the operator ignores must get exactly zero gradient, and
garbage (NaN) in them must not change any result.
"""
import numpy as np
import pytest

import gspn_inputs as gi
import oracle
import paper_2606_00746_amd as gspn
from gpu_util import check_half_ulp, ignored_taps, report, require_gpu, to_host, tolerance, upload

pytestmark = pytest.mark.gpu

GRAD_KEYS = ("dx", "dw", "dlam", "du")


def run_gpu(inputs, wl, backward, layout="pixel"):
    """Run the library on pixel-major host inputs (per-direction tensors in
    `layout` on the device); returns pixel-major results."""
    torch = require_gpu()
    print(f"[case] {wl.name} B={wl.B} C={wl.C} G={wl.G} {wl.H}x{wl.W} dirs={wl.dirs} "
          f"{wl.dtype} layout={layout}", flush=True)
    t = upload(inputs, wl.dtype, wl.dirs, layout)
    y = gspn.scan_fwd(t["x"], t["w"], t["lam"], t["u"], wl.dirs, layout=layout)
    out = {"y": y}
    if backward:
        dx, dw, dlam, du = gspn.scan_bwd(t["x"], t["w"], t["lam"], t["u"], t["dy"], wl.dirs,
                                         layout=layout)
        out.update(dx=dx, dw=dw, dlam=dlam, du=du)
    torch.cuda.synchronize()
    res = {k: to_host(v) for k, v in out.items()}
    if layout == "blocked":
        for k in ("dw", "dlam", "du"):
            if k in res:
                res[k] = gi.from_line_major(res[k], wl.dirs, wl.H, wl.W)
    return res


def check_against_oracle(inputs, got, wl, backward, tag=""):
    tol = tolerance(wl.dtype)
    ref_y = oracle.scan_fwd(inputs["x"], inputs["w"], inputs["lam"], inputs["u"], wl.dirs)
    err = report(tag, "y", got["y"], ref_y)
    assert err <= tol, f"{tag} y err {err:.3g} > {tol}"
    if backward:
        ref = oracle.scan_bwd(inputs["x"], inputs["w"], inputs["lam"], inputs["u"], inputs["dy"],
                              wl.dirs)
        for k in GRAD_KEYS:
            err = report(tag, k, got[k], ref[k])
            assert err <= tol, f"{tag} {k} err {err:.3g} > {tol}"
        ign = ignored_taps(wl.dirs, wl.H, wl.W)          # [D,3,H,W]
        dw = got["dw"]                                    # [D,B,G,3,H,W]
        mask = np.broadcast_to(ign[:, None, None], dw.shape)
        assert np.all(dw[mask] == 0.0), f"{tag} dw not zero on ignored taps"


def case(name, B, C, G, H, W, dirs=15, dtype="bf16", backward=True, gate="sigmoid", sigma=1.0,
         seed=5):
    return gi.Workload(name, B, C, G, H, W, dtype, dirs, backward, gate, sigma, seed)


# reduced-batch versions of the five workloads: the oracle checks every output
REDUCED = [
    gi.workload(0),
    gi.workload(0).with_(name="tiny-f32-bwd", backward=True),
    gi.workload(1).with_(B=2),
    gi.workload(2).with_(B=2),
    gi.workload(3).with_(B=1, C=64, G=2),
    gi.workload(4).with_(C=8, G=2),
]

EDGE = [
    case("1x1", 1, 3, 3, 1, 1),
    case("row", 2, 5, 1, 1, 7),
    case("column", 1, 6, 2, 9, 1),
    case("13x7-G=C", 1, 4, 4, 13, 7),
    case("17x33-ragged-channels", 3, 7, 7, 17, 33),
    case("31x20-dirs5", 1, 10, 5, 31, 20, dirs=5),
    case("64x63-dirs10", 2, 12, 3, 64, 63, dirs=10),
    case("16x16-cpg64", 1, 128, 2, 16, 16),
    case("f32-40x24", 2, 6, 3, 40, 24, dtype="f32", gate="normal"),
    case("f32-9x12-R2L", 1, 5, 1, 9, 12, dirs=8, dtype="f32", gate="normal"),
    case("general-65x3", 1, 2, 1, 65, 3),
    case("general-70x100", 1, 4, 2, 70, 100),
    case("general-f32-3x130", 1, 3, 1, 3, 130, dtype="f32", gate="normal"),
    # the largest side the library takes (4096): a single row, 4096-step
    # scans of narrow planes
    case("maxside-row-1x4096", 1, 2, 1, 1, 4096),
    case("maxside-f32-4096x2", 1, 2, 2, 4096, 2, dtype="f32", gate="normal"),
    case("maxside-4096x8-dirs9", 1, 1, 1, 4096, 8, dirs=9),
    case("peaky-48x48", 1, 8, 2, 48, 48, sigma=2.0),
    # register-streamed path (bf16, 56x56 / 64x64): direction subsets, ragged
    # channel chunks (idle waves), fewer than three waves per workgroup
    case("med64-dirs5-cpg20", 1, 40, 2, 64, 64, dirs=5),
    case("med64-R2L-cpg2", 2, 4, 2, 64, 64, dirs=8),
    case("med56-dirs6-cpg1", 1, 3, 3, 56, 56, dirs=6),
    case("med64-all-cpg9", 1, 18, 2, 64, 64),
    case("med56-T2B-cpg12", 2, 24, 2, 56, 56, dirs=1),
    case("med64-peaky", 1, 16, 1, 64, 64, sigma=2.0),
    # lines longer than a wave (forward: several positions per lane, fp32
    # direction planes summed by a tiled kernel): ragged position groups,
    # unused groups, both orientations, direction subsets, peaky weights
    case("wide-72x136", 1, 4, 2, 72, 136),
    case("wide-256x64-fwd", 1, 3, 1, 256, 64, backward=False),
    case("wide-128x128-dirs9", 1, 6, 3, 128, 128, dirs=9, backward=False),
    case("wide-200x248-peaky", 1, 2, 1, 200, 248, sigma=2.0, backward=False),
    case("wide-96x80-R2L", 2, 4, 4, 96, 80, dirs=8),
    case("wide-128x192-dirs6", 1, 4, 4, 128, 192, dirs=6, backward=False),
    case("wide-256x128-dirs9-peaky", 1, 2, 1, 256, 128, dirs=9, sigma=2.0, backward=False),
    # pixel-major vertical directions read in place, 4 columns per lane: 2
    # lanes active (W = 8), 50 lanes (W = 200)
    case("wide-200x8-fwd", 2, 3, 3, 200, 8, backward=False),
    case("wide-8x200-dirs3", 1, 4, 2, 8, 200, dirs=3, backward=False),
    # few channel planes of 256 x 256: the forward cuts every scan into
    # chunks of whole line blocks, end states from zero, carries through w,
    # then the chunks again from their carries (16, 16 and 8 chunks)
    case("chunk-256x256-c8", 1, 8, 2, 256, 256, backward=False),
    case("chunk-256x256-dirs6-peaky", 1, 4, 4, 256, 256, dirs=6, sigma=2.0, backward=False),
    case("chunk8-256x256-c20-R2L", 1, 20, 4, 256, 256, dirs=8, backward=False),
    # planes of at most 16 x 16 (whole planes staged in LDS, four channels per
    # wave): idle channel slots, one channel per group, groups split into
    # chunks (fp32 partials), every size, direction subsets, peaky weights
    case("tiny-14x14-cpg6-dirs6", 2, 12, 2, 14, 14, dirs=6),
    case("tiny-8x8-R2L-cpg1", 1, 3, 3, 8, 8, dirs=8),
    case("tiny-12x12-peaky", 1, 20, 4, 12, 12, sigma=2.0),
    case("tiny-16x16-cpg72", 1, 144, 2, 16, 16),
    case("tiny-14x14-T2B-cpg33", 1, 33, 1, 14, 14, dirs=1),
    # one channel per group (per-channel weights): workgroups of up to eight
    # independent channels, fewer than eight channels, direction subsets
    case("med64-G=C", 1, 16, 16, 64, 64),
    # the same kernels at the other square sides they are built for
    case("med48-all-cpg12", 2, 24, 2, 48, 48),
    case("med40-dirs10-cpg3", 1, 6, 2, 40, 40, dirs=10),
    case("med32-cpg32", 1, 64, 2, 32, 32),
    case("med24-G=C-dirs5", 2, 5, 5, 24, 24, dirs=5),
    case("med32-peaky-R2L", 1, 8, 1, 32, 32, dirs=8, sigma=2.0),
    case("med64-G=C-3ch-dirs9", 2, 3, 3, 64, 64, dirs=9),
    case("med56-G=C-dirs6", 2, 12, 12, 56, 56, dirs=6),
    # shapes whose backward takes 4 slots per step (two 4-channel workgroups
    # per CU): 3 chunks of 4, one chunk of 4 (no partials), a direction subset
    case("med48-ns4-cpg12", 1, 24, 2, 48, 48),
    case("med64-ns4-cpg4", 2, 16, 4, 64, 64),
    case("med40-ns4-cpg12-dirs6", 1, 12, 1, 40, 40, dirs=6),
    # both vertical directions (the second takes x and dy from the first's
    # registers) at the sides no other case runs them on: 9 channels per group
    # (uneven chunks), and with a horizontal direction run before them
    case("med40-vertical-pair-cpg9", 1, 18, 2, 40, 40, dirs=3),
    case("med24-dirs11-cpg3", 2, 6, 2, 24, 24, dirs=11),
]


@pytest.mark.parametrize("wl", REDUCED + EDGE, ids=lambda w: w.name)
def test_parity_against_oracle(wl):
    inputs = gi.make_inputs(wl, with_dy=wl.backward)
    got = run_gpu(inputs, wl, wl.backward)
    check_against_oracle(inputs, got, wl, wl.backward, wl.name)


# the producer layout (blocked line-major per-direction tensors) on every
# kernel family
BLOCKED = [
    gi.workload(0).with_(name="tiny-f32-bwd", backward=True),
    gi.workload(1).with_(B=2),
    gi.workload(2).with_(B=2),
    gi.workload(3).with_(B=1, C=64, G=2),
    gi.workload(4).with_(C=8, G=2),
    case("13x7-G=C", 1, 4, 4, 13, 7),
    case("general-70x100", 1, 4, 2, 70, 100),
    case("wide-72x136", 1, 4, 2, 72, 136),
    case("med64-G=C", 1, 16, 16, 64, 64),
    case("med56-T2B-cpg12", 2, 24, 2, 56, 56, dirs=1),
    case("med40-vertical-pair-cpg9", 1, 18, 2, 40, 40, dirs=3),
    case("chunk-256x256-c8", 1, 8, 2, 256, 256, backward=False),
]


@pytest.mark.parametrize("wl", BLOCKED, ids=lambda w: w.name)
def test_blocked_layout_parity(wl):
    inputs = gi.make_inputs(wl, with_dy=wl.backward)
    got = run_gpu(inputs, wl, wl.backward, layout="blocked")
    check_against_oracle(inputs, got, wl, wl.backward, wl.name + " blocked")


@pytest.mark.parametrize("wl", [gi.workload(3).with_(B=1, C=64, G=2),
                                case("tiny-14x14-cpg6-dirs6", 2, 12, 2, 14, 14, dirs=6),
                                case("general-f32-3x130", 1, 3, 1, 3, 130, dtype="f32",
                                     gate="normal")], ids=lambda w: w.name)
def test_layouts_agree_bitwise(wl):
    """Both layouts run the same arithmetic: identical results."""
    inputs = gi.make_inputs(wl, with_dy=True)
    a = run_gpu(inputs, wl, True)
    b = run_gpu(inputs, wl, True, layout="blocked")
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("wl", [case("nan-taps-14x14", 2, 8, 2, 14, 14),
                                case("nan-taps-64x64", 1, 4, 1, 64, 64),
                                case("nan-taps-general", 1, 2, 1, 3, 80),
                                case("nan-taps-wide", 1, 2, 1, 72, 136)], ids=lambda w: w.name)
def test_ignored_taps_may_hold_nan(wl):
    inputs = gi.make_inputs(wl, with_dy=True)
    clean = run_gpu(inputs, wl, True)
    dirty = dict(inputs)
    w = inputs["w"].copy()
    ign = ignored_taps(wl.dirs, wl.H, wl.W)
    w[np.broadcast_to(ign[:, None, None], w.shape)] = np.nan
    dirty["w"] = w
    got = run_gpu(dirty, wl, True)
    for k in ("y",) + GRAD_KEYS:
        assert np.array_equal(got[k], clean[k]), k


def test_deterministic_bitwise():
    wl = gi.workload(3).with_(B=1, C=64, G=2)
    inputs = gi.make_inputs(wl)
    a = run_gpu(inputs, wl, True)
    b = run_gpu(inputs, wl, True)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


# full-size workloads: every output computed on the GPU, sampled
# (batch, group) units checked against the oracle
@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_full_size_sampled_units(idx):
    wl = gi.workload(idx)
    inputs = gi.make_inputs(wl)
    got = run_gpu(inputs, wl, wl.backward)
    rng = np.random.default_rng(idx)
    units = {(0, 0), (wl.B - 1, wl.G - 1), (int(rng.integers(wl.B)), int(rng.integers(wl.G)))}
    # groups spread over the planes: kernels that take the planes in rounds
    # (the 256 x 256 forward) get a unit checked in every round
    units |= {(0, g) for g in range(0, wl.G, max(1, wl.G // 4))}
    cpg = wl.C // wl.G
    for b, g in sorted(units):
        sl = oracle.slice_group(inputs, b, g, wl.G)
        cs = slice(g * cpg, (g + 1) * cpg)
        part = {"y": got["y"][b:b + 1, cs]}
        if wl.backward:
            part.update(dx=got["dx"][b:b + 1, cs], dw=got["dw"][:, b:b + 1, g:g + 1],
                        dlam=got["dlam"][:, b:b + 1, cs], du=got["du"][:, b:b + 1, cs])
        unit_wl = wl.with_(B=1, C=cpg, G=1)
        check_against_oracle(sl, part, unit_wl, wl.backward, f"{wl.name} unit b={b} g={g}")
    assert np.all(np.isfinite(got["y"]))


def test_wide_rounds_ragged():
    """The 256 x 256 forward takes its planes in rounds of as many as the
    device runs at once (256 on this GPU); 300 planes end with a short round,
    and the weight group of planes 250..274 spans the boundary between the
    rounds.  Units on both sides of it and in the last round, against the
    oracle."""
    wl = case("wide256-300planes", 3, 100, 4, 256, 256, backward=False)
    inputs = gi.make_inputs(wl)
    got = run_gpu(inputs, wl, False)
    cpg = wl.C // wl.G
    for b, g in [(0, 0), (2, 1), (2, 2), (2, 3)]:
        sl = oracle.slice_group(inputs, b, g, wl.G)
        cs = slice(g * cpg, (g + 1) * cpg)
        check_against_oracle(sl, {"y": got["y"][b:b + 1, cs]}, wl.with_(B=1, C=cpg, G=1), False,
                             f"{wl.name} unit b={b} g={g}")
    assert np.all(np.isfinite(got["y"]))


@pytest.mark.parametrize("wl", [case("med56-cpg12", 1, 24, 2, 56, 56),
                                case("med64-cpg32", 1, 64, 2, 64, 64),
                                case("med48-cpg12-dirs6", 2, 24, 2, 48, 48, dirs=6)],
                         ids=lambda w: w.name)
def test_slot_plans_agree(wl):
    """The register-streamed backward under both launch plans (4 channels per
    workgroup, or up to 8): each plan bitwise reproducible; dx, dlam and du
    bit for bit the same across plans (nothing there depends on the plan);
    dw, whose sum over a group's channels the plan associates differently,
    within half a bf16 ulp of the exact value under both, so at most one ulp
    apart."""
    torch = require_gpu()
    print(f"[case] slot plans {wl.name}", flush=True)
    inputs = gi.make_inputs(wl, with_dy=True)
    t = upload(inputs, wl.dtype, wl.dirs)
    res = {}
    for slots in (4, 8, 4):
        out = gspn.scan_bwd(t["x"], t["w"], t["lam"], t["u"], t["dy"], wl.dirs, slots=slots)
        torch.cuda.synchronize()
        got = dict(zip(GRAD_KEYS, (to_host(v) for v in out)))
        if slots in res:
            for k in GRAD_KEYS:
                assert np.array_equal(got[k], res[slots][k]), f"slots={slots} {k} not repeatable"
        res[slots] = got
    for k in ("dx", "dlam", "du"):
        assert np.array_equal(res[4][k], res[8][k]), k
    ref = oracle.scan_bwd(inputs["x"], inputs["w"], inputs["lam"], inputs["u"], inputs["dy"],
                          wl.dirs)
    ab = {k: np.abs(v) for k, v in inputs.items()}
    mag = oracle.scan_bwd(ab["x"], inputs["w"], ab["lam"], ab["u"], ab["dy"], wl.dirs)
    K = 16 * (wl.H + wl.C // wl.G)
    for slots in (4, 8):
        check_half_ulp(f"{wl.name} slots={slots} dw", res[slots]["dw"], ref["dw"], mag["dw"], K)
    diff = np.abs(res[4]["dw"] - res[8]["dw"])
    print(f"[err] {wl.name} dw elements differing between plans: "
          f"{float(np.mean(diff > 0)):.2e}", flush=True)
