"""GPU parity of the latent-space sublayer (C-GSPN, Sec. 5) through the C ABI
against the fp64 oracle, on seeded inputs.

* gspn_project (Eqs. (latent_down), (latent_up)): bf16 result of an fp32
  accumulation against the exact product: within one bf16 rounding plus the
  fp32 summation error, |got - ref| <= 2^-8 |ref| + 1e-4 max|ref|.
* gspn_latent_params (Eq. (latent_params) + Eq. (row_stochastic_norm)): u and
  lambda as above; normalized w within 2^-8 (weights lie in [0, 1]) and exactly
  0 on taps that leave the grid.
* gspn_latent_fwd (the whole sublayer): normwise error <= 2e-2 against the
  oracle that rounds the stored stage results (x_c, u, lambda, w, y_c) to
  bf16 at the same points as the library.
"""
import numpy as np
import pytest

import gspn_inputs as gi
import oracle
import paper_2606_00746_amd as gspn
from gpu_util import normwise_err, require_gpu, to_device, to_host

pytestmark = pytest.mark.gpu


def _lw(name, B, C, Cc, H, W, dirs=15, seed=31):
    return gi.LatentWorkload(name, B, C, Cc, H, W, dirs, seed)


def _close_bf16(got, ref, tag):
    scale = float(np.abs(ref).max()) or 1.0
    bad = np.abs(got - ref) > 2.0 ** -8 * np.abs(ref) + 1e-4 * scale
    assert not bad.any(), (f"{tag}: {int(bad.sum())} of {bad.size} outside bound, "
                           f"max err {float(np.abs(got - ref).max()):.3g}")


# (B, M, K, H, W): ragged pixel tiles (H*W not a multiple of 128), ragged row
# tiles (M not a multiple of 64), K of one partial stage, several stages and
# the paper's widths
PROJECT_CASES = [
    (1, 8, 8, 1, 1),
    (2, 64, 64, 5, 7),
    (1, 70, 24, 9, 16),
    (2, 3, 1152, 13, 11),
    (1, 1152, 64, 12, 12),
    (3, 128, 136, 16, 8),
    (1, 64, 1152, 37, 37),
    # K > 64, not a multiple of 64, with K-rows at every 2-byte offset from
    # 16-byte alignment (H * W odd): the stage kernel's 16-byte pieces
    (3, 40, 104, 7, 9),
    (2, 17, 200, 5, 5),
]


@pytest.mark.parametrize("B,M,K,H,W", PROJECT_CASES)
def test_project_matches_oracle(B, M, K, H, W):
    require_gpu()
    lw = _lw("proj", B, K, 8, H, W, seed=M + 7 * K)
    rng_in = gi.make_latent_inputs(lw.with_(Cc=8))
    x = rng_in["x"]                                          # [B, K, H, W]
    a = gi.make_latent_inputs(lw.with_(B=1, C=K, Cc=M, H=1, W=1))["p_down"]   # [M, K]
    y = to_host(gspn.project(to_device(a, "bf16"), to_device(x, "bf16")))
    _close_bf16(y, oracle.project(a, x), f"project {B}x{M}x{K} {H}x{W}")


LATENT_CASES = [
    _lw("tiny-5x7", 1, 16, 8, 5, 7),
    _lw("vit-37x37", 2, 64, 16, 37, 37),
    _lw("rect-12x20-dirs5", 1, 64, 64, 12, 20, dirs=5),
    _lw("odd-9x8-dirs10", 2, 24, 24, 9, 8, dirs=10),
    _lw("tall-70x9-dirs3", 1, 32, 8, 70, 9, dirs=3),
    _lw("paper-width-20x20", 1, 1152, 64, 20, 20),
    # more than 64 latent channels: the parameter product takes K in stages
    _lw("cc128-9x10-dirs5", 1, 128, 128, 9, 10, dirs=5),
]


@pytest.mark.parametrize("lw", LATENT_CASES, ids=lambda w: w.name)
def test_latent_params_match_oracle(lw):
    require_gpu()
    inp = gi.make_latent_inputs(lw)
    xc = gi.round_to_bf16(oracle.project(inp["p_down"], inp["x"]).astype(np.float32))
    dev = {k: to_device(v, "bf16") for k, v in inp.items()}
    u, lam, w = gspn.latent_params(to_device(xc, "bf16"), dev["l_u"], dev["l_lam"], dev["l_w"],
                                   lw.dirs)
    D, B, Cc, H, W = lw.ndirs, lw.B, lw.Cc, lw.H, lw.W
    got_u = gi.from_line_major(to_host(u).reshape(D, B, Cc, H * W), lw.dirs, H, W)
    got_l = gi.from_line_major(to_host(lam).reshape(D, B, Cc, H * W), lw.dirs, H, W)
    got_w = gi.from_line_major(to_host(w).reshape(D, B, Cc, 3, H * W), lw.dirs, H, W)
    ref = oracle.latent_params(xc, inp["l_u"], inp["l_lam"], inp["l_w"], lw.dirs)
    _close_bf16(got_u, ref["u"], f"{lw.name} u")
    _close_bf16(got_l, ref["lam"], f"{lw.name} lam")
    assert float(np.abs(got_w - ref["w"]).max()) <= 2.0 ** -8, f"{lw.name} w"
    assert np.all(got_w[ref["w"] == 0.0] == 0.0), f"{lw.name} off-grid taps not 0"


# sides that are not multiples of 8 run the latent scan on a grid padded to
# whole 8-line blocks: scans that start in the padding (B2T, R2L), wide
# padded grids, square and oblong ones
FWD_CASES = LATENT_CASES + [
    _lw("r2l-only-14x30", 3, 16, 16, 14, 30, dirs=8),
    _lw("b2t-r2l-37x45", 1, 32, 32, 37, 45, dirs=10),
    _lw("pad-to-wide-73x73", 1, 64, 64, 73, 73),
    _lw("pad-to-64-57x61-dirs6", 2, 32, 32, 57, 61, dirs=6),
]


@pytest.mark.parametrize("lw", FWD_CASES, ids=lambda w: w.name)
def test_latent_fwd_matches_oracle(lw):
    require_gpu()
    inp = gi.make_latent_inputs(lw)
    dev = {k: to_device(v, "bf16") for k, v in inp.items()}
    y = to_host(gspn.latent_fwd(dev["x"], dev["p_down"], dev["l_u"], dev["l_lam"], dev["l_w"],
                                dev["p_up"], lw.dirs))
    ref = oracle.latent_fwd(inp["x"], inp["p_down"], inp["l_u"], inp["l_lam"], inp["l_w"],
                            inp["p_up"], lw.dirs, storage="bf16")
    err = normwise_err(y, ref)
    assert err <= 2e-2, f"{lw.name} y err {err:.3g}"


@pytest.mark.parametrize("lw", gi.LATENT_WORKLOADS, ids=lambda w: w.name)
def test_latent_full_size_sampled_images(lw):
    """The paper's token grids at their full size (B = 32, C = 1152, Cc = 64),
    in the one call the benchmark times: every image is independent, so the
    oracle checks the first and the last."""
    require_gpu()
    print(f"[case] latent full size {lw.name}", flush=True)
    inp = gi.make_latent_inputs(lw)
    dev = {k: to_device(v, "bf16") for k, v in inp.items()}
    y = gspn.latent_fwd(dev["x"], dev["p_down"], dev["l_u"], dev["l_lam"], dev["l_w"],
                        dev["p_up"], lw.dirs)
    for b in (0, lw.B - 1):
        ref = oracle.latent_fwd(inp["x"][b:b + 1], inp["p_down"], inp["l_u"], inp["l_lam"],
                                inp["l_w"], inp["p_up"], lw.dirs, storage="bf16")
        err = normwise_err(to_host(y[b:b + 1]), ref)
        print(f"[err] {lw.name} image {b}: normwise {err:.3g}", flush=True)
        assert err <= 2e-2, f"image {b} y err {err:.3g}"
