"""bf16 results within half a bf16 ulp of the exact result, element by element.

The kernels read bf16 inputs, compute in fp32 and round every output once,
to nearest even.  The oracle computes the exact result r (fp64) from the same
bf16 inputs, and the bound for each element is

    |got - r| <= 0.5 ulp_bf16(max(|r|, |got|)) + 2^-24 K m

with m the element's magnitude (the oracle on |x|, |lambda|, |u|, |dy| and
the non-negative weights: every term of the result taken with its absolute
value) and K = 16 (max(H, W) + C/G) for fp32's accumulated rounding.  A
kernel that truncates instead of rounding, rounds twice, or drops a term is
off by up to a whole ulp on a large share of the elements and fails.

Where the library itself stores an intermediate in bf16 (the normalized
weights and their gradient in the _norm entry points), the oracle starts
from the stored values the call left in its workspace: the same bf16-rounded
stores.  Those stores are checked on their own against the exact
normalization, to the same bound.
"""
import numpy as np
import pytest

import gspn_inputs as gi
import oracle
import paper_2606_00746_amd as gspn
from gpu_util import check_half_ulp, require_gpu, to_device, to_host, upload

pytestmark = pytest.mark.gpu


def case(name, B, C, G, H, W, dirs=15, backward=True):
    return gi.Workload(name, B, C, G, H, W, "bf16", dirs, backward, "sigmoid", 1.0, 13)


# one case per kernel family, pixel-major (and the blocked layout once)
CASES = [
    ("tiny-14x14", case("tiny-14x14", 2, 12, 2, 14, 14), "pixel"),
    ("small-40x24", case("small-40x24", 1, 8, 2, 40, 24), "pixel"),
    ("med-64x64-cpg32", case("med-64x64-cpg32", 1, 64, 2, 64, 64), "pixel"),
    ("med-64x64-cpg32-blocked", case("med-64x64-cpg32", 1, 64, 2, 64, 64), "blocked"),
    ("med-56x56-ns4", case("med-56x56-ns4", 1, 24, 2, 56, 56), "pixel"),
    ("med-64x64-G=C", case("med-64x64-G=C", 1, 16, 16, 64, 64), "pixel"),
    ("wide-72x136", case("wide-72x136", 1, 4, 2, 72, 136), "pixel"),
    ("chunked-256x256-fwd", case("chunked-256x256", 1, 8, 2, 256, 256, backward=False), "pixel"),
    ("general-70x100", case("general-70x100", 1, 4, 2, 70, 100), "pixel"),
]


def _abs_inputs(inp):
    out = {k: np.abs(v) for k, v in inp.items()}
    out["w"] = inp["w"]                      # non-negative already
    return out


@pytest.mark.parametrize("name,wl,layout", CASES, ids=[c[0] for c in CASES])
def test_outputs_within_half_ulp(name, wl, layout):
    torch = require_gpu()
    print(f"[case] bf16-exact {name} B={wl.B} C={wl.C} G={wl.G} {wl.H}x{wl.W} "
          f"layout={layout}", flush=True)
    inp = gi.make_inputs(wl, with_dy=wl.backward)
    assert np.all(inp["w"] >= 0)
    t = upload(inp, "bf16", wl.dirs, layout)
    got = {"y": gspn.scan_fwd(t["x"], t["w"], t["lam"], t["u"], wl.dirs, layout=layout)}
    if wl.backward:
        got.update(zip(("dx", "dw", "dlam", "du"),
                       gspn.scan_bwd(t["x"], t["w"], t["lam"], t["u"], t["dy"], wl.dirs,
                                     layout=layout)))
    torch.cuda.synchronize()
    got = {k: to_host(v) for k, v in got.items()}
    if layout == "blocked":
        for k in ("dw", "dlam", "du"):
            if k in got:
                got[k] = gi.from_line_major(got[k], wl.dirs, wl.H, wl.W)
    K = 16 * (max(wl.H, wl.W) + wl.C // wl.G)
    ab = _abs_inputs(inp)
    ref = {"y": oracle.scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], wl.dirs)}
    mag = {"y": oracle.scan_fwd(ab["x"], ab["w"], ab["lam"], ab["u"], wl.dirs)}
    if wl.backward:
        ref.update(oracle.scan_bwd(inp["x"], inp["w"], inp["lam"], inp["u"], inp["dy"], wl.dirs))
        mag.update(oracle.scan_bwd(ab["x"], ab["w"], ab["lam"], ab["u"], ab["dy"], wl.dirs))
    for k in got:
        check_half_ulp(f"{name} {k}", got[k], ref[k], mag[k], K)


def _ws_bf16(ws, offset, shape):
    """bf16 values the call left in its workspace at byte `offset`."""
    n = int(np.prod(shape))
    bits = ws[offset:offset + 2 * n].cpu().numpy().view(np.uint16)
    return gi.from_bf16_bits(bits).astype(np.float64).reshape(shape)


@pytest.mark.parametrize("wl", [case("norm-med-64x64", 1, 64, 2, 64, 64),
                                case("norm-med-56x56-G=C-dirs13", 1, 8, 8, 56, 56, dirs=13),
                                case("norm-tiny-14x14", 2, 12, 2, 14, 14)],
                         ids=lambda w: w.name)
def test_norm_stores_and_outputs_within_half_ulp(wl):
    torch = require_gpu()
    print(f"[case] bf16-exact norm {wl.name}", flush=True)
    inp = gi.make_inputs(wl, with_dy=True)
    wt = gi.make_logits(wl)
    t = upload(inp, "bf16", wl.dirs)
    wtd = to_device(wt, "bf16")
    wt = to_host(wtd)                          # the logits as the library reads them
    D = wl.ndirs
    wshape = (D, wl.B, wl.G, 3, wl.H, wl.W)
    nbytes = 2 * int(np.prod(wshape))
    ws = torch.zeros(gspn.workspace_size(gspn.OP_BWD_NORM, t["x"], wtd, wl.dirs) + 4096,
                     dtype=torch.uint8, device="cuda")
    y = gspn.scan_fwd_norm(t["x"], wtd, t["lam"], t["u"], wl.dirs, workspace=ws)
    torch.cuda.synchronize()
    # the register-streamed shapes (bf16 squares of side 24..64, a multiple
    # of 8) form the weights directly in the blocked order their scan reads
    blocked_w = wl.H == wl.W and wl.H % 8 == 0 and 24 <= wl.H <= 64

    def stored_w():
        v = _ws_bf16(ws, 0, wshape)
        if not blocked_w:
            return v
        return gi.from_line_major(v.reshape(wshape[:-2] + (wl.H * wl.W,)), wl.dirs, wl.H, wl.W)

    w_st = stored_w()
    dx, dwt, dlam, du = gspn.scan_bwd_norm(t["x"], wtd, t["lam"], t["u"], t["dy"], wl.dirs,
                                           workspace=ws)
    torch.cuda.synchronize()
    dw_st = _ws_bf16(ws, (nbytes + 255) // 256 * 256, wshape)
    K = 16 * (max(wl.H, wl.W) + wl.C // wl.G)
    # the stored weights against the exact normalization (the forward's and
    # the backward's copies are the same computation)
    w_ex = oracle.normalize_w(wt, wl.dirs)
    check_half_ulp(f"{wl.name} stored w", w_st, w_ex, np.ones_like(w_ex), 64)
    assert np.array_equal(w_st, stored_w())
    # the scan on the stored weights
    ab = _abs_inputs(inp)
    ref = oracle.scan_bwd(inp["x"], w_st, inp["lam"], inp["u"], inp["dy"], wl.dirs)
    mag = oracle.scan_bwd(ab["x"], w_st, ab["lam"], ab["u"], ab["dy"], wl.dirs)
    check_half_ulp(f"{wl.name} y", to_host(y),
                   oracle.scan_fwd(inp["x"], w_st, inp["lam"], inp["u"], wl.dirs),
                   oracle.scan_fwd(ab["x"], w_st, ab["lam"], ab["u"], wl.dirs), K)
    for k, v in (("dx", dx), ("dlam", dlam), ("du", du)):
        check_half_ulp(f"{wl.name} {k}", to_host(v), ref[k], mag[k], K)
    check_half_ulp(f"{wl.name} stored dw", dw_st, ref["dw"], mag["dw"], K)
    # the logits' gradient from the stored dw and w
    # (|dwt_m| <= |dw_m| + max_k |dw_k|: sigma' <= sigma <= S and the w_k sum to 1)
    dwt_ref = oracle.normalize_w_bwd(wt, dw_st, wl.dirs)
    dwt_mag = np.abs(dw_st) + np.abs(dw_st).max(axis=3, keepdims=True)
    check_half_ulp(f"{wl.name} dwt", to_host(dwt), dwt_ref, dwt_mag, 64)
