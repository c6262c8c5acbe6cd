"""gspn_scan_bwd_static (the backward for callers that cannot allocate; its
workspace is the library's fixed device array) against gspn_scan_bwd with a
caller workspace, through the C ABI, on two calls in a row, the second with a
smaller input.  Both run the same kernels in the same order, so the results
must agree bit for bit."""
import numpy as np
import pytest

import gspn_inputs as gi
import paper_2606_00746_amd as gspn
from gpu_util import require_gpu, to_device

pytestmark = pytest.mark.gpu


def _run(wl, static):
    torch = require_gpu()
    inp = gi.make_inputs(wl, with_dy=True)
    t = {k: to_device(v, wl.dtype) for k, v in inp.items()}
    out = [torch.full_like(t[k], float("nan")) for k in ("x", "w", "lam", "u")]
    ptrs = [t[k].data_ptr() for k in ("x", "w", "lam", "u", "dy")] + [o.data_ptr() for o in out]
    dt = gspn.BF16 if wl.dtype == "bf16" else gspn.F32
    sizes = (wl.dirs, wl.B, wl.C, wl.G, wl.H, wl.W, dt)
    stream = torch.cuda.current_stream().cuda_stream
    st, need = gspn.gspn_workspace_size(gspn.OP_BWD, *sizes)
    assert st == 0
    if static:
        assert 0 < need <= gspn._native.STATIC_SCRATCH_BYTES     # the array is used
        st = gspn.gspn_scan_bwd_static(*ptrs, *sizes, stream)
    else:
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        st = gspn.gspn_scan_bwd(*ptrs, *sizes, ws.data_ptr(), need, stream)
    assert st == 0, gspn.gspn_strerror(st)
    torch.cuda.synchronize()
    return [o.cpu() for o in out]


# a group split over several workgroups (fp32 partial sums in the workspace),
# then a smaller problem on the array the first call left behind
CASES = [gi.workload(3).with_(name="64x64-b2-c64-g2", B=2, C=64, G=2),
         gi.workload(3).with_(name="64x64-b1-c32-g2-dirs6", B=1, C=32, G=2, dirs=6)]


def test_static_backward_matches_workspace_backward():
    torch = require_gpu()
    for wl in CASES:
        print(f"[case] {wl.name}", flush=True)
        ref = _run(wl, static=False)
        got = _run(wl, static=True)
        for k, a, b in zip(("dx", "dw", "dlam", "du"), got, ref):
            assert not np.isnan(a.float().numpy()).any(), k      # every element written
            assert np.array_equal(a.view(torch.int16).numpy(), b.view(torch.int16).numpy()), k
