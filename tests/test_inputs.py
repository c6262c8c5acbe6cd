"""The seeded input generator: determinism, recipe and storage rounding."""
import numpy as np
import pytest

import gspn_inputs as gi


def test_deterministic_and_seed_dependent():
    wl = gi.workload(0)
    a = gi.make_inputs(wl)
    b = gi.make_inputs(wl)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    c = gi.make_inputs(wl.with_(seed=9))
    assert not np.array_equal(a["x"], c["x"])


def test_recipe_statistics():
    wl = gi.workload(1).with_(B=4)
    t = gi.make_inputs(wl)
    x = t["x"]
    assert abs(float(x.mean())) < 0.01 and abs(float(x.std()) - 1.0) < 0.01
    lam = t["lam"]
    assert lam.min() > 0.0 and lam.max() < 1.0          # sigmoid gate
    assert abs(float(lam.mean()) - 0.5) < 0.01
    assert t["dy"].shape == x.shape
    # all values bf16-representable
    for k, v in t.items():
        gi.to_bf16_bits(v)


@pytest.mark.parametrize("idx", [0, 1, 4])
def test_taps_are_masked_softmax(idx):
    wl = gi.workload(idx)
    if wl.H > 64:
        wl = wl.with_(B=1, C=wl.G, H=9, W=11)
    t = gi.make_inputs(wl)
    w = t["w"].astype(np.float64)
    H, W = wl.H, wl.W
    s = 0
    for bit in gi.DIR_BITS:
        if not wl.dirs & bit:
            continue
        vertical = bit in (gi.T2B, gi.B2T)
        ws = w[s]
        # out-of-grid taps are exactly zero
        if vertical:
            assert np.all(ws[:, :, 0, :, 0] == 0) and np.all(ws[:, :, 2, :, W - 1] == 0)
        else:
            assert np.all(ws[:, :, 0, 0, :] == 0) and np.all(ws[:, :, 2, H - 1, :] == 0)
        assert np.all(ws >= 0)
        tol = 1e-6 if wl.dtype == "f32" else 3 * 2.0 ** -8
        np.testing.assert_allclose(ws.sum(axis=2), 1.0, atol=tol)
        s += 1


def test_peaky_logits_for_extreme_resolution():
    """sigma = 2 logits concentrate the weight on one neighbour far more often."""
    small = gi.workload(1).with_(B=1, C=12, H=32, W=32)
    peaky = gi.workload(4).with_(B=1, C=32, H=32, W=32)
    m1 = gi.make_inputs(small)["w"].max(axis=3).mean()
    m2 = gi.make_inputs(peaky)["w"].max(axis=3).mean()
    assert m2 > m1 + 0.1


def test_bf16_helpers_round_trip():
    a = np.array([1.0, -2.5, 3.0e-3, 65504.0], dtype=np.float32)
    r = gi.round_to_bf16(a)
    np.testing.assert_array_equal(gi.from_bf16_bits(gi.to_bf16_bits(r)), r)
    # ties to even: 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7
    t = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], dtype=np.float32)
    np.testing.assert_array_equal(gi.round_to_bf16(t), np.array([1.0, 1.0 + 2.0 ** -6], np.float32))
    with pytest.raises(ValueError):
        gi.to_bf16_bits(np.array([1.0 + 2.0 ** -10], dtype=np.float32))


def _blocked_offset(l, p, L, P):
    """Blocked line-major offset written out: 8-line blocks, positions adjacent."""
    q = l // 8
    n = min(8, L - 8 * q)
    return 8 * P * q + n * p + l % 8


@pytest.mark.parametrize("H,W", [(3, 5), (11, 19), (16, 8), (24, 17)])
def test_line_major_round_trip_and_layout(H, W):
    rng = np.random.default_rng(3)
    a = rng.standard_normal((4, 2, 2, H, W))
    lm = gi.to_line_major(a, 15)
    assert lm.shape == (4, 2, 2, H * W)
    for r in range(H):
        for c in range(W):
            # vertical directions scan rows: line r, position c
            assert lm[0, 1, 0, _blocked_offset(r, c, H, W)] == a[0, 1, 0, r, c]
            assert lm[1, 0, 1, _blocked_offset(r, c, H, W)] == a[1, 0, 1, r, c]
            # horizontal directions scan columns: line c, position r
            assert lm[2, 1, 1, _blocked_offset(c, r, W, H)] == a[2, 1, 1, r, c]
            assert lm[3, 0, 1, _blocked_offset(c, r, W, H)] == a[3, 0, 1, r, c]
    np.testing.assert_array_equal(gi.from_line_major(lm, 15, H, W), a)
    # subsets keep slot order
    b = a[:2]
    np.testing.assert_array_equal(gi.from_line_major(gi.to_line_major(b, 5), 5, H, W), b)
