"""Pins of the oracle's latent-space sublayer (Sec. 5, Eqs. (latent_down),
(latent_params), (latent_recurrence), (latent_up)) against hand-worked values,
an independent sigmoid and symmetries -- CPU only."""
import numpy as np
import pytest
from scipy.special import expit

import oracle


def test_round_bf16_ties_and_known_values():
    # 8 significant bits, ties to the even neighbour
    got = oracle.round_bf16([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 3.14159, 0.0,
                             1 + 2 ** -8 + 2 ** -20])
    assert got.tolist() == [1.0, 1.0, 1 + 2 ** -6, -1.0, 3.140625, 0.0, 1 + 2 ** -7]


def test_round_bf16_matches_torch_on_float32_values():
    torch = pytest.importorskip("torch")
    v = np.random.default_rng(3).standard_normal(10000).astype(np.float32) * 100
    ref = torch.from_numpy(v).to(torch.bfloat16).double().numpy()
    assert np.array_equal(oracle.round_bf16(v), ref)


def test_project_hand_worked():
    a = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])          # M = 3, K = 2
    x = np.array([[[[1.0, 2.0]], [[-1.0, 0.5]]]])               # B = 1, K = 2, H = 1, W = 2
    y = oracle.project(a, x)
    assert y.shape == (1, 3, 1, 2)
    assert y[0, :, 0, 0].tolist() == [-1.0, -1.0, -1.0]
    assert y[0, :, 0, 1].tolist() == [3.0, 8.0, 13.0]


def test_latent_single_pixel_hand_worked():
    # one pixel: every direction sees only its first line, h = lambda * x_c
    x = np.array([1.0, 2.0]).reshape(1, 2, 1, 1)
    p_down = np.array([[1.0, 0.0], [1.0, 1.0]])                 # x_c = (1, 3)
    l_u = np.array([[[1.0, 1.0], [0.0, 2.0]],                   # T2B: u = (4, 6)
                    [[0.0, 1.0], [1.0, 0.0]]])                  # L2R: u = (3, 1)
    l_lam = np.array([[[2.0, 0.0], [1.0, -1.0]],                # T2B: lambda = (2, -2)
                      [[1.0, 0.0], [0.0, 1.0]]])                # L2R: lambda = (1, 3)
    l_w = np.random.default_rng(0).standard_normal((2, 2, 3, 2))   # unused on a first line
    p_up = np.array([[1.0, 0.0], [1.0, 1.0]])
    # y_c = (4*2*1 + 3*1*1, 6*(-2)*3 + 1*3*3) = (11, -27); y = (11, -16)
    y = oracle.latent_fwd(x, p_down, l_u, l_lam, l_w, p_up, dirs=1 | 4)
    assert y.reshape(-1).tolist() == [11.0, -16.0]


def test_latent_weights_from_logits_hand_worked():
    # 2 x 2 map, one channel, top-to-bottom only, identity projections:
    # u = lambda = x, tap logits (al, be, ga) * x.  Row 0: y = x^3.
    a, b, c, d = 1.0, 2.0, 0.5, -1.0
    al, be, ga = 0.3, -0.7, 1.1
    x = np.array([[a, b], [c, d]]).reshape(1, 1, 2, 2)
    one = np.ones((1, 1, 1))
    l_w = np.array([al, be, ga]).reshape(1, 1, 3, 1)
    y = oracle.latent_fwd(x, np.ones((1, 1)), one, one, l_w, np.ones((1, 1)), dirs=1)
    h0 = (a * a, b * b)
    # (1, 0): taps 1 and 2 are on the grid
    s1, s2 = expit(be * c), expit(ga * c)
    y10 = c * ((s1 * h0[0] + s2 * h0[1]) / (s1 + s2) + c * c)
    # (1, 1): taps 0 and 1 are on the grid
    s0, s1 = expit(al * d), expit(be * d)
    y11 = d * ((s0 * h0[0] + s1 * h0[1]) / (s0 + s1) + d * d)
    np.testing.assert_allclose(y.reshape(2, 2), [[a ** 3, b ** 3], [y10, y11]], rtol=1e-13)


def _random_sublayer(rng, B=2, C=6, Cc=4, H=5, W=6, dirs=15):
    D = bin(dirs).count("1")
    return dict(x=rng.standard_normal((B, C, H, W)), p_down=rng.standard_normal((Cc, C)),
                l_u=rng.standard_normal((D, Cc, Cc)), l_lam=rng.standard_normal((D, Cc, Cc)),
                l_w=rng.standard_normal((D, Cc, 3, Cc)), p_up=rng.standard_normal((C, Cc)))


def test_latent_invariant_under_latent_channel_permutation():
    rng = np.random.default_rng(1)
    s = _random_sublayer(rng)
    y = oracle.latent_fwd(**s, dirs=15)
    pi = rng.permutation(s["p_down"].shape[0])
    t = dict(x=s["x"], p_down=s["p_down"][pi], l_u=s["l_u"][:, pi][:, :, pi],
             l_lam=s["l_lam"][:, pi][:, :, pi], l_w=s["l_w"][:, pi][:, :, :, pi],
             p_up=s["p_up"][:, pi])
    np.testing.assert_allclose(oracle.latent_fwd(**t, dirs=15), y, rtol=1e-12, atol=1e-12)


def test_latent_equivariant_under_output_channel_permutation_and_linear_in_p_up():
    rng = np.random.default_rng(2)
    s = _random_sublayer(rng, dirs=6)
    y = oracle.latent_fwd(**s, dirs=6)
    pi = rng.permutation(s["p_up"].shape[0])
    t = dict(s, p_up=s["p_up"][pi])
    np.testing.assert_allclose(oracle.latent_fwd(**t, dirs=6), y[:, pi], rtol=1e-12, atol=1e-12)
    t = dict(s, p_up=2.5 * s["p_up"])
    np.testing.assert_allclose(oracle.latent_fwd(**t, dirs=6), 2.5 * y, rtol=1e-12, atol=1e-12)


def test_latent_params_layout_and_normalization():
    rng = np.random.default_rng(4)
    s = _random_sublayer(rng, dirs=9)
    xc = oracle.project(s["p_down"], s["x"])
    prm = oracle.latent_params(xc, s["l_u"], s["l_lam"], s["l_w"], dirs=9)
    B, Cc, H, W = xc.shape
    assert prm["u"].shape == (2, B, Cc, H, W) and prm["w"].shape == (2, B, Cc, 3, H, W)
    # u of direction slot 1 (R2L), channel 2, at pixel (3, 4): row 2 of its L_u
    assert np.isclose(prm["u"][1, 0, 2, 3, 4], s["l_u"][1, 2] @ xc[0, :, 3, 4])
    # taps on the grid sum to one; R2L (slot 1) has no tap 0 on row 0
    wsum = prm["w"].sum(axis=3)
    np.testing.assert_allclose(wsum, 1.0, rtol=1e-12)
    assert np.all(prm["w"][1, :, :, 0, 0, :] == 0.0)
    assert np.all(prm["w"][0, :, :, 2, :, W - 1] == 0.0)   # T2B: no tap 2 in the last column


def test_latent_bf16_storage_is_close_to_float64():
    rng = np.random.default_rng(5)
    s = _random_sublayer(rng, B=1, C=8, Cc=8, H=7, W=7)
    y64 = oracle.latent_fwd(**s, dirs=15)
    y16 = oracle.latent_fwd(**s, dirs=15, storage="bf16")
    scale = np.abs(y64).max()
    assert 0 < np.abs(y16 - y64).max() < 0.05 * scale
