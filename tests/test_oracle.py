"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these tests re-types the oracle's loops.  They check it against
  * the block lower-triangular operator of Sec. 3, Eq. (global), evaluated
    with exact rational arithmetic on tiny grids (recurrence and first line);
  * closed forms: identity propagation gives a lambda-weighted running sum
    along the scan axis; a pure top-left tap gives a diagonal running sum
    (tap orientation, Sec. 3 "top-left, top-center, top-right");
  * the row-stochastic invariant (Sec. 3, Eq. (row_stochastic_norm)): a
    constant injection b gives h_i = (i+1) b;
  * frame identities between the four directions (flips / transposes);
  * the channel-sharing reduction of Sec. 4.2, Eq. (2dsp) (G=1 equals G=C with
    replicated weights);
  * linearity, central finite differences and adjoint identities for the
    backward pass.
All tests run on the CPU.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle

T2B, B2T, L2R, R2L = 1, 2, 4, 8
DIRS = (T2B, B2T, L2R, R2L)


def ndirs(mask):
    return bin(mask).count("1")


def valid_tap_mask(d, H, W):
    """[3, H, W] boolean: tap k of the weight at (row, col) stays inside the grid."""
    m = np.zeros((3, H, W), dtype=bool)
    for k in range(3):
        for r in range(H):
            for c in range(W):
                if d in (T2B, B2T):
                    m[k, r, c] = 0 <= c + k - 1 < W
                else:
                    m[k, r, c] = 0 <= r + k - 1 < H
    return m


def first_line_mask(d, H, W):
    """[H, W] boolean: the pixel lies on the first line scanned by direction d."""
    m = np.zeros((H, W), dtype=bool)
    if d == T2B:
        m[0, :] = True
    elif d == B2T:
        m[H - 1, :] = True
    elif d == L2R:
        m[:, 0] = True
    else:
        m[:, W - 1] = True
    return m


def random_problem(rng, B, C, G, H, W, dirs, garbage=True):
    """Random fp64 inputs; ignored taps hold large garbage values when asked."""
    D = ndirs(dirs)
    x = rng.standard_normal((B, C, H, W))
    lam = rng.standard_normal((D, B, C, H, W))
    u = rng.standard_normal((D, B, C, H, W))
    w = np.empty((D, B, G, 3, H, W))
    for s, d in enumerate([d for d in DIRS if dirs & d]):
        m = valid_tap_mask(d, H, W)
        raw = rng.uniform(0.1, 1.0, size=(B, G, 3, H, W)) * m
        raw /= raw.sum(axis=2, keepdims=True)
        if garbage:
            junk = rng.uniform(-1e3, 1e3, size=raw.shape)
            raw = np.where(m, raw, junk)
            raw = np.where(first_line_mask(d, H, W)[None, None, None], junk, raw)
        w[s] = raw
    return x, w, lam, u


# ---------------------------------------------------------------------------
# frame maps between a direction and the top-to-bottom frame (test-side)
# ---------------------------------------------------------------------------

def to_t2b(d, a):
    """Re-index a [..., H, W] tensor so that direction d becomes top-to-bottom."""
    if d == T2B:
        return a
    if d == B2T:
        return a[..., ::-1, :]
    if d == L2R:
        return np.swapaxes(a, -1, -2)
    return np.swapaxes(a[..., :, ::-1], -1, -2)


def from_t2b(d, a):
    if d == T2B:
        return a
    if d == B2T:
        return a[..., ::-1, :]
    if d == L2R:
        return np.swapaxes(a, -1, -2)
    return np.swapaxes(a, -1, -2)[..., :, ::-1]


# ---------------------------------------------------------------------------
# Eq. (global): dense block lower-triangular operator, exact rationals
# ---------------------------------------------------------------------------

def _frac_matmul(A, B):
    n, m, p = len(A), len(B), len(B[0])
    return [[sum((A[i][k] * B[k][j] for k in range(m)), Fraction(0)) for j in range(p)]
            for i in range(n)]


def dense_t2b_states(x, lam, w):
    """h for one top-to-bottom scan of one channel via H_v = G X_v.

    x, lam: [L][P] Fractions; w: [L][P][3] Fractions (taps outside the grid
    are never read).  Block G_ij = (w_i w_{i-1} ... w_{j+1}) Lambda_j for j <= i.
    """
    L, P = len(x), len(x[0])
    ident = [[Fraction(int(a == b)) for b in range(P)] for a in range(P)]

    def wmat(i):
        M = [[Fraction(0)] * P for _ in range(P)]
        for j in range(P):
            for k in range(3):
                jj = j + k - 1
                if 0 <= jj < P:
                    M[j][jj] = w[i][j][k]
        return M

    h = []
    for i in range(L):
        hi = [Fraction(0)] * P
        for j in range(i + 1):
            prod = ident
            for tau in range(j + 1, i + 1):
                prod = _frac_matmul(wmat(tau), prod)
            lamx = [[lam[j][p] * x[j][p]] for p in range(P)]
            contrib = _frac_matmul(prod, lamx)
            hi = [hi[p] + contrib[p][0] for p in range(P)]
        h.append(hi)
    return h


def _rand_frac(rng, lo, hi, den=8):
    return Fraction(int(rng.integers(lo * den, hi * den + 1)), den)


@pytest.mark.parametrize("d", DIRS)
@pytest.mark.parametrize("H,W", [(3, 4), (4, 3), (1, 3), (3, 1)])
def test_dense_operator_exact(d, H, W):
    """Every direction equals Eq. (global) evaluated exactly in the t2b frame."""
    rng = np.random.default_rng(100 + d * 7 + H * 3 + W)
    xs = np.array([[_rand_frac(rng, -3, 3) for _ in range(W)] for _ in range(H)], dtype=object)
    ls = np.array([[_rand_frac(rng, -2, 2) for _ in range(W)] for _ in range(H)], dtype=object)
    ws = np.array([[[_rand_frac(rng, 0, 1, 16) for _ in range(W)] for _ in range(H)]
                   for _ in range(3)], dtype=object)               # [3][H][W]
    # the oracle, u = 1 and a single direction: y = h
    x = xs.astype(np.float64)[None, None]
    lam = ls.astype(np.float64)[None, None, None]
    w = ws.astype(np.float64)[None, None, None]
    u = np.ones_like(lam)
    y = oracle.scan_fwd(x, w, lam, u, d)[0, 0]
    # the dense operator in the t2b frame
    xf, lf = to_t2b(d, xs), to_t2b(d, ls)
    wf = np.stack([to_t2b(d, ws[k]) for k in range(3)], axis=-1)  # [L][P][3]
    L, P = xf.shape
    h = dense_t2b_states([[xf[i][j] for j in range(P)] for i in range(L)],
                         [[lf[i][j] for j in range(P)] for i in range(L)],
                         [[[wf[i][j][k] for k in range(3)] for j in range(P)] for i in range(L)])
    expect = from_t2b(d, np.array([[float(v) for v in row] for row in h]))
    np.testing.assert_allclose(y, expect, rtol=1e-13, atol=1e-13)


def test_dense_operator_four_directions_grouped():
    """Merged 4-direction output with G < C equals the sum of dense scans."""
    rng = np.random.default_rng(7)
    B, C, G, H, W = 1, 4, 2, 3, 3
    x, w, lam, u = random_problem(rng, B, C, G, H, W, 15)
    y = oracle.scan_fwd(x, w, lam, u, 15)
    expect = np.zeros_like(y)
    for s, d in enumerate(DIRS):
        for c in range(C):
            g = c // (C // G)
            xf = to_t2b(d, x[0, c])
            lf = to_t2b(d, lam[s, 0, c])
            wf = np.stack([to_t2b(d, w[s, 0, g, k]) for k in range(3)], axis=-1)
            L, P = xf.shape
            h = dense_t2b_states([[Fraction(float(v)) for v in row] for row in xf],
                                 [[Fraction(float(v)) for v in row] for row in lf],
                                 [[[Fraction(float(wf[i, j, k])) for k in range(3)]
                                   for j in range(P)] for i in range(L)])
            hs = from_t2b(d, np.array([[float(v) for v in row] for row in h]))
            expect[0, c] += u[s, 0, c] * hs
    np.testing.assert_allclose(y, expect, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------------------
# closed forms and invariants
# ---------------------------------------------------------------------------

def _cumsum_scan(d, a):
    """Running sum along the scan axis of direction d, in scan order."""
    if d == T2B:
        return np.cumsum(a, axis=-2)
    if d == B2T:
        return np.cumsum(a[..., ::-1, :], axis=-2)[..., ::-1, :]
    if d == L2R:
        return np.cumsum(a, axis=-1)
    return np.cumsum(a[..., :, ::-1], axis=-1)[..., :, ::-1]


@pytest.mark.parametrize("dirs", [1, 2, 4, 8, 15, 5, 10])
def test_identity_weights_give_running_sum(dirs):
    rng = np.random.default_rng(dirs)
    B, C, G, H, W = 2, 6, 3, 7, 9
    x, w, lam, u = random_problem(rng, B, C, G, H, W, dirs)
    w[:] = 0.0
    w[:, :, :, 1] = 1.0
    # garbage on the ignored first line must not matter
    for s, d in enumerate([d for d in DIRS if dirs & d]):
        w[s][..., first_line_mask(d, H, W)] = 123.0
    y = oracle.scan_fwd(x, w, lam, u, dirs)
    expect = np.zeros_like(y)
    for s, d in enumerate([d for d in DIRS if dirs & d]):
        expect += u[s] * _cumsum_scan(d, lam[s] * x)
    np.testing.assert_allclose(y, expect, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d", DIRS)
def test_top_left_tap_gives_diagonal_sum(d):
    """Only tap 0 set: h_i[j] = sum_{t <= min(i, j)} (lam x)[i-t][j-t] in the scan frame."""
    rng = np.random.default_rng(11 + d)
    B, C, G, H, W = 1, 2, 1, 6, 5
    x, w, lam, u = random_problem(rng, B, C, G, H, W, d, garbage=False)
    w[:] = 0.0
    w[:, :, :, 0] = 1.0
    u[:] = 1.0
    y = oracle.scan_fwd(x, w, lam, u, d)
    lx = to_t2b(d, lam[0] * x)                     # [B, C, L, P]
    L, P = lx.shape[-2:]
    expect = np.zeros_like(lx)
    for i in range(L):
        for j in range(P):
            for t in range(min(i, j) + 1):
                expect[..., i, j] += lx[..., i - t, j - t]
    np.testing.assert_allclose(y, from_t2b(d, expect), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d", DIRS)
def test_row_stochastic_constant_injection(d):
    """Rows of w sum to 1 and lam x = b everywhere  =>  h_i = (i+1) b."""
    rng = np.random.default_rng(21 + d)
    B, C, G, H, W = 1, 3, 1, 8, 6
    x, w, lam, u = random_problem(rng, B, C, G, H, W, d)
    b = 0.75
    lam[:] = 1.0
    x[:] = b
    y = oracle.scan_fwd(x, w, lam, u, d)
    steps = to_t2b(d, np.zeros((H, W)))
    idx = np.arange(steps.shape[0])[:, None] + np.zeros_like(steps)
    expect = u[0] * from_t2b(d, (idx + 1) * b)
    np.testing.assert_allclose(y, expect, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("d", [B2T, L2R, R2L])
def test_direction_frames_reduce_to_top_to_bottom(d):
    """A direction on the inputs equals top-to-bottom on re-indexed inputs."""
    rng = np.random.default_rng(31 + d)
    B, C, G, H, W = 2, 4, 2, 5, 7
    x, w, lam, u = random_problem(rng, B, C, G, H, W, d)
    y = oracle.scan_fwd(x, w, lam, u, d)
    xt = np.ascontiguousarray(to_t2b(d, x))
    wt = np.ascontiguousarray(to_t2b(d, w))
    lt = np.ascontiguousarray(to_t2b(d, lam))
    ut = np.ascontiguousarray(to_t2b(d, u))
    yt = oracle.scan_fwd(xt, wt, lt, ut, T2B)
    np.testing.assert_allclose(y, from_t2b(d, yt), rtol=1e-12, atol=1e-12)


def test_shared_weights_equal_replicated_per_channel_weights():
    """Eq. (2dsp): G = 1 is the per-channel recurrence with identical w_c."""
    rng = np.random.default_rng(41)
    B, C, H, W = 2, 6, 6, 5
    x, w1, lam, u = random_problem(rng, B, C, 1, H, W, 15)
    wC = np.repeat(w1, C, axis=2)
    np.testing.assert_allclose(oracle.scan_fwd(x, w1, lam, u, 15),
                               oracle.scan_fwd(x, wC, lam, u, 15), rtol=1e-13, atol=1e-13)
    # and an intermediate grouping
    w3 = np.repeat(w1, 3, axis=2)
    np.testing.assert_allclose(oracle.scan_fwd(x, w1, lam, u, 15),
                               oracle.scan_fwd(x, w3, lam, u, 15), rtol=1e-13, atol=1e-13)


def test_single_row_and_single_column():
    rng = np.random.default_rng(51)
    # H = 1: vertical scans are one step, h_0 = lam x.
    x, w, lam, u = random_problem(rng, 1, 3, 1, 1, 6, T2B | B2T)
    y = oracle.scan_fwd(x, w, lam, u, T2B | B2T)
    np.testing.assert_allclose(y, (u[0] * lam[0] + u[1] * lam[1]) * x, rtol=1e-13)
    # W = 1 (line length 1) for vertical scans: only the centre tap is valid;
    # with the generator's renormalisation it is 1 -> running sum.
    x, w, lam, u = random_problem(rng, 1, 3, 1, 6, 1, T2B)
    w[:, :, :, 1] = 1.0
    y = oracle.scan_fwd(x, w, lam, u, T2B)
    np.testing.assert_allclose(y, u[0] * np.cumsum(lam[0] * x, axis=-2), rtol=1e-13)


def test_linear_in_x():
    rng = np.random.default_rng(61)
    x1, w, lam, u = random_problem(rng, 2, 4, 2, 6, 5, 15)
    x2 = rng.standard_normal(x1.shape)
    a, b = 0.7, -1.3
    lhs = oracle.scan_fwd(a * x1 + b * x2, w, lam, u, 15)
    rhs = a * oracle.scan_fwd(x1, w, lam, u, 15) + b * oracle.scan_fwd(x2, w, lam, u, 15)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-11, atol=1e-11)


# ---------------------------------------------------------------------------
# backward
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dirs,shape", [(15, (1, 4, 2, 4, 3)), (15, (1, 2, 1, 3, 5)),
                                        (T2B | L2R, (2, 2, 2, 3, 3)), (R2L, (1, 1, 1, 4, 4))])
def test_backward_matches_central_differences(dirs, shape):
    B, C, G, H, W = shape
    rng = np.random.default_rng(71 + dirs + H)
    x, w, lam, u = random_problem(rng, B, C, G, H, W, dirs)
    r = rng.standard_normal((B, C, H, W))
    grads = oracle.scan_bwd(x, w, lam, u, r, dirs)
    params = {"x": x, "w": w, "lam": lam, "u": u}
    eps = 1e-6

    def loss(p):
        return float(np.sum(oracle.scan_fwd(p["x"], p["w"], p["lam"], p["u"], dirs) * r))

    for name, arr in params.items():
        fd = np.zeros_like(arr)
        flat = arr.reshape(-1)
        for i in range(flat.size):
            old = flat[i]
            flat[i] = old + eps
            lp = loss(params)
            flat[i] = old - eps
            lm = loss(params)
            flat[i] = old
            fd.reshape(-1)[i] = (lp - lm) / (2 * eps)
        g = grads["d" + name]
        scale = max(1.0, np.abs(fd).max())
        assert np.abs(g - fd).max() <= 1e-6 * scale, name
    # ignored taps (outside the grid, first line) have exactly zero gradient
    for s, d in enumerate([d for d in DIRS if dirs & d]):
        ignored = ~valid_tap_mask(d, H, W) | first_line_mask(d, H, W)[None]
        assert np.all(grads["dw"][s][:, :, ignored] == 0.0)


def test_backward_adjoint_identities():
    """y is linear in x, in each lam_d and in each u_d separately."""
    rng = np.random.default_rng(81)
    B, C, G, H, W = 2, 8, 2, 12, 10
    x, w, lam, u = random_problem(rng, B, C, G, H, W, 15)
    dy = rng.standard_normal((B, C, H, W))
    y = oracle.scan_fwd(x, w, lam, u, 15)
    g = oracle.scan_bwd(x, w, lam, u, dy, 15)
    ydy = float(np.sum(y * dy))
    assert abs(ydy - float(np.sum(x * g["dx"]))) <= 1e-10 * abs(ydy) + 1e-10
    # h_d is linear in lam_d and y in u_d, one direction at a time
    for s in range(4):
        ys = u[s] * (oracle.scan_fwd(x, w[s:s + 1], lam[s:s + 1], np.ones_like(u[s:s + 1]),
                                     DIRS[s]))
        ref = float(np.sum(ys * dy))
        assert abs(ref - float(np.sum(lam[s] * g["dlam"][s]))) <= 1e-10 * abs(ref) + 1e-10
        assert abs(ref - float(np.sum(u[s] * g["du"][s]))) <= 1e-10 * abs(ref) + 1e-10
    # a directional derivative along w
    v = rng.standard_normal(w.shape)
    eps = 1e-6
    lp = float(np.sum(oracle.scan_fwd(x, w + eps * v, lam, u, 15) * dy))
    lm = float(np.sum(oracle.scan_fwd(x, w - eps * v, lam, u, 15) * dy))
    fd = (lp - lm) / (2 * eps)
    assert abs(fd - float(np.sum(g["dw"] * v))) <= 1e-6 * max(1.0, abs(fd))


def test_group_slice_is_self_contained():
    """Outputs of one (batch, group) unit depend only on that unit's inputs."""
    rng = np.random.default_rng(91)
    B, C, G, H, W = 3, 6, 3, 5, 4
    x, w, lam, u = random_problem(rng, B, C, G, H, W, 15)
    dy = rng.standard_normal((B, C, H, W))
    full_y = oracle.scan_fwd(x, w, lam, u, 15)
    full_g = oracle.scan_bwd(x, w, lam, u, dy, 15)
    inputs = {"x": x, "w": w, "lam": lam, "u": u, "dy": dy}
    b, g = 2, 1
    sl = oracle.slice_group(inputs, b, g, G)
    cs = slice(g * 2, g * 2 + 2)
    np.testing.assert_array_equal(oracle.scan_fwd(sl["x"], sl["w"], sl["lam"], sl["u"], 15),
                                  full_y[b:b + 1, cs])
    part = oracle.scan_bwd(sl["x"], sl["w"], sl["lam"], sl["u"], sl["dy"], 15)
    np.testing.assert_array_equal(part["dx"], full_g["dx"][b:b + 1, cs])
    np.testing.assert_array_equal(part["dw"], full_g["dw"][:, b:b + 1, g:g + 1])
    np.testing.assert_array_equal(part["dlam"], full_g["dlam"][:, b:b + 1, cs])


# ---------------------------------------------------------------------------
# weights from logits, Sec. 3, Eq. (row_stochastic_norm)
# ---------------------------------------------------------------------------

def _logits(rng, dirs, B, G, H, W, scale=1.0):
    return rng.standard_normal((ndirs(dirs), B, G, 3, H, W)) * scale


@pytest.mark.parametrize("d", DIRS)
def test_norm_equal_logits_closed_form(d):
    # equal logits: every tap of N(j) gets 1 / |N(j)| (1/3 inside, 1/2 at the
    # ends of a line), taps off the grid get 0
    H, W = 4, 5
    w = oracle.normalize_w(np.full((1, 2, 1, 3, H, W), 0.7), d)
    m = valid_tap_mask(d, H, W)
    expect = m / m.sum(axis=0, keepdims=True)
    assert np.allclose(w[0, 0, 0], expect, rtol=0, atol=1e-15)
    assert np.allclose(w[0, 1, 0], expect, rtol=0, atol=1e-15)


@pytest.mark.parametrize("dirs", [1, 6, 15])
def test_norm_rows_sum_to_one_and_ratios_are_sigmoid_ratios(dirs):
    from scipy.special import expit
    rng = np.random.default_rng(11)
    H, W = 5, 7
    wt = _logits(rng, dirs, 2, 3, H, W, scale=2.0)
    w = oracle.normalize_w(wt, dirs)
    for s, d in enumerate([d for d in DIRS if dirs & d]):
        m = valid_tap_mask(d, H, W)
        ws = w[s]
        assert np.all(ws[:, :, ~m] == 0.0)
        assert np.allclose(ws.sum(axis=2), 1.0, rtol=0, atol=1e-14)
        # w_k / w_1 = sigma(wt_k) / sigma(wt_1) (the centre tap is always on the grid)
        sg = expit(wt[s])
        for k in (0, 2):
            r = np.where(m[k], ws[:, :, k] / ws[:, :, 1], 0.0)
            e = np.where(m[k], sg[:, :, k] / sg[:, :, 1], 0.0)
            assert np.allclose(r, e, rtol=1e-13, atol=0)


def test_norm_saturated_neighbours_give_one_weight():
    # two taps with very negative logits: the third carries the whole row
    H, W = 3, 4
    wt = np.full((1, 1, 1, 3, H, W), -800.0)
    wt[0, 0, 0, 1] = 0.3
    w = oracle.normalize_w(wt, T2B)
    assert np.allclose(w[0, 0, 0, 1], 1.0, rtol=0, atol=1e-15)
    assert np.all(np.abs(w[0, 0, 0, 0]) < 1e-300) and np.all(np.abs(w[0, 0, 0, 2]) < 1e-300)


def test_norm_clamp_reading():
    # every sigmoid of N(j) far below 1e-30: the denominator is held at 1e-30,
    # so the row no longer sums to one (the reading of the unstated clamp)
    from scipy.special import expit
    wt = np.full((1, 1, 1, 3, 2, 3), -80.0)
    w = oracle.normalize_w(wt, T2B)
    m = valid_tap_mask(T2B, 2, 3)
    assert np.allclose(w[0, 0, 0][m], expit(-80.0) / 1e-30, rtol=1e-12, atol=0)
    # just above the clamp the row sums to one again
    w2 = oracle.normalize_w(np.full((1, 1, 1, 3, 2, 3), -60.0), T2B)
    assert np.allclose(w2[0, 0, 0].sum(axis=0), 1.0, rtol=0, atol=1e-14)


@pytest.mark.parametrize("dirs,scale", [(15, 1.5), (5, 3.0), (2, 1.0)])
def test_norm_backward_matches_central_differences(dirs, scale):
    rng = np.random.default_rng(5)
    H, W = 3, 4
    wt = _logits(rng, dirs, 1, 2, H, W, scale)
    dw = rng.standard_normal(wt.shape)
    g = oracle.normalize_w_bwd(wt, dw, dirs)
    eps = 1e-6
    for idx in [tuple(rng.integers(0, n) for n in wt.shape) for _ in range(40)]:
        wp, wm = wt.copy(), wt.copy()
        wp[idx] += eps
        wm[idx] -= eps
        fd = (np.sum(dw * oracle.normalize_w(wp, dirs)) -
              np.sum(dw * oracle.normalize_w(wm, dirs))) / (2 * eps)
        assert abs(fd - g[idx]) < 1e-7 * (1 + abs(fd)), (idx, fd, g[idx])


def test_norm_backward_under_the_clamp_matches_central_differences():
    rng = np.random.default_rng(6)
    wt = -75.0 + 0.5 * rng.standard_normal((1, 1, 1, 3, 2, 3))
    dw = rng.standard_normal(wt.shape)
    g = oracle.normalize_w_bwd(wt, dw, T2B)
    eps = 1e-4
    for idx in np.ndindex(*wt.shape):
        wp, wm = wt.copy(), wt.copy()
        wp[idx] += eps
        wm[idx] -= eps
        fd = (np.sum(dw * oracle.normalize_w(wp, T2B)) -
              np.sum(dw * oracle.normalize_w(wm, T2B))) / (2 * eps)
        assert abs(fd - g[idx]) <= 1e-6 * (abs(fd) + abs(g[idx])) + 1e-300, (idx, fd, g[idx])
