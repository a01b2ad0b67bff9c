"""Pins for the oracle's learnable modulation and softened ternarization.

Each check ties the oracle to something other than itself: 50-digit mpmath
evaluations of Eq. 5 and its derivatives, the limits and properties the paper
states for f (Sec. 2.3), closed forms on hand-built groups (Eq. 3), exact
rational evaluation of Eq. 2, BitNet's absmean rule as the special case of
identity modulation (Sec. 2.2), finite differences of the forward for the
factor gradients, and a hand-computed packed byte.
"""
from fractions import Fraction

import mpmath
import numpy as np
import pytest

from oracle import lmst

mpmath.mp.dps = 50


def mp_f(x, s, D):
    """Eq. 5 at 50 significant digits; inside the dead zone the two tanh
    terms cancel to within exp(-2 s |x - D|), so the working precision is
    raised until the difference is resolved."""
    def ev():
        xx, ss, DD = mpmath.mpf(x), mpmath.mpf(s), mpmath.mpf(D)
        return (mpmath.tanh(ss * (xx - DD)) + mpmath.tanh(ss * (xx + DD))) / (2 * mpmath.tanh(ss))
    extra = int(4 * float(s) * (abs(float(D)) + abs(float(x))) / 2.3) + 10
    with mpmath.workdps(max(mpmath.mp.dps, 50) + extra):
        v = ev()
    return v


def rel(a, b):
    a, b = float(a), float(b)
    if b == 0:
        return abs(a)
    return abs(a - b) / abs(b)


GRID_S = [0.05, 0.625, 1.0, 3.75, 7.0, 15.0, 30.0, 100.0]
GRID_D = [0.05, 0.5, 0.9, 1.5]
GRID_X = [-5.0, -1.3, -0.5, -0.49, -1e-3, 0.0, 1e-6, 0.01, 0.3, 0.49999, 0.5, 0.50001, 0.7, 2.0]


def test_f_matches_mpmath():
    worst = 0.0
    for s in GRID_S:
        for D in GRID_D:
            xs = np.array(GRID_X)
            f = lmst.transition(xs, s, D)
            for x, v in zip(xs, f):
                ref = mp_f(x, s, D)
                if ref == 0:
                    assert v == 0
                    continue
                worst = max(worst, rel(v, ref))
    assert worst < 1e-13, worst


def test_derivatives_match_mpmath():
    worst = 0.0
    for s in [0.3, 3.75, 15.0, 30.0]:
        for D in [0.25, 0.5, 1.2]:
            xs = np.array([-1.1, -0.4, 0.05, 0.45, 0.55, 1.3])
            _, fW, fD = lmst.transition_parts(xs, s, D)
            for x, a, b in zip(xs, fW, fD):
                rW = mpmath.diff(lambda t: mp_f(t, s, D), x)
                rD = mpmath.diff(lambda t: mp_f(x, s, t), D)
                worst = max(worst, rel(a, rW), rel(b, rD) if abs(rD) > 1e-300 else 0)
    assert worst < 1e-12, worst


def test_naive_formula_cancels_but_stable_does_not():
    # the paper's formula evaluated directly loses digits inside the dead zone
    x, s, D = 0.01, 30.0, 0.5
    naive = (np.tanh(s * (x - D)) + np.tanh(s * (x + D))) / (2 * np.tanh(s))
    ref = mp_f(x, s, D)
    assert rel(naive, ref) > 1e-6
    assert rel(lmst.transition(np.array([x]), s, D)[0], ref) < 1e-13


def test_f_odd_and_monotone():
    pos = np.linspace(0, 3, 1001)[1:]
    xs = np.concatenate([-pos[::-1], [0.0], pos])           # exactly symmetric grid
    for s in [0.1, 1, 4.95, 30]:
        f, fW, fD = lmst.transition_parts(xs, s, 0.5)
        np.testing.assert_array_equal(f, -f[::-1])          # odd (Sec. 2.3, property 1)
        assert np.all(fW > 0)                                # increasing in W
        assert np.all(np.diff(f) >= 0)
        np.testing.assert_array_equal(fD, -fD[::-1])


def test_small_s_gives_identity():
    # property (2): s -> 0 approaches the identity mapping
    xs = np.array([-0.9, -0.3, 0.0, 0.3, 0.7])
    f = lmst.transition(xs, 1e-6, 0.5)
    np.testing.assert_allclose(f, xs, rtol=0, atol=1e-10)
    assert abs(lmst.transition(np.array([0.3]), 1e-6, 0.5)[0] - 0.3) < 1e-12


def test_large_s_gives_hard_ternarization():
    # property (4): s -> inf approaches Q of Eq. 2 away from |W| = Delta
    xs = np.array([-2.0, -0.6, -0.4, 0.0, 0.2, 0.45, 0.55, 1.7])
    Q = np.where(xs > 0.5, 1.0, np.where(xs < -0.5, -1.0, 0.0))
    np.testing.assert_allclose(lmst.transition(xs, 1e4, 0.5), Q, atol=1e-12)
    # on the boundary the limit is +-1/2
    np.testing.assert_allclose(lmst.transition(np.array([-0.5, 0.5]), 1e4, 0.5), [-0.5, 0.5],
                               atol=1e-12)


def test_sharpness_increases_with_s():
    # property (3): as s grows the curve gets steeper (largest slope grows)
    # and moves monotonically toward the hard ternarization of Eq. 2
    xs = np.linspace(-2, 2, 40001)
    Q = np.where(xs > 0.5, 1.0, np.where(xs < -0.5, -1.0, 0.0))
    prev_slope, prev_dist = 0.0, np.inf
    for s in [0.05, 0.5, 1, 2, 4, 8, 16, 30, 60]:
        f, fW, _ = lmst.transition_parts(xs, s, 0.5)
        slope, dist = fW.max(), np.abs(f - Q).mean()
        assert slope > prev_slope and dist < prev_dist
        prev_slope, prev_dist = slope, dist
    # the steepest point sits on the threshold with slope ~ s/2 for large s
    assert abs(prev_slope - 30.0) < 1e-9


def test_output_bound_is_coth():
    # sup f = coth(s); the paper's "within [-1, 1] at s = 4.95" holds to 1e-4
    for s in [1.0, 4.95, 10.0]:
        big = lmst.transition(np.array([60.0 / s]), s, 0.5)[0]
        assert rel(big, 1 / np.tanh(s)) < 1e-14
    assert abs((1 / np.tanh(4.95) - 1) - 1.0035e-4) < 1e-7
    assert 1 / np.tanh(4.9518) - 1 <= 1.0e-4 + 1e-9


def test_f_at_one_never_exceeds_one():
    for s in np.linspace(0.05, 100, 400):
        assert lmst.transition(np.array([1.0]), s, 0.5)[0] <= 1.0 + 1e-15


# ---------------------------------------------------------------- statistics

def test_stats_closed_forms():
    a = 0.03125
    # (i) 64 x (+a) and 64 x (-a): mu0 = 0, alpha0 = a
    W = np.array([a] * 64 + [-a] * 64).reshape(1, 128)
    mu0, al0 = lmst.group_stats(W)
    assert mu0[0] == 0 and al0[0] == a
    # (ii) {3,1,-1,-3} repeated: mu0 = 0, alpha0 = 2, W_hat = W/2
    W2 = np.tile([3.0, 1.0, -1.0, -3.0], 32).reshape(1, 128)
    mu0, al0 = lmst.group_stats(W2)
    assert mu0[0] == 0 and al0[0] == 2
    r = lmst.modulate_ternarize(W2, 128, 0.0, 1.0, 1.0, lmst.HARD)
    # W_hat = {1.5, .5, -.5, -1.5} and Delta = .5: the ties at +-.5 give 0
    np.testing.assert_array_equal(r["codes"][0, :4], [1, 0, 0, -1])
    # (iii) shifting by c moves mu0 by c and leaves alpha0 and the codes alone
    W3 = W2 + 8.0
    mu3, al3 = lmst.group_stats(W3)
    assert mu3[0] == 8.0 and al3[0] == 2.0
    r3 = lmst.modulate_ternarize(W3, 128, 0.0, 1.0, 1.0, lmst.HARD)
    np.testing.assert_array_equal(r3["codes"], r["codes"])
    # (iv) a constant group: alpha0 = 0, codes 0, fake weight 0, finite
    W4 = np.full((1, 128), 0.25)
    r4 = lmst.modulate_ternarize(W4, 128, 0.2, 1.0, 1.0, lmst.HARD)
    assert r4["alpha0"][0] == 0
    assert np.all(r4["codes"] == 0) and np.all(r4["W_fake"] == 0)
    r5 = lmst.modulate_ternarize(W4, 128, 0.2, 1.0, 1.0, lmst.SOFT, s=30.0)
    assert np.all(r5["W_fake"] == 0)


def test_stats_equal_plain_mean_on_random():
    rng = np.random.default_rng(1)
    W = rng.standard_normal((64, 512)) * 0.02
    W = W.astype(np.float32).astype(np.float64)
    for g in (16, 64, 128, 256, 512):
        mu0, al0 = lmst.group_stats(W, g)
        Wg = W.reshape(-1, g)
        np.testing.assert_allclose(mu0, Wg.mean(1), rtol=1e-6, atol=1e-12)
        np.testing.assert_allclose(al0, np.abs(Wg - mu0[:, None]).mean(1), rtol=1e-6)


def test_canonical_sum_order():
    # the fixed order is pairwise; check it on values whose sum depends on order
    x = np.zeros(128)
    x[0], x[4], x[64] = 1e16, 1.0, -1e16
    # (0,4) pair first: 1e16 + 1 rounds to 1e16; then + (-1e16) -> 0
    assert lmst.canonical_sum(x) == 0.0
    y = np.arange(128, dtype=np.float64)
    assert lmst.canonical_sum(y) == y.sum()


def test_absmean_special_case():
    # identity modulation on a zero-mean group is BitNet's absmean rule:
    # alpha = mean|W|, T = RoundClip(W/alpha, -1, 1) (round half to even)
    rng = np.random.default_rng(7)
    half = rng.standard_normal((32, 64)) * 0.02
    half = half.astype(np.float32).astype(np.float64)
    W = np.concatenate([half, -half[:, ::-1]], axis=1)    # each row sums to exactly 0
    r = lmst.modulate_ternarize(W, 128, 0.0, 1.0, 1.0, lmst.HARD)
    assert np.all(r["mu0"] == 0)
    gam = np.abs(W).mean(1)
    np.testing.assert_allclose(r["alpha"], gam, rtol=1e-7)
    ref = np.clip(np.round(W / r["alpha"][:, None]), -1, 1)
    np.testing.assert_array_equal(r["codes"], ref)


# ---------------------------------------------------------------- hard codes

def test_hard_codes_exact_rational():
    rng = np.random.default_rng(3)
    W = rng.standard_normal((4, 128)).astype(np.float32).astype(np.float64) * 0.02
    for dmu, dal, dde in [(0.0, 1.0, 1.0), (0.3, 0.7, 1.4), (-0.8, 2.0, 0.3)]:
        r = lmst.modulate_ternarize(W, 128, dmu, dal, dde, lmst.HARD)
        codes = r["codes"].reshape(-1, 128)
        for j in range(codes.shape[0]):
            mu = Fraction(r["mu"][j])
            al = Fraction(r["alpha"][j])
            D = Fraction(r["delta"][j])
            for i in range(128):
                wh = (Fraction(W.reshape(-1, 128)[j, i]) - mu) / al
                q = 1 if wh > D else (-1 if wh < -D else 0)
                assert codes[j, i] == q


def test_hard_outputs_are_ternary_times_scale():
    rng = np.random.default_rng(5)
    W = rng.standard_normal((8, 256)) * 0.02
    r = lmst.modulate_ternarize(W, 128, 0.1, 1.2, 0.8, lmst.HARD)
    assert set(np.unique(r["codes"])) <= {-1, 0, 1}
    Wf = r["W_fake"].reshape(-1, 128)
    al = r["alpha"][:, None]
    assert np.all((Wf == 0) | (Wf == al) | (Wf == -al))


def test_modulation_formula():
    # Eq. 3-4 on one group with simple numbers
    mu, al, de = lmst.modulation(np.array([0.5]), np.array([2.0]), np.array([0.25]),
                                 np.array([1.5]), np.array([0.75]), 0.5)
    assert mu[0] == 1.0 and al[0] == 3.0 and de[0] == 0.375


def test_identity_mode_returns_w():
    W = np.random.default_rng(2).standard_normal((2, 128))
    r = lmst.modulate_ternarize(W, 128, 0.3, 0.5, 2.0, lmst.IDENTITY)
    np.testing.assert_array_equal(r["W_fake"], W)


# --------------------------------------------------------------- gradients

def _objective(G, W, g, fac, mode, s, strides=(1, 1, 1)):
    r = lmst.modulate_ternarize(W, g, fac[0], fac[1], fac[2], mode, s=s, strides=strides)
    return float(np.sum(G * r["W_fake"]))


@pytest.mark.parametrize("s", [0.7, 7.0, 30.0])
def test_factor_grads_finite_differences(s):
    rng = np.random.default_rng(11)
    W = rng.standard_normal((2, 256)) * 0.02
    G = rng.standard_normal(W.shape)
    n = 4
    fac = [rng.uniform(-0.3, 0.3, n), np.exp(rng.uniform(-0.3, 0.3, n)),
           np.exp(rng.uniform(-0.3, 0.3, n))]
    ga = lmst.factor_grads(G, W, 128, *fac, lmst.SOFT, s=s)
    for which in range(3):
        for j in range(n):
            h = 1e-6
            fp = [f.copy() for f in fac]
            fm = [f.copy() for f in fac]
            fp[which][j] += h
            fm[which][j] -= h
            # modulation rounds mu, alpha, Delta to fp32; use unrounded fp64
            # factors through a finite step large against that rounding
            num = (_objective_exact(G, W, fp, s) - _objective_exact(G, W, fm, s)) / (2 * h)
            assert abs(num - ga[which][j]) <= 1e-6 * max(1.0, abs(num)), (which, j, num, ga[which][j])


def _objective_exact(G, W, fac, s, g=128):
    """Same forward in plain float64 without the fp32 rounding of the
    per-group scalars (a smooth function of the factors)."""
    Wg = W.reshape(-1, g)
    mu0, al0 = lmst.group_stats(W, g)
    mu = mu0 + fac[0] * al0
    al = fac[1] * al0
    D = fac[2] * 0.5
    xh = (Wg - mu[:, None]) / al[:, None]
    T = lmst.transition(xh, s, D[:, None])
    return float(np.sum(G.reshape(-1, g) * al[:, None] * T))


def test_factor_grads_shared_is_sum():
    rng = np.random.default_rng(12)
    W = rng.standard_normal((2, 256)) * 0.02
    G = rng.standard_normal(W.shape)
    per = lmst.factor_grads(G, W, 128, np.zeros(4), np.ones(4), np.ones(4), lmst.SOFT, s=5.0)
    sh = lmst.factor_grads(G, W, 128, np.zeros(1), np.ones(1), np.ones(1), lmst.SOFT, s=5.0,
                           strides=(0, 0, 0))
    for a, b in zip(per, sh):
        assert abs(a.sum() - b[0]) < 1e-12 * max(1, abs(b[0]))


def test_hard_ste_closed_form():
    # s_bwd = 0: f_W = 1, f_D = 0, so dmu = -alpha0 sum G and
    # dalpha = alpha0 (sum G T - sum G W_hat), dDelta = 0
    W = np.tile([3.0, 1.0, -1.0, -3.0], 32).reshape(1, 128) * 2.0 ** -6   # exact values
    G = np.tile([1.0, 2.0, 0.5, -1.0], 32).reshape(1, 128)
    gm, ga, gd = lmst.factor_grads(G, W, 128, 0.0, 1.0, 1.0, lmst.HARD, s_bwd=0.0)
    al0 = 2.0 * 2.0 ** -6
    wh = np.tile([1.5, 0.5, -0.5, -1.5], 32)
    T = np.tile([1.0, 0.0, 0.0, -1.0], 32)
    Gf = G.reshape(-1)
    assert gm[0] == al0 * (-Gf.sum())
    assert ga[0] == al0 * ((Gf * T).sum() - (Gf * wh).sum())
    assert gd[0] == 0


def test_hard_surrogate_uses_s_bwd():
    rng = np.random.default_rng(13)
    W = rng.standard_normal((1, 128)) * 0.02
    G = rng.standard_normal(W.shape)
    soft = lmst.factor_grads(G, W, 128, 0.0, 1.0, 1.0, lmst.SOFT, s=30.0)
    hard = lmst.factor_grads(G, W, 128, 0.0, 1.0, 1.0, lmst.HARD, s_bwd=30.0)
    # mu and Delta terms do not involve T: identical
    assert abs(soft[0][0] - hard[0][0]) < 1e-12 * max(1, abs(soft[0][0]))
    assert abs(soft[2][0] - hard[2][0]) < 1e-12 * max(1, abs(soft[2][0]))


def test_identity_mode_has_no_factor_gradient():
    W = np.random.default_rng(2).standard_normal((1, 128))
    G = np.ones_like(W)
    for v in lmst.factor_grads(G, W, 128, 0.0, 1.0, 1.0, lmst.IDENTITY):
        assert np.all(v == 0)


# ---------------------------------------------------------------------- pack

def test_pack_hand_byte():
    # T = (+1, 0, -1, 0) -> codes (2, 1, 0, 1) -> 0b01_00_01_10 = 0x46
    p = lmst.pack_ternary(np.array([[1, 0, -1, 0]], np.int8))
    assert p.shape == (1, 1) and p[0, 0] == 0x46


def test_pack_roundtrip():
    rng = np.random.default_rng(4)
    c = rng.integers(-1, 2, size=(7, 64)).astype(np.int8)
    np.testing.assert_array_equal(lmst.unpack_ternary(lmst.pack_ternary(c), 64), c)
    with pytest.raises(ValueError):
        lmst.pack_ternary(np.array([[2, 0, 0, 0]], np.int8))
