"""Pins for the oracle's sliding-window reconstruction (Eq. 7 over several
blocks).

* the window step's factor and input gradients against central finite
  differences of the window loss (a dropped block, a wrong chaining order or
  a lost residual path in the backward fails them);
* the one-block window is the single-block step, and a one-block sliding
  calibration is the block calibration run on the full-precision activations
  (an independent code path);
* the identity branch reconstructs exactly; the window spans cover every
  block in order.
"""
import numpy as np
import pytest

import synthgen as sg
from oracle import block, calib, lmst, window

TINY = sg.small_dense(batch=1, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)


def _weights(cfg, seed):
    return {k: sg.bf16_bits_to_f32(v).astype(np.float64)
            for k, v in sg.block_weights(cfg, seed).items()}


def _x(cfg, seed=0):
    return sg.bf16_bits_to_f32(sg.activations(cfg, seed)).astype(np.float64)


def _smooth_fake(W, fac, s, g=128):
    """alpha * f(W_hat) with the per-group scalars kept in float64 (no fp32
    rounding), so that central differences in the factors are clean."""
    Wg = W.reshape(-1, g)
    mu0, al0 = lmst.group_stats(W, g)
    mu = mu0 + fac[0] * al0
    al = fac[1] * al0
    D = fac[2] * 0.5
    xh = (Wg - mu[:, None]) / al[:, None]
    return (al[:, None] * lmst.transition(xh, s, D[:, None])).reshape(W.shape)


def _rand_factors(Wd, seed):
    rng = np.random.default_rng(seed)
    out = {}
    for k, w in Wd.items():
        n = w.size // 128
        out[k] = [rng.uniform(-0.2, 0.2, n), np.exp(rng.uniform(-0.2, 0.2, n)),
                  np.exp(rng.uniform(-0.2, 0.2, n))]
    return out


def test_window_spans():
    assert window.window_spans(5, 2) == [(0, 2), (1, 3), (2, 4), (3, 5)]
    assert window.window_spans(5, 2, stride=2) == [(0, 2), (2, 4), (3, 5)]
    assert window.window_spans(3, 3) == [(0, 3)]
    assert window.window_spans(2, 4) == [(0, 2)]
    assert window.window_spans(4, 1) == [(0, 1), (1, 2), (2, 3), (3, 4)]
    for n, l, st in [(7, 3, 1), (7, 3, 2), (9, 4, 3), (6, 2, 2), (8, 3, 3)]:
        sp = window.window_spans(n, l, st)
        covered = sorted({b for a, e in sp for b in range(a, e)})
        assert covered == list(range(n))
        assert all(e - a == min(l, n) for a, e in sp)
        assert [a for a, _ in sp] == sorted(a for a, _ in sp)
        assert sp[-1][1] == n
    with pytest.raises(ValueError):
        window.window_spans(0, 2)
    with pytest.raises(ValueError):
        window.window_spans(6, 2, stride=3)


@pytest.mark.parametrize("s", [3.75, 30.0])
def test_window_factor_grads_finite_differences(s):
    Wds = [_weights(TINY, 0), _weights(TINY, 1)]
    x = _x(TINY)
    facs = [_rand_factors(Wds[0], 5), _rand_factors(Wds[1], 6)]
    res = window.window_step(x, Wds, facs, TINY, lmst.SOFT, s=s)
    y_fp = res["y_fp"]

    def loss_of(fk):
        Wfs = [{k: _smooth_fake(W[k], f[k], s) for k in W} for W, f in zip(Wds, fk)]
        return block.recon_loss(window.window_forward(x, Wfs, TINY)[0], y_fp)[0]

    probe = [(0, "Wq", 0, 3), (0, "Wo", 1, 7), (0, "Wd", 2, 100), (1, "Wk", 0, 0),
             (1, "Wu", 1, 2), (1, "Wg", 2, 11)]
    for b, name, which, j in probe:
        h = 1e-5
        fp = [{k: [a.copy() for a in v] for k, v in f.items()} for f in facs]
        fm = [{k: [a.copy() for a in v] for k, v in f.items()} for f in facs]
        fp[b][name][which][j] += h
        fm[b][name][which][j] -= h
        num = (loss_of(fp) - loss_of(fm)) / (2 * h)
        ana = res["fgrads"][b][name][which][j]
        scale = max(abs(num), 1e-3 * np.abs(res["fgrads"][b][name][which]).max())
        assert abs(num - ana) <= 1e-4 * scale, (b, name, which, j, num, ana)


def test_window_input_gradient_finite_differences():
    Wds = [_weights(TINY, 0), _weights(TINY, 1), _weights(TINY, 2)]
    x = _x(TINY)
    facs = [{k: sg.perturbed_factors(i, w.size // 128) for k, w in Wd.items()}
            for i, Wd in enumerate(Wds)]
    res = window.window_step(x, Wds, facs, TINY, lmst.SOFT, s=15.0)
    for (i, j) in [(0, 0), (3, 77), (5, 127)]:
        h = 1e-6
        xp, xm = x.copy(), x.copy()
        xp[i, j] += h
        xm[i, j] -= h
        lp = block.recon_loss(window.window_forward(xp, res["W_fake"], TINY)[0], res["y_fp"])[0]
        lm = block.recon_loss(window.window_forward(xm, res["W_fake"], TINY)[0], res["y_fp"])[0]
        num = (lp - lm) / (2 * h)
        assert abs(num - res["dx"][i, j]) <= 1e-5 * max(abs(num), 1e-8), (i, j, num)


def test_one_block_window_is_the_block_step():
    W = _weights(TINY, 0)
    x = _x(TINY)
    fac = {k: sg.perturbed_factors(3, w.size // 128) for k, w in W.items()}
    a = window.window_step(x, [W], [fac], TINY, lmst.SOFT, s=7.5, s_bwd=30.0)
    b = calib.dense_step(x, W, fac, TINY, lmst.SOFT, s=7.5, s_bwd=30.0)
    assert a["loss"] == b["loss"]
    np.testing.assert_array_equal(a["dx"], b["dx"])
    for k in W:
        for i in range(3):
            np.testing.assert_array_equal(a["fgrads"][0][k][i], b["fgrads"][k][i])


def test_window_identity_is_exact():
    Wds = [_weights(TINY, 0), _weights(TINY, 1)]
    x = _x(TINY)
    facs = [{k: sg.perturbed_factors(i, w.size // 128) for k, w in Wd.items()}
            for i, Wd in enumerate(Wds)]
    res = window.window_step(x, Wds, facs, TINY, lmst.IDENTITY)
    assert res["loss"] == 0.0
    assert not np.any(res["dx"])
    # the window output is the blocks applied in order
    y = block.block_forward(block.block_forward(x, Wds[0], TINY)[0], Wds[1], TINY)[0]
    np.testing.assert_array_equal(res["y_fp"], y)


def test_one_block_sliding_calibration_is_block_calibration():
    """l = 1: block 1 is calibrated alone on the full-precision output of
    block 0, exactly what the block calibration does with that input."""
    cfg = sg.small_dense(batch=1, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    xcfg = sg.small_dense(batch=2, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    Wds = [_weights(cfg, 0), _weights(cfg, 1)]
    x_all = _x(xcfg)
    r = window.sliding_calibration(x_all, Wds, cfg, l=1, n_epochs=3)
    assert [h["span"] for h in r["history"]] == [(0, 1), (1, 2)]
    x1 = np.concatenate([block.block_forward(x_all[b * 6:(b + 1) * 6], Wds[0], cfg)[0]
                         for b in range(2)])
    ref0 = calib.dense_calibration(x_all, Wds[0], cfg, 3)
    ref1 = calib.dense_calibration(x1, Wds[1], cfg, 3)
    assert r["history"][0]["losses"] == ref0["losses"]
    assert r["history"][1]["losses"] == ref1["losses"]
    for k in Wds[1]:
        for i in range(3):
            np.testing.assert_array_equal(r["factors"][0][k][i], ref0["factors"][k][i])
            np.testing.assert_array_equal(r["factors"][1][k][i], ref1["factors"][k][i])


def test_sliding_calibration_reduces_window_loss_and_keeps_constraints():
    cfg = TINY
    xcfg = sg.small_dense(batch=2, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    Wds = [_weights(cfg, i) for i in range(3)]
    r = window.sliding_calibration(_x(xcfg), Wds, cfg, l=2, n_epochs=4, lr0=1e-2)
    assert [h["span"] for h in r["history"]] == [(0, 2), (1, 3)]
    for h in r["history"]:
        assert len(h["losses"]) == 4 * 2 and all(np.isfinite(h["losses"]))
        assert h["losses"][0] > 0
    for f in r["factors"]:
        for k, (dm, da, dd) in f.items():
            assert np.all(np.abs(dm) < 1) and np.all(da > 0) and np.all(dd > 0)
    # block 1 lies in both windows: its factors moved away from the start
    assert any(np.any(f[0] != 0) for f in r["factors"][1].values())
