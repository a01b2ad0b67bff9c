"""Host logic of the calibration loop (no GPU): the time state of Eq. 6 per
epoch and the linear learning-rate decay, against the values the paper's
formulas give and against the oracle's own implementation."""
import numpy as np
import pytest

import synthgen as sg
from oracle import block, calib, lmst


def test_epoch_state_values():
    """Sec. 2.3 / App. B.1: s = (t / gamma) s0 while t <= gamma, hard after;
    t_e = (e + 1)/n.  Five epochs at gamma 0.8, s0 30: s = 7.5, 15, 22.5, 30,
    then hard; sixty epochs: 48 soft epochs from s = 0.625 to 30, 12 hard."""
    got = [calib.epoch_state(e, 5) for e in range(5)]
    assert [m for m, _ in got] == [lmst.SOFT] * 4 + [lmst.HARD]
    np.testing.assert_allclose([s for _, s in got[:4]], [7.5, 15.0, 22.5, 30.0], rtol=1e-15)
    sixty = [calib.epoch_state(e, 60) for e in range(60)]
    soft = [s for m, s in sixty if m == lmst.SOFT]
    assert len(soft) == 48 and abs(soft[0] - 0.625) < 1e-12 and abs(soft[-1] - 30.0) < 1e-12


@pytest.mark.parametrize("n", [1, 5, 10, 60])
def test_host_schedule_matches_oracle(n):
    from paper_2606_26650_amd import calibrate
    for e in range(n):
        assert calibrate.time_state(e, n) == calib.epoch_state(e, n)
    for k in range(n):
        assert calibrate.linear_lr(k, n) == calib.linear_lr(k, n)


def test_dense_calibration_is_step_plus_adamw():
    """One epoch of one batch: the loop reduces to one reconstruction step and
    one AdamW update of every factor at the first learning rate."""
    cfg = sg.small_dense(batch=1, seq=8, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    W = {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in sg.block_weights(cfg, 0).items()}
    x = sg.bf16_bits_to_f32(sg.activations(cfg, 0)).astype(np.float64)
    out = calib.dense_calibration(x, W, cfg, n_epochs=1, gamma=0.8)
    mode, s = calib.epoch_state(0, 1)
    assert mode == lmst.HARD  # t = 1 > gamma
    fac0 = {n: [np.zeros(w.size // 128), np.ones(w.size // 128), np.ones(w.size // 128)]
            for n, w in W.items()}
    r = calib.dense_step(x, W, fac0, cfg, mode, s=None, s_bwd=30.0)
    assert out["losses"] == [r["loss"]]
    for n in W:
        for i, kind in enumerate(("mu", "pos", "pos")):
            p, _, _ = calib.adamw_step(fac0[n][i], r["fgrads"][n][i], np.zeros_like(fac0[n][i]),
                                       np.zeros_like(fac0[n][i]), 1, 1e-3, kind=kind)
            np.testing.assert_array_equal(out["factors"][n][i], p)


@pytest.mark.parametrize("n,l,stride", [(1, 1, 1), (5, 2, 1), (5, 2, 2), (36, 4, 1), (36, 4, 3),
                                        (7, 3, 3), (3, 8, 1)])
def test_host_window_spans_match_oracle(n, l, stride):
    """The sliding-window geometry the GPU driver walks is the oracle's."""
    from oracle import window as ow
    from paper_2606_26650_amd import window
    assert window.window_spans(n, l, stride) == ow.window_spans(n, l, stride)


def test_host_window_spans_reject_bad_geometry():
    from paper_2606_26650_amd import window
    for args in [(0, 2, 1), (4, 0, 1), (4, 2, 0), (6, 2, 3)]:
        with pytest.raises(ValueError):
            window.window_spans(*args)
