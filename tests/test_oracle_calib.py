"""Pins of the oracle's optimiser and learning-rate schedule (App. B.1:
AdamW, learning rate 1e-3 decayed linearly to zero; Sec. 2.2 constraints
-1 < d_mu < 1, d_alpha > 0, d_Delta > 0 enforced by clamping).

Independent of the oracle's own arithmetic: torch's AdamW (weight decay 0)
in float64, the closed form of Adam's first update, and hand values of the
linear decay.  Gradient magnitudes span 1e-9 (below eps, where eps decides
the step) to 1e2 and change sign between steps, so a dropped bias
correction, eps inside the square root, g instead of g^2 in the second
moment or a wrong beta fail here."""
import numpy as np
import pytest
import torch

from oracle import calib

LR = 1e-3
GRADS = np.array([
    [1e-9, -3e-7, 1e-4, -2.5e-2, 1.0, -7.0, 120.0, 0.0],
    [-2e-9, 5e-7, 1e-4, 3e-2, -1.0, -6.0, 80.0, 1e-3],
    [3e-9, 1e-6, -2e-4, 1e-2, 0.5, 9.0, -150.0, -1e-3],
    [0.0, -1e-6, 3e-4, -4e-2, -0.25, 1.0, 60.0, 2e-5],
])
# positive and >= 0.05: the d_alpha / d_Delta clamp at 1e-4 stays inactive
P0 = np.array([0.1, 0.2, 0.5, 0.3, 1.0, 1.5, 0.7, 0.05])


def _f32(a):
    return np.asarray(a, np.float32).astype(np.float64)


def _torch_adamw_step(p, g, m, v, step, lr):
    """One float64 torch AdamW step (weight decay 0) from the given state;
    ``step`` is 1-based (torch's state counts the steps already taken)."""
    t = torch.tensor(p, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([t], lr=lr, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0,
                            foreach=False)
    if step > 1:
        opt.state[t] = {"step": torch.tensor(float(step - 1), dtype=torch.float64),
                        "exp_avg": torch.tensor(m, dtype=torch.float64),
                        "exp_avg_sq": torch.tensor(v, dtype=torch.float64)}
    t.grad = torch.tensor(g, dtype=torch.float64)
    opt.step()
    st = opt.state[t]
    return (t.detach().numpy().copy(), st["exp_avg"].numpy().copy(),
            st["exp_avg_sq"].numpy().copy())


def test_adamw_single_steps_match_torch():
    """Every step, from the oracle's own (fp32) state, equals torch's float64
    AdamW step rounded once to fp32: at most half an fp32 ulp apart."""
    p, m, v = _f32(P0), np.zeros(8), np.zeros(8)
    for k, g in enumerate(GRADS, start=1):
        tp, tm, tv = _torch_adamw_step(p, g, m, v, k, LR)
        op, om, ov = calib.adamw_step(p, g, m, v, k, LR, kind="pos")
        for got, ref in ((op, tp), (om, tm), (ov, tv)):
            ulp = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
            assert np.all(np.abs(got - ref) <= 0.5 * ulp + 1e-300), (k, got, ref)
        p, m, v = op, om, ov


def test_adamw_trajectory_matches_torch():
    """Four steps with a linearly decaying learning rate against torch's
    float64 trajectory (the oracle rounds its state to fp32 each step)."""
    t = torch.tensor(_f32(P0), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([t], lr=LR, betas=(0.9, 0.999), eps=1e-8, weight_decay=0.0,
                            foreach=False)
    p, m, v = _f32(P0), np.zeros(8), np.zeros(8)
    n = len(GRADS)
    for k, g in enumerate(GRADS, start=1):
        lr = calib.linear_lr(k - 1, n)
        for grp in opt.param_groups:
            grp["lr"] = lr
        t.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        p, m, v = calib.adamw_step(p, g, m, v, k, lr, kind="pos")
    np.testing.assert_allclose(p, t.detach().numpy(), rtol=0, atol=1e-6)


def test_adamw_first_step_closed_form():
    """Adam's first update is lr * g / (|g| + eps): m_hat = g, v_hat = g^2."""
    g = GRADS[0]
    p, m, v = calib.adamw_step(_f32(P0), g, np.zeros(8), np.zeros(8), 1, LR, kind="pos")
    ref = _f32(P0) - LR * g / (np.abs(g) + 1e-8)
    np.testing.assert_allclose(p, _f32(ref), rtol=0, atol=0)
    np.testing.assert_allclose(m, _f32(0.1 * g), rtol=0, atol=0)
    np.testing.assert_allclose(v, _f32(0.001 * g * g), rtol=0, atol=0)
    # a gradient of eps/10 moves the factor by lr/11; one far above eps by lr
    assert abs(abs(p[0] - _f32(P0)[0]) - LR / 11) < 1e-7
    assert abs(abs(p[6] - _f32(P0)[6]) - LR) < 1e-6


def test_adamw_clamps():
    """Sec. 2.2 constraints after the update: d_mu into [-1 + 1e-4, 1 - 1e-4],
    d_alpha and d_Delta at least 1e-4."""
    p = np.array([0.99995, -0.99995, 0.3])
    g = np.array([-1.0, 1.0, 1.0])
    out, _, _ = calib.adamw_step(p, g, np.zeros(3), np.zeros(3), 1, LR, kind="mu")
    np.testing.assert_array_equal(out, _f32([1 - 1e-4, -(1 - 1e-4), 0.3 - LR]))
    q = np.array([2e-4, 5e-4, 1.0])
    out, _, _ = calib.adamw_step(q, np.array([1.0, 1.0, -1.0]), np.zeros(3), np.zeros(3), 1, LR,
                                 kind="pos")
    np.testing.assert_array_equal(out, _f32([1e-4, 1e-4, 1.0 + LR]))


@pytest.mark.parametrize("n", [1, 2, 10, 171])
def test_linear_lr_values(n):
    """lr0 at the first update, decaying by lr0/n per update, lr0/n at the
    last one (it would reach zero one update later)."""
    assert calib.linear_lr(0, n) == LR
    assert abs(calib.linear_lr(n - 1, n) - LR / n) <= 1e-18
    if n % 2 == 0:
        assert abs(calib.linear_lr(n // 2, n) - LR / 2) <= 1e-18
    lrs = [calib.linear_lr(k, n) for k in range(n)]
    assert all(a > b for a, b in zip(lrs, lrs[1:]))
    assert abs(sum(lrs) - LR * (n + 1) / 2) <= 1e-15
