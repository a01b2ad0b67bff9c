"""One calibration step end to end, the time-state schedule and AdamW, float64.

Parity of the calibration trajectory against the paper is UNPINNED: the paper
prints no trajectory, only its hyper-parameters (App. B.1: AdamW, lr 1e-3
decayed linearly to zero, s0 = 30, gamma = 0.8, Delta0 = 0.5).  The optimizer
and the learning-rate schedule themselves are pinned independently of this
module (tests/test_oracle_calib.py: torch's float64 AdamW step by step and over
a trajectory, the closed-form first step, the clamps, and linear_lr at its end
points and midpoint).
"""
from __future__ import annotations

import numpy as np

from . import block, lmst, moe

DMU_LIM = 1.0 - 1e-4
POS_MIN = 1e-4


def schedule(k, n_steps, gamma=0.8, s0=30.0):
    """Eq. 6 branch for step k (1-based) of n_steps.  READING: the normalised
    time is t = k/n_steps; SOFT with s = (t/gamma)*s0 while t <= gamma, HARD
    after.  (t = 0, the identity branch, is only the starting point.)"""
    t = k / n_steps
    if t <= gamma:
        return lmst.SOFT, (t / gamma) * s0
    return lmst.HARD, 0.0


def adamw_step(p, grad, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, kind="mu"):
    """READING: AdamW with betas (0.9, 0.999), eps 1e-8 and no weight decay
    (decay would pull d_alpha and d_Delta to zero), then the constraints of
    Sec. 2.2 enforced by clamping: -1 < d_mu < 1, d_alpha > 0, d_Delta > 0.
    ``step`` is 1-based.  Returns fp32-rounded (p, m, v)."""
    p = np.asarray(p, np.float64)
    g = np.asarray(grad, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1 - beta2) * g * g
    mh = m / (1 - beta1 ** step)
    vh = v / (1 - beta2 ** step)
    p = p - lr * mh / (np.sqrt(vh) + eps)
    if kind == "mu":
        p = np.clip(p, -DMU_LIM, DMU_LIM)
    else:
        p = np.maximum(p, POS_MIN)
    return lmst.f32(p), lmst.f32(m), lmst.f32(v)


def epoch_state(e, n_epochs, gamma=0.8, s0=30.0):
    """Eq. 6 branch for 0-based epoch e: READING t_e = (e + 1)/n_epochs (the
    identity branch t = 0 is only the starting point)."""
    return schedule(e + 1, n_epochs, gamma, s0)


def linear_lr(k0, n_steps, lr0=1e-3):
    """Linear decay to zero: step k0 (0-based) uses lr0 * (1 - k0/n_steps)."""
    return lr0 * (1.0 - k0 / n_steps)


# ------------------------------------------------------------- step helpers

def fake_weights(Wd, factors, g, mode, s, strides=(1, 1, 1), delta0=0.5):
    out = {}
    for name, W in Wd.items():
        dm, da, dd = factors[name]
        out[name] = lmst.modulate_ternarize(W, g, dm, da, dd, mode, s=s, delta0=delta0,
                                            strides=strides)["W_fake"]
    return out


def factor_grads_all(dW, Wd, factors, g, mode, s, s_bwd, strides=(1, 1, 1), delta0=0.5):
    out = {}
    for name, W in Wd.items():
        dm, da, dd = factors[name]
        out[name] = lmst.factor_grads(dW[name], W, g, dm, da, dd, mode, s=s, s_bwd=s_bwd,
                                      delta0=delta0, strides=strides)
    return out


def dense_step(x, Wd, factors, cfg, mode, s=None, s_bwd=0.0, g=128, y_fp=None, a8=False):
    """LM+ST of all seven linears -> block forward with alpha*T -> loss
    against the full-precision block output on the same x -> backward to the
    input and to every linear's factors.  a8: the quantized block also
    fake-quantizes its activations (W1.58A8); the target stays the
    full-precision block."""
    Wf = fake_weights(Wd, factors, g, mode, s)
    if y_fp is None:
        y_fp, _ = block.block_forward(x, Wd, cfg)
    y_q, cache = block.block_forward(x, Wf, cfg, a8)
    loss, dy = block.recon_loss(y_q, y_fp)
    dx, dW = block.block_backward(dy, cache, Wf, cfg)
    fg = factor_grads_all(dW, Wd, factors, g, mode, s, s_bwd)
    return dict(W_fake=Wf, y_fp=y_fp, y_q=y_q, loss=loss, dy=dy, dx=dx, dW=dW, fgrads=fg)


def moe_step(x, Wd, factors, logits, cfg, mode, s=None, s_bwd=0.0, g=128, y_fp=None):
    Wf = fake_weights(Wd, factors, g, mode, s)
    if y_fp is None:
        y_fp, _ = moe.moe_block_forward(x, Wd, logits, cfg)
    y_q, cache = moe.moe_block_forward(x, Wf, logits, cfg)
    loss, dy = block.recon_loss(y_q, y_fp)
    dx, dW = moe.moe_block_backward(dy, cache, Wf, cfg)
    fg = factor_grads_all(dW, Wd, factors, g, mode, s, s_bwd)
    return dict(W_fake=Wf, y_fp=y_fp, y_q=y_q, loss=loss, dy=dy, dx=dx, dW=dW, fgrads=fg,
                route=cache[2:])


def single_linear_calibration(W, X, n_steps=10, g=128, strides=(1, 1, 1), gamma=0.8, s0=30.0,
                              lr0=1e-3, delta0=0.5):
    """Single linear, MSE to its full-precision output, n_steps of LM+ST with
    AdamW (the 256x256 fp32 workload).  Returns the per-step record."""
    W = np.asarray(W, np.float64)
    X = np.asarray(X, np.float64)
    ng = W.size // g
    nf = [ng if st == 1 else 1 for st in strides]
    p = [np.zeros(nf[0]), np.ones(nf[1]), np.ones(nf[2])]
    mom = [np.zeros(n) for n in nf]
    vel = [np.zeros(n) for n in nf]
    y_fp = X @ W.T
    rec = []
    for k in range(1, n_steps + 1):
        mode, s = schedule(k, n_steps, gamma, s0)
        r = lmst.modulate_ternarize(W, g, p[0], p[1], p[2], mode, s=s, delta0=delta0,
                                    strides=strides)
        y = X @ r["W_fake"].T
        loss, dy = block.recon_loss(y, y_fp)
        G = dy.T @ X
        grads = lmst.factor_grads(G, W, g, p[0], p[1], p[2], mode, s=s, s_bwd=s0,
                                  delta0=delta0, strides=strides)
        lr = linear_lr(k - 1, n_steps, lr0)
        for i, kind in enumerate(("mu", "pos", "pos")):
            p[i], mom[i], vel[i] = adamw_step(p[i], grads[i], mom[i], vel[i], k, lr, kind=kind)
        rec.append(dict(k=k, mode=mode, s=s, loss=loss, grads=grads,
                        factors=[q.copy() for q in p]))
    return rec


def dense_calibration(x_all, Wd, cfg, n_epochs, gamma=0.8, s0=30.0, lr0=1e-3, g=128):
    """Calibration of one dense block (Sec. 2.2-2.4, App. B.1): epochs over
    the calibration set x_all (batches of cfg.batch consecutive samples),
    the Eq. 6 time state per epoch, one AdamW update of every factor per
    batch with the learning rate decayed linearly to zero over all updates,
    the hard branch's backward at s0.  Factors start at the identity
    modulation.  Returns the per-step losses and the final factors."""
    tpb = cfg.batch * cfg.seq
    nb = x_all.shape[0] // tpb
    total = n_epochs * nb
    fac = {n: [np.zeros(W.size // g), np.ones(W.size // g), np.ones(W.size // g)]
           for n, W in Wd.items()}
    mom = {n: [np.zeros(W.size // g) for _ in range(3)] for n, W in Wd.items()}
    vel = {n: [np.zeros(W.size // g) for _ in range(3)] for n, W in Wd.items()}
    xs = [x_all[b * tpb:(b + 1) * tpb] for b in range(nb)]
    y_fp = [block.block_forward(x, Wd, cfg)[0] for x in xs]
    losses, step = [], 0
    for e in range(n_epochs):
        mode, s = epoch_state(e, n_epochs, gamma, s0)
        for b in range(nb):
            r = dense_step(xs[b], Wd, fac, cfg, mode, s=s if s else None, s_bwd=s0, g=g,
                           y_fp=y_fp[b])
            losses.append(r["loss"])
            step += 1
            lr = linear_lr(step - 1, total, lr0)
            for n in Wd:
                for i, kind in enumerate(("mu", "pos", "pos")):
                    fac[n][i], mom[n][i], vel[n][i] = adamw_step(
                        fac[n][i], r["fgrads"][n][i], mom[n][i], vel[n][i], step, lr, kind=kind)
    return dict(losses=losses, factors=fac)
