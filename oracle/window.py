"""Sliding-layer output reconstruction over a window of consecutive blocks
(Sec. 2.4, Eq. 7), float64.  Test infrastructure only: the HIP path never
imports it.

Eq. 7 matches the output of the whole window computed with alpha*T against
the output of the same window with the full-precision weights, both on the
same input X.  A window of one block is the single-block step.

READINGS (the paper defers the window geometry to SliderQuant and states
neither its size nor its stride):
  * windows of ``l`` consecutive blocks moving by ``stride`` blocks (default
    1: the paper shows at least 20 windows for a 36-layer model), the last
    window ending at the last block;
  * X of a window is the full-precision model's activation entering its first
    block, so windows are independent of each other's quantisation;
  * each window runs the whole Eq. 6 schedule (its own epochs, time state and
    linear learning-rate decay) with fresh AdamW moments; a block that lies
    in several windows keeps its factors from one window to the next.

Parity of the sliding schedule against the paper is UNPINNED (no trajectory
is printed); the window step itself is pinned by finite differences and by
its one-block special case (tests/test_oracle_window.py).
"""
from __future__ import annotations

import numpy as np

from . import block, calib


def window_spans(n_blocks, l, stride=1):
    """[first, last) block ranges of the windows, in calibration order."""
    if n_blocks <= 0 or l <= 0 or stride <= 0:
        raise ValueError("n_blocks, l and stride must be positive")
    if stride > l:
        raise ValueError("a stride longer than the window would skip blocks")
    if l >= n_blocks:
        return [(0, n_blocks)]
    spans = [(a, a + l) for a in range(0, n_blocks - l + 1, stride)]
    if spans[-1][1] != n_blocks:
        spans.append((n_blocks - l, n_blocks))
    return spans


def window_forward(x, Ws, cfg):
    """Output of the blocks with weights Ws[0], Ws[1], ... applied in turn,
    plus every block's input and cache for the backward."""
    xs, caches = [], []
    h = x
    for W in Ws:
        xs.append(h)
        h, c = block.block_forward(h, W, cfg)
        caches.append(c)
    return h, xs, caches


def window_backward(dy, caches, Ws, cfg):
    """Chain rule through the window: the gradient of the window output
    enters the last block; each block's input gradient is the output
    gradient of the block before it.  Returns (dx of the window input,
    [dW of every block])."""
    dWs = [None] * len(Ws)
    d = dy
    for i in range(len(Ws) - 1, -1, -1):
        d, dWs[i] = block.block_backward(d, caches[i], Ws[i], cfg)
    return d, dWs


def window_step(x, Wds, factors, cfg, mode, s=None, s_bwd=0.0, g=128, y_fp=None):
    """LM+ST of every linear of every block of the window -> window forward
    with alpha*T -> Eq. 7 loss against the full-precision window output on
    the same x -> backward to x and to every factor."""
    Wfs = [calib.fake_weights(Wd, fac, g, mode, s) for Wd, fac in zip(Wds, factors)]
    if y_fp is None:
        y_fp = window_forward(x, Wds, cfg)[0]
    y_q, xs, caches = window_forward(x, Wfs, cfg)
    loss, dy = block.recon_loss(y_q, y_fp)
    dx, dWs = window_backward(dy, caches, Wfs, cfg)
    fg = [calib.factor_grads_all(dW, Wd, fac, g, mode, s, s_bwd)
          for dW, Wd, fac in zip(dWs, Wds, factors)]
    return dict(W_fake=Wfs, y_fp=y_fp, y_q=y_q, loss=loss, dy=dy, dx=dx, dW=dWs, fgrads=fg,
                inputs=xs)


def sliding_calibration(x_all, Wds, cfg, l, n_epochs, stride=1, gamma=0.8, s0=30.0, lr0=1e-3,
                        g=128):
    """Calibrates blocks Wds[0..n) window by window (readings in the module
    header).  x_all holds the calibration samples entering block 0, batches
    of cfg.batch consecutive samples.  Returns the per-window loss histories
    and the final factors of every block."""
    n = len(Wds)
    tpb = cfg.batch * cfg.seq
    nb = x_all.shape[0] // tpb
    fac = [{k: [np.zeros(W.size // g), np.ones(W.size // g), np.ones(W.size // g)]
            for k, W in Wd.items()} for Wd in Wds]
    # full-precision activations entering each block
    acts = [x_all]
    for i in range(n - 1):
        acts.append(np.concatenate([block.block_forward(acts[i][b * tpb:(b + 1) * tpb], Wds[i],
                                                        cfg)[0] for b in range(nb)]))
    history = []
    for a, e_ in window_spans(n, l, stride):
        Wwin = Wds[a:e_]
        xs = [acts[a][b * tpb:(b + 1) * tpb] for b in range(nb)]
        y_fp = [window_forward(x, Wwin, cfg)[0] for x in xs]
        mom = [{k: [np.zeros(W.size // g) for _ in range(3)] for k, W in Wd.items()} for Wd in Wwin]
        vel = [{k: [np.zeros(W.size // g) for _ in range(3)] for k, W in Wd.items()} for Wd in Wwin]
        total, step, losses = n_epochs * nb, 0, []
        for ep in range(n_epochs):
            mode, s = calib.epoch_state(ep, n_epochs, gamma, s0)
            for b in range(nb):
                r = window_step(xs[b], Wwin, fac[a:e_], cfg, mode, s=s if s else None,
                                s_bwd=s0, g=g, y_fp=y_fp[b])
                losses.append(r["loss"])
                step += 1
                lr = calib.linear_lr(step - 1, total, lr0)
                for j in range(e_ - a):
                    f, m, v = fac[a + j], mom[j], vel[j]
                    for k in f:
                        for i, kind in enumerate(("mu", "pos", "pos")):
                            f[k][i], m[k][i], v[k][i] = calib.adamw_step(
                                f[k][i], r["fgrads"][j][k][i], m[k][i], v[k][i], step, lr,
                                kind=kind)
        history.append(dict(span=(a, e_), losses=losses))
    return dict(history=history, factors=fac)
