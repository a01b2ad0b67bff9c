"""Routed mixture-of-experts block, float64.

The attention half is the dense block's.  The MLP half routes each token to
the top-k experts of given router logits (the routing module is left
unquantised, App. B.2; READING: its logits are a fixed input of the step, so
no gradient flows to them), weights the chosen experts by a softmax over the
k selected logits, and sums the experts' SwiGLU outputs.  Each expert's
gate/up/down weights are fake-ternarised like any dense linear.
"""
from __future__ import annotations

import numpy as np

from . import block


def route(logits, top_k):
    """Top-k expert ids per token (largest logit first; equal logits: lower
    expert id first) and their renormalised softmax weights."""
    lg = np.asarray(logits, np.float64)
    idx = np.argsort(-lg, axis=1, kind="stable")[:, :top_k]
    sel = np.take_along_axis(lg, idx, 1)
    e = np.exp(sel - sel.max(1, keepdims=True))
    return idx, e / e.sum(1, keepdims=True)


def moe_mlp_forward(h1, Wg, Wu, Wd, idx, wts):
    """Wg, Wu [E][F][h]; Wd [E][h][F]."""
    xn2, r2 = block.rmsnorm(h1)
    out = np.zeros_like(h1)
    per = {}
    for e in range(Wg.shape[0]):
        tok, slot = np.nonzero(idx == e)
        if tok.size == 0:
            continue
        xe = xn2[tok]
        gt = xe @ Wg[e].T
        up = xe @ Wu[e].T
        a = block.silu(gt) * up
        ye = a @ Wd[e].T
        out[tok] += wts[tok, slot][:, None] * ye
        per[e] = dict(tok=tok, slot=slot, gt=gt, up=up, a=a, xe=xe)
    return h1 + out, dict(h1=h1, xn2=xn2, r2=r2, per=per)


def moe_mlp_backward(dy, c, Wg, Wu, Wd, wts):
    E = Wg.shape[0]
    dWg, dWu, dWd = np.zeros_like(Wg), np.zeros_like(Wu), np.zeros_like(Wd)
    dxn2 = np.zeros_like(c["xn2"])
    for e, p in c["per"].items():
        dye = wts[p["tok"], p["slot"]][:, None] * dy[p["tok"]]
        dWd[e] = dye.T @ p["a"]
        da = dye @ Wd[e]
        dgt = da * p["up"] * block.silu_grad(p["gt"])
        dup = da * block.silu(p["gt"])
        dWg[e] = dgt.T @ p["xe"]
        dWu[e] = dup.T @ p["xe"]
        np.add.at(dxn2, p["tok"], dgt @ Wg[e] + dup @ Wu[e])
    dh1 = dy + block.rmsnorm_bwd(c["h1"], c["r2"], dxn2)
    return dh1, dict(Wg=dWg, Wu=dWu, Wd=dWd)


def moe_block_forward(x, W, logits, cfg):
    h1, ca = block.attn_forward(x, W, cfg)
    idx, wts = route(logits, cfg.top_k)
    y, cm = moe_mlp_forward(h1, W["Wg"], W["Wu"], W["Wd"], idx, wts)
    return y, (ca, cm, idx, wts)


def moe_block_backward(dy, cache, W, cfg):
    ca, cm, idx, wts = cache
    dh1, gm = moe_mlp_backward(dy, cm, W["Wg"], W["Wu"], W["Wd"], wts)
    dx, ga = block.attn_backward(dh1, ca, W, cfg)
    ga.update(gm)
    return dx, ga


def moe_block_forward_rows(x, W, expert, logits, cfg, rows):
    """Block output for the token rows ``rows``.  ``W`` holds the attention
    weights; ``expert(e)`` returns expert e's (gate, up, down) weights, so
    only the experts these tokens are routed to are ever formed.  Per token
    this is moe_mlp_forward's arithmetic (checked against it)."""
    rows = [int(t) for t in rows]
    h1 = block.attn_forward_rows(x, W, cfg, rows)
    idx, wts = route(np.asarray(logits)[rows], cfg.top_k)
    xn2, _ = block.rmsnorm(h1)
    y = h1.copy()
    cache = {}
    for i in range(len(rows)):
        for j in range(cfg.top_k):
            e = int(idx[i, j])
            if e not in cache:
                cache[e] = expert(e)
            Wg, Wu, Wd = cache[e]
            a = block.silu(xn2[i] @ Wg.T) * (xn2[i] @ Wu.T)
            y[i] += wts[i, j] * (a @ Wd.T)
    return y
