"""Pins for the oracle's block forward/backward, loss and routing.

The hand-written backward is checked against torch.autograd (float64, CPU:
an independent differentiator) and the whole calibration step against
central finite differences of the Eq. 7 loss in the factors.  Forward pieces
are checked against invariants that hold by construction of each operation.
"""
import numpy as np
import pytest
import torch

import synthgen as sg
from oracle import block, calib, lmst, moe

TINY = sg.small_dense(batch=1, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
SMALL = sg.small_dense(batch=2, seq=9, hidden=128, n_q=4, n_kv=2, head_dim=32, ffn=256)


def _weights(cfg, seed=0):
    return {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in sg.block_weights(cfg, seed).items()}


def _x(cfg, seed=0):
    return sg.bf16_bits_to_f32(sg.activations(cfg, seed)).astype(np.float64)


# ------------------------------------------------------------ torch mirror

def _t_rms(x):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + block.EPS)


def _t_rope(x, S, d, theta):
    half = d // 2
    inv = theta ** (-(2.0 * torch.arange(half, dtype=torch.float64)) / d)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * inv[None]
    c, s = torch.cos(ang)[None, :, None], torch.sin(ang)[None, :, None]
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], -1)


def _t_attn_half(x, W, cfg):
    B, S, Hq, Hkv, d = cfg.batch, cfg.seq, cfg.n_q, cfg.n_kv, cfg.head_dim
    xn = _t_rms(x)
    q = (xn @ W["Wq"].T).reshape(B, S, Hq, d)
    k = (xn @ W["Wk"].T).reshape(B, S, Hkv, d)
    v = (xn @ W["Wv"].T).reshape(B, S, Hkv, d)
    if cfg.qk_norm:
        q, k = _t_rms(q), _t_rms(k)
    q, k = _t_rope(q, S, d, cfg.rope_theta), _t_rope(k, S, d, cfg.rope_theta)
    G = Hq // Hkv
    k = k.repeat_interleave(G, dim=2)
    v = v.repeat_interleave(G, dim=2)
    sc = torch.einsum("bqhd,bkhd->bhqk", q, k) / d ** 0.5
    mask = torch.triu(torch.ones(S, S, dtype=torch.bool), 1)
    p = torch.softmax(sc.masked_fill(mask, float("-inf")), -1)
    o = torch.einsum("bhqk,bkhd->bqhd", p, v).reshape(B * S, Hq * d)
    return x + o @ W["Wo"].T


def _t_block(x, W, cfg):
    h1 = _t_attn_half(x, W, cfg)
    xn2 = _t_rms(h1)
    a = torch.nn.functional.silu(xn2 @ W["Wg"].T) * (xn2 @ W["Wu"].T)
    return h1 + a @ W["Wd"].T


def test_block_backward_matches_autograd():
    cfg = SMALL
    W = _weights(cfg)
    x = _x(cfg)
    dy = np.random.default_rng(3).standard_normal((cfg.tokens, cfg.hidden))
    y, cache = block.block_forward(x, W, cfg)
    dx, dW = block.block_backward(dy, cache, W, cfg)
    tx = torch.tensor(x, requires_grad=True)
    tW = {k: torch.tensor(v, requires_grad=True) for k, v in W.items()}
    ty = _t_block(tx, tW, cfg)
    np.testing.assert_allclose(ty.detach().numpy(), y, rtol=1e-12, atol=1e-12)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-12)
    for k in W:
        np.testing.assert_allclose(dW[k], tW[k].grad.numpy(), rtol=1e-10, atol=1e-12)


def test_moe_backward_matches_autograd():
    cfg = sg.small_moe(batch=1, seq=12, hidden=128, n_q=2, n_kv=1, head_dim=64, n_experts=4,
                       top_k=2, expert_ffn=64)
    W = _weights(cfg)
    x = _x(cfg)
    logits = sg.router_logits(cfg)
    dy = np.random.default_rng(4).standard_normal((cfg.tokens, cfg.hidden))
    y, cache = moe.moe_block_forward(x, W, logits, cfg)
    dx, dW = moe.moe_block_backward(dy, cache, W, cfg)
    idx, wts = cache[2], cache[3]
    tx = torch.tensor(x, requires_grad=True)
    tW = {k: torch.tensor(v, requires_grad=True) for k, v in W.items()}
    h1 = _t_attn_half(tx, tW, cfg)
    xn2 = _t_rms(h1)
    out = torch.zeros_like(h1)
    for t in range(cfg.tokens):
        for j in range(cfg.top_k):
            e = int(idx[t, j])
            xe = xn2[t]
            a = torch.nn.functional.silu(tW["Wg"][e] @ xe) * (tW["Wu"][e] @ xe)
            out = out.index_add(0, torch.tensor([t]), (float(wts[t, j]) * (tW["Wd"][e] @ a))[None])
    ty = h1 + out
    np.testing.assert_allclose(ty.detach().numpy(), y, rtol=1e-12, atol=1e-12)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-12)
    for k in W:
        np.testing.assert_allclose(dW[k], tW[k].grad.numpy(), rtol=1e-10, atol=1e-12)


# ------------------------------------------------- whole-step finite difference

def _smooth_fake(W, fac, s, g=128):
    Wg = W.reshape(-1, g)
    mu0, al0 = lmst.group_stats(W, g)
    mu = mu0 + fac[0] * al0
    al = fac[1] * al0
    D = fac[2] * 0.5
    xh = (Wg - mu[:, None]) / al[:, None]
    return (al[:, None] * lmst.transition(xh, s, D[:, None])).reshape(W.shape)


@pytest.mark.parametrize("s", [3.75, 30.0])
def test_step_factor_grads_finite_differences(s):
    cfg = TINY
    W = _weights(cfg)
    x = _x(cfg)
    rng = np.random.default_rng(5)
    fac = {}
    for k, w in W.items():
        n = w.size // 128
        fac[k] = [rng.uniform(-0.2, 0.2, n), np.exp(rng.uniform(-0.2, 0.2, n)),
                  np.exp(rng.uniform(-0.2, 0.2, n))]
    res = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=s)
    y_fp = res["y_fp"]

    def loss_of(fk):
        Wf = {k: _smooth_fake(W[k], fk[k], s) for k in W}
        y, _ = block.block_forward(x, Wf, cfg)
        return block.recon_loss(y, y_fp)[0]

    probe = [("Wq", 0, 3), ("Wk", 1, 0), ("Wv", 2, 5), ("Wo", 0, 7), ("Wg", 1, 11),
             ("Wu", 2, 2), ("Wd", 0, 100)]
    for name, which, j in probe:
        h = 1e-5
        fp = {k: [a.copy() for a in v] for k, v in fac.items()}
        fm = {k: [a.copy() for a in v] for k, v in fac.items()}
        fp[name][which][j] += h
        fm[name][which][j] -= h
        num = (loss_of(fp) - loss_of(fm)) / (2 * h)
        ana = res["fgrads"][name][which][j]
        scale = max(abs(num), 1e-3 * np.abs(res["fgrads"][name][which]).max())
        assert abs(num - ana) <= 1e-4 * scale, (name, which, j, num, ana)


def test_step_input_gradient_finite_differences():
    cfg = TINY
    W = _weights(cfg)
    x = _x(cfg)
    fac = {k: sg.perturbed_factors(0, w.size // 128) for k, w in W.items()}
    res = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0)
    Wf = res["W_fake"]
    for (i, j) in [(0, 0), (3, 77), (5, 127)]:
        h = 1e-6
        xp, xm = x.copy(), x.copy()
        xp[i, j] += h
        xm[i, j] -= h
        # the target is fixed (cached full-precision output of the original x)
        lp = block.recon_loss(block.block_forward(xp, Wf, cfg)[0], res["y_fp"])[0]
        lm = block.recon_loss(block.block_forward(xm, Wf, cfg)[0], res["y_fp"])[0]
        num = (lp - lm) / (2 * h)
        assert abs(num - res["dx"][i, j]) <= 1e-5 * max(abs(num), 1e-8), (i, j, num, res["dx"][i, j])


# ------------------------------------------------------------ forward pins

def test_identity_mode_loss_is_zero():
    cfg = TINY
    W = _weights(cfg)
    x = _x(cfg)
    fac = {k: sg.perturbed_factors(0, w.size // 128) for k, w in W.items()}
    res = calib.dense_step(x, W, fac, cfg, lmst.IDENTITY)
    assert res["loss"] == 0.0 and np.all(res["dy"] == 0)
    for v in res["fgrads"].values():
        assert all(np.all(a == 0) for a in v)


def test_attention_first_token_and_rows():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((1, 5, 2, 8))
    k = rng.standard_normal((1, 5, 1, 8))
    v = rng.standard_normal((1, 5, 1, 8))
    O, P = block.causal_attention(q, k, v)
    # causal: the first query sees only the first key
    np.testing.assert_allclose(O[0, 0, 0], v[0, 0, 0], rtol=0, atol=1e-15)
    np.testing.assert_allclose(P.sum(-1), 1.0, rtol=1e-14)
    assert np.all(np.triu(P[0, 0], 1) == 0)


def test_rmsnorm_unit_rms_and_rope_properties():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 64)) * 3
    y, _ = block.rmsnorm(x)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1.0, rtol=1e-6)
    cos, sin = block.rope_tables(16, 64, 1e6)
    q = rng.standard_normal((1, 16, 1, 64))
    qr = block.rope(q, cos, sin)
    np.testing.assert_allclose(np.linalg.norm(qr, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
    # position 0 is untouched; the score between two rotated vectors depends
    # only on their position difference
    np.testing.assert_allclose(qr[0, 0], q[0, 0], rtol=0, atol=0)
    a, b = rng.standard_normal(64), rng.standard_normal(64)
    A = block.rope(np.tile(a, (1, 16, 1, 1)), cos, sin)[0, :, 0]
    Bv = block.rope(np.tile(b, (1, 16, 1, 1)), cos, sin)[0, :, 0]
    np.testing.assert_allclose(A[5] @ Bv[2], A[12] @ Bv[9], rtol=1e-10)


def test_loss_closed_form_single_linear():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((32, 16))
    W = rng.standard_normal((8, 16))
    E = rng.standard_normal((8, 16))
    eps = 1e-3
    loss, dy = block.recon_loss(X @ (W + eps * E).T, X @ W.T)
    ref = np.mean((X @ (eps * E).T) ** 2)
    assert abs(loss - ref) <= 1e-12 * ref
    assert loss >= 0


# -------------------------------------------------------------- routing

def test_route_brute_force():
    rng = np.random.default_rng(9)
    lg = rng.standard_normal((50, 16)).astype(np.float32)
    lg[3, 5] = lg[3, 9] = 4.0                   # a tie: lower expert id first
    idx, w = moe.route(lg, 4)
    for t in range(50):
        order = sorted(range(16), key=lambda e: (-float(lg[t, e]), e))[:4]
        assert list(idx[t]) == order
        sel = np.array([float(lg[t, e]) for e in order])
        ref = np.exp(sel) / np.exp(sel).sum()
        np.testing.assert_allclose(w[t], ref, rtol=1e-12)
    assert list(idx[3][:2]) == [5, 9]
    counts = np.bincount(idx.reshape(-1), minlength=16)
    assert counts.sum() == 50 * 4


def test_single_linear_schedule_and_steps():
    W, X = sg.single_linear_case(0)
    rec = calib.single_linear_calibration(W, X[:256], n_steps=10)
    modes = [r["mode"] for r in rec]
    assert modes == [lmst.SOFT] * 8 + [lmst.HARD] * 2
    np.testing.assert_allclose([r["s"] for r in rec[:8]], [3.75 * k for k in range(1, 9)])
    for r in rec:
        dm, da, dd = r["factors"]
        assert np.all(np.abs(dm) < 1) and np.all(da > 0) and np.all(dd > 0)
        assert np.isfinite(r["loss"])


# ------------------------------------------------------ selected-token forward

@pytest.mark.parametrize("cfg", [SMALL, sg.small_dense(batch=3, seq=7, hidden=128, n_q=4, n_kv=1,
                                                       head_dim=32, ffn=192, qk_norm=False)])
def test_block_forward_rows_matches_full(cfg):
    """The selected-token forward (used for full-size sampled checks) equals
    rows of the whole-block forward and of the torch mirror, including the
    first and last token of every sample."""
    W, x = _weights(cfg), _x(cfg)
    S = cfg.seq
    rows = sorted({0, S - 1, S, 2 * S - 1, cfg.tokens - 1, 3, S + 2})
    got = block.block_forward_rows(x, W, cfg, rows)
    ref = block.block_forward(x, W, cfg)[0][rows]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    tw = {k: torch.from_numpy(v) for k, v in W.items()}
    mirror = _t_block(torch.from_numpy(x), tw, cfg).numpy()[rows]
    np.testing.assert_allclose(got, mirror, rtol=1e-10, atol=1e-12)


def test_moe_forward_rows_matches_full():
    cfg = sg.small_moe(batch=2, seq=12, hidden=128, n_q=4, n_kv=2, head_dim=32, n_experts=6,
                       top_k=2, expert_ffn=64, router_bias_std=1.0)
    W, x = _weights(cfg), _x(cfg)
    logits = sg.router_logits(cfg, 0)
    rows = [0, 5, 11, 12, 23]
    got = moe.moe_block_forward_rows(x, W, lambda e: (W["Wg"][e], W["Wu"][e], W["Wd"][e]),
                                     logits, cfg, rows)
    ref = moe.moe_block_forward(x, W, logits, cfg)[0][rows]
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
