"""Decoder-block forward/backward and the output-reconstruction loss, float64.

Sec. 2.4 (Eq. 7): the window output computed with fake-ternary weights
alpha*T is matched in squared L2 norm to the output computed with the
full-precision weights, on the same calibration input.  The window here is
one decoder block.  The paper uses the host models' own blocks and does not
write them out; READING: a pre-norm block with RMSNorm (unit weight,
eps 1e-6), q/k/v projections, optional per-head RMSNorm on q and k,
rotary embedding (rotate-half pairs (i, i + d/2)), causal grouped-query
softmax attention scaled by 1/sqrt(head_dim), output projection, residual,
RMSNorm, SwiGLU MLP silu(gate)*up, down projection, residual.  No biases.
The loss is the mean of the squared differences over every output element.

Activations are [tokens][features] with tokens = batch*seq, sample-major.
The backward is written out by hand (chain rule); the tests check it against
finite differences and against torch.autograd.
"""
from __future__ import annotations

import numpy as np

from . import actquant

EPS = 1e-6
LINEARS = ("Wq", "Wk", "Wv", "Wo", "Wg", "Wu", "Wd")


# ---------------------------------------------------------------- pieces

def rmsnorm(x, eps=EPS):
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)
    return x * r[..., None], r


def rmsnorm_bwd(x, r, dy):
    n = x.shape[-1]
    return r[..., None] * dy - x * (r ** 3)[..., None] * (np.sum(dy * x, -1, keepdims=True) / n)


def rope_tables(seq, head_dim, theta):
    half = head_dim // 2
    inv = theta ** (-(2.0 * np.arange(half)) / head_dim)
    ang = np.arange(seq)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x, cos, sin):
    """x [B, S, H, d]; pairs (i, i + d/2) rotated by angle pos*theta^(-2i/d)."""
    h = x.shape[-1] // 2
    c, s = cos[None, :, None, :], sin[None, :, None, :]
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def rope_bwd(dy, cos, sin):
    h = dy.shape[-1] // 2
    c, s = cos[None, :, None, :], sin[None, :, None, :]
    d1, d2 = dy[..., :h], dy[..., h:]
    return np.concatenate([d1 * c + d2 * s, -d1 * s + d2 * c], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def silu_grad(x):
    sg = 1.0 / (1.0 + np.exp(-x))
    return sg * (1.0 + x * (1.0 - sg))


def causal_attention(q, k, v):
    """q [B,S,Hq,d], k/v [B,S,Hkv,d]; query head h reads kv head h // (Hq/Hkv).
    Returns O [B,S,Hq,d] and the probabilities P [B,Hq,S,S]."""
    B, S, Hq, d = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    scale = 1.0 / np.sqrt(d)
    mask = np.triu(np.ones((S, S), bool), 1)
    O = np.empty_like(q)
    P = np.empty((B, Hq, S, S))
    for b in range(B):
        for h in range(Hq):
            sc = q[b, :, h, :] @ k[b, :, h // G, :].T * scale
            sc[mask] = -np.inf
            m = sc.max(1, keepdims=True)
            e = np.exp(sc - m)
            p = e / e.sum(1, keepdims=True)
            P[b, h] = p
            O[b, :, h, :] = p @ v[b, :, h // G, :]
    return O, P


def causal_attention_bwd(q, k, v, P, dO):
    B, S, Hq, d = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    scale = 1.0 / np.sqrt(d)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for b in range(B):
        for h in range(Hq):
            kv = h // G
            p = P[b, h]
            do = dO[b, :, h, :]
            dv[b, :, kv, :] += p.T @ do
            dp = do @ v[b, :, kv, :].T
            ds = p * (dp - np.sum(dp * p, 1, keepdims=True))
            dq[b, :, h, :] = ds @ k[b, :, kv, :] * scale
            dk[b, :, kv, :] += ds.T @ q[b, :, h, :] * scale
    return dq, dk, dv


# ---------------------------------------------------------- attention half

def _aq(x, group):
    """W1.58A8 activation fake quantization of a stored (bf16) activation:
    the quantizer of oracle/actquant.py applied to the bf16 value."""
    x32 = np.asarray(x, np.float64).astype(np.float32)
    return actquant.quantize(actquant.bf16_round(x32), group)[0]


def _q8(a8, name, x, group):
    """The W1.58A8 quantized value of activation ``name``: the quantizer on
    the oracle's own value, or, when ``a8`` is a dict, the quantized
    activation given there (same shape), so that a comparison can take the
    quantizer's code decisions from another computation of the same step."""
    if isinstance(a8, dict):
        q = np.asarray(a8[name], np.float64)
        assert q.shape == x.shape, (name, q.shape, x.shape)
        return q
    return _aq(x, group)


def attn_forward(x, W, cfg, a8=False):
    """x [M][h] -> h1 = x + o_proj(attention(...)).  W maps names to [d_out][d_in].
    a8: the inputs of q|k|v and o, and Q, K, V of the attention products, are
    fake-quantized to 8 bits (per token; per token and head for Q, K, V) and
    the cache holds the quantized values (the backward is straight-through).
    a8 may be a dict of given quantized activations (see _q8): "xn1", "qr",
    "kr", "v", "attn", "xn2", "a"."""
    B, S = cfg.batch, cfg.seq
    Hq, Hkv, hd = cfg.n_q, cfg.n_kv, cfg.head_dim
    c = {"x": x}
    xn1, r1 = rmsnorm(x)
    if a8:
        xn1 = _q8(a8, "xn1", xn1, xn1.shape[-1])
    c.update(xn1=xn1, r1=r1)
    q = (xn1 @ W["Wq"].T).reshape(B, S, Hq, hd)
    k = (xn1 @ W["Wk"].T).reshape(B, S, Hkv, hd)
    v = (xn1 @ W["Wv"].T).reshape(B, S, Hkv, hd)
    c.update(q_raw=q, k_raw=k, v=v)
    if cfg.qk_norm:
        q, rq = rmsnorm(q)
        k, rk = rmsnorm(k)
        c.update(rq=rq, rk=rk)
    cos, sin = rope_tables(S, hd, cfg.rope_theta)
    c.update(cos=cos, sin=sin, q_n=q, k_n=k)
    qr, kr = rope(q, cos, sin), rope(k, cos, sin)
    if a8:
        qr, kr, v = _q8(a8, "qr", qr, hd), _q8(a8, "kr", kr, hd), _q8(a8, "v", v, hd)
        c["v"] = v
    c.update(qr=qr, kr=kr)
    O, P = causal_attention(qr, kr, v)
    c["P"] = P
    attn = O.reshape(B * S, Hq * hd)
    if a8:
        attn = _q8(a8, "attn", attn, attn.shape[-1])
    c["attn"] = attn
    h1 = x + attn @ W["Wo"].T
    return h1, c


def attn_backward(dh1, c, W, cfg):
    """Returns dx and the fake-weight gradients of q, k, v, o."""
    B, S = cfg.batch, cfg.seq
    Hq, Hkv, hd = cfg.n_q, cfg.n_kv, cfg.head_dim
    g = {}
    g["Wo"] = dh1.T @ c["attn"]
    dO = (dh1 @ W["Wo"]).reshape(B, S, Hq, hd)
    dqr, dkr, dv = causal_attention_bwd(c["qr"], c["kr"], c["v"], c["P"], dO)
    dq = rope_bwd(dqr, c["cos"], c["sin"])
    dk = rope_bwd(dkr, c["cos"], c["sin"])
    if cfg.qk_norm:
        dq = rmsnorm_bwd(c["q_raw"], c["rq"], dq)
        dk = rmsnorm_bwd(c["k_raw"], c["rk"], dk)
    dq = dq.reshape(B * S, Hq * hd)
    dk = dk.reshape(B * S, Hkv * hd)
    dv = dv.reshape(B * S, Hkv * hd)
    xn1 = c["xn1"]
    g["Wq"], g["Wk"], g["Wv"] = dq.T @ xn1, dk.T @ xn1, dv.T @ xn1
    dxn1 = dq @ W["Wq"] + dk @ W["Wk"] + dv @ W["Wv"]
    dx = dh1 + rmsnorm_bwd(c["x"], c["r1"], dxn1)
    return dx, g


# ---------------------------------------------------------------- MLP half

def mlp_forward(h1, W, a8=False):
    xn2, r2 = rmsnorm(h1)
    if a8:
        xn2 = _q8(a8, "xn2", xn2, xn2.shape[-1])
    gt = xn2 @ W["Wg"].T
    up = xn2 @ W["Wu"].T
    a = silu(gt) * up
    if a8:
        a = _q8(a8, "a", a, a.shape[-1])
    y = h1 + a @ W["Wd"].T
    return y, dict(h1=h1, xn2=xn2, r2=r2, gt=gt, up=up, a=a)


def mlp_backward(dy, c, W):
    g = {}
    g["Wd"] = dy.T @ c["a"]
    da = dy @ W["Wd"]
    dgt = da * c["up"] * silu_grad(c["gt"])
    dup = da * silu(c["gt"])
    g["Wg"] = dgt.T @ c["xn2"]
    g["Wu"] = dup.T @ c["xn2"]
    dxn2 = dgt @ W["Wg"] + dup @ W["Wu"]
    dh1 = dy + rmsnorm_bwd(c["h1"], c["r2"], dxn2)
    return dh1, g


# ------------------------------------------------------------------ block

def block_forward(x, W, cfg, a8=False):
    h1, ca = attn_forward(x, W, cfg, a8)
    y, cm = mlp_forward(h1, W, a8)
    return y, (ca, cm)


def block_backward(dy, cache, W, cfg):
    ca, cm = cache
    dh1, gm = mlp_backward(dy, cm, W)
    dx, ga = attn_backward(dh1, ca, W, cfg)
    ga.update(gm)
    return dx, ga


# ------------------------------------------------- selected tokens only

def attn_forward_rows(x, W, cfg, rows):
    """h1 = x + o_proj(attention) for the token rows ``rows`` only (Eq. 7's
    window forward restricted to some outputs).  Causal attention lets token
    s of sample b see tokens 0..s of b alone, so the keys and values of that
    prefix and the query of token s are all it needs; every step is the one
    attn_forward takes, applied to that subset (checked against it)."""
    S = cfg.seq
    Hq, Hkv, hd = cfg.n_q, cfg.n_kv, cfg.head_dim
    G = Hq // Hkv
    cos, sin = rope_tables(S, hd, cfg.rope_theta)
    rows = [int(t) for t in rows]
    out = np.empty((len(rows), x.shape[1]))
    by_sample = {}
    for i, t in enumerate(rows):
        by_sample.setdefault(t // S, []).append(i)
    for b, idxs in by_sample.items():
        last = max(rows[i] % S for i in idxs)
        xn, _ = rmsnorm(x[b * S: b * S + last + 1])
        k = (xn @ W["Wk"].T).reshape(1, last + 1, Hkv, hd)
        v = (xn @ W["Wv"].T).reshape(1, last + 1, Hkv, hd)
        if cfg.qk_norm:
            k, _ = rmsnorm(k)
        kr = rope(k, cos[:last + 1], sin[:last + 1])
        for i in idxs:
            s = rows[i] % S
            q = (xn[s:s + 1] @ W["Wq"].T).reshape(1, 1, Hq, hd)
            if cfg.qk_norm:
                q, _ = rmsnorm(q)
            qr = rope(q, cos[s:s + 1], sin[s:s + 1])
            o = np.empty((Hq, hd))
            for h in range(Hq):
                sc = kr[0, :s + 1, h // G, :] @ qr[0, 0, h, :] / np.sqrt(hd)
                e = np.exp(sc - sc.max())
                o[h] = (e / e.sum()) @ v[0, :s + 1, h // G, :]
            out[i] = x[rows[i]] + o.reshape(-1) @ W["Wo"].T
    return out


def block_forward_rows(x, W, cfg, rows):
    """Block output for the token rows ``rows`` (the MLP half is per token)."""
    return mlp_forward(attn_forward_rows(x, W, cfg, rows), W)[0]


def recon_loss(y_q, y_fp):
    """Eq. 7 as a mean over all n outputs: L = (1/n) sum (y_q - y_fp)^2 and
    dL/dy_q = 2 (y_q - y_fp)/n."""
    d = np.asarray(y_q, np.float64) - np.asarray(y_fp, np.float64)
    n = d.size
    return float(np.sum(d * d) / n), 2.0 * d / n
