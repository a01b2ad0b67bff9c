"""Learnable modulation + softened ternarization, float64 reference.

Follows Sec. 2.1 (Eq. 1-2), Sec. 2.2 (Eq. 3-4), Sec. 2.3 (Eq. 5-6) and the
group-wise scheme of App. B.2.  Readings of points the paper leaves open are
marked READING; they are listed with their reasons in the design notes.

Weights arrive as the exact values of their storage type (bf16 or fp32)
widened to float64.  Group j of a [d_out][d_in] matrix is the j-th run of g
consecutive elements of its row-major flattening (App. B.2); with d_in a
multiple of g a group is a g-wide slice of one row.
"""
from __future__ import annotations

import numpy as np

IDENTITY, SOFT, HARD = 0, 1, 2
FLT_MIN = float(np.finfo(np.float32).tiny)


def f32(x):
    """Round float64 to float32 (IEEE round-to-nearest-even) and widen back."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


# ------------------------------------------------------------------ groups

def as_groups(W, g):
    W = np.asarray(W, dtype=np.float64)
    if W.size % g:
        raise ValueError("weight count not a multiple of the group size")
    return W.reshape(-1, g)


def canonical_sum(a):
    """Sum over the last axis (length g = 8*L, L a power of two) in a fixed
    order: inside each run of 8 the pairs (j, j+4), (j, j+2), (j, j+1); then the
    L partial sums folded in halves.  READING: the paper defines the group
    mean; this fixed order makes the float64 sum reproducible bit for bit."""
    a = np.asarray(a, dtype=np.float64)
    g = a.shape[-1]
    L = g // 8
    if L * 8 != g or L & (L - 1):
        raise ValueError("group size must be 8 times a power of two")
    a = a.reshape(a.shape[:-1] + (L, 8))
    a = a[..., :4] + a[..., 4:]
    a = a[..., :2] + a[..., 2:]
    a = a[..., 0] + a[..., 1]
    while L > 1:
        L //= 2
        a = a[..., :L] + a[..., L:]
    return a[..., 0]


def group_stats(W, g=128):
    """Eq. 3: mu0 = mean of the group, alpha0 = mean |W - mu0|.
    Both accumulated in float64 (canonical_sum), scaled by 1/g and rounded to
    fp32; alpha0 uses the fp32 mu0.  Returns (mu0, alpha0) as float64 arrays of
    fp32 values, one per group."""
    Wg = as_groups(W, g)
    mu0 = f32(canonical_sum(Wg) * (1.0 / g))
    alpha0 = f32(canonical_sum(np.abs(Wg - mu0[:, None])) * (1.0 / g))
    return mu0, alpha0


def expand(v, n_groups, stride):
    """Per-group view of a factor: stride 1 = one value per group, stride 0 =
    one shared scalar (App. B.2 keeps parameters per group; the shared form
    serves the single-threshold variant)."""
    v = np.asarray(v, dtype=np.float64).reshape(-1)
    if stride == 0 or v.size == 1:
        return np.full(n_groups, v[0])
    if v.size < n_groups:
        raise ValueError("fewer factor values than groups")
    return v[:n_groups]


def modulation(mu0, alpha0, d_mu, d_alpha, d_delta, delta0=0.5):
    """Eq. 3-4: mu = mu0 + d_mu*alpha0, alpha = d_alpha*alpha0,
    Delta = d_Delta*Delta0.  Each is formed in float64 from fp32 operands and
    rounded once to fp32 (the products are exact in float64).  READING: fp32
    storage of the per-group scalars."""
    mu = f32(mu0 + np.asarray(d_mu, np.float64) * alpha0)
    alpha = f32(np.asarray(d_alpha, np.float64) * alpha0)
    delta = f32(np.asarray(d_delta, np.float64) * np.float64(np.float32(delta0)))
    return mu, alpha, delta


def safe_alpha(alpha):
    """READING for a constant group (alpha0 = 0, or alpha = 0): divide by
    max(alpha, smallest normal fp32) so every transformed weight stays finite."""
    return np.maximum(alpha, FLT_MIN)


def transformed(W, g, mu, alpha):
    """Eq. 3: W_hat = (W - mu)/alpha, float64, per element."""
    Wg = as_groups(W, g)
    return (Wg - mu[:, None]) / safe_alpha(alpha)[:, None]


# ------------------------------------------------------------ Eq. 5 and 2

def transition_parts(x_hat, s, delta):
    """Transition function of Eq. 5,
        f(W; s, D) = [tanh(s(W - D)) + tanh(s(W + D))] / (2 tanh s),
    with its partial derivatives f_W = df/dW and f_D = df/dD, evaluated in a
    cancellation-free form.  With x = |W|, a = s(x - D), b = s(x + D),
    qa = exp(-2|a|), qb = exp(-2b), E = 1 - exp(-4 s x), E_D = 1 - exp(-4 s D):
        tanh a + tanh b = 2E/((1+qa)(1+qb))          if x >= D
                        = 2 qa E/((1+qa)(1+qb))       if x <  D
        sech^2 a = 4 qa/(1+qa)^2,  sech^2 b = 4 qb/(1+qb)^2
        qb = qa (1 - E_D) (x >= D)  or  qa (1 - E) (x < D)
        sech^2 b - sech^2 a = 4 (qb - qa)(1 - qa qb)/((1+qa)^2 (1+qb)^2)
    f is odd in W, f_W even, f_D odd.  ``delta`` broadcasts against x_hat."""
    xh = np.asarray(x_hat, dtype=np.float64)
    s = np.float64(s)
    D = np.broadcast_to(np.asarray(delta, dtype=np.float64), xh.shape)
    x = np.abs(xh)
    sg = np.sign(xh)
    d = x - D
    ge = d >= 0
    qa = np.exp(-2.0 * s * np.abs(d))
    E = -np.expm1(-4.0 * s * x)
    ED = -np.expm1(-4.0 * s * D)
    eb = np.where(ge, ED, E)              # 1 - qb/qa
    qb = qa * (1.0 - eb)
    k = 1.0 / (2.0 * np.tanh(s))
    pa, pb = 1.0 + qa, 1.0 + qb
    f = sg * (2.0 * E * np.where(ge, 1.0, qa)) / (pa * pb) * k
    fW = s * (4.0 * qa / (pa * pa) + 4.0 * qb / (pb * pb)) * k
    one_m_qaqb = np.where(ge, E, ED)      # 1 - qa*qb
    fD = sg * s * 4.0 * (-qa * eb) * one_m_qaqb / (pa * pa * pb * pb) * k
    return f, fW, fD


def transition(x_hat, s, delta):
    return transition_parts(x_hat, s, delta)[0]


def hard_codes(W, g, mu, alpha, delta):
    """Eq. 2 and Eq. 4: T = Q(W_hat; Delta) = +1 if W_hat > Delta, 0 if
    |W_hat| <= Delta, -1 if W_hat < -Delta, with W_hat = (W - mu)/alpha.
    Decided without a division: r = W - mu and theta = Delta*alpha (exact
    product) in float64, then r > theta / r < -theta.  An exact tie gives 0."""
    Wg = as_groups(W, g)
    r = Wg - mu[:, None]
    theta = (delta * safe_alpha(alpha))[:, None]
    return ((r > theta).astype(np.int8) - (r < -theta).astype(np.int8))


# ---------------------------------------------------------- forward (a1-a3)

def modulate_ternarize(W, g, d_mu, d_alpha, d_delta, mode, s=None, delta0=0.5,
                       strides=(1, 1, 1), stats=None):
    """One LM+ST forward for a weight matrix (Eq. 3-6 with W ~ alpha*T, no mu,
    Sec. 2.2).  Returns dict with float64 ``W_fake`` shaped like W, the group
    stats, the per-group (mu, alpha, Delta) and, in HARD mode, the int8 codes.

    mode IDENTITY (t = 0):        W_fake = W
    mode SOFT (0 < t <= gamma):   W_fake = alpha * f(W_hat; s, Delta)
    mode HARD (gamma < t <= 1):   W_fake = alpha * Q(W_hat; Delta)
    """
    W = np.asarray(W, dtype=np.float64)
    mu0, alpha0 = group_stats(W, g) if stats is None else stats
    n = mu0.shape[0]
    dm = expand(d_mu, n, strides[0])
    da = expand(d_alpha, n, strides[1])
    dd = expand(d_delta, n, strides[2])
    mu, alpha, delta = modulation(mu0, alpha0, dm, da, dd, delta0)
    out = dict(mu0=mu0, alpha0=alpha0, mu=mu, alpha=alpha, delta=delta)
    if mode == IDENTITY:
        out["W_fake"] = W.copy()
        return out
    if mode == SOFT:
        if not (s is not None and s > 0):
            raise ValueError("SOFT mode needs s > 0")
        T = transition(transformed(W, g, mu, alpha), s, delta[:, None])
        out["T"] = T.reshape(W.shape)
    elif mode == HARD:
        codes = hard_codes(W, g, mu, alpha, delta)
        out["codes"] = codes.reshape(W.shape)
        T = codes.astype(np.float64)
        out["T"] = T.reshape(W.shape)
    else:
        raise ValueError("bad mode")
    out["W_fake"] = (alpha[:, None] * T).reshape(W.shape)
    return out


# --------------------------------------------------------- backward (a10)

def factor_grads(G, W, g, d_mu, d_alpha, d_delta, mode, s=None, s_bwd=0.0, delta0=0.5,
                 strides=(1, 1, 1), stats=None):
    """Gradients of a loss L with dL/dW_fake = G with respect to the three
    learnable factors of Eq. 3-4 (W is frozen; only the factors learn).

    From W_fake = alpha*T(W_hat), W_hat = (W - mu)/alpha:
        dL/dmu    = -sum G f_W
        dL/dalpha =  sum G T - sum G f_W W_hat
        dL/dDelta =  alpha sum G f_D
    and mu = mu0 + d_mu alpha0, alpha = d_alpha alpha0, Delta = d_Delta Delta0:
        dL/dd_mu = alpha0 dL/dmu,  dL/dd_alpha = alpha0 dL/dalpha,
        dL/dd_Delta = Delta0 dL/dDelta.
    SOFT uses f's derivatives at s.  HARD takes T = Q and, READING of the
    hard-stage rule of Sec. 2.3, the surrogate derivatives of f at s_bwd
    (s_bwd = 0 gives the straight-through f_W = 1, f_D = 0).  IDENTITY has no
    dependence on the factors.  Shared (stride 0) factors get the sum over
    groups.  Returns three float64 arrays (length n_groups, or 1 if shared)."""
    W = np.asarray(W, dtype=np.float64)
    Gg = as_groups(G, g)
    mu0, alpha0 = group_stats(W, g) if stats is None else stats
    n = mu0.shape[0]
    dm = expand(d_mu, n, strides[0])
    da = expand(d_alpha, n, strides[1])
    dd = expand(d_delta, n, strides[2])
    mu, alpha, delta = modulation(mu0, alpha0, dm, da, dd, delta0)
    if mode == IDENTITY:
        z = np.zeros(n)
        gm, ga, gd = z, z.copy(), z.copy()
    else:
        xh = transformed(W, g, mu, alpha)
        if mode == SOFT:
            T, fW, fD = transition_parts(xh, s, delta[:, None])
        elif mode == HARD:
            T = hard_codes(W, g, mu, alpha, delta).astype(np.float64)
            if s_bwd > 0:
                _, fW, fD = transition_parts(xh, s_bwd, delta[:, None])
            else:
                fW, fD = np.ones_like(xh), np.zeros_like(xh)
        else:
            raise ValueError("bad mode")
        S_T = (Gg * T).sum(1)
        S_W = (Gg * fW * xh).sum(1)
        S_1 = (Gg * fW).sum(1)
        S_D = (Gg * fD).sum(1)
        gm = alpha0 * (-S_1)
        ga = alpha0 * (S_T - S_W)
        gd = np.float64(np.float32(delta0)) * (alpha * S_D)
    res = []
    for v, st in zip((gm, ga, gd), strides):
        res.append(np.array([v.sum()]) if st == 0 else v)
    return tuple(res)


# ------------------------------------------------------------- pack (a11)

def pack_ternary(codes):
    """Deployment storage of T in {-1,0,+1} (App. B.2, zero-point free):
    READING of the bit layout, which the paper leaves open: code c = T + 1 in
    {0,1,2}; byte b of a row holds elements 4b..4b+3, element 4b+j in bits
    2j..2j+1 (least significant first).  Returns uint8 [d_out][d_in/4]."""
    c = np.asarray(codes).astype(np.int64) + 1
    if c.min(initial=1) < 0 or c.max(initial=1) > 2:
        raise ValueError("codes must be in {-1,0,1}")
    d_out, d_in = c.shape
    c = c.reshape(d_out, d_in // 4, 4)
    b = c[..., 0] | (c[..., 1] << 2) | (c[..., 2] << 4) | (c[..., 3] << 6)
    return b.astype(np.uint8)


def unpack_ternary(packed, d_in):
    p = np.asarray(packed).astype(np.int64)
    out = np.stack([(p >> (2 * j)) & 3 for j in range(4)], axis=-1)
    return (out.reshape(p.shape[0], d_in) - 1).astype(np.int8)
