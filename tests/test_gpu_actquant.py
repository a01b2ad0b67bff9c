"""GPU parity of the W1.58A8 activation fake quantization: the standalone
quantizer bit for bit against the oracle on the same inputs (codes decided in
fp32 on both sides), Q/K/V quantization inside the attention preparation,
and the a8 calibration step of a dense block against the oracle's a8 step."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, median_rel, to_dev_bf16, to_dev_f32
from oracle import actquant, calib, lmst

pytestmark = pytest.mark.gpu


def _ties(rows, n, seed):
    """Rows whose quotients x/s land exactly on half-integers: the max is
    127 c and the others (j + 0.5) c with c a power of two (exact in bf16)."""
    rng = np.random.default_rng(seed)
    out = np.empty((rows, n), np.float32)
    for r in range(rows):
        c = np.float32(2.0 ** -rng.integers(2, 10))
        j = rng.integers(-126, 126, n).astype(np.float32) + np.float32(0.5)
        out[r] = j * c
        out[r, rng.integers(0, n)] = np.float32(127) * c * (1 if rng.random() < 0.5 else -1)
    return out


@pytest.mark.parametrize("rows,n,group", [(37, 2048, 2048), (16, 6144, 128), (5, 17408, 17408),
                                          (64, 256, 64)])
def test_act_quant_bitexact(catq, rows, n, group):
    import torch
    rng = np.random.default_rng(rows * n)
    x = np.concatenate([rng.standard_t(4, (rows - 2, n)).astype(np.float32) * 0.7,
                        _ties(2, n, rows)])
    x[0, :group] = 0.0                                     # an all-zero group
    xb = sg.f32_to_bf16_bits(x)
    xq_ref, q_ref, s_ref = actquant.quantize(f64(xb), group)
    xd = to_dev_bf16(xb)
    y = torch.empty_like(xd)
    catq.catq_aux_act_quant(xd, y, group)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(y), xq_ref)
    catq.catq_aux_act_quant(xd, xd, group)                 # in place
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(xd), xq_ref)
    # fp32 input: the quantizer on the fp32 values
    xf = x.copy()
    yq = torch.empty(rows, n, dtype=torch.bfloat16, device="cuda")
    catq.catq_aux_act_quant(to_dev_f32(xf), yq, group)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(yq), actquant.quantize(xf.astype(np.float64), group)[0])


def test_attention_operands_quantized(catq):
    """With act_quant the saved Q, K, V heads are the quantizer applied to
    the unquantized heads (the same preparation otherwise), per (token,
    head); the quantizer runs in fp32 on both sides, so they agree exactly."""
    import torch
    cfg = sg.small_dense(batch=2, seq=136, n_q=4, n_kv=2, head_dim=128)
    M, d = cfg.tokens, cfg.head_dim
    ld = (cfg.n_q + 2 * cfg.n_kv) * d
    qkv = to_dev_bf16(sg.normal_bf16(1, "X", (M, ld)))
    outs = []
    for aq in (False, True):
        desc = catq.attn_desc(cfg.batch, cfg.seq, cfg.n_q, cfg.n_kv, d, True, cfg.rope_theta,
                              act_quant=aq)
        saved = torch.zeros(catq.catq_attn_saved_bytes(desc), dtype=torch.uint8, device="cuda")
        o = torch.empty(M, cfg.n_q * d, dtype=torch.bfloat16, device="cuda")
        catq.catq_aux_attention_fwd(desc, qkv, o, saved)
        torch.cuda.synchronize()
        outs.append(saved)
    # saved layout: Q heads, K heads, q/k rstd, rope cos, sin, V heads (each
    # region rounded up to 256 bytes)
    ru = lambda b: (b + 255) // 256 * 256
    B, S = cfg.batch, cfg.seq
    nq, nk = B * cfg.n_q * S * d, B * cfg.n_kv * S * d
    o_k = ru(nq * 2)
    o_v = o_k + ru(nk * 2) + ru(B * S * (cfg.n_q + cfg.n_kv) * 4) + 2 * ru(S * (d // 2) * 4)
    for off, cnt in ((0, nq), (o_k, nk), (o_v, nk)):
        plain = outs[0][off:off + 2 * cnt].view(torch.bfloat16).float().cpu().numpy()
        quant = outs[1][off:off + 2 * cnt].view(torch.bfloat16).float().cpu().numpy()
        np.testing.assert_array_equal(quant.astype(np.float64).reshape(-1, d),
                                      actquant.quantize(plain.astype(np.float64).reshape(-1, d), d)[0])


@pytest.mark.parametrize("mode,s", [(lmst.SOFT, 15.0), (lmst.HARD, 0.0)])
def test_a8_dense_step(catq, mode, s):
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = sg.small_dense(batch=2, seq=136, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    W = sg.block_weights(cfg, 0)
    blk = DenseBlock(cfg, W, a8=True)
    fac = {}
    lin_id = {"qkv": 0, "o": 1, "gu": 2, "d": 3}
    for name, L in blk.lin.items():
        f = sg.perturbed_factors(1, L.n_groups, extra=(lin_id[name],))
        L.set_factors(*f)
        parts = [DenseBlock.split_fused(cfg, name, a) for a in f]
        for k in parts[0]:
            fac[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    xb = sg.activations(cfg, 0)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    loss = blk.step(x, y_fp, mode=mode, s=s, s_bwd=30.0)
    torch.cuda.synchronize()
    Wo = {k: f64(v) for k, v in W.items()}
    ref = calib.dense_step(f64(xb), Wo, fac, cfg, mode, s=s if s else None, s_bwd=30.0, a8=True)
    tol = 2e-2
    assert max_norm_err(host(y_fp), ref["y_fp"]) <= tol
    assert max_norm_err(host(blk.y), ref["y_q"]) <= tol
    assert abs(loss.item() - ref["loss"]) <= tol * ref["loss"], (loss.item(), ref["loss"])
    assert max_norm_err(host(blk.dx), ref["dx"]) <= tol
    # Factor gradients: the two sides quantize activations that differ by the
    # upstream bf16 rounding, so a code whose quotient lies within that
    # rounding of a half-integer lands one step apart (1/127 of its group's
    # maximum, ~15% of the codes at 2^-8 relative noise).  In G = dY^T X_q
    # that is about 1% of extra relative noise, which the signed per-group
    # sums of the factor gradients amplify: their bound is doubled.
    tol_g = 2 * tol
    for name, L in blk.lin.items():
        parts = [DenseBlock.split_fused(cfg, name, host(a)) for a in (L.g_mu, L.g_alpha, L.g_delta)]
        for k in parts[0]:
            for i in range(3):
                g = np.asarray(parts[i][k]).reshape(-1)
                err = max_norm_err(g, ref["fgrads"][k][i])
                assert err <= tol_g, (k, i, err, median_rel(g, ref["fgrads"][k][i]))
    # the a8 step and its two-stream schedule agree bit for bit
    a = blk.step(x, y_fp, mode=mode, s=s, s_bwd=30.0, overlap=False).clone()
    g1 = [L.g_delta.clone() for L in blk.lin.values()]
    b = blk.step(x, y_fp, mode=mode, s=s, s_bwd=30.0, overlap=True).clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    for u, L in zip(g1, blk.lin.values()):
        assert torch.equal(u, L.g_delta)
