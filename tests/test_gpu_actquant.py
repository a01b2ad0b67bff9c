"""GPU parity of the W1.58A8 activation fake quantization: the standalone
quantizer bit for bit against the oracle on the same inputs (codes decided in
fp32 on both sides), Q/K/V quantization inside the attention preparation,
and the a8 calibration step of a dense block against the oracle's a8 step
fed the GPU's quantized activations."""
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


def _saved_heads(saved, cfg):
    """Q, K, V heads as the attention preparation saved them (quantized when
    act_quant is on), in the oracle's [B][S][H][d] layout.  Saved layout: Q
    heads, K heads, q/k rstd, rope cos, sin, V heads ([B][H][S][d] each,
    regions rounded up to 256 bytes)."""
    ru = lambda b: (b + 255) // 256 * 256
    B, S, d = cfg.batch, cfg.seq, cfg.head_dim
    nq, nk = B * cfg.n_q * S * d, B * cfg.n_kv * S * d
    o_k = ru(nq * 2)
    o_v = o_k + ru(nk * 2) + ru(B * S * (cfg.n_q + cfg.n_kv) * 4) + 2 * ru(S * (d // 2) * 4)
    out = []
    for off, cnt, H in ((0, nq, cfg.n_q), (o_k, nk, cfg.n_kv), (o_v, nk, cfg.n_kv)):
        t = saved[off:off + 2 * cnt].view(torch_bf16()).float().cpu().numpy().astype(np.float64)
        out.append(t.reshape(B, H, S, d).transpose(0, 2, 1, 3))
    return out


def torch_bf16():
    import torch
    return torch.bfloat16


@pytest.mark.parametrize("mode,s", [(lmst.SOFT, 15.0), (lmst.HARD, 0.0)])
def test_a8_dense_step(catq, mode, s):
    """The a8 calibration step against the oracle's a8 step fed the GPU's own
    quantized activations (so both sides take the same code decisions; the
    quantizer itself is checked bit for bit above): output, loss, input
    gradient and every factor gradient at 2e-2.  Reported: the oracle on its
    own quantization, whose codes near a rounding boundary land one step
    (1/127 of the group maximum) away from the GPU's because the two
    quantize activations that differ by upstream bf16 rounding."""
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
    qr, kr, v = _saved_heads(blk.saved, cfg)
    given = {"xn1": host(blk.xn1), "qr": qr, "kr": kr, "v": v, "attn": host(blk.attn_q),
             "xn2": host(blk.xn2), "a": host(blk.a)}
    got_g = {}
    for name, L in blk.lin.items():
        parts = [DenseBlock.split_fused(cfg, name, host(a)) for a in (L.g_mu, L.g_alpha, L.g_delta)]
        for k in parts[0]:
            got_g[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    Wo = {k: f64(v) for k, v in W.items()}
    sv = s if s else None
    tol = 2e-2
    ref = calib.dense_step(f64(xb), Wo, fac, cfg, mode, s=sv, s_bwd=30.0, a8=given)
    own = calib.dense_step(f64(xb), Wo, fac, cfg, mode, s=sv, s_bwd=30.0, a8=True)
    for r in (ref, own):
        assert max_norm_err(host(y_fp), r["y_fp"]) <= tol
        assert max_norm_err(host(blk.y), r["y_q"]) <= tol
        assert abs(loss.item() - r["loss"]) <= tol * r["loss"], (loss.item(), r["loss"])
        assert max_norm_err(host(blk.dx), r["dx"]) <= tol
    worst = worst_own = 0.0
    for k in got_g:
        for i in range(3):
            err = max_norm_err(got_g[k][i], ref["fgrads"][k][i])
            worst = max(worst, err)
            assert err <= tol, (k, i, err, median_rel(got_g[k][i], ref["fgrads"][k][i]))
            worst_own = max(worst_own, max_norm_err(got_g[k][i], own["fgrads"][k][i]))
    print(f"[a8] factor-gradient error {worst:.4f} on the GPU's quantized activations, "
          f"{worst_own:.4f} on the oracle's own", flush=True)
    assert worst_own <= 5e-2
    # the a8 step and its two-stream schedule agree bit for bit
    a = blk.step(x, y_fp, mode=mode, s=s, s_bwd=30.0, overlap=False).clone()
    g1 = [L.g_delta.clone() for L in blk.lin.values()]
    b = blk.step(x, y_fp, mode=mode, s=s, s_bwd=30.0, overlap=True).clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    for u, L in zip(g1, blk.lin.values()):
        assert torch.equal(u, L.g_delta)
