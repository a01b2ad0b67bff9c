"""Oracle parity of the calibration step at the benchmarked sizes.

* The whole reconstruction step of the Qwen3-1.7B-shaped block (4 samples x
  2048 tokens, all 50.3M weights), soft at s = 15 and hard with the
  backward at s0 = 30, on seeded perturbed factors: loss, block output, the
  input gradient of every token and all 21 factor-gradient arrays of the
  seven linears against the float64 oracle (Eq. 3-7, Sec. 2.2-2.4).  The
  oracle runs the samples one at a time (they are independent in the
  block) and sums their weight gradients before the factor-gradient pass.
* The fused attention in the launch configuration the full-size blocks use
  (the dK/dV kernel summing several q heads per block, sequences of 2048 and
  4096) against the oracle's causal GQA attention, on sampled (sample, kv
  head) groups: every query row of O and dQ and every key row of dK and dV
  of the group's heads.
"""
import dataclasses
import gc

import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, median_rel, to_dev_bf16
from oracle import block, calib, lmst

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

LIN_ID = {"qkv": 0, "o": 1, "gu": 2, "d": 3}
TOL = 2e-2


def _oracle_step_by_sample(xo, Wo, fac, cfg, mode, s, s_bwd):
    """The oracle's block step over cfg.batch samples run one at a time:
    the loss is the mean of the per-sample means, so the output gradient,
    the input gradient and the weight gradients of the batch are the
    per-sample ones divided by the batch size."""
    one = dataclasses.replace(cfg, batch=1)
    Wf = calib.fake_weights(Wo, fac, 128, mode, s)
    B, S = cfg.batch, cfg.seq
    losses, dxs, yqs = [], [], []
    dW = {k: np.zeros_like(v) for k, v in Wo.items()}
    for b in range(B):
        xb = xo[b * S:(b + 1) * S]
        y_fp, _ = block.block_forward(xb, Wo, one)
        y_q, cache = block.block_forward(xb, Wf, one)
        loss, dy = block.recon_loss(y_q, y_fp)
        dx, dWb = block.block_backward(dy / B, cache, Wf, one)
        del cache
        losses.append(loss)
        dxs.append(dx)
        yqs.append(y_q)
        for k in dW:
            dW[k] += dWb[k]
        print(f"[oracle] sample {b} done", flush=True)
    fg = calib.factor_grads_all(dW, Wo, fac, 128, mode, s, s_bwd)
    return dict(loss=float(np.mean(losses)), dx=np.concatenate(dxs), y_q=np.concatenate(yqs),
                fgrads=fg)


@pytest.fixture(scope="module")
def c2_block():
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = sg.QWEN3_1P7B
    W = sg.block_weights(cfg, 0)
    blk = DenseBlock(cfg, W)
    fac = {}
    for name, L in blk.lin.items():
        f = sg.perturbed_factors(21, L.n_groups, extra=(LIN_ID[name],))
        L.set_factors(*f)
        parts = [DenseBlock.split_fused(cfg, name, a) for a in f]
        for k in parts[0]:
            fac[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    xb = sg.activations(cfg, 0)
    yield cfg, W, blk, fac, xb
    del blk
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode,s", [(lmst.SOFT, 15.0), (lmst.HARD, None)], ids=["soft15", "hard"])
def test_full_size_step_parity_qwen3_1p7b(catq, c2_block, mode, s):
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg, W, blk, fac, xb = c2_block
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    print(f"[c2 step] mode={mode} s={s}: GPU step", flush=True)
    loss = blk.step(x, y_fp, mode=mode, s=s if s else 15.0, s_bwd=30.0, recompute_stats=True)
    torch.cuda.synchronize()
    got_loss, got_y, got_dx = loss.item(), host(blk.y), host(blk.dx)
    got_g = {}
    for name, L in blk.lin.items():
        parts = [DenseBlock.split_fused(cfg, name, host(a)) for a in (L.g_mu, L.g_alpha, L.g_delta)]
        for k in parts[0]:
            got_g[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    del x, y_fp
    Wo = {k: f64(v) for k, v in W.items()}
    ref = _oracle_step_by_sample(f64(xb), Wo, fac, cfg, mode, s, 30.0)
    print(f"[c2 step] loss GPU {got_loss:.6e} oracle {ref['loss']:.6e}", flush=True)
    assert abs(got_loss - ref["loss"]) <= TOL * ref["loss"]
    assert max_norm_err(got_y, ref["y_q"]) <= TOL
    err_dx = max_norm_err(got_dx, ref["dx"])
    print(f"[c2 step] dx error {err_dx:.4f} (median rel {median_rel(got_dx, ref['dx']):.2e})",
          flush=True)
    assert err_dx <= TOL
    assert sorted(got_g) == sorted(Wo) and len(got_g) == 7
    worst = 0.0
    for k in sorted(got_g):
        for i in range(3):
            err = max_norm_err(got_g[k][i], ref["fgrads"][k][i])
            worst = max(worst, err)
            assert err <= TOL, (k, i, err, median_rel(got_g[k][i], ref["fgrads"][k][i]))
    print(f"[c2 step] worst of the 21 factor-gradient errors {worst:.4f}", flush=True)


# ----------------------------------------------------------------- attention

def _oracle_group_attention(qkv, S, G, d, qk_norm, theta, dO):
    """Causal attention of one (sample, kv head) group: qkv holds the
    group's G q heads, its k head and v head as [S][(G + 2) d]; dO is
    [S][G d].  Heads are independent apart from sharing k and v, so the
    group is the whole problem for the oracle's batch-1, one-kv-head case."""
    q = qkv[:, :G * d].reshape(1, S, G, d)
    k = qkv[:, G * d:(G + 1) * d].reshape(1, S, 1, d)
    v = qkv[:, (G + 1) * d:].reshape(1, S, 1, d)
    if qk_norm:
        qn, rq = block.rmsnorm(q)
        kn, rk = block.rmsnorm(k)
    else:
        qn, kn = q, k
    cos, sin = block.rope_tables(S, d, theta)
    qr, kr = block.rope(qn, cos, sin), block.rope(kn, cos, sin)
    O, P = block.causal_attention(qr, kr, v)
    dqr, dkr, dv = block.causal_attention_bwd(qr, kr, v, P, dO.reshape(1, S, G, d))
    del P
    dq, dk = block.rope_bwd(dqr, cos, sin), block.rope_bwd(dkr, cos, sin)
    if qk_norm:
        dq, dk = block.rmsnorm_bwd(q, rq, dq), block.rmsnorm_bwd(k, rk, dk)
    return O.reshape(S, G * d), dq.reshape(S, G * d), dk.reshape(S, d), dv.reshape(S, d)


@pytest.mark.parametrize("geom", [
    # (B, S, Hq, Hkv, d, qk_norm, theta, sampled (sample, kv head) groups)
    (4, 2048, 16, 8, 128, True, 1e6, [(0, 0), (3, 7), (2, 3)]),   # 1.7B-shaped: 2 q heads/block
    (2, 4096, 40, 8, 128, True, 1e6, [(1, 7), (0, 2)]),           # 14B-shaped: 5 q heads/block
    (4, 2048, 32, 8, 128, False, 5e5, [(3, 5)]),                  # 8B-shaped: 4 q heads/block
    (2, 2048, 64, 4, 128, True, 1e6, [(0, 3), (1, 0)]),           # 235B-shaped: 16 heads over 4 blocks
], ids=["qwen3-1.7b", "qwen3-14b", "llama3-8b", "qwen3-235b"])
def test_attention_parity_block_geometry(catq, geom):
    import torch
    B, S, Hq, Hkv, d, qk, theta, groups = geom
    G = Hq // Hkv
    M = B * S
    ld = (Hq + 2 * Hkv) * d
    qb = sg.normal_bf16(1, "X", (M, ld))
    gb = sg.normal_bf16(2, "Y", (M, Hq * d), std=0.1)
    qkv, dO = to_dev_bf16(qb), to_dev_bf16(gb)
    desc = catq.attn_desc(B, S, Hq, Hkv, d, qk, theta)
    saved = torch.empty(catq.catq_attn_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(catq.catq_attn_bwd_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    o = torch.empty(M, Hq * d, dtype=torch.bfloat16, device="cuda")
    dqkv = torch.empty(M, ld, dtype=torch.bfloat16, device="cuda")
    print(f"[attention] B={B} S={S} Hq={Hq} Hkv={Hkv}", flush=True)
    catq.catq_aux_attention_fwd(desc, qkv, o, saved)
    catq.catq_aux_attention_bwd(desc, qkv, o, saved, dO, dqkv, ws)
    torch.cuda.synchronize()
    for b, h in groups:
        rows = slice(b * S, (b + 1) * S)
        qc = slice(h * G * d, (h + 1) * G * d)
        kc = slice((Hq + h) * d, (Hq + h + 1) * d)
        vc = slice((Hq + Hkv + h) * d, (Hq + Hkv + h + 1) * d)
        grp = np.concatenate([qb[rows, qc], qb[rows, kc], qb[rows, vc]], 1)
        Or, dq, dk, dv = _oracle_group_attention(f64(grp), S, G, d, qk, theta, f64(gb[rows, qc]))
        for what, got, ref in (("O", o[rows, qc], Or), ("dQ", dqkv[rows, qc], dq),
                               ("dK", dqkv[rows, kc], dk), ("dV", dqkv[rows, vc], dv)):
            err = max_norm_err(host(got), ref)
            print(f"[attention] group ({b}, {h}) {what} error {err:.4f}", flush=True)
            assert err <= TOL, (b, h, what, err)
