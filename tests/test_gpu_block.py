"""GPU parity of attention, the dense and routed-expert block steps, and the
fp32 single-linear calibration against the oracle."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, median_rel, to_dev_bf16, to_dev_f32
from oracle import block, calib, lmst, moe

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------- attention

def _oracle_attention(qkv, cfg, dO):
    B, S, Hq, Hkv, d = cfg.batch, cfg.seq, cfg.n_q, cfg.n_kv, cfg.head_dim
    q = qkv[:, :Hq * d].reshape(B, S, Hq, d)
    k = qkv[:, Hq * d:(Hq + Hkv) * d].reshape(B, S, Hkv, d)
    v = qkv[:, (Hq + Hkv) * d:].reshape(B, S, Hkv, d)
    if cfg.qk_norm:
        qn, rq = block.rmsnorm(q)
        kn, rk = block.rmsnorm(k)
    else:
        qn, kn = q, k
    cos, sin = block.rope_tables(S, d, cfg.rope_theta)
    qr, kr = block.rope(qn, cos, sin), block.rope(kn, cos, sin)
    O, P = block.causal_attention(qr, kr, v)
    dOr = dO.reshape(B, S, Hq, d)
    dqr, dkr, dv = block.causal_attention_bwd(qr, kr, v, P, dOr)
    dq, dk = block.rope_bwd(dqr, cos, sin), block.rope_bwd(dkr, cos, sin)
    if cfg.qk_norm:
        dq, dk = block.rmsnorm_bwd(q, rq, dq), block.rmsnorm_bwd(k, rk, dk)
    dqkv = np.concatenate([dq.reshape(B * S, -1), dk.reshape(B * S, -1), dv.reshape(B * S, -1)], 1)
    return O.reshape(B * S, Hq * d), dqkv


@pytest.mark.parametrize("S,d,qk", [(80, 64, True), (136, 128, True), (264, 64, False),
                                    (512, 128, True), (200, 256, True), (1000, 128, False)])
def test_attention_parity(catq, S, d, qk):
    import torch
    cfg = sg.small_dense(batch=2, seq=S, n_q=4, n_kv=2, head_dim=d, qk_norm=qk)
    M = cfg.tokens
    ld = (cfg.n_q + 2 * cfg.n_kv) * d
    qb = sg.normal_bf16(1, "X", (M, ld))
    gb = sg.normal_bf16(2, "Y", (M, cfg.n_q * d), std=0.1)
    qkv, dO = to_dev_bf16(qb), to_dev_bf16(gb)
    desc = catq.attn_desc(cfg.batch, S, cfg.n_q, cfg.n_kv, d, qk, cfg.rope_theta)
    saved = torch.empty(catq.catq_attn_saved_bytes(desc), dtype=torch.uint8, device="cuda")
    ws = torch.empty(catq.catq_attn_bwd_workspace_bytes(desc), dtype=torch.uint8, device="cuda")
    o = torch.empty(M, cfg.n_q * d, dtype=torch.bfloat16, device="cuda")
    dqkv = torch.empty(M, ld, dtype=torch.bfloat16, device="cuda")
    catq.catq_aux_attention_fwd(desc, qkv, o, saved)
    catq.catq_aux_attention_bwd(desc, qkv, o, saved, dO, dqkv, ws)
    torch.cuda.synchronize()
    Oref, dref = _oracle_attention(f64(qb), cfg, f64(gb))
    assert max_norm_err(host(o), Oref) <= 2e-2
    assert max_norm_err(host(dqkv), dref) <= 2e-2


# ------------------------------------------------------------ dense block

def _dense_setup(cfg, seed=0, fac_seed=1):
    from paper_2606_26650_amd.block import DenseBlock
    W = sg.block_weights(cfg, seed)
    blk = DenseBlock(cfg, W)
    fac = _set_factors(blk, DenseBlock.split_fused, cfg, fac_seed)
    Wo = {k: f64(v) for k, v in W.items()}
    xb = sg.activations(cfg, seed)
    return blk, Wo, fac, xb


LIN_ID = {"qkv": 0, "o": 1, "gu": 2, "d": 3}


def _set_factors(blk, split, cfg, seed):
    """Draw factors per fused matrix, load them, and return the oracle's
    per-linear view {name: [d_mu, d_alpha, d_delta]}."""
    fac = {}
    for name, L in blk.lin.items():
        f = sg.perturbed_factors(seed, L.n_groups, extra=(LIN_ID[name],))
        L.set_factors(*f)
        parts = [split(cfg, name, a) for a in f]
        for k in parts[0]:
            fac[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    return fac


def _split_grads(split, cfg, name, L):
    parts = [split(cfg, name, host(a)) for a in (L.g_mu, L.g_alpha, L.g_delta)]
    return {k: [np.asarray(parts[i][k]).reshape(-1) for i in range(3)] for k in parts[0]}


def _check_step(catq, cfg, mode, s, s_bwd=30.0, tol=2e-2):
    import torch
    blk, Wo, fac, xb = _dense_setup(cfg)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    loss = blk.step(x, y_fp, mode=mode, s=s, s_bwd=s_bwd)
    torch.cuda.synchronize()
    ref = calib.dense_step(f64(xb), Wo, fac, cfg, mode, s=s, s_bwd=s_bwd)
    assert max_norm_err(host(y_fp), ref["y_fp"]) <= tol
    assert max_norm_err(host(blk.y), ref["y_q"]) <= tol
    if mode == lmst.IDENTITY:
        assert loss.item() == 0.0
        return blk, ref
    assert abs(loss.item() - ref["loss"]) <= tol * ref["loss"], (loss.item(), ref["loss"])
    assert max_norm_err(host(blk.dx), ref["dx"]) <= tol
    from paper_2606_26650_amd.block import DenseBlock
    for name, L in blk.lin.items():
        for k, v in _split_grads(DenseBlock.split_fused, cfg, name, L).items():
            for i in range(3):
                err = max_norm_err(v[i], ref["fgrads"][k][i])
                assert err <= tol, (k, i, err, median_rel(v[i], ref["fgrads"][k][i]))
    return blk, ref


@pytest.mark.parametrize("s", [0.625, 15.0, 30.0])
def test_dense_block_soft(catq, s):
    cfg = sg.small_dense(batch=2, seq=136, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    _check_step(catq, cfg, lmst.SOFT, s)


def test_dense_block_hard(catq):
    cfg = sg.small_dense(batch=1, seq=200, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    _check_step(catq, cfg, lmst.HARD, None)


def test_dense_block_identity(catq):
    cfg = sg.small_dense(batch=1, seq=64, hidden=256, n_q=2, n_kv=1, head_dim=128, ffn=256)
    _check_step(catq, cfg, lmst.IDENTITY, None)


def test_dense_block_llama_shape_no_qknorm(catq):
    cfg = sg.small_dense(batch=2, seq=128, hidden=512, n_q=4, n_kv=1, head_dim=128, ffn=768,
                         qk_norm=False, x_law="normal")
    _check_step(catq, cfg, lmst.SOFT, 15.0)


def test_finalize_codes_and_pack(catq):
    """Final hard ternarisation + 2-bit pack of every weight of the block,
    bit-exact against the oracle on the same factors."""
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = sg.small_dense(batch=1, seq=32, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    blk, Wo, fac, xb = _dense_setup(cfg)
    bufs = blk.finalize(blk.finalize_buffers())
    torch.cuda.synchronize()
    for name in blk.lin:
        codes = bufs[name]["codes"].cpu().numpy()
        packed = bufs[name]["packed"].cpu().numpy()
        alpha = bufs[name]["alpha"].cpu().numpy().astype(np.float64)
        cs = DenseBlock.split_fused(cfg, name, codes)
        ps = DenseBlock.split_fused(cfg, name, packed)
        al = DenseBlock.split_fused(cfg, name, alpha.reshape(codes.shape[0], -1))
        for k in cs:
            r = lmst.modulate_ternarize(Wo[k], 128, *fac[k], lmst.HARD)
            np.testing.assert_array_equal(cs[k], r["codes"])
            np.testing.assert_array_equal(ps[k], lmst.pack_ternary(r["codes"]))
            np.testing.assert_array_equal(al[k].reshape(-1), r["alpha"])
    # without int8 codes the finalize writes the packed codes in one launch:
    # the same bytes and scales
    fused = blk.finalize(blk.finalize_buffers(codes=False))
    torch.cuda.synchronize()
    assert "codes" not in fused["_flat"]
    assert torch.equal(fused["_flat"]["packed"], bufs["_flat"]["packed"])
    assert torch.equal(fused["_flat"]["alpha"], bufs["_flat"]["alpha"])


def test_block_step_deterministic(catq):
    import torch
    cfg = sg.small_dense(batch=2, seq=256, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    blk, Wo, fac, xb = _dense_setup(cfg)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    res = []
    for _ in range(2):
        l = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
        res.append((l, blk.dx.clone(), [L.g_alpha.clone() for L in blk.lin.values()]))
    torch.cuda.synchronize()
    assert torch.equal(res[0][0], res[1][0])
    assert torch.equal(res[0][1].view(torch.int16), res[1][1].view(torch.int16))
    for a, b in zip(res[0][2], res[1][2]):
        assert torch.equal(a, b)


@pytest.mark.parametrize("kind", ["dense", "moe"])
def test_overlapped_step_matches_serial(catq, kind):
    """The two-stream schedule (weight-gradient halves and the finalize on a
    side stream) gives bit for bit the one-stream results."""
    import torch
    if kind == "dense":
        cfg = sg.small_dense(batch=2, seq=128, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
        blk, _, _, xb = _dense_setup(cfg)
    else:
        cfg = sg.small_moe(batch=1, seq=96, hidden=256, n_q=4, n_kv=2, head_dim=64, n_experts=8,
                           top_k=2, expert_ffn=128, router_bias_std=1.0)
        blk, _, _, xb, _ = _moe_setup(cfg)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    out = []
    for overlap in (False, True):
        fin = blk.finalize_buffers()
        l = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0, overlap=overlap, finalize=fin).clone()
        torch.cuda.synchronize()
        out.append((l, blk.dx.clone(), [t.clone() for L in blk.lin.values()
                                        for t in (L.g_mu, L.g_alpha, L.g_delta)],
                    fin["_flat"]["packed"].clone(), fin["_flat"]["alpha"].clone()))
    a, b = out
    assert torch.equal(a[0], b[0])
    assert torch.equal(a[1].view(torch.int16), b[1].view(torch.int16))
    for u, v in zip(a[2], b[2]):
        assert torch.equal(u, v)
    assert torch.equal(a[3], b[3]) and torch.equal(a[4], b[4])


@pytest.mark.parametrize("kind", ["dense", "moe"])
@pytest.mark.parametrize("overlap", [False, True])
def test_step_without_input_gradient(catq, kind, overlap):
    """A calibrated block's input is fixed data, so the calibration skips
    the gradient of the block input (Eq. 7 optimises only the factors): the
    loss and every factor gradient are bit for bit those of the full step,
    and the input-gradient buffer is left untouched."""
    import torch
    if kind == "dense":
        cfg = sg.small_dense(batch=2, seq=128, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
        blk, _, _, xb = _dense_setup(cfg)
    else:
        cfg = sg.small_moe(batch=1, seq=96, hidden=256, n_q=4, n_kv=2, head_dim=64, n_experts=8,
                           top_k=2, expert_ffn=128, router_bias_std=1.0)
        blk, _, _, xb, _ = _moe_setup(cfg)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    out = []
    for input_grad in (True, False):
        blk.dx.fill_(7.0)
        l = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0, overlap=overlap,
                     input_grad=input_grad).clone()
        torch.cuda.synchronize()
        out.append((l, blk.dx.clone(), [t.clone() for L in blk.lin.values()
                                        for t in (L.g_mu, L.g_alpha, L.g_delta)]))
    (la, dxa, ga), (lb, dxb, gb) = out
    assert torch.equal(la, lb)
    for u, v in zip(ga, gb):
        assert torch.equal(u, v)
    assert not torch.all(dxa == 7.0)
    assert torch.all(dxb == 7.0)


def test_full_size_block_properties(catq):
    """The 1.7B-shaped block at its real size (4 x 2048 tokens): identity
    branch gives loss 0, soft step gives a finite positive loss and finite
    gradients, twice bitwise identical."""
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = sg.QWEN3_1P7B
    blk = DenseBlock(cfg, sg.block_weights(cfg, 0))
    x = to_dev_bf16(sg.activations(cfg, 0))
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    l0 = blk.step(x, y_fp, mode=lmst.IDENTITY).item()
    assert l0 == 0.0
    l1 = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
    g1 = [L.g_delta.clone() for L in blk.lin.values()]
    l2 = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(l1).all() and l1.item() > 0 and torch.equal(l1, l2)
    for a, L in zip(g1, blk.lin.values()):
        assert torch.isfinite(a).all() and torch.equal(a, L.g_delta)


# --------------------------------------------------------------- MoE block

def _moe_setup(cfg, seed=0):
    from paper_2606_26650_amd.block import MoEBlock
    W = sg.block_weights(cfg, seed)
    logits = sg.router_logits(cfg, seed)
    blk = MoEBlock(cfg, W, logits)
    fac = _set_factors(blk, MoEBlock.split_fused, cfg, 3)
    Wo = {k: f64(v) for k, v in W.items()}
    return blk, Wo, fac, sg.activations(cfg, seed), logits


@pytest.mark.parametrize("bias", [0.0, 1.5])
def test_moe_block_step(catq, bias):
    import torch
    from paper_2606_26650_amd.block import MoEBlock
    cfg = sg.small_moe(batch=1, seq=96, hidden=256, n_q=4, n_kv=2, head_dim=64, n_experts=8,
                       top_k=2, expert_ffn=128, router_bias_std=bias)
    blk, Wo, fac, xb, logits = _moe_setup(cfg)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    loss = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0)
    torch.cuda.synchronize()
    # routing: ids and offsets exact
    idx, wts = moe.route(logits, cfg.top_k)
    np.testing.assert_array_equal(blk.ids.cpu().numpy(), idx)
    np.testing.assert_allclose(blk.wts.cpu().numpy(), wts, rtol=1e-5)
    counts = np.bincount(idx.reshape(-1), minlength=cfg.n_experts)
    np.testing.assert_array_equal(blk.offs.cpu().numpy(),
                                  np.concatenate([[0], np.cumsum(counts)]))
    ref = calib.moe_step(f64(xb), Wo, fac, logits, cfg, lmst.SOFT, s=15.0, s_bwd=30.0)
    assert abs(loss.item() - ref["loss"]) <= 2e-2 * ref["loss"]
    assert max_norm_err(host(blk.dx), ref["dx"]) <= 2e-2
    for name, L in blk.lin.items():
        for k, v in _split_grads(MoEBlock.split_fused, cfg, name, L).items():
            for i in range(3):
                r = np.asarray(ref["fgrads"][k][i]).reshape(-1)
                assert max_norm_err(v[i], r) <= 2e-2, (k, i)


# ------------------------------------------------------- fp32 single linear

@pytest.mark.parametrize("strides", [(1, 1, 1), (1, 1, 0)], ids=["per-group", "shared-delta"])
def test_single_linear_fp32_calibration(catq, strides):
    """10 LM+ST calibration steps of the 256x256 fp32 linear (8 soft steps at
    s = 3.75k, 2 hard with the backward at s0 = 30), AdamW, per-group factors
    or one threshold factor shared by the matrix (stride 0).  Gated at every
    step on the GPU's own factors (Sec. 2.2-2.3, Eq. 3-6): the oracle's loss
    within 1e-5 relative and its factor gradients within 1e-4 (max-norm); the
    GPU's AdamW update against the oracle's on the same state.  The final
    codes equal the oracle's hard decision on the GPU's final factors bit for
    bit.  Reported: the oracle's own 10-step trajectory (losses within
    1e-3)."""
    import torch
    from calib_checks import check_adamw
    W, X = sg.single_linear_case(0)
    M, K = X.shape
    N = W.shape[0]
    Wd, Xd = to_dev_f32(W), to_dev_f32(X)
    ng = N * K // 128
    nf = [ng if st else 1 for st in strides]
    dm = torch.zeros(nf[0], device="cuda")
    da = torch.ones(nf[1], device="cuda")
    dd = torch.ones(nf[2], device="cuda")
    params = [dm, da, dd]
    mom = [torch.zeros(n, device="cuda") for n in nf]
    vel = [torch.zeros(n, device="cuda") for n in nf]
    g = [torch.zeros(n, device="cuda") for n in nf]
    stats = torch.zeros(ng, 2, device="cuda")
    wf = torch.empty(N, K, device="cuda")
    y_fp = torch.empty(M, N, device="cuda")
    y = torch.empty(M, N, device="cuda")
    dy = torch.empty(M, N, device="cuda")
    loss = torch.zeros(1, device="cuda")
    codes = torch.empty(N, K, dtype=torch.int8, device="cuda")
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K), dtype=torch.uint8, device="cuda")
    lws = torch.empty(catq.catq_workspace_size(1, M * N, 1, 1), dtype=torch.uint8, device="cuda")
    catq.catq_fakeq_linear_fwd(Xd, Wd, y_fp, M, N, K)
    W64, X64 = W.astype(np.float64), X.astype(np.float64)
    yref_fp = X64 @ W64.T
    losses, worst = [], [0.0, 0.0]
    for k in range(1, 11):
        mode, s = calib.schedule(k, 10)
        p = catq.lmst_params(mode=mode, s=s if s else 1.0, s_bwd=30.0, strides=strides)
        catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0 if k == 1 else 1, W_fake=wf)
        catq.catq_fakeq_linear_fwd(Xd, wf, y, M, N, K)
        catq.catq_block_recon_loss(y, y_fp, loss, dy, lws)
        catq.catq_fakeq_linear_bwd(dy, Xd, wf, M, N, K, Wd, stats, dm, da, dd, p, *g, ws)
        lr = calib.linear_lr(k - 1, 10)
        before = dict(p=[host(t) for t in params], m=[host(t) for t in mom],
                      v=[host(t) for t in vel], g=[host(t) for t in g], step=k, lr=lr)
        losses.append(loss.item())
        r = lmst.modulate_ternarize(W64, 128, *before["p"], mode, s=s, strides=strides)
        rl, rdy = block.recon_loss(X64 @ r["W_fake"].T, yref_fp)
        rg = lmst.factor_grads(rdy.T @ X64, W64, 128, *before["p"], mode, s=s, s_bwd=30.0,
                               strides=strides)
        worst[0] = max(worst[0], abs(losses[-1] - rl) / rl)
        assert abs(losses[-1] - rl) <= 1e-5 * rl, (k, losses[-1], rl)
        for i in range(3):
            err = max_norm_err(before["g"][i], np.asarray(rg[i]).reshape(-1))
            worst[1] = max(worst[1], err)
            assert err <= 1e-4, (k, i, err)
        for i, (P_, lo, hi) in enumerate([(dm, -1 + 1e-4, 1 - 1e-4), (da, 1e-4, 1e30),
                                          (dd, 1e-4, 1e30)]):
            catq.catq_aux_adamw(P_, g[i], mom[i], vel[i], k, lr, lo=lo, hi=hi)
        check_adamw(dict(before=before, after=dict(p=[host(t) for t in params],
                                                   m=[host(t) for t in mom],
                                                   v=[host(t) for t in vel])))
    catq.catq_modulate_ternarize(Wd, dm, da, dd, catq.lmst_params(mode=catq.HARD, strides=strides),
                                 stats, 1, W_fake=None, codes=codes)
    torch.cuda.synchronize()
    print(f"[fp32 linear {strides}] worst loss error {worst[0]:.2e}, "
          f"worst factor-gradient error {worst[1]:.2e}", flush=True)
    assert np.all(host(da) > 0) and np.all(host(dd) > 0) and np.all(np.abs(host(dm)) < 1)
    fin = [host(t) for t in params]
    rc = lmst.modulate_ternarize(W64, 128, *fin, lmst.HARD, strides=strides)["codes"]
    np.testing.assert_array_equal(codes.cpu().numpy(), rc)
    # reported: the oracle's own trajectory
    own = calib.single_linear_calibration(W64, X64, 10, strides=strides)
    for k, (l, r) in enumerate(zip(losses, own)):
        assert abs(l - r["loss"]) <= 1e-3 * r["loss"], (k, l, r["loss"])
