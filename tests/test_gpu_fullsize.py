"""Full-size GPU checks of the block step for every decoder-block workload
(Qwen3-1.7B-, Llama-3-8B-, Qwen3-14B-shaped dense blocks and the
Qwen3-235B-A22B-shaped routed-expert block, uniform and skewed routing), in
the launch configuration the benchmark times (one LM+ST launch over the
block's weight arena, the direct-to-LDS GEMMs, fused attention).

The oracle cannot run a whole block at these sizes, so the checks are:
  * sampled rows of every fused weight through LM+ST (SOFT, statistics
    computed) and the hard finalize: statistics, codes, packed bytes and
    group scales bit-exact, fake weights within bf16 rounding;
  * sampled tokens of the block output through the identity branch (the
    full-precision target) against the oracle's selected-token forward,
    including the last token of every sample (the longest causal rows);
    compared on y - x, the block's own contribution;
  * exact routing (MoE);
  * properties every step has at any size: identity loss exactly 0, a
    finite positive soft loss, finite factor gradients, bitwise determinism.
Factor gradients at full size are checked on sampled rows with seeded output
gradients in the linear-layer tests."""
import gc

import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, to_dev_bf16
from oracle import block, lmst, moe

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

LIN_ID = {"qkv": 0, "o": 1, "gu": 2, "d": 3}
DENSE = {"qwen3-1.7b": sg.QWEN3_1P7B, "llama3-8b": sg.LLAMA3_8B, "qwen3-14b": sg.QWEN3_14B}


def _tokens(cfg, n, seed):
    """n random tokens plus the last token of every sample."""
    r = np.random.default_rng(seed)
    last = {(b + 1) * cfg.seq - 1 for b in range(cfg.batch)}
    return sorted(last | {int(t) for t in r.integers(0, cfg.tokens, n)})


def _fused_rows(W, cfg, name, rows):
    """Rows of a fused matrix (q|k|v, o, gate|up, down; experts stacked) as
    bf16 bits, read from the seeded weights."""
    if name == "o":
        return W["Wo"].reshape(-1, W["Wo"].shape[-1])[rows]
    if name == "d":
        return W["Wd"].reshape(-1, W["Wd"].shape[-1])[rows]
    if name == "qkv":
        full = np.concatenate([W["Wq"], W["Wk"], W["Wv"]], 0)
        return full[rows]
    if W["Wg"].ndim == 2:  # dense gate|up
        F = W["Wg"].shape[0]
        return np.stack([W["Wg"][r] if r < F else W["Wu"][r - F] for r in rows])
    E, F, _ = W["Wg"].shape  # experts: [E][2F][h] per expert
    out = []
    for r in rows:
        e, j = divmod(int(r), 2 * F)
        out.append(W["Wg"][e, j] if j < F else W["Wu"][e, j - F])
    return np.stack(out)


def _load_factors(blk, seed):
    fac = {}
    for name, L in blk.lin.items():
        f = sg.perturbed_factors(seed, L.n_groups, extra=(LIN_ID[name],))
        L.set_factors(*f)
        fac[name] = f
    return fac


def _check_weight_rows(catq, blk, W, cfg, fac, seed):
    import torch
    r = np.random.default_rng(seed)
    pick = {}
    for name, L in blk.lin.items():
        nrows, d_in = L.W.shape
        gpr = d_in // 128
        rows = np.sort(r.choice(nrows, 12, replace=False))
        grp = (rows[:, None] * gpr + np.arange(gpr)[None]).reshape(-1)
        pick[name] = (rows, grp, torch.from_numpy(rows).cuda(), torch.from_numpy(grp).cuda())
    blk.modulate_all(blk.params(lmst.SOFT, s=15.0), recompute_stats=True)
    torch.cuda.synchronize()
    soft = {n: (host(L.W_fake[pick[n][2]]), L.stats[pick[n][3]].cpu().numpy().astype(np.float64))
            for n, L in blk.lin.items()}
    bufs = blk.finalize(blk.finalize_buffers())
    torch.cuda.synchronize()
    for name, L in blk.lin.items():
        rows, grp, rows_t, grp_t = pick[name]
        Wr = f64(_fused_rows(W, cfg, name, rows))
        fr = [f[grp] for f in fac[name]]
        ref = lmst.modulate_ternarize(Wr, 128, *fr, lmst.SOFT, s=15.0)
        wf, st = soft[name]
        np.testing.assert_array_equal(st[:, 0], ref["mu0"], err_msg=name)
        np.testing.assert_array_equal(st[:, 1], ref["alpha0"], err_msg=name)
        assert np.all(np.abs(wf - ref["W_fake"]) <= 2.0 ** -8 * np.abs(ref["W_fake"]) + 1e-30), name
        rh = lmst.modulate_ternarize(Wr, 128, *fr, lmst.HARD)
        b = bufs[name]
        np.testing.assert_array_equal(b["codes"][rows_t].cpu().numpy(), rh["codes"], err_msg=name)
        np.testing.assert_array_equal(b["packed"][rows_t].cpu().numpy(),
                                      lmst.pack_ternary(rh["codes"]), err_msg=name)
        np.testing.assert_array_equal(b["alpha"][grp_t].cpu().numpy().astype(np.float64),
                                      rh["alpha"], err_msg=name)
    # the one-launch finalize (no int8 codes) writes the same bytes and scales
    fused = blk.finalize(blk.finalize_buffers(codes=False))
    torch.cuda.synchronize()
    assert torch.equal(fused["_flat"]["packed"], bufs["_flat"]["packed"])
    assert torch.equal(fused["_flat"]["alpha"], bufs["_flat"]["alpha"])
    del bufs, fused


def _check_step_properties(blk, x, y_fp):
    import torch
    l0 = blk.step(x, y_fp, mode=lmst.IDENTITY).item()
    assert l0 == 0.0
    l1 = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
    g1 = [L.g_delta.clone() for L in blk.lin.values()]
    dx1 = blk.dx.clone()
    l2 = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
    torch.cuda.synchronize()
    assert torch.isfinite(l1).all() and l1.item() > 0 and torch.equal(l1, l2)
    assert torch.equal(dx1.view(torch.int16), blk.dx.view(torch.int16))
    for a, L in zip(g1, blk.lin.values()):
        assert torch.isfinite(a).all() and torch.equal(a, L.g_delta)


@pytest.mark.parametrize("name", list(DENSE))
def test_full_size_dense_block(catq, name):
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = DENSE[name]
    W = sg.block_weights(cfg, 0)
    blk = DenseBlock(cfg, W)
    fac = _load_factors(blk, 11)
    xb = sg.activations(cfg, 0)
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    torch.cuda.synchronize()
    toks = _tokens(cfg, 6, 2)
    Wo = {k: f64(v) for k, v in W.items()}
    xo = f64(xb)
    ref = block.block_forward_rows(xo, Wo, cfg, toks)
    got = host(y_fp)[toks]
    err = max_norm_err(got - xo[toks], ref - xo[toks])
    assert err <= 2e-2, (name, err)
    del Wo, xo
    _check_weight_rows(catq, blk, W, cfg, fac, 3)
    _check_step_properties(blk, x, y_fp)
    del blk, x, y_fp
    gc.collect()
    torch.cuda.empty_cache()


@pytest.fixture(scope="module")
def moe_full():
    """The routed-expert block at full size (2.42B expert weights), built once."""
    import torch
    from paper_2606_26650_amd.block import MoEBlock
    cfg = sg.QWEN3_235B_MOE
    print("[moe] drawing 2.4B expert weights", flush=True)
    W = sg.block_weights(cfg, 0)
    print("[moe] building the block", flush=True)
    blk = MoEBlock(cfg, W, sg.router_logits(cfg, 0))
    fac = _load_factors(blk, 13)
    xb = sg.activations(cfg, 0)
    yield cfg, W, blk, fac, xb
    del blk
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("bias", [0.0, 0.5])
def test_full_size_moe_block(catq, moe_full, bias):
    import dataclasses

    import torch
    cfg0, W, blk, fac, xb = moe_full
    cfg = dataclasses.replace(cfg0, router_bias_std=bias)
    logits = sg.router_logits(cfg, 0)
    blk.logits.copy_(torch.from_numpy(np.ascontiguousarray(logits)))
    x = to_dev_bf16(xb)
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    torch.cuda.synchronize()
    idx, wts = moe.route(logits, cfg.top_k)
    np.testing.assert_array_equal(blk.ids.cpu().numpy(), idx)
    np.testing.assert_allclose(blk.wts.cpu().numpy(), wts, rtol=1e-5)
    counts = np.bincount(idx.reshape(-1), minlength=cfg.n_experts)
    np.testing.assert_array_equal(blk.offs.cpu().numpy(), np.concatenate([[0], np.cumsum(counts)]))
    if bias > 0:
        assert counts.max() > 4 * counts.min() + 1  # the skew actually happened
    toks = _tokens(cfg, 4, 5)
    Wa = {k: f64(W[k]) for k in ("Wq", "Wk", "Wv", "Wo")}
    xo = f64(xb)
    ref = moe.moe_block_forward_rows(
        xo, Wa, lambda e: (f64(W["Wg"][e]), f64(W["Wu"][e]), f64(W["Wd"][e])), logits, cfg, toks)
    got = host(y_fp)[toks]
    err = max_norm_err(got - xo[toks], ref - xo[toks])
    assert err <= 2e-2, (bias, err)
    if bias == 0.0:
        _check_weight_rows(catq, blk, W, cfg, fac, 7)
    _check_step_properties(blk, x, y_fp)
