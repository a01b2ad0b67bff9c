"""GPU parity of the sliding-window reconstruction (Eq. 7 over several
blocks): the window step against the oracle's window step, the two-stream
schedule against the one-stream one, and the window-by-window calibration
checked step by step against the oracle on the GPU's own factors."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, median_rel, to_dev_bf16
from oracle import block, calib, lmst, window

pytestmark = pytest.mark.gpu

LIN_ID = {"qkv": 0, "o": 1, "gu": 2, "d": 3}


def _blocks(cfg, n, fac_seed0=None):
    """n dense blocks with weights drawn from seeds 0..n-1; factors loaded
    when fac_seed0 is given.  Returns GPU blocks, oracle weights, oracle
    factors."""
    from paper_2606_26650_amd.block import DenseBlock
    blks, Wos, facs = [], [], []
    for i in range(n):
        W = sg.block_weights(cfg, i)
        blk = DenseBlock(cfg, W)
        fac = {}
        if fac_seed0 is not None:
            for name, L in blk.lin.items():
                f = sg.perturbed_factors(fac_seed0 + i, L.n_groups, extra=(LIN_ID[name],))
                L.set_factors(*f)
                parts = [DenseBlock.split_fused(cfg, name, a) for a in f]
                for k in parts[0]:
                    fac[k] = [np.asarray(parts[j][k]).reshape(-1) for j in range(3)]
        blks.append(blk)
        Wos.append({k: f64(v) for k, v in W.items()})
        facs.append(fac)
    return blks, Wos, facs


def _split(cfg, name, arrs):
    from paper_2606_26650_amd.block import DenseBlock
    parts = [DenseBlock.split_fused(cfg, name, host(a)) for a in arrs]
    return {k: [np.asarray(parts[i][k]).reshape(-1) for i in range(3)] for k in parts[0]}


@pytest.mark.parametrize("mode,s", [(lmst.SOFT, 15.0), (lmst.HARD, 0.0)])
def test_window_step_parity(catq, mode, s):
    import torch
    from paper_2606_26650_amd.window import Window
    cfg = sg.small_dense(batch=2, seq=136, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    blks, Wos, facs = _blocks(cfg, 2, fac_seed0=1)
    xb = sg.activations(cfg, 0)
    x = to_dev_bf16(xb)
    win = Window(blks)
    y_fp = win.new_output()
    win.target(x, y_fp)
    loss = win.step(x, y_fp, mode=mode, s=s, s_bwd=30.0)
    torch.cuda.synchronize()
    print(f"[window] mode={mode} s={s} loss={loss.item():.6e}", flush=True)
    ref = window.window_step(f64(xb), Wos, facs, cfg, mode, s=s if s else None, s_bwd=30.0)
    tol = 2e-2
    assert max_norm_err(host(y_fp), ref["y_fp"]) <= tol
    assert max_norm_err(host(win.y), ref["y_q"]) <= tol
    assert max_norm_err(host(blks[0].y), ref["inputs"][1]) <= tol
    assert abs(loss.item() - ref["loss"]) <= tol * ref["loss"], (loss.item(), ref["loss"])
    assert max_norm_err(host(win.dx), ref["dx"]) <= tol
    assert max_norm_err(host(blks[1].dx), _inner_dy(ref, cfg)) <= tol
    # Factor gradients.  The last block is gated end to end.  An earlier
    # block b is gated on its own backward given the gradient that reaches
    # its output (the GPU's input gradient of block b + 1): end to end its
    # factor gradients sit on a floor set by the bf16 forward of both
    # windows (the loss gradient is a small difference of two bf16
    # pipelines that passed through n - b blocks).  An exact float64
    # emulation of every bf16 rounding the GPU performs gives 0.017 on block
    # 0 of this case, independent of the token count, so that figure is
    # reported, with a loose tripwire only.
    n = len(blks)
    xs = [ref["inputs"][0]] + [ref["inputs"][b] for b in range(1, n)]
    for b, blk in enumerate(blks):
        if b == n - 1:
            gate = ref["fgrads"][b]
        else:
            _, cache = block.block_forward(xs[b], ref["W_fake"][b], cfg)
            _, dW = block.block_backward(host(blks[b + 1].dx), cache, ref["W_fake"][b], cfg)
            gate = calib.factor_grads_all(dW, Wos[b], facs[b], 128, mode, s if s else None, 30.0)
        worst = worst_e2e = 0.0
        for name, L in blk.lin.items():
            for k, v in _split(cfg, name, (L.g_mu, L.g_alpha, L.g_delta)).items():
                for i in range(3):
                    err = max_norm_err(v[i], gate[k][i])
                    worst = max(worst, err)
                    assert err <= tol, (b, k, i, err, median_rel(v[i], gate[k][i]))
                    worst_e2e = max(worst_e2e, max_norm_err(v[i], ref["fgrads"][b][k][i]))
        print(f"[window] block {b}: worst factor-gradient error {worst:.4f} (gated), "
              f"{worst_e2e:.4f} end to end", flush=True)
        assert worst_e2e <= 5e-2


def _inner_dy(ref, cfg):
    """Gradient of the loss at the output of the first block: the input
    gradient of the last block, from the oracle's own backward."""
    from oracle import block
    _, xs, caches = window.window_forward(ref["inputs"][0], ref["W_fake"], cfg)
    d, _ = block.block_backward(ref["dy"], caches[1], ref["W_fake"][1], cfg)
    return d


def test_window_overlap_matches_serial(catq):
    import torch
    from paper_2606_26650_amd.window import Window
    cfg = sg.small_dense(batch=2, seq=128, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    blks, _, _ = _blocks(cfg, 3, fac_seed0=4)
    x = to_dev_bf16(sg.activations(cfg, 0))
    win = Window(blks)
    y_fp = win.new_output()
    win.target(x, y_fp)
    out = []
    for overlap in (False, True):
        fin = win.finalize_buffers()
        l = win.step(x, y_fp, mode=lmst.SOFT, s=15.0, overlap=overlap, finalize=fin).clone()
        torch.cuda.synchronize()
        out.append((l, win.dx.clone(), [t.clone() for b in blks for L in b.lin.values()
                                        for t in (L.g_mu, L.g_alpha, L.g_delta)],
                    [f["_flat"]["packed"].clone() for f in fin]))
    a, b = out
    assert torch.equal(a[0], b[0])
    assert torch.equal(a[1].view(torch.int16), b[1].view(torch.int16))
    for u, v in zip(a[2], b[2]):
        assert torch.equal(u, v)
    for u, v in zip(a[3], b[3]):
        assert torch.equal(u, v)


N_SAMPLES, N_EPOCHS = 4, 3


def test_sliding_calibration_against_oracle(catq):
    """Window-by-window calibration of three blocks (l = 2, stride 1).  Gated
    per optimiser step on the GPU's own state: the oracle's window step on
    the factors the GPU held (loss; every block's factor gradients from its
    own backward of the gradient reaching its output, for the last block the
    loss gradient; end to end they carry the earlier block's forward noise
    through the loss gradient and are reported, under a 5e-2 tripwire) and
    the oracle's AdamW on the same factors, gradients and moments; the final
    codes against the oracle's hard decision on the GPU's final factors, bit
    for bit.  Reported: the oracle's own trajectory."""
    import torch
    from calib_checks import StepRecorder, check_adamw, per_linear
    from oracle import block
    from paper_2606_26650_amd.block import DenseBlock
    from paper_2606_26650_amd.window import SlidingCalibrator
    cfg = sg.small_dense(batch=2, seq=64, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    xcfg = sg.small_dense(batch=N_SAMPLES, seq=64, hidden=256, n_q=4, n_kv=2, head_dim=64,
                          ffn=384)
    blks, Wos, _ = _blocks(cfg, 3)
    xb = sg.activations(xcfg, 0)
    cal = SlidingCalibrator(blks, to_dev_bf16(xb), l=2, n_epochs=N_EPOCHS)
    rec = StepRecorder()

    def obs(phase, c, b, mode, s, lr):
        rec.span = cal.span
        rec(phase, c, b, mode, s, lr)
        if phase == "grads":   # gradients reaching the outputs of the window's blocks
            rec.steps[-1]["dy_in"] = ([host(blk.dx) for blk in c.blk.blocks[1:]] +
                                      [host(c.blk.blocks[-1].dy)])

    cal.observer = obs
    bufs = cal.run()
    torch.cuda.synchronize()
    assert [sp for sp, _ in cal.history] == [(0, 2), (1, 3)]
    tpb = cfg.batch * cfg.seq
    nb = N_SAMPLES // cfg.batch
    acts = [f64(xb)]
    for i in range(2):
        acts.append(np.concatenate([block.block_forward(acts[i][b * tpb:(b + 1) * tpb], Wos[i],
                                                        cfg)[0] for b in range(nb)]))
    assert len(rec.steps) == 2 * N_EPOCHS * nb
    worst, worst_e2e = {}, {}
    for r in rec.steps:
        bef, (a, e) = r["before"], r["span"]
        xw = acts[a][bef["batch"] * tpb:(bef["batch"] + 1) * tpb]
        facs = [per_linear(blks[a + j], DenseBlock.split_fused, cfg, bef["p"][3 * j:3 * j + 3])
                for j in range(e - a)]
        s = bef["s"] if bef["s"] else None
        ref = window.window_step(xw, Wos[a:e], facs, cfg, bef["mode"], s=s, s_bwd=30.0)
        assert abs(bef["loss"] - ref["loss"]) <= 2e-2 * ref["loss"], ((a, e), bef["step"])
        for j in range(e - a):
            grads = per_linear(blks[a + j], DenseBlock.split_fused, cfg, bef["g"][3 * j:3 * j + 3])
            # each block on its own backward from the gradient that reaches its
            # output (the last block: the loss gradient the GPU computed)
            _, cache = block.block_forward(ref["inputs"][j], ref["W_fake"][j], cfg)
            _, dW = block.block_backward(r["dy_in"][j], cache, ref["W_fake"][j], cfg)
            gate = calib.factor_grads_all(dW, Wos[a + j], facs[j], 128, bef["mode"], s, 30.0)
            for k in grads:
                for i in range(3):
                    err = max_norm_err(grads[k][i], gate[k][i])
                    worst[j] = max(worst.get(j, 0.0), err)
                    assert err <= 2e-2, ((a, e), bef["step"], j, k, i, err)
                    e2e = max_norm_err(grads[k][i], ref["fgrads"][j][k][i])
                    worst_e2e[j] = max(worst_e2e.get(j, 0.0), e2e)
        check_adamw(r)
    print(f"[sliding] worst factor-gradient error per window position {worst} (gated), "
          f"{worst_e2e} end to end", flush=True)
    assert max(worst_e2e.values()) <= 5e-2
    for i, blk in enumerate(blks):
        for name, L in blk.lin.items():
            gf = _split(cfg, name, (L.d_mu, L.d_alpha, L.d_delta))
            codes = DenseBlock.split_fused(cfg, name, bufs[i][name]["codes"].cpu().numpy())
            for k, c in codes.items():
                rc = lmst.modulate_ternarize(Wos[i][k], 128, *gf[k], lmst.HARD)["codes"]
                np.testing.assert_array_equal(c, rc)
    # reported: the oracle's own trajectory
    ref = window.sliding_calibration(f64(xb), Wos, cfg, l=2, n_epochs=N_EPOCHS)
    assert [h["span"] for h in ref["history"]] == [(0, 2), (1, 3)]
    dev = max(abs(a - b) / b for (_, got), h in zip(cal.history, ref["history"])
              for a, b in zip(got, h["losses"]))
    print(f"[sliding] own trajectories: loss deviation {dev:.2e}", flush=True)
    assert dev <= 2e-2
