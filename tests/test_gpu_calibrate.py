"""GPU calibration loop of a dense block (Eq. 6 schedule per epoch, AdamW
with clamping, linear learning-rate decay, checkpoints) against the oracle.

Gated, per optimiser step on the GPU's own state: the factors the GPU held
are fed to the oracle's step, whose loss and factor gradients must match the
GPU's at the bf16 tolerance; the GPU's AdamW update must match the oracle's
AdamW on the same factors, gradients and moments; the final hard codes must
equal the oracle's codes on the GPU's final factors bit for bit.  Reported,
and loosely bounded: the oracle's own trajectory (losses per step, code
flips at the end)."""
import numpy as np
import pytest

import synthgen as sg
from calib_checks import StepRecorder, check_adamw, per_linear
from helpers import f64, host, max_norm_err, to_dev_bf16
from oracle import block, calib, lmst

pytestmark = pytest.mark.gpu

CFG = sg.small_dense(batch=2, seq=64, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
N_SAMPLES, N_EPOCHS = 4, 5
TOL = 2e-2


def _setup():
    from paper_2606_26650_amd.block import DenseBlock
    from paper_2606_26650_amd.calibrate import BlockCalibrator
    W = sg.block_weights(CFG, 0)
    xb = sg.activations(sg.small_dense(batch=N_SAMPLES, seq=64, hidden=256, n_q=4, n_kv=2,
                                       head_dim=64, ffn=384), 0)
    blk = DenseBlock(CFG, W)
    cal = BlockCalibrator(blk, to_dev_bf16(xb), N_EPOCHS)
    return W, xb, blk, cal


def test_block_calibration_against_oracle(catq):
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    W, xb, blk, cal = _setup()
    rec = StepRecorder()
    cal.observer = rec
    losses = cal.run()
    bufs = cal.finalize()
    torch.cuda.synchronize()
    Wo = {k: f64(v) for k, v in W.items()}
    x = f64(xb)
    tpb = CFG.batch * CFG.seq
    xs = [x[b * tpb:(b + 1) * tpb] for b in range(N_SAMPLES // CFG.batch)]
    y_fp = [block.block_forward(xi, Wo, CFG)[0] for xi in xs]
    assert len(rec.steps) == len(losses) == N_EPOCHS * len(xs)
    worst_g = worst_a = 0.0
    for r in rec.steps:
        bef = r["before"]
        fac = per_linear(blk, DenseBlock.split_fused, CFG, bef["p"])
        grads = per_linear(blk, DenseBlock.split_fused, CFG, bef["g"])
        s = bef["s"] if bef["s"] else None
        ref = calib.dense_step(xs[bef["batch"]], Wo, fac, CFG, bef["mode"], s=s, s_bwd=30.0,
                               y_fp=y_fp[bef["batch"]])
        assert abs(bef["loss"] - ref["loss"]) <= TOL * ref["loss"], (bef["step"], bef["loss"],
                                                                     ref["loss"])
        for k in grads:
            for i in range(3):
                err = max_norm_err(grads[k][i], ref["fgrads"][k][i])
                worst_g = max(worst_g, err)
                assert err <= TOL, (bef["step"], k, i, err)
        worst_a = max(worst_a, check_adamw(r))
    print(f"[calibration] worst factor-gradient error {worst_g:.4f}, "
          f"worst AdamW deviation {worst_a:.3f} of its bound", flush=True)
    # final codes: the oracle's hard decision on the GPU's final factors, exact
    gf = per_linear(blk, DenseBlock.split_fused, CFG, [host(t) for t in cal.params])
    for name in blk.lin:
        codes = DenseBlock.split_fused(CFG, name, bufs[name]["codes"].cpu().numpy())
        for k, c in codes.items():
            rc = lmst.modulate_ternarize(Wo[k], 128, *gf[k], lmst.HARD)["codes"]
            np.testing.assert_array_equal(c, rc)
    # reported: the oracle's own trajectory (chaotic only at threshold flips)
    own = calib.dense_calibration(x, Wo, CFG, N_EPOCHS)
    dev = max(abs(a - b) / b for a, b in zip(losses, own["losses"]))
    flips = total_w = 0
    for name in blk.lin:
        codes = DenseBlock.split_fused(CFG, name, bufs[name]["codes"].cpu().numpy())
        for k, c in codes.items():
            rc = lmst.modulate_ternarize(Wo[k], 128, *own["factors"][k], lmst.HARD)["codes"]
            flips += int((c != rc).sum())
            total_w += c.size
    print(f"[calibration] own trajectories: loss deviation {dev:.2e}, "
          f"code flips {flips}/{total_w}", flush=True)
    assert dev <= TOL and flips <= 1e-2 * total_w


def test_calibration_resume_is_bitwise(catq, tmp_path):
    """Two epochs, checkpoint, a fresh block resumes from the file: the final
    factors and the loss history equal the uninterrupted run's bit for bit."""
    import torch
    _, _, blk_a, cal_a = _setup()
    cal_a.run()
    _, _, blk_b, cal_b = _setup()
    cal_b.run_epoch()
    cal_b.run_epoch()
    path = str(tmp_path / "ckpt.npz")
    cal_b.save(path)
    _, _, blk_c, cal_c = _setup()
    cal_c.load(path)
    assert cal_c.epoch == 2 and cal_c.step_no == 2 * (N_SAMPLES // CFG.batch)
    cal_c.run()
    torch.cuda.synchronize()
    for pa, pc in zip(cal_a.params, cal_c.params):
        assert torch.equal(pa, pc)
    np.testing.assert_array_equal(cal_a.loss_history(), cal_c.loss_history())
