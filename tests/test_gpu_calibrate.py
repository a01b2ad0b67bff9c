"""GPU calibration loop of a dense block (Eq. 6 schedule per epoch, AdamW
with clamping, linear learning-rate decay, checkpoints) against the oracle's
own calibration loop.  The two sides follow their own trajectories: nothing
the GPU computes is fed to the oracle.  Per-step losses are compared with the
bf16 tolerance; factors within the AdamW drift bound (an update moves a
factor by about lr at most per step when its gradient keeps its sign, a sign
flip of a near-zero gradient by up to 2 lr), and the final hard codes of the
two trajectories may differ only on a small fraction of weights near a
threshold."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, to_dev_bf16
from oracle import calib, lmst

pytestmark = pytest.mark.gpu

CFG = sg.small_dense(batch=2, seq=64, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
N_SAMPLES, N_EPOCHS = 4, 5


def _setup():
    from paper_2606_26650_amd.block import DenseBlock
    from paper_2606_26650_amd.calibrate import BlockCalibrator
    W = sg.block_weights(CFG, 0)
    xb = sg.activations(sg.small_dense(batch=N_SAMPLES, seq=64, hidden=256, n_q=4, n_kv=2,
                                       head_dim=64, ffn=384), 0)
    blk = DenseBlock(CFG, W)
    cal = BlockCalibrator(blk, to_dev_bf16(xb), N_EPOCHS)
    return W, xb, blk, cal


def _gpu_factors(blk):
    from paper_2606_26650_amd.block import DenseBlock
    out = {}
    for name, L in blk.lin.items():
        parts = [DenseBlock.split_fused(CFG, name, host(a)) for a in (L.d_mu, L.d_alpha, L.d_delta)]
        for k in parts[0]:
            out[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    return out


def test_block_calibration_against_oracle(catq):
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    W, xb, blk, cal = _setup()
    losses = cal.run()
    bufs = cal.finalize()
    torch.cuda.synchronize()
    Wo = {k: f64(v) for k, v in W.items()}
    ref = calib.dense_calibration(f64(xb), Wo, CFG, N_EPOCHS)
    assert len(losses) == len(ref["losses"]) == N_EPOCHS * (N_SAMPLES // CFG.batch)
    for k, (a, b) in enumerate(zip(losses, ref["losses"])):
        assert abs(a - b) <= 2e-2 * b, (k, a, b)
    total = len(losses)
    drift = 2.0 * sum(calib.linear_lr(k, total) for k in range(total))
    gf = _gpu_factors(blk)
    for k in Wo:
        for i in range(3):
            d = np.abs(gf[k][i] - ref["factors"][k][i])
            assert d.max() <= drift, (k, i, d.max(), drift)
    assert np.all(np.abs(np.concatenate([f[0] for f in gf.values()])) < 1)
    assert np.all(np.concatenate([np.concatenate(f[1:]) for f in gf.values()]) > 0)
    # final hard codes of each trajectory: flips only near thresholds
    flips = total_w = 0
    for name in blk.lin:
        codes = DenseBlock.split_fused(CFG, name, bufs[name]["codes"].cpu().numpy())
        for k, c in codes.items():
            rc = lmst.modulate_ternarize(Wo[k], 128, *ref["factors"][k], lmst.HARD)["codes"]
            flips += int((c != rc).sum())
            total_w += c.size
    assert flips <= 1e-2 * total_w, (flips, total_w)


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
