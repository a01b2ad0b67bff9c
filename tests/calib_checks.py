"""Per-step checks of a GPU calibration against the oracle on the GPU's own
state: at every optimiser step the factors the GPU held are fed to the
oracle's step (loss and factor gradients compared), and the GPU's AdamW
update is compared with the oracle's AdamW on the same factors, gradients
and moments (App. B.1; Sec. 2.2 clamps)."""
import numpy as np

from helpers import host
from oracle import calib

KINDS = ("mu", "pos", "pos")


class StepRecorder:
    """Observer for BlockCalibrator: host copies of the flat factor,
    gradient and moment arrays around every AdamW update."""

    def __init__(self):
        self.steps = []
        self.span = None

    def __call__(self, phase, cal, b, mode, s, lr):
        snap = dict(p=[host(t) for t in cal.params], m=[host(t) for t in cal.m],
                    v=[host(t) for t in cal.v])
        if phase == "grads":
            snap.update(g=[host(t) for t in cal.grads], batch=b, mode=mode, s=s, lr=lr,
                        step=cal.step_no, loss=float(cal.losses[-1].item()))
            self.steps.append(dict(before=snap, span=self.span))
        else:
            self.steps[-1]["after"] = snap


def per_linear(blk, split, cfg, flat3):
    """{oracle linear name: [a, b, c]} from three flat per-group arrays of a
    block's weight arena."""
    A = blk.arena
    out = {}
    for name, (o, n, _) in A.spans.items():
        parts = [split(cfg, name, np.asarray(a[o // A.g:(o + n) // A.g])) for a in flat3]
        for k in parts[0]:
            out[k] = [np.asarray(parts[i][k]).reshape(-1) for i in range(3)]
    return out


def check_adamw(rec):
    """The GPU's update of every flat factor array against the oracle's
    AdamW from the same factors, gradients and moments.  fp32 arithmetic on
    the GPU against float64 rounded once: a few fp32 ulps of the operands."""
    bef, aft = rec["before"], rec["after"]
    worst = 0.0
    for i in range(len(bef["p"])):
        p0, g, m0, v0 = bef["p"][i], bef["g"][i], bef["m"][i], bef["v"][i]
        rp, rm, rv = calib.adamw_step(p0, g, m0, v0, bef["step"], bef["lr"], kind=KINDS[i % 3])
        tol_m = 4e-7 * (0.9 * np.abs(m0) + 0.1 * np.abs(g)) + 1e-37
        tol_v = 4e-7 * (0.999 * np.abs(v0) + 0.001 * g * g) + 1e-37
        tol_p = 4e-7 * (np.abs(p0) + np.abs(rp)) + 1e-5 * np.abs(rp - p0) + 1e-12
        for got, ref, tol, what in ((aft["m"][i], rm, tol_m, "m"), (aft["v"][i], rv, tol_v, "v"),
                                    (aft["p"][i], rp, tol_p, "p")):
            d = np.abs(got - ref)
            bad = d > tol
            assert not bad.any(), (bef["step"], i, what, int(bad.sum()), float(d.max()))
            worst = max(worst, float(np.max(d / np.maximum(tol, 1e-300))))
    return worst
