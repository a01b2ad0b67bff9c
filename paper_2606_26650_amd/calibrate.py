"""Block-wise CAT-Q calibration around the reconstruction step.

Sec. 2.3 (Eq. 6) drives the transition with a normalised time state t of the
current calibration epoch: the identity branch at t = 0, the softened
ternarisation with sharpness s = (t / gamma) * s0 while t <= gamma, the hard
quantiser after.  App. B.1 fixes the optimiser (AdamW, learning rate 1e-3
decayed linearly to zero), s0 = 30, gamma = 0.8 and Delta0 = 0.5; Sec. 2.2
constrains the factors (-1 < delta_mu < 1, delta_alpha > 0, delta_Delta > 0).

Readings where the paper is silent: t_e = (e + 1) / n_epochs for epoch e (so
the first epoch is already soft, the identity branch only being the start);
AdamW with betas (0.9, 0.999), eps 1e-8 and no weight decay, the constraints
enforced by clamping after each update (delta_mu into [-1 + 1e-4, 1 - 1e-4],
delta_alpha and delta_Delta to >= 1e-4); in hard epochs the backward uses the
transition's derivatives at s0 (the last soft sharpness, Sec. 2.3).

Everything on the device runs through the C ABI; this module only sequences
the calls and keeps the host-side bookkeeping (epochs, learning rate,
checkpoints).
"""
from __future__ import annotations

import os

import numpy as np
import torch

from . import HARD, SOFT, catq_aux_adamw

DMU_LIM = 1.0 - 1e-4
POS_MIN = 1e-4


def time_state(epoch: int, n_epochs: int, gamma: float = 0.8, s0: float = 30.0):
    """(mode, s) of Eq. 6 for 0-based ``epoch``: t = (epoch + 1) / n_epochs."""
    t = (epoch + 1) / n_epochs
    if t <= gamma:
        return SOFT, (t / gamma) * s0
    return HARD, 0.0


def linear_lr(step: int, total: int, lr0: float = 1e-3) -> float:
    """Learning rate of 0-based optimiser ``step`` out of ``total``."""
    return lr0 * (1.0 - step / total)


class BlockCalibrator:
    """Calibrates one block (a DenseBlock or MoEBlock driver), or a window of
    blocks, on a cached set of calibration samples already resident on the
    device.

    ``x_all`` is [n_samples * seq][hidden] bf16; batches are consecutive runs
    of ``block.cfg.batch`` samples.  The full-precision targets of every batch
    are computed once (identity branch) and kept on the device."""

    def __init__(self, block, x_all: torch.Tensor, n_epochs: int, gamma: float = 0.8,
                 s0: float = 30.0, lr0: float = 1e-3, overlap: bool | None = None):
        self.blk = block
        # the step's side stream (see the block drivers); None: the driver's
        # overlap_default
        self.overlap = block.overlap_default if overlap is None else overlap
        cfg = block.cfg
        self.tok_per_batch = cfg.batch * cfg.seq
        if x_all.shape[0] % self.tok_per_batch:
            raise ValueError("the calibration set must hold whole batches of samples")
        self.x_all = x_all
        self.n_batches = x_all.shape[0] // self.tok_per_batch
        self.n_epochs, self.gamma, self.s0, self.lr0 = n_epochs, gamma, s0, lr0
        self.total_steps = n_epochs * self.n_batches
        arenas = getattr(block, "arenas", None) or [block.arena]
        self.params = [t for A in arenas for t in (A.d_mu, A.d_alpha, A.d_delta)]
        self.grads = [t for A in arenas for t in (A.g_mu, A.g_alpha, A.g_delta)]
        self.bounds = [(-DMU_LIM, DMU_LIM), (POS_MIN, 1e30), (POS_MIN, 1e30)] * len(arenas)
        self.m = [torch.zeros_like(p) for p in self.params]
        self.v = [torch.zeros_like(p) for p in self.params]
        self.step_no = 0          # optimiser steps taken
        self.epoch = 0            # next epoch to run
        self.losses = []          # one device scalar per step (copied)
        # optional callable(phase, calibrator, batch, mode, s, lr): "grads"
        # after a step's backward (factors and moments not yet updated),
        # "update" after its AdamW launches
        self.observer = None
        self.targets = [block.new_output() for _ in range(self.n_batches)]
        for b in range(self.n_batches):
            block.target(self.batch(b), self.targets[b])

    def batch(self, b: int) -> torch.Tensor:
        return self.x_all[b * self.tok_per_batch:(b + 1) * self.tok_per_batch]

    def run_epoch(self):
        """One pass over the calibration set at this epoch's time state."""
        mode, s = time_state(self.epoch, self.n_epochs, self.gamma, self.s0)
        for b in range(self.n_batches):
            # the calibration input is fixed data: no gradient of the block input
            loss = self.blk.step(self.batch(b), self.targets[b], mode=mode, s=s, s_bwd=self.s0,
                                 recompute_stats=self.step_no == 0, overlap=self.overlap,
                                 input_grad=False)
            self.losses.append(loss.clone())
            self.step_no += 1
            lr = linear_lr(self.step_no - 1, self.total_steps, self.lr0)
            if self.observer is not None:
                self.observer("grads", self, b, mode, s, lr)
            for p, g, m, v, (lo, hi) in zip(self.params, self.grads, self.m, self.v, self.bounds):
                catq_aux_adamw(p, g, m, v, self.step_no, lr, lo=lo, hi=hi)
            if self.observer is not None:
                self.observer("update", self, b, mode, s, lr)
        self.epoch += 1

    def reset(self):
        """Back to the start of the schedule: identity factors (Sec. 2.2 at
        delta_mu = 0, delta_alpha = delta_Delta = 1), zero moments, no steps
        taken; the cached targets are kept."""
        for i in range(0, len(self.params), 3):
            self.params[i].zero_()
            self.params[i + 1].fill_(1.0)
            self.params[i + 2].fill_(1.0)
        for t in self.m + self.v:
            t.zero_()
        self.step_no = self.epoch = 0
        self.losses = []

    def run(self, checkpoint_dir: str | None = None):
        while self.epoch < self.n_epochs:
            self.run_epoch()
            if checkpoint_dir:
                self.save(os.path.join(checkpoint_dir, f"factors_epoch{self.epoch:03d}.npz"))
        return self.loss_history()

    def loss_history(self) -> np.ndarray:
        return torch.cat(self.losses).cpu().numpy() if self.losses else np.zeros(0, np.float32)

    # ------------------------------------------------------------ checkpoint
    def save(self, path: str):
        """Factors, optimiser moments and the position in the schedule."""
        torch.cuda.synchronize()
        np.savez(path, epoch=self.epoch, step=self.step_no,
                 **{f"p{i}": t.cpu().numpy() for i, t in enumerate(self.params)},
                 **{f"m{i}": t.cpu().numpy() for i, t in enumerate(self.m)},
                 **{f"v{i}": t.cpu().numpy() for i, t in enumerate(self.v)},
                 losses=self.loss_history())

    def load(self, path: str):
        with np.load(path, allow_pickle=False) as z:
            for i in range(len(self.params)):
                self.params[i].copy_(torch.from_numpy(z[f"p{i}"]))
                self.m[i].copy_(torch.from_numpy(z[f"m{i}"]))
                self.v[i].copy_(torch.from_numpy(z[f"v{i}"]))
            self.epoch = int(z["epoch"])
            self.step_no = int(z["step"])
            self.losses = [torch.from_numpy(z["losses"]).to(self.params[0].device)] \
                if z["losses"].size else []
        if hasattr(self.blk, "invalidate_stats"):   # recomputed on the next step
            self.blk.invalidate_stats()
        else:
            self.blk.stats_ready = False

    def finalize(self):
        """Final hard ternarisation and 2-bit packing of every weight."""
        return self.blk.finalize(self.blk.finalize_buffers())
