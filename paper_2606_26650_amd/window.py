"""Sliding-layer output reconstruction (Sec. 2.4, Eq. 7) over a window of
consecutive decoder blocks, and the window-by-window calibration around it.

Eq. 7 compares the output of the whole window computed with alpha*T against
the full-precision window output on the same input.  A window step is LM+ST
of every block, the blocks' forwards in turn (each block's fp32 output is the
next block's input), one loss at the end, and the blocks' backwards in
reverse order, each block's input gradient being the output gradient of the
block before it.  Every step runs in the library's kernels; this module only
orders the calls.

Readings where the paper is silent (it takes the window geometry from
SliderQuant without stating it): windows of ``l`` blocks moving by ``stride``
blocks (default 1), the last window ending at the last block; the input of a
window is the full-precision model's activation entering its first block;
each window runs the whole Eq. 6 schedule with fresh AdamW moments, and a
block lying in several windows keeps its factors from one to the next.
"""
from __future__ import annotations

import os

import torch

from . import IDENTITY, SOFT, catq_block_recon_loss
from .calibrate import BlockCalibrator


def window_spans(n_blocks: int, l: int, stride: int = 1):
    """[first, last) block ranges of the windows, in calibration order."""
    if n_blocks <= 0 or l <= 0 or stride <= 0:
        raise ValueError("n_blocks, l and stride must be positive")
    if stride > l:
        raise ValueError("a stride longer than the window would skip blocks")
    if l >= n_blocks:
        return [(0, n_blocks)]
    spans = list(range(0, n_blocks - l + 1, stride))
    if spans[-1] + l != n_blocks:
        spans.append(n_blocks - l)
    return [(a, a + l) for a in spans]


class Window:
    """Consecutive blocks (DenseBlock or MoEBlock drivers of one geometry)
    calibrated jointly.  Presents the interface BlockCalibrator drives:
    cfg, arenas, new_output, target, step, finalize_buffers/finalize."""

    def __init__(self, blocks):
        if not blocks:
            raise ValueError("a window needs at least one block")
        self.blocks = list(blocks)
        self.cfg = self.blocks[0].cfg
        side = self.blocks[0].side_stream()
        for b in self.blocks:
            if b.M != self.blocks[0].M or b.cfg.hidden != self.cfg.hidden:
                raise ValueError("the blocks of a window must share tokens and hidden size")
            b.side = side    # one side stream: the window joins it once

    @property
    def arenas(self):
        return [b.arena for b in self.blocks]

    @property
    def loss(self):
        return self.blocks[-1].loss

    @property
    def dx(self):
        return self.blocks[0].dx

    @property
    def y(self):
        return self.blocks[-1].y

    def invalidate_stats(self):
        for b in self.blocks:
            b.stats_ready = False

    def params(self, mode, s=15.0, s_bwd=30.0):
        return self.blocks[0].params(mode, s, s_bwd)

    def modulate_all(self, p, recompute_stats=False):
        for b in self.blocks:
            b.modulate_all(p, recompute_stats)

    def forward(self, x, out=None):
        h = x
        for b in self.blocks[:-1]:
            h = b.forward(h)
        return self.blocks[-1].forward(h, out)

    def new_output(self):
        return self.blocks[-1].new_output()

    def target(self, x, out):
        """Full-precision window output on x (IDENTITY branch everywhere)."""
        self.modulate_all(self.params(IDENTITY))
        return self.forward(x, out)

    def finalize_buffers(self, codes=True):
        return [b.finalize_buffers(codes) for b in self.blocks]

    def finalize(self, bufs):
        """Hard codes, group scales and 2-bit packing of every block."""
        return [b.finalize(f) for b, f in zip(self.blocks, bufs)]

    @property
    def overlap_default(self):
        """The step's default schedule: that of the window's blocks."""
        return self.blocks[0].overlap_default

    def step(self, x, y_fp, mode=SOFT, s=15.0, s_bwd=30.0, recompute_stats=False, overlap=None,
             finalize=None, input_grad=True):
        """LM+ST of every block -> window forward -> Eq. 7 loss -> backward
        through the blocks in reverse.  Loss stays on the device.
        ``finalize`` (buffers from finalize_buffers) also runs every block's
        hard ternarisation + packing after LM+ST (on the side stream with
        ``overlap``; None takes overlap_default).  ``input_grad`` false skips
        the gradient of the window input (the first block's dx); the later
        blocks' input gradients are always formed."""
        if overlap is None:
            overlap = self.overlap_default
        p = self.params(mode, s, s_bwd)
        self.modulate_all(p, recompute_stats)
        main = torch.cuda.current_stream()
        b0 = self.blocks[0]
        if finalize is not None:
            side = b0.side_stream() if overlap else main
            if side is not main:
                b0.order("window_finalize", main, side)
            with torch.cuda.stream(side):
                self.finalize(finalize)
        last = self.blocks[-1]
        self.forward(x)
        catq_block_recon_loss(last.y, y_fp, last.loss, last.dy, last.loss_ws)
        ins = [x] + [b.y for b in self.blocks[:-1]]
        n = len(self.blocks)
        for i in range(n - 1, -1, -1):
            dy = None if i == n - 1 else self.blocks[i + 1].dx
            self.blocks[i].backward(ins[i], p, overlap, dy=dy, join=(i == 0),
                                    input_grad=input_grad or i > 0)
        if finalize is not None and overlap:
            b0.order("window_finalize_join", b0.side_stream(), main)
        return last.loss


class SlidingCalibrator:
    """Calibrates ``blocks`` window by window (readings in the module
    header).  ``x_all`` holds the calibration samples entering the first
    block, [n_samples * seq][hidden], bf16 or fp32, resident on the device;
    batches are consecutive runs of cfg.batch samples."""

    def __init__(self, blocks, x_all: torch.Tensor, l: int, n_epochs: int, stride: int = 1,
                 gamma: float = 0.8, s0: float = 30.0, lr0: float = 1e-3):
        self.blocks = list(blocks)
        self.spans = window_spans(len(self.blocks), l, stride)
        self.x_all = x_all
        self.n_epochs, self.gamma, self.s0, self.lr0 = n_epochs, gamma, s0, lr0
        cfg = self.blocks[0].cfg
        self.tok_per_batch = cfg.batch * cfg.seq
        if x_all.shape[0] % self.tok_per_batch:
            raise ValueError("the calibration set must hold whole batches of samples")
        self.history = []     # (span, loss history) per finished window
        # optional observer handed to each window's BlockCalibrator (see
        # there); self.span names the window being calibrated
        self.observer = None
        self.span = None

    def _fp_forward(self, blk, acts):
        """Full-precision output of one block on every batch (fp32)."""
        out = torch.empty(acts.shape[0], blk.cfg.hidden, dtype=torch.float32, device=acts.device)
        for b0 in range(0, acts.shape[0], self.tok_per_batch):
            blk.target(acts[b0:b0 + self.tok_per_batch], out[b0:b0 + self.tok_per_batch])
        return out

    def run(self, checkpoint_dir: str | None = None, finalize: bool = True):
        """All windows in order; returns {block index: finalize buffers} when
        ``finalize`` (each block is hard-ternarised and packed once its last
        window is done), else {}."""
        acts, at = self.x_all, 0
        last_window = {i: w for w, (a, e) in enumerate(self.spans) for i in range(a, e)}
        done = {}
        for w, (a, e) in enumerate(self.spans):
            while at < a:
                acts = self._fp_forward(self.blocks[at], acts)
                at += 1
            win = Window(self.blocks[a:e])
            cal = BlockCalibrator(win, acts, self.n_epochs, self.gamma, self.s0, self.lr0)
            cal.observer = self.observer
            self.span = (a, e)
            ck = None
            if checkpoint_dir:
                ck = os.path.join(checkpoint_dir, f"window{w:03d}_blocks{a:03d}-{e:03d}")
                os.makedirs(ck, exist_ok=True)
            losses = cal.run(ck)
            self.history.append(((a, e), losses))
            if finalize:
                for i in range(a, e):
                    if last_window[i] == w:
                        blk = self.blocks[i]
                        done[i] = blk.finalize(blk.finalize_buffers())
        return done
