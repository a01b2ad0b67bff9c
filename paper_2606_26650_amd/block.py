"""One CAT-Q block-wise reconstruction step driven through the C ABI.

The driver owns device buffers (torch tensors used as plain HBM allocations)
and issues the library calls in order on one stream; it computes nothing
itself.  The seven linears of a decoder block are stored as four fused
matrices, q|k|v, o, gate|up and down: groups never straddle rows, so
learnable modulation and its gradients are unchanged by the fusion, while
the GEMMs get larger and the input gradient of q, k and v (and of gate and
up) comes out of one contraction.

Step (Sec. 2.2-2.4):
  LM+ST of every weight (Eq. 3-6) -> block forward with alpha*T ->
  reconstruction loss against the full-precision output on the same input
  (Eq. 7) -> backward to the block input and to the factors of every group,
  and (finalize) hard codes (Eq. 2) + 2-bit packing with the group scales.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (BF16, HARD, IDENTITY, SOFT, attn_desc, catq_aux_act_quant, catq_aux_attention_bwd,
               catq_aux_attention_fwd, catq_aux_moe_combine, catq_aux_moe_combine_bwd,
               catq_aux_moe_gather, catq_aux_moe_route, catq_aux_moe_route_workspace_bytes,
               catq_aux_moe_scatter_add, catq_aux_rmsnorm_bwd, catq_aux_rmsnorm_fwd,
               catq_aux_swiglu_bwd, catq_aux_swiglu_fwd, catq_attn_bwd_workspace_bytes,
               catq_attn_saved_bytes, catq_block_recon_loss, catq_fakeq_linear_bwd,
               catq_fakeq_down_swiglu_bwd, catq_fakeq_gateup_swiglu_fwd, catq_fakeq_linear_fwd,
               catq_modulate_ternarize, catq_pack_ternary, catq_ternarize_pack,
               catq_workspace_size, lmst_params, WS_LINEAR_BWD, WS_LOSS)

DEV = "cuda"


def bf16_tensor(bits: np.ndarray, device=DEV) -> torch.Tensor:
    """Device bf16 tensor holding exactly the given uint16 bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def empty(shape, dtype=torch.bfloat16):
    return torch.empty(shape, dtype=dtype, device=DEV)


class QLinear:
    """A weight under learnable modulation: W frozen, three factor arrays
    (per group), cached group statistics, fake weight and factor gradients.
    ``W`` is [rows][d_in] (experts stacked along rows).  ``store`` supplies
    views of a block arena for every per-weight array (else they are
    allocated here)."""

    FIELDS = ("d_mu", "d_alpha", "d_delta", "stats", "W_fake", "g_mu", "g_alpha", "g_delta")

    def __init__(self, W: torch.Tensor, d_out: int, d_in: int, g: int = 128, n_experts: int = 1,
                 store: dict | None = None):
        self.W = W
        self.d_out, self.d_in, self.E = d_out, d_in, n_experts
        self.g = g
        ng = W.numel() // g
        self.n_groups = ng
        if store is not None:
            for k in self.FIELDS:
                setattr(self, k, store[k])
            return
        self.d_mu = torch.zeros(ng, dtype=torch.float32, device=DEV)
        self.d_alpha = torch.ones(ng, dtype=torch.float32, device=DEV)
        self.d_delta = torch.ones(ng, dtype=torch.float32, device=DEV)
        self.stats = torch.zeros(ng, 2, dtype=torch.float32, device=DEV)
        self.W_fake = torch.empty_like(W)
        self.g_mu = torch.zeros_like(self.d_mu)
        self.g_alpha = torch.zeros_like(self.d_mu)
        self.g_delta = torch.zeros_like(self.d_mu)

    def set_factors(self, dmu, dal, dde):
        self.d_mu.copy_(torch.as_tensor(dmu, dtype=torch.float32))
        self.d_alpha.copy_(torch.as_tensor(dal, dtype=torch.float32))
        self.d_delta.copy_(torch.as_tensor(dde, dtype=torch.float32))

    def modulate(self, p, stats_mode, codes=None, alpha_out=None, W_fake="self"):
        wf = self.W_fake if W_fake == "self" else W_fake
        catq_modulate_ternarize(self.W, self.d_mu, self.d_alpha, self.d_delta, p, self.stats,
                                stats_mode, W_fake=wf, codes=codes, alpha_out=alpha_out)


class WeightArena:
    """Every weight of a block in one flat allocation, with its factors,
    statistics, fake weight and gradients alongside.  Groups never straddle
    rows, so the flat view of the concatenated row-major matrices holds
    exactly the per-matrix groups in order: LM+ST, the hard finalize and the
    packing can each run as one launch over the whole block."""

    def __init__(self, mats: list, g: int):
        # mats: (name, tensor [rows][d_in], d_out, d_in, n_experts)
        self.g = g
        total = sum(t.numel() for _, t, *_ in mats)
        self.P, self.n_groups = total, total // g
        self.W = torch.empty(total, dtype=torch.bfloat16, device=DEV)
        self.W_fake = torch.empty_like(self.W)
        ng = self.n_groups
        self.d_mu = torch.zeros(ng, dtype=torch.float32, device=DEV)
        self.d_alpha = torch.ones(ng, dtype=torch.float32, device=DEV)
        self.d_delta = torch.ones(ng, dtype=torch.float32, device=DEV)
        self.stats = torch.zeros(ng, 2, dtype=torch.float32, device=DEV)
        self.g_mu = torch.zeros(ng, dtype=torch.float32, device=DEV)
        self.g_alpha = torch.zeros_like(self.g_mu)
        self.g_delta = torch.zeros_like(self.g_mu)
        self.spans = {}
        self.lin = {}
        o = 0
        for name, t, d_out, d_in, E in mats:
            n = t.numel()
            shape = (n // d_in, d_in)
            self.W[o:o + n].copy_(t.reshape(-1))
            go, gn = o // g, n // g
            store = {"W_fake": self.W_fake[o:o + n].view(shape),
                     "stats": self.stats[go:go + gn]}
            for k in ("d_mu", "d_alpha", "d_delta", "g_mu", "g_alpha", "g_delta"):
                store[k] = getattr(self, k)[go:go + gn]
            self.lin[name] = QLinear(self.W[o:o + n].view(shape), d_out, d_in, g, E, store)
            self.spans[name] = (o, n, shape)
            o += n

    def flat(self, t):
        """[P] (or [P]-sized) tensor seen as [P/g][g] for the flat calls."""
        return t.view(self.P // self.g, self.g) if t is not None else None

    def modulate(self, p, stats_mode, W_fake="self", codes=None, alpha_out=None):
        wf = self.W_fake if W_fake == "self" else W_fake
        catq_modulate_ternarize(self.flat(self.W), self.d_mu, self.d_alpha, self.d_delta, p,
                                self.stats, stats_mode, W_fake=self.flat(wf),
                                codes=self.flat(codes), alpha_out=alpha_out)

    def ternarize_pack(self, p, stats_mode, packed, alpha_out):
        """Hard codes of every weight straight to 2-bit storage (one launch)."""
        catq_ternarize_pack(self.flat(self.W), self.d_mu, self.d_alpha, self.d_delta, p,
                            self.stats, stats_mode, packed.view(self.P // self.g, self.g // 4),
                            alpha_out=alpha_out)


class DenseBlock:
    """Pre-norm decoder block (RMSNorm, fused q|k|v, QK-norm, RoPE, causal GQA
    attention, o, residual, RMSNorm, fused gate|up, SwiGLU, down, residual)."""

    # Schedule of a step when the caller names none: one stream.  Every
    # product of a dense block fills the chip on its own, and two of them at
    # once on two streams share the caches and ran the calibration step
    # 1-3% slower (14B- and 1.7B-shaped blocks).
    overlap_default = False

    def __init__(self, cfg, weights: dict, g: int = 128, a8: bool = False):
        """a8: the W1.58A8 setting -- the inputs of the four linears and Q, K,
        V of the attention products are fake-quantized to 8 bits in the
        step's forward (straight-through backward); the full-precision
        target is not."""
        self.cfg = cfg
        c = cfg
        hd, h = c.head_dim, c.hidden
        self.a8 = a8
        self._act = a8
        # SwiGLU forward and backward inside the gate|up and down GEMM
        # epilogues (same bits as the separate kernels; off: separate kernels)
        self.fuse_swiglu = True
        self.Nqkv = (c.n_q + 2 * c.n_kv) * hd
        self.M = c.batch * c.seq
        self.g = g
        dev_w = {k: bf16_tensor(v) for k, v in weights.items()}
        self.arena = WeightArena([
            ("qkv", torch.cat([dev_w["Wq"], dev_w["Wk"], dev_w["Wv"]], 0), self.Nqkv, h, 1),
            ("o", dev_w["Wo"], h, c.n_q * hd, 1),
            ("gu", torch.cat([dev_w["Wg"], dev_w["Wu"]], 0), 2 * c.ffn, h, 1),
            ("d", dev_w["Wd"], h, c.ffn, 1),
        ], g)
        self.lin = self.arena.lin
        del dev_w
        M = self.M
        self.desc = attn_desc(c.batch, c.seq, c.n_q, c.n_kv, hd, c.qk_norm, c.rope_theta)
        self.desc_a8 = attn_desc(c.batch, c.seq, c.n_q, c.n_kv, hd, c.qk_norm, c.rope_theta,
                                 act_quant=True) if a8 else None
        self.fwd_desc = self.desc
        # activations
        self.xn1, self.rstd1 = empty((M, h)), empty((M,), torch.float32)
        self.qkv = empty((M, self.Nqkv))
        self.attn = empty((M, c.n_q * hd))
        self.attn_q = empty((M, c.n_q * hd)) if a8 else None   # quantized o input
        self.h1 = empty((M, h), torch.float32)      # residual stream kept in fp32
        self.xn2, self.rstd2 = empty((M, h)), empty((M,), torch.float32)
        self.gu = empty((M, 2 * c.ffn))
        self.a = empty((M, c.ffn))
        self.y = empty((M, h), torch.float32)
        self.saved = torch.empty(catq_attn_saved_bytes(self.desc), dtype=torch.uint8, device=DEV)
        # gradients
        self.dy = empty((M, h))
        self.da = empty((M, c.ffn))
        self.dgu = empty((M, 2 * c.ffn))
        self.dxn2 = empty((M, h))
        self.dh1 = empty((M, h))
        self.dattn = empty((M, c.n_q * hd))
        self.dqkv = empty((M, self.Nqkv))
        self.dxn1 = empty((M, h))
        self.dx = empty((M, h))
        self.attn_ws = torch.empty(catq_attn_bwd_workspace_bytes(self.desc), dtype=torch.uint8,
                                   device=DEV)
        ws = max(catq_workspace_size(WS_LINEAR_BWD, M, L.d_out, L.d_in) for L in self.lin.values())
        self.lin_ws = torch.empty(ws, dtype=torch.uint8, device=DEV)
        self.loss_ws = torch.empty(catq_workspace_size(WS_LOSS, M, 1, 1), dtype=torch.uint8,
                                   device=DEV)
        self.loss = torch.zeros(1, dtype=torch.float32, device=DEV)
        self.stats_ready = False
        self.side = None
        self._events = {}

    def side_stream(self):
        """Second stream (default priority) for the weight-gradient halves and
        the hard finalize, which then overlap the input-gradient chain."""
        if self.side is None:
            self.side = torch.cuda.Stream(device=DEV)
        return self.side

    def order(self, key, before, after):
        """Make stream ``after`` wait for the work issued so far on ``before``,
        through an event kept per ``key`` (created on first use, then
        re-recorded: a step captured into a graph creates no events)."""
        ev = self._events.get(key)
        if ev is None:
            ev = self._events[key] = torch.cuda.Event()
        ev.record(before)
        after.wait_event(ev)

    # ------------------------------------------------------------------ LM+ST
    def params(self, mode, s=15.0, s_bwd=30.0, strides=(1, 1, 1)):
        return lmst_params(self.g, mode, 0.5, s if s else 1.0, s_bwd, strides)

    def modulate_all(self, p, recompute_stats=False):
        """LM+ST of every weight: one launch over the arena (per-linear calls
        when a factor is shared, since a shared factor is per matrix)."""
        mode_stats = 0 if (recompute_stats or not self.stats_ready) else 1
        if all(st == 1 for st in p.factor_stride):
            self.arena.modulate(p, mode_stats)
        else:
            for L in self.lin.values():
                L.modulate(p, mode_stats)
        self.stats_ready = True

    # ---------------------------------------------------------------- forward
    def forward(self, x, out=None):
        """Block forward with the current fake weights; returns the output."""
        c, M = self.cfg, self.M
        h = c.hidden
        y = self.y if out is None else out
        act = self._act
        catq_aux_rmsnorm_fwd(x, self.xn1, self.rstd1)
        if act:
            catq_aux_act_quant(self.xn1, self.xn1)
        L = self.lin["qkv"]
        catq_fakeq_linear_fwd(self.xn1, L.W_fake, self.qkv, M, self.Nqkv, h)
        self.fwd_desc = self.desc_a8 if act else self.desc
        catq_aux_attention_fwd(self.fwd_desc, self.qkv, self.attn, self.saved)
        self.o_in = self.attn
        if act:
            catq_aux_act_quant(self.attn, self.attn_q)
            self.o_in = self.attn_q
        L = self.lin["o"]
        catq_fakeq_linear_fwd(self.o_in, L.W_fake, self.h1, M, h, c.n_q * c.head_dim, residual=x)
        catq_aux_rmsnorm_fwd(self.h1, self.xn2, self.rstd2)
        if act:
            catq_aux_act_quant(self.xn2, self.xn2)
        L = self.lin["gu"]
        if self.fuse_swiglu:
            catq_fakeq_gateup_swiglu_fwd(self.xn2, L.W_fake, self.gu, self.a, M, c.ffn, h)
        else:
            catq_fakeq_linear_fwd(self.xn2, L.W_fake, self.gu, M, 2 * c.ffn, h)
            catq_aux_swiglu_fwd(self.gu, self.a)
        if act:
            catq_aux_act_quant(self.a, self.a)
        L = self.lin["d"]
        catq_fakeq_linear_fwd(self.a, L.W_fake, y, M, h, c.ffn, residual=self.h1)
        return y

    def new_output(self):
        return empty((self.M, self.cfg.hidden), torch.float32)

    def target(self, x, out):
        """Full-precision block output on the same input (IDENTITY branch,
        activations not quantized)."""
        self.modulate_all(self.params(IDENTITY))
        self._act = False
        try:
            return self.forward(x, out)
        finally:
            self._act = self.a8

    # --------------------------------------------------------------- backward
    def backward(self, x, p, overlap=True, dy=None, join=True, input_grad=True):
        """Backward to the block input and to every factor.  With ``overlap``
        each linear's weight-gradient half (G = dY^T X and the factor
        gradients) runs on the side stream as soon as dY is ready, while the
        main stream carries on with dX and the glue; the main stream waits
        for the side stream at the end (unless ``join`` is false: a window
        of blocks joins once, after its first block).  ``dy`` is the
        gradient of the block output (default: the loss's, in self.dy).
        ``input_grad`` false skips the gradient of the block input (self.dx):
        the factors' gradients do not need it when the input is fixed data
        (a calibrated block, or the first block of a window), so the q|k|v
        projection runs its weight-gradient half only."""
        c, M = self.cfg, self.M
        h = c.hidden
        ws = self.lin_ws
        main = torch.cuda.current_stream()
        side = self.side_stream() if overlap else None

        def lbwd(name, dY, X, dX):
            L = self.lin[name]
            if side is None:
                catq_fakeq_linear_bwd(dY, X, L.W_fake, M, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                      L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha, L.g_delta, ws,
                                      dX=dX)
                return
            self.order(name, main, side)
            with torch.cuda.stream(side):
                catq_fakeq_linear_bwd(dY, X, L.W_fake, M, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                      L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha, L.g_delta, ws)
            catq_fakeq_linear_bwd(dY, X, L.W_fake, M, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                  L.d_alpha, L.d_delta, p, None, None, None, None, dX=dX)

        def lbwd_weights(name, dY, X):
            # the weight-gradient half alone (on the side stream with overlap)
            L = self.lin[name]
            if side is not None:
                self.order(name, main, side)
            with torch.cuda.stream(side if side is not None else main):
                catq_fakeq_linear_bwd(dY, X, L.W_fake, M, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                      L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha, L.g_delta, ws)

        dy = self.dy if dy is None else dy
        if self.fuse_swiglu:
            # the down projection's weight-gradient half as usual; its input
            # gradient with the SwiGLU backward in the GEMM epilogue
            L = self.lin["d"]
            if side is not None:
                self.order("d", main, side)
            with torch.cuda.stream(side if side is not None else main):
                catq_fakeq_linear_bwd(dy, self.a, L.W_fake, M, L.d_out, L.d_in, L.W, L.stats,
                                      L.d_mu, L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha,
                                      L.g_delta, ws)
            catq_fakeq_down_swiglu_bwd(dy, L.W_fake, self.gu, self.dgu, M, h, c.ffn, da=self.da)
        else:
            lbwd("d", dy, self.a, self.da)
            catq_aux_swiglu_bwd(self.gu, self.da, self.dgu)
        lbwd("gu", self.dgu, self.xn2, self.dxn2)
        catq_aux_rmsnorm_bwd(self.h1, self.rstd2, self.dxn2, self.dh1, dres=dy)
        lbwd("o", self.dh1, self.o_in, self.dattn)
        catq_aux_attention_bwd(self.fwd_desc, self.qkv, self.attn, self.saved, self.dattn,
                               self.dqkv, self.attn_ws)
        if input_grad:
            lbwd("qkv", self.dqkv, self.xn1, self.dxn1)
            catq_aux_rmsnorm_bwd(x, self.rstd1, self.dxn1, self.dx, dres=self.dh1)
        else:
            lbwd_weights("qkv", self.dqkv, self.xn1)
        if side is not None and join:
            self.order("join", side, main)

    # ------------------------------------------------------------------- step
    def step(self, x, y_fp, mode=SOFT, s=15.0, s_bwd=30.0, recompute_stats=False, overlap=None,
             finalize=None, input_grad=True):
        """LM+ST -> forward -> loss -> backward.  Loss stays on the device.
        ``overlap`` (None: the block's overlap_default) puts the
        weight-gradient halves on the side stream.  ``finalize`` (buffers
        from finalize_buffers) also runs the hard ternarisation + packing,
        on the side stream (with overlap) once LM+ST has the statistics (it
        reads only W, the statistics and the factors).  ``input_grad`` false
        leaves self.dx unwritten (see backward)."""
        if overlap is None:
            overlap = self.overlap_default
        p = self.params(mode, s, s_bwd)
        self.modulate_all(p, recompute_stats)
        if finalize is not None:
            main = torch.cuda.current_stream()
            side = self.side_stream() if overlap else main
            if side is not main:
                self.order("finalize", main, side)
            with torch.cuda.stream(side):
                self.finalize(finalize)
        self.forward(x)
        catq_block_recon_loss(self.y, y_fp, self.loss, self.dy, self.loss_ws)
        self.backward(x, p, overlap, input_grad=input_grad)
        if finalize is not None and overlap:
            self.order("finalize_join", self.side_stream(), torch.cuda.current_stream())
        return self.loss

    def finalize_buffers(self, codes=True):
        """Flat scales / packed bytes (and int8 codes unless ``codes`` is
        false) for the whole arena, with per-linear views."""
        A = self.arena
        flat = dict(alpha=torch.empty(A.n_groups, dtype=torch.float32, device=DEV),
                    packed=torch.empty(A.P // 4, dtype=torch.uint8, device=DEV))
        if codes:
            flat["codes"] = torch.empty(A.P, dtype=torch.int8, device=DEV)
        out = {"_flat": flat}
        for name, (o, n, shape) in A.spans.items():
            out[name] = dict(alpha=flat["alpha"][o // A.g:(o + n) // A.g],
                             packed=flat["packed"][o // 4:(o + n) // 4].view(shape[0], shape[1] // 4))
            if codes:
                out[name]["codes"] = flat["codes"][o:o + n].view(shape)
        return out

    def finalize(self, bufs):
        """Hard codes (Eq. 2), group scales and 2-bit packing of every weight:
        with int8 codes requested, the HARD LM+ST writing them and then the
        packing (one launch each over the arena); without, one launch that
        writes the packed codes directly (same bits)."""
        p = self.params(HARD)
        A, f = self.arena, bufs["_flat"]
        stats_mode = 1 if self.stats_ready else 0
        if "codes" in f:
            A.modulate(p, stats_mode, W_fake=None, codes=f["codes"], alpha_out=f["alpha"])
            catq_pack_ternary(A.flat(f["codes"]), f["packed"].view(A.P // A.g, A.g // 4))
        else:
            A.ternarize_pack(p, stats_mode, f["packed"], f["alpha"])
        self.stats_ready = True
        return bufs

    # ------------------------------------------------------------ oracle map
    @staticmethod
    def split_fused(cfg, name, arr):
        """Split a fused-matrix array (rows or per-group values) into the
        per-linear pieces, in q, k, v / gate, up order."""
        hd = cfg.head_dim
        if name == "qkv":
            sizes = [cfg.n_q * hd, cfg.n_kv * hd, cfg.n_kv * hd]
            names = ["Wq", "Wk", "Wv"]
        elif name == "gu":
            sizes = [cfg.ffn, cfg.ffn]
            names = ["Wg", "Wu"]
        elif name == "o":
            return {"Wo": arr}
        else:
            return {"Wd": arr}
        return _split_rows(arr, sizes, names)


class MoEBlock:
    """Decoder block whose MLP routes every token to its top-k experts (router
    logits given, left unquantised); attention half as in DenseBlock."""

    # Two streams by default: the experts' weight-gradient products, with the
    # factor gradients in their vector-bound epilogues, overlap the
    # input-gradient chain (about 1% faster than one stream on the
    # 235B-A22B-shaped block, even and skewed expert loads).
    overlap_default = True

    def __init__(self, cfg, weights: dict, logits: np.ndarray, g: int = 128):
        self.cfg = c = cfg
        hd, h = c.head_dim, c.hidden
        self.Nqkv = (c.n_q + 2 * c.n_kv) * hd
        self.M = c.batch * c.seq
        self.R = self.M * c.top_k  # routed rows
        self.g = g
        dev_w = {k: bf16_tensor(v) for k, v in weights.items()}
        E, F = c.n_experts, c.expert_ffn
        self.arena = WeightArena([
            ("qkv", torch.cat([dev_w["Wq"], dev_w["Wk"], dev_w["Wv"]], 0), self.Nqkv, h, 1),
            ("o", dev_w["Wo"], h, c.n_q * hd, 1),
            # experts' gate|up fused per expert: [E][2F][h]
            ("gu", torch.cat([dev_w["Wg"], dev_w["Wu"]], 1), 2 * F, h, E),
            ("d", dev_w["Wd"], h, F, E),
        ], g)
        self.lin = self.arena.lin
        del dev_w
        M, R = self.M, self.R
        self.logits = torch.from_numpy(np.ascontiguousarray(logits)).to(DEV)
        self.desc = attn_desc(c.batch, c.seq, c.n_q, c.n_kv, hd, c.qk_norm, c.rope_theta)
        self.ids = torch.empty((M, c.top_k), dtype=torch.int32, device=DEV)
        self.wts = torch.empty((M, c.top_k), dtype=torch.float32, device=DEV)
        self.perm = torch.empty((M, c.top_k), dtype=torch.int32, device=DEV)
        self.offs = torch.empty(E + 1, dtype=torch.int64, device=DEV)
        self.route_ws = torch.empty(catq_aux_moe_route_workspace_bytes(M, E, c.top_k),
                                    dtype=torch.uint8, device=DEV)
        self.xn1, self.rstd1 = empty((M, h)), empty((M,), torch.float32)
        self.qkv = empty((M, self.Nqkv))
        self.attn = empty((M, c.n_q * hd))
        self.h1 = empty((M, h), torch.float32)      # residual stream kept in fp32
        self.xn2, self.rstd2 = empty((M, h)), empty((M,), torch.float32)
        self.xg = empty((R, h))
        self.gu = empty((R, 2 * F))
        self.a = empty((R, F))
        self.yg = empty((R, h))
        self.y = empty((M, h), torch.float32)
        self.saved = torch.empty(catq_attn_saved_bytes(self.desc), dtype=torch.uint8, device=DEV)
        self.dy = empty((M, h))
        self.dyg = empty((R, h))
        self.da = empty((R, F))
        self.dgu = empty((R, 2 * F))
        self.dxg = empty((R, h))
        self.dxn2 = empty((M, h))
        self.dh1 = empty((M, h))
        self.dattn = empty((M, c.n_q * hd))
        self.dqkv = empty((M, self.Nqkv))
        self.dxn1 = empty((M, h))
        self.dx = empty((M, h))
        self.attn_ws = torch.empty(catq_attn_bwd_workspace_bytes(self.desc), dtype=torch.uint8,
                                   device=DEV)
        ws = max(catq_workspace_size(WS_LINEAR_BWD, M, self.Nqkv, h),
                 catq_workspace_size(WS_LINEAR_BWD, M, h, c.n_q * hd),
                 catq_workspace_size(WS_LINEAR_BWD, R, 2 * F, h, E),
                 catq_workspace_size(WS_LINEAR_BWD, R, h, F, E))
        self.lin_ws = torch.empty(ws, dtype=torch.uint8, device=DEV)
        self.loss_ws = torch.empty(catq_workspace_size(WS_LOSS, M, 1, 1), dtype=torch.uint8,
                                   device=DEV)
        self.loss = torch.zeros(1, dtype=torch.float32, device=DEV)
        self.stats_ready = False
        self.side = None
        self._events = {}

    params = DenseBlock.params
    side_stream = DenseBlock.side_stream
    order = DenseBlock.order
    modulate_all = DenseBlock.modulate_all
    new_output = DenseBlock.new_output
    finalize_buffers = DenseBlock.finalize_buffers
    finalize = DenseBlock.finalize

    def route(self):
        catq_aux_moe_route(self.logits, self.cfg.top_k, self.ids, self.wts, self.perm, self.offs,
                           self.route_ws)

    def forward(self, x, out=None):
        c, M, R = self.cfg, self.M, self.R
        h, E, F, k = c.hidden, c.n_experts, c.expert_ffn, c.top_k
        y = self.y if out is None else out
        catq_aux_rmsnorm_fwd(x, self.xn1, self.rstd1)
        catq_fakeq_linear_fwd(self.xn1, self.lin["qkv"].W_fake, self.qkv, M, self.Nqkv, h)
        catq_aux_attention_fwd(self.desc, self.qkv, self.attn, self.saved)
        catq_fakeq_linear_fwd(self.attn, self.lin["o"].W_fake, self.h1, M, h, c.n_q * c.head_dim,
                              residual=x)
        catq_aux_rmsnorm_fwd(self.h1, self.xn2, self.rstd2)
        self.route()
        catq_aux_moe_gather(self.xn2, self.perm, k, self.xg)
        catq_fakeq_linear_fwd(self.xg, self.lin["gu"].W_fake, self.gu, R, 2 * F, h, n_experts=E,
                              row_offsets=self.offs)
        catq_aux_swiglu_fwd(self.gu, self.a)
        catq_fakeq_linear_fwd(self.a, self.lin["d"].W_fake, self.yg, R, h, F, n_experts=E,
                              row_offsets=self.offs)
        catq_aux_moe_combine(self.yg, self.perm, self.wts, self.h1, y, k)
        return y

    def target(self, x, out):
        self.modulate_all(self.params(IDENTITY))
        return self.forward(x, out)

    def backward(self, x, p, overlap=True, dy=None, join=True, input_grad=True):
        """As DenseBlock.backward, with the routed-expert MLP half."""
        c, M, R = self.cfg, self.M, self.R
        h, E, F, k = c.hidden, c.n_experts, c.expert_ffn, c.top_k
        ws = self.lin_ws
        main = torch.cuda.current_stream()
        side = self.side_stream() if overlap else None

        def lbwd(name, dY, X, dX, rows, E_=1, offs=None):
            L = self.lin[name]
            if side is None:
                catq_fakeq_linear_bwd(dY, X, L.W_fake, rows, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                      L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha, L.g_delta, ws,
                                      dX=dX, n_experts=E_, row_offsets=offs)
                return
            self.order(name, main, side)
            with torch.cuda.stream(side):
                catq_fakeq_linear_bwd(dY, X, L.W_fake, rows, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                      L.d_alpha, L.d_delta, p, L.g_mu, L.g_alpha, L.g_delta, ws,
                                      n_experts=E_, row_offsets=offs)
            catq_fakeq_linear_bwd(dY, X, L.W_fake, rows, L.d_out, L.d_in, L.W, L.stats, L.d_mu,
                                  L.d_alpha, L.d_delta, p, None, None, None, None, dX=dX,
                                  n_experts=E_, row_offsets=offs)

        dy = self.dy if dy is None else dy
        catq_aux_moe_combine_bwd(dy, self.perm, self.wts, self.dyg, k)
        lbwd("d", self.dyg, self.a, self.da, R, E, self.offs)
        catq_aux_swiglu_bwd(self.gu, self.da, self.dgu)
        lbwd("gu", self.dgu, self.xg, self.dxg, R, E, self.offs)
        catq_aux_moe_scatter_add(self.dxg, self.perm, self.dxn2, k)
        catq_aux_rmsnorm_bwd(self.h1, self.rstd2, self.dxn2, self.dh1, dres=dy)
        lbwd("o", self.dh1, self.attn, self.dattn, M)
        catq_aux_attention_bwd(self.desc, self.qkv, self.attn, self.saved, self.dattn, self.dqkv,
                               self.attn_ws)
        if input_grad:
            lbwd("qkv", self.dqkv, self.xn1, self.dxn1, M)
            catq_aux_rmsnorm_bwd(x, self.rstd1, self.dxn1, self.dx, dres=self.dh1)
        else:
            L = self.lin["qkv"]
            if side is not None:
                self.order("qkv", main, side)
            with torch.cuda.stream(side if side is not None else main):
                catq_fakeq_linear_bwd(self.dqkv, self.xn1, L.W_fake, M, L.d_out, L.d_in, L.W,
                                      L.stats, L.d_mu, L.d_alpha, L.d_delta, p, L.g_mu,
                                      L.g_alpha, L.g_delta, ws)
        if side is not None and join:
            self.order("join", side, main)

    step = DenseBlock.step

    @staticmethod
    def split_fused(cfg, name, arr):
        """Per-linear pieces of a fused array; expert arrays are [E*rows][...]
        (or per-group values in the same order)."""
        hd = cfg.head_dim
        if name == "qkv":
            return _split_rows(arr, [cfg.n_q * hd, cfg.n_kv * hd, cfg.n_kv * hd],
                               ["Wq", "Wk", "Wv"])
        if name == "o":
            return {"Wo": arr}
        E, F = cfg.n_experts, cfg.expert_ffn
        if name == "gu":
            per = arr.reshape(E, 2 * F, -1)
            return {"Wg": per[:, :F].reshape(E * F, -1), "Wu": per[:, F:].reshape(E * F, -1)}
        return {"Wd": arr}


class StepGraph:
    """One calibration step (on one stream or both, as ``step_kw`` asks)
    captured as a HIP graph and replayed: the step's ~35 launches then cost one graph launch.  Inputs
    and outputs are the captured buffers: change them in place between
    replays (the factors are updated in place by the optimiser).  The step
    is run once eagerly first, so the side stream, the events and the
    cached statistics exist before capture."""

    def __init__(self, blk, x, y_fp, **step_kw):
        blk.step(x, y_fp, **step_kw)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.loss = blk.step(x, y_fp, **step_kw)
        torch.cuda.synchronize()

    def replay(self):
        self.graph.replay()
        return self.loss


def _split_rows(arr, sizes, names):
    total = sum(sizes)
    per_row = arr.shape[0] // total
    out, r = {}, 0
    for n, sz in zip(names, sizes):
        out[n] = arr[r * per_row:(r + sz) * per_row]
        r += sz
    return out
