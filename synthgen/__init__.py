"""Seeded synthetic inputs shared by the CPU oracle and the HIP path.

This module only draws and materialises numbers: weights, calibration
activations, router logits and learnable-factor values.  It holds none of the
quantisation method's arithmetic, so both the oracle and the GPU path can
consume the very same bytes without sharing any of the method's code.

Every tensor comes from its own PCG64 stream, ``default_rng([seed, tensor_id])``
(plus a sample index for calibration samples), drawn in float64 and rounded
to the storage type (fp32, or bf16 through fp32 with round-to-nearest-even).
bf16 tensors are carried as ``uint16`` bit patterns.

The paper calibrates on 512 C4 samples of 2048 tokens and pre-trained model
weights (Sec. 3.1, App. B.1); neither is available here.  The recipes below
take the shapes of those workloads (decoder blocks shaped like Qwen3-1.7B,
Llama-3-8B, Qwen3-14B and Qwen3-235B-A22B) with synthetic value laws.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

# tensor ids: one independent stream per named tensor
_TID = {
    "Wq": 1, "Wk": 2, "Wv": 3, "Wo": 4, "Wg": 5, "Wu": 6, "Wd": 7,
    "X": 20, "router": 21, "router_bias": 22, "W": 30,
    "dmu": 40, "dalpha": 41, "ddelta": 42, "G": 43, "Y": 44, "codes": 45,
    "outlier_cols": 50,
}
LINEARS = ("Wq", "Wk", "Wv", "Wo", "Wg", "Wu", "Wd")


def rng(seed: int, name: str, *extra: int) -> np.random.Generator:
    """Independent PCG64 stream for tensor ``name``."""
    return np.random.default_rng([int(seed), _TID[name]] + [int(e) for e in extra])


# ---------------------------------------------------------------- bf16 bits

def f32_to_bf16_bits(x) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest even), as uint16."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(np.asarray(b, dtype=np.uint16))
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_bf16_bits(x64) -> np.ndarray:
    return f32_to_bf16_bits(np.asarray(x64, dtype=np.float64).astype(np.float32))


# ---------------------------------------------------------------- configs

@dataclasses.dataclass(frozen=True)
class DenseBlockCfg:
    """Pre-norm decoder block shape (no biases)."""
    name: str
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    ffn: int
    qk_norm: bool
    rope_theta: float
    batch: int
    seq: int
    w_std: float
    w_outlier_frac: float = 0.0       # fraction of entries per matrix scaled x10
    x_law: str = "student_t4"         # "student_t4" | "normal"

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    def linear_shapes(self) -> Dict[str, tuple]:
        h, hd = self.hidden, self.head_dim
        return {
            "Wq": (self.n_q * hd, h), "Wk": (self.n_kv * hd, h), "Wv": (self.n_kv * hd, h),
            "Wo": (h, self.n_q * hd), "Wg": (self.ffn, h), "Wu": (self.ffn, h),
            "Wd": (h, self.ffn),
        }

    def n_weights(self) -> int:
        return sum(a * b for a, b in self.linear_shapes().values())


@dataclasses.dataclass(frozen=True)
class MoEBlockCfg:
    """Decoder block whose MLP is a routed mixture of SwiGLU experts."""
    name: str
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    n_experts: int
    top_k: int
    expert_ffn: int
    qk_norm: bool
    rope_theta: float
    batch: int
    seq: int
    w_std: float
    router_bias_std: float = 0.0      # >0 gives skewed per-expert loads
    x_law: str = "student_t4"

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    def attn_shapes(self) -> Dict[str, tuple]:
        h, hd = self.hidden, self.head_dim
        return {"Wq": (self.n_q * hd, h), "Wk": (self.n_kv * hd, h),
                "Wv": (self.n_kv * hd, h), "Wo": (h, self.n_q * hd)}

    def expert_shapes(self) -> Dict[str, tuple]:
        return {"Wg": (self.n_experts, self.expert_ffn, self.hidden),
                "Wu": (self.n_experts, self.expert_ffn, self.hidden),
                "Wd": (self.n_experts, self.hidden, self.expert_ffn)}


# Workloads shaped like the paper's models (Sec. 3.1): one decoder block each.
QWEN3_1P7B = DenseBlockCfg("qwen3-1.7b-block", 2048, 16, 8, 128, 6144, True, 1e6,
                           batch=4, seq=2048, w_std=0.02)
LLAMA3_8B = DenseBlockCfg("llama3-8b-block", 4096, 32, 8, 128, 14336, False, 5e5,
                          batch=4, seq=2048, w_std=0.015, w_outlier_frac=1e-3,
                          x_law="normal")
QWEN3_14B = DenseBlockCfg("qwen3-14b-block", 5120, 40, 8, 128, 17408, True, 1e6,
                          batch=2, seq=4096, w_std=0.015)
QWEN3_235B_MOE = MoEBlockCfg("qwen3-235b-a22b-moe-block", 4096, 64, 4, 128, 128, 8, 1536,
                             True, 1e6, batch=2, seq=2048, w_std=0.02)
QWEN3_235B_MOE_SKEW = dataclasses.replace(QWEN3_235B_MOE, name="qwen3-235b-a22b-moe-block-skew",
                                          router_bias_std=0.5)


def small_dense(batch=2, seq=80, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384,
                qk_norm=True, w_std=0.02, x_law="student_t4", name="small-dense"):
    """Reduced block that keeps every structural feature (GQA, QK-norm, ragged tiles)."""
    return DenseBlockCfg(name, hidden, n_q, n_kv, head_dim, ffn, qk_norm, 1e6,
                         batch=batch, seq=seq, w_std=w_std, x_law=x_law)


def small_moe(batch=2, seq=48, hidden=256, n_q=4, n_kv=2, head_dim=64, n_experts=8, top_k=2,
              expert_ffn=128, router_bias_std=0.0, name="small-moe"):
    return MoEBlockCfg(name, hidden, n_q, n_kv, head_dim, n_experts, top_k, expert_ffn, True,
                       1e6, batch=batch, seq=seq, w_std=0.02, router_bias_std=router_bias_std)


# ---------------------------------------------------------------- draws

def normal_weight(seed: int, name: str, shape, std: float, outlier_frac: float = 0.0,
                  dtype: str = "bf16", extra=()) -> np.ndarray:
    """N(0, std^2) weight; ``outlier_frac`` of the entries (uniform, without
    replacement) are multiplied by 10."""
    g = rng(seed, name, *extra)
    w = g.standard_normal(shape) * std
    if outlier_frac > 0:
        n = w.size
        k = max(1, int(round(n * outlier_frac)))
        idx = g.choice(n, size=k, replace=False)
        w.reshape(-1)[idx] *= 10.0
    return to_bf16_bits(w) if dtype == "bf16" else w.astype(np.float32)


def block_weights(cfg, seed: int = 0) -> Dict[str, np.ndarray]:
    """All quantised weights of a block as bf16 bit patterns, [d_out][d_in]
    (experts: [E][d_out][d_in])."""
    out = {}
    if isinstance(cfg, DenseBlockCfg):
        for n, shp in cfg.linear_shapes().items():
            out[n] = normal_weight(seed, n, shp, cfg.w_std, cfg.w_outlier_frac)
    else:
        for n, shp in cfg.attn_shapes().items():
            out[n] = normal_weight(seed, n, shp, cfg.w_std)
        for n, shp in cfg.expert_shapes().items():
            out[n] = normal_weight(seed, n, shp, cfg.w_std)
    return out


def activations(cfg, seed: int = 0, sample0: int = 0) -> np.ndarray:
    """Block input X as bf16 bits [batch*seq][hidden]; sample ``sample0+b`` for
    batch row b, each sample from its own stream (so a calibration set is the
    concatenation of per-sample draws)."""
    rows = []
    for b in range(cfg.batch):
        g = rng(seed, "X", sample0 + b)
        if cfg.x_law == "student_t4":
            x = g.standard_t(4.0, size=(cfg.seq, cfg.hidden))
        else:
            x = g.standard_normal((cfg.seq, cfg.hidden))
        rows.append(to_bf16_bits(x))
    return np.concatenate(rows, axis=0)


def router_logits(cfg: MoEBlockCfg, seed: int = 0) -> np.ndarray:
    """Router logits fp32 [tokens][n_experts], N(0,1) plus an optional
    per-expert bias N(0, router_bias_std^2) that skews expert loads."""
    g = rng(seed, "router")
    lg = g.standard_normal((cfg.tokens, cfg.n_experts))
    if cfg.router_bias_std > 0:
        lg = lg + rng(seed, "router_bias").standard_normal(cfg.n_experts) * cfg.router_bias_std
    return lg.astype(np.float32)


def init_factors(n_groups: int):
    """Identity modulation: delta_mu = 0, delta_alpha = 1, delta_Delta = 1."""
    return (np.zeros(n_groups, np.float32), np.ones(n_groups, np.float32),
            np.ones(n_groups, np.float32))


def perturbed_factors(seed: int, n_groups: int, spread: float = 0.3, extra=()):
    """Factors drawn around the identity modulation inside the paper's
    constraints (-1 < d_mu < 1, d_alpha > 0, d_Delta > 0)."""
    dmu = rng(seed, "dmu", *extra).uniform(-spread, spread, n_groups)
    dal = np.exp(rng(seed, "dalpha", *extra).uniform(-spread, spread, n_groups))
    dde = np.exp(rng(seed, "ddelta", *extra).uniform(-spread, spread, n_groups))
    return dmu.astype(np.float32), dal.astype(np.float32), dde.astype(np.float32)


def single_linear_case(seed: int = 0):
    """Single 256x256 fp32 linear: W ~ N(0, 0.02^2); calibration activations
    8 samples x 128 tokens, N(0,1) with 4 outlier channels scaled x20."""
    W = rng(seed, "W").standard_normal((256, 256)) * 0.02
    X = rng(seed, "X").standard_normal((8 * 128, 256))
    cols = rng(seed, "outlier_cols").choice(256, 4, replace=False)
    X[:, cols] *= 20.0
    return W.astype(np.float32), X.astype(np.float32)


def uniform_f32(seed: int, name: str, shape, lo=-1.0, hi=1.0, extra=()) -> np.ndarray:
    return rng(seed, name, *extra).uniform(lo, hi, shape).astype(np.float32)


def normal_bf16(seed: int, name: str, shape, std=1.0, extra=()) -> np.ndarray:
    return to_bf16_bits(rng(seed, name, *extra).standard_normal(shape) * std)
