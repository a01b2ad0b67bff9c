"""Activation fake quantization for the W1.58A8 setting, float64 with the
decisions taken in fp32.  Test infrastructure only: the HIP path never
imports it.

The paper (Sec. 3, W1.58A8 results) quantizes all intermediate activations
in the same calibration, except the softmax output, but does not define the
activation quantizer.

READING: symmetric 8-bit absmax fake quantization per group of consecutive
values (a token's feature vector for a linear layer's input, a token's head
vector for the attention operands Q, K and V):
    s = fp32(max|x| / 127)         (0 for an all-zero group)
    q = round-half-even(fp32(x / s)) in [-127, 127]     (q = 0 when s = 0)
    x_q = bf16(fp32(q * s))
The backward is straight-through: dL/dx = dL/dx_q.  The inputs are the
stored activations (bf16 or fp32 values), so both sides take every decision
on the same numbers in the same precision.
"""
from __future__ import annotations

import numpy as np


def bf16_round(x32):
    """fp32 -> nearest bf16 (ties to even), returned as float64."""
    b = np.asarray(x32, np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def quantize(x, group):
    """x [..., n] (values exactly representable in fp32), groups of `group`
    consecutive values along the last axis.  Returns (x_q float64 holding
    bf16 values, codes int8, scales fp32 per group)."""
    x = np.asarray(x, np.float64)
    n = x.shape[-1]
    if n % group:
        raise ValueError("the last axis must hold whole groups")
    xg = x.reshape(*x.shape[:-1], n // group, group).astype(np.float32)
    amax = np.abs(xg).max(axis=-1, keepdims=True)
    s = (amax / np.float32(127.0)).astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(s > 0, xg / np.where(s > 0, s, np.float32(1)), np.float32(0)).astype(np.float32)
    q = np.clip(np.rint(r), -127, 127).astype(np.float32)
    xq32 = (q * s).astype(np.float32)
    xq = bf16_round(xq32).reshape(x.shape)
    return xq, q.astype(np.int8).reshape(x.shape), s[..., 0]
