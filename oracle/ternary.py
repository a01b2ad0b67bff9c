"""Deployment-side linear layer on the 2-bit storage of the final
ternarisation, float64.  Test infrastructure only: the HIP path never imports
it.

App. B.2 stores each weight as a ternary value T in {-1, 0, +1} plus one scale
alpha per group of g consecutive weights of a row (no zero point), so the
layer computes Y = X (alpha * T)^T.  The 2-bit layout is the one the pack
step writes: code c = T + 1, byte b of a row holds elements 4b..4b+3, element
4b + j in bits 2j..2j+1, least significant first.

READING: code 3 is never written for a valid weight (the pack step stores it
only for an out-of-range input); here it decodes to 0, i.e. contributes
nothing.
"""
from __future__ import annotations

import numpy as np


def unpack_codes(packed, d_in):
    """uint8 [rows][d_in / 4] -> codes int64 [rows][d_in] in {0, 1, 2, 3}."""
    p = np.asarray(packed, dtype=np.uint8).astype(np.int64)
    if p.ndim != 2 or p.shape[1] * 4 != d_in:
        raise ValueError("packed must be [rows][d_in / 4]")
    return np.stack([(p >> (2 * j)) & 3 for j in range(4)], axis=-1).reshape(p.shape[0], d_in)


def ternary_values(packed, d_in):
    """T = c - 1 for c in {0, 1, 2}; 0 for the invalid code 3."""
    c = unpack_codes(packed, d_in)
    return np.where(c == 3, 0, c - 1).astype(np.float64)


def dequantize(packed, alpha, d_in, g=128):
    """W = alpha * T with alpha [rows][d_in / g] (or flat) repeated over its
    group's g weights."""
    T = ternary_values(packed, d_in)
    a = np.asarray(alpha, dtype=np.float64).reshape(T.shape[0], d_in // g)
    return np.repeat(a, g, axis=1) * T


def ternary_linear(X, packed, alpha, d_in, g=128):
    """Y = X W^T for the dequantised W, X [M][d_in]."""
    return np.asarray(X, dtype=np.float64) @ dequantize(packed, alpha, d_in, g).T


def abs_terms(X, packed, alpha, d_in, g=128):
    """sum_k |X[m,k] W[n,k]|: the scale of the rounding error of any fp32
    summation of the products."""
    return np.abs(np.asarray(X, dtype=np.float64)) @ np.abs(dequantize(packed, alpha, d_in, g)).T
