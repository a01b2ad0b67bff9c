"""Shared helpers for the GPU parity tests (tolerances, host/device moves)."""
import numpy as np

import synthgen as sg


def f64(bits):
    """Oracle view of bf16 bit patterns: their exact values in float64."""
    return sg.bf16_bits_to_f32(bits).astype(np.float64)


def to_dev_bf16(bits):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.cuda().view(torch.bfloat16)


def to_dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host(t):
    """Device tensor -> float64 numpy (bf16 widened exactly)."""
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        return t.float().cpu().numpy().astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def max_norm_err(g, r):
    """max|g - r| / max|r| over the tensor (the GEMM / loss / gradient metric)."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    den = np.abs(r).max()
    return float(np.abs(g - r).max() / (den if den > 0 else 1.0))


def elem_rel_ok(g, r, tol, floor=1e-30):
    """|g - r| <= tol |r| elementwise, or both below the underflow floor."""
    g = np.asarray(g, np.float64)
    r = np.asarray(r, np.float64)
    ok = (np.abs(g - r) <= tol * np.abs(r)) | ((np.abs(g) < floor) & (np.abs(r) < floor))
    return bool(ok.all()), float(np.max(np.abs(g - r) / np.maximum(np.abs(r), floor)))


def median_rel(g, r):
    g = np.asarray(g, np.float64).ravel()
    r = np.asarray(r, np.float64).ravel()
    m = np.abs(r) > 0
    return float(np.median(np.abs(g[m] - r[m]) / np.abs(r[m]))) if m.any() else 0.0
