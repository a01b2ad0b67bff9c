"""Pins for the oracle's packed-ternary linear layer (App. B.2 storage).

* a hand-decoded byte (0x46 = codes 2, 1, 0, 1 = T +1, 0, -1, 0) and rows of
  it against the closed-form product with X = 0, 1, 2, ...;
* one nonzero code at each position of a byte and of a row: y is +-alpha x_k
  of exactly that k (a wrong bit position or element order fails it);
* the scale of a group applies to exactly its g weights (g = 128 and 256);
* the deployment product equals the calibration's hard fake-weight product:
  codes and scales from the hard ternarisation, packed by the pack step,
  decoded here, give X (alpha T)^T = X W_fake^T of the hard branch.
"""
import numpy as np
import pytest

import synthgen as sg
from oracle import lmst, ternary


def test_hand_decoded_byte():
    assert ternary.unpack_codes(np.array([[0x46]], np.uint8), 4).tolist() == [[2, 1, 0, 1]]
    np.testing.assert_array_equal(ternary.ternary_values(np.array([[0x46]], np.uint8), 4),
                                  [[1, 0, -1, 0]])
    # a row of 128 weights, bytes 0x46: T = (+1, 0, -1, 0) * 32, alpha = 0.5,
    # x_k = k: y = 0.5 * sum_i (4i - (4i + 2)) = 0.5 * 32 * (-2) = -32
    packed = np.full((1, 32), 0x46, np.uint8)
    x = np.arange(128, dtype=np.float64)[None]
    assert ternary.ternary_linear(x, packed, [0.5], 128)[0, 0] == -32.0
    # all codes 0 (T = -1), alpha 1: y = -sum x
    assert ternary.ternary_linear(x, np.zeros((1, 32), np.uint8), [1.0], 128)[0, 0] == -8128.0
    # all codes 1 (T = 0): y = 0
    assert ternary.ternary_linear(x, np.full((1, 32), 0x55, np.uint8), [3.0], 128)[0, 0] == 0.0


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4, 63, 127, 128, 200, 255])
def test_single_code_position(k):
    d_in = 256
    packed = np.full((1, d_in // 4), 0x55, np.uint8)           # all T = 0
    packed[0, k // 4] = (0x55 & ~(3 << (2 * (k % 4)))) | (2 << (2 * (k % 4)))   # T_k = +1
    x = (np.arange(d_in, dtype=np.float64) + 1.0)[None] * 0.25
    alpha = np.array([1.5, 2.5])
    y = ternary.ternary_linear(x, packed, alpha, d_in)[0, 0]
    assert y == alpha[k // 128] * x[0, k]
    packed[0, k // 4] = 0x55 & ~(3 << (2 * (k % 4)))             # T_k = -1
    assert ternary.ternary_linear(x, packed, alpha, d_in)[0, 0] == -alpha[k // 128] * x[0, k]


def test_invalid_code_contributes_nothing():
    packed = np.full((1, 32), 0xFF, np.uint8)   # every code 3
    assert ternary.ternary_linear(np.ones((1, 128)), packed, [1.0], 128)[0, 0] == 0.0


@pytest.mark.parametrize("g", [128, 256])
def test_group_scale_span(g):
    d_in = 512
    rng = np.random.default_rng(1)
    codes = rng.integers(0, 3, (3, d_in))
    packed = lmst.pack_ternary((codes - 1).astype(np.int8))
    alpha = rng.uniform(0.5, 2.0, (3, d_in // g))
    x = rng.standard_normal((2, d_in))
    y = ternary.ternary_linear(x, packed, alpha, d_in, g)
    ref = np.zeros((2, 3))
    for n in range(3):
        for k in range(d_in):
            ref[:, n] += x[:, k] * alpha[n, k // g] * (codes[n, k] - 1)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_deployment_product_is_the_hard_branch_product():
    W = sg.bf16_bits_to_f32(sg.normal_bf16(3, "W", (48, 384), std=0.02)).astype(np.float64)
    fac = sg.perturbed_factors(2, W.size // 128)
    hard = lmst.modulate_ternarize(W, 128, *fac, lmst.HARD)
    packed = lmst.pack_ternary(hard["codes"])
    x = np.random.default_rng(4).standard_normal((5, 384))
    y = ternary.ternary_linear(x, packed, hard["alpha"], 384)
    np.testing.assert_allclose(y, x @ hard["W_fake"].T, rtol=1e-12, atol=1e-15)
    np.testing.assert_array_equal(ternary.dequantize(packed, hard["alpha"], 384), hard["W_fake"])


def test_abs_terms_bounds_the_product():
    rng = np.random.default_rng(5)
    packed = rng.integers(0, 256, (4, 64)).astype(np.uint8)
    alpha = rng.uniform(0.1, 1.0, (4, 2))
    x = rng.standard_normal((3, 256))
    y = ternary.ternary_linear(x, packed, alpha, 256)
    s = ternary.abs_terms(x, packed, alpha, 256)
    assert np.all(np.abs(y) <= s + 1e-12) and np.all(s > 0)
