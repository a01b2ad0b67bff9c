"""Pins for the W1.58A8 activation fake quantization (reading: symmetric
8-bit absmax per group, round half to even, straight-through backward) and
its place in the oracle's block.

* hand-computed groups (ties to even, the group maximum at +-127, an
  all-zero group, a negative maximum);
* the bf16 rounding helper against exhaustive ties and torch's conversion;
* properties at any size: codes in [-127, 127], each group attains |q| = 127,
  |x - x_q| <= s/2 plus the bf16 rounding of the product;
* the a8 block: its straight-through gradients are the plain block's
  gradients evaluated at the quantized activations (checked through torch
  autograd with the quantizer as a custom straight-through function), and it
  differs from the full-precision block by the small amount 8-bit
  activations cost.
"""
import numpy as np
import pytest
import torch

import synthgen as sg
from oracle import actquant, block, calib, lmst


def test_hand_group_ties_to_even():
    x = np.array([[127.0, -63.5, 0.5, 1.5, 2.5, -0.5, 0.0, 126.5]])
    xq, q, s = actquant.quantize(x, 8)
    assert s[0, 0] == np.float32(1.0)
    np.testing.assert_array_equal(q, [[127, -64, 0, 2, 2, 0, 0, 126]])
    np.testing.assert_array_equal(xq, [[127, -64, 0, 2, 2, 0, 0, 126]])


def test_hand_groups_zero_and_negative_max():
    x = np.array([[0.0, 0.0, 0.0, 0.0, -2.54, 1.27, 0.0, 0.02]])
    xq, q, s = actquant.quantize(x, 4)
    np.testing.assert_array_equal(q[0, :4], 0)
    np.testing.assert_array_equal(xq[0, :4], 0)
    assert s[0, 0] == 0
    s1 = np.float32(np.float32(2.54) / np.float32(127))
    assert s[0, 1] == s1
    assert q[0, 4] == -127 and q[0, 5] == 64  # 1.27 / 0.02 = 63.5 (fp32) -> even 64
    assert xq[0, 4] == actquant.bf16_round(np.float32(-127) * s1)


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32),
                        # exact ties: 8 significant bits + a half
                        (np.arange(256, 512, dtype=np.float32) + 0.5) * np.float32(2.0 ** -8)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(actquant.bf16_round(x), ref)


@pytest.mark.parametrize("group", [64, 128, 2048])
def test_properties(group):
    rng = np.random.default_rng(group)
    x = actquant.bf16_round(rng.standard_t(4, (7, 4096)).astype(np.float32) * 3)
    xq, q, s = actquant.quantize(x, group)
    assert q.min() >= -127 and q.max() <= 127
    qg = np.abs(q.reshape(7, -1, group).astype(np.int32)).max(-1)
    assert np.all(qg == 127)
    sg_ = np.repeat(s.astype(np.float64), group, axis=-1)
    assert np.all(np.abs(x - xq) <= sg_ / 2 + 2.0 ** -8 * np.abs(xq) + 1e-30)


class _STE(torch.autograd.Function):
    """The reading's quantizer (on the bf16-stored activation) with a
    straight-through backward."""

    @staticmethod
    def forward(ctx, x, group):
        x32 = x.detach().numpy().astype(np.float32)
        xq = actquant.quantize(actquant.bf16_round(x32), group)[0]
        return torch.from_numpy(xq)

    @staticmethod
    def backward(ctx, g):
        return g, None


def test_a8_block_gradients_are_straight_through():
    """The a8 block's hand-written backward against torch autograd of a
    mirror built from torch ops and the straight-through quantizer."""
    cfg = sg.small_dense(batch=1, seq=6, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    W = {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in sg.block_weights(cfg, 0).items()}
    x = sg.bf16_bits_to_f32(sg.activations(cfg, 0)).astype(np.float64)
    y, cache = block.block_forward(x, W, cfg, a8=True)
    dy = np.random.default_rng(1).standard_normal(y.shape)
    dx, dW = block.block_backward(dy, cache, W, cfg)

    B, S, Hq, Hkv, hd = cfg.batch, cfg.seq, cfg.n_q, cfg.n_kv, cfg.head_dim
    tx = torch.tensor(x, requires_grad=True)
    tW = {k: torch.tensor(v, requires_grad=True) for k, v in W.items()}

    def rms(t):
        return t * torch.rsqrt((t * t).mean(-1, keepdim=True) + block.EPS)

    def aq(t, g):
        return _STE.apply(t, g)

    cos, sin = block.rope_tables(S, hd, cfg.rope_theta)
    cos, sin = torch.tensor(cos)[None, :, None], torch.tensor(sin)[None, :, None]

    def rope(t):
        h = hd // 2
        return torch.cat([t[..., :h] * cos - t[..., h:] * sin, t[..., h:] * cos + t[..., :h] * sin], -1)

    xn1 = aq(rms(tx), cfg.hidden)
    q = rope(rms((xn1 @ tW["Wq"].T).reshape(B, S, Hq, hd)))
    k = rope(rms((xn1 @ tW["Wk"].T).reshape(B, S, Hkv, hd)))
    v = (xn1 @ tW["Wv"].T).reshape(B, S, Hkv, hd)
    q, k, v = aq(q, hd), aq(k, hd), aq(v, hd)
    G = Hq // Hkv
    kk = k.repeat_interleave(G, dim=2)
    vv = v.repeat_interleave(G, dim=2)
    sc = torch.einsum("bshd,bthd->bhst", q, kk) / np.sqrt(hd)
    mask = torch.triu(torch.ones(S, S, dtype=torch.bool), 1)
    P = torch.softmax(sc.masked_fill(mask, -np.inf), -1)
    O = torch.einsum("bhst,bthd->bshd", P, vv).reshape(B * S, Hq * hd)
    h1 = tx + aq(O, Hq * hd) @ tW["Wo"].T
    xn2 = aq(rms(h1), cfg.hidden)
    gt, up = xn2 @ tW["Wg"].T, xn2 @ tW["Wu"].T
    a = aq(torch.nn.functional.silu(gt) * up, cfg.ffn)
    ty = h1 + a @ tW["Wd"].T
    np.testing.assert_allclose(ty.detach().numpy(), y, rtol=1e-12, atol=1e-12)
    ty.backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-9, atol=1e-11)
    for k_ in W:
        np.testing.assert_allclose(dW[k_], tW[k_].grad.numpy(), rtol=1e-9, atol=1e-11)


def test_a8_step_is_close_to_the_w16_step():
    cfg = sg.small_dense(batch=1, seq=8, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128)
    W = {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in sg.block_weights(cfg, 0).items()}
    x = sg.bf16_bits_to_f32(sg.activations(cfg, 0)).astype(np.float64)
    fac = {k: sg.perturbed_factors(1, w.size // 128) for k, w in W.items()}
    a = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0, s_bwd=30.0, a8=True)
    b = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0, s_bwd=30.0)
    np.testing.assert_array_equal(a["y_fp"], b["y_fp"])      # the target is the W16A16 block
    d = np.abs(a["y_q"] - b["y_q"]).max() / np.abs(b["y_q"] - x).max()
    assert 0 < d < 0.05
    assert 0 < abs(a["loss"] - b["loss"]) < 0.2 * b["loss"]


def test_given_quantized_activations_reproduce_the_a8_step():
    """The a8 path fed its own quantized activations as a dict (the form a
    comparison uses to take another computation's code decisions) gives the
    a8 step bit for bit: every quantization point is wired to its name."""
    from oracle import block, calib, lmst
    cfg = sg.small_dense(batch=2, seq=24, hidden=128, n_q=4, n_kv=2, head_dim=64, ffn=256)
    W = {k: sg.bf16_bits_to_f32(v).astype(np.float64) for k, v in sg.block_weights(cfg, 0).items()}
    x = sg.bf16_bits_to_f32(sg.activations(cfg, 0)).astype(np.float64)
    fac = {k: list(sg.perturbed_factors(3, v.size // 128)) for k, v in W.items()}
    ref = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0, s_bwd=30.0, a8=True)
    Wf = calib.fake_weights(W, fac, 128, lmst.SOFT, 15.0)
    _, (ca, cm) = block.block_forward(x, Wf, cfg, True)
    given = {"xn1": ca["xn1"], "qr": ca["qr"], "kr": ca["kr"], "v": ca["v"], "attn": ca["attn"],
             "xn2": cm["xn2"], "a": cm["a"]}
    got = calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0, s_bwd=30.0, a8=given)
    assert got["loss"] == ref["loss"]
    np.testing.assert_array_equal(got["dx"], ref["dx"])
    for k in W:
        for i in range(3):
            np.testing.assert_array_equal(got["fgrads"][k][i], ref["fgrads"][k][i])
    # a different given activation changes the step (the values are used)
    given["a"] = given["a"] * 1.01
    assert calib.dense_step(x, W, fac, cfg, lmst.SOFT, s=15.0, s_bwd=30.0,
                            a8=given)["loss"] != ref["loss"]
