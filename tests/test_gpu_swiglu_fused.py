"""The SwiGLU MLP's fused GEMM epilogues against the separate kernels and the
oracle.

* gate|up projection with silu(gate) * up in the epilogue: gu and a bit for
  bit equal to the plain GEMM followed by the SwiGLU kernel (the fused launch
  runs the same 256 x 256 kernel on the shapes it takes, with the weight rows
  read in gate/up pairs), and sampled rows against the oracle;
* down projection's input gradient with the SwiGLU backward in the epilogue:
  d[gate | up] bit for bit equal to the plain dX GEMM followed by the SwiGLU
  backward kernel, and sampled rows against the oracle's MLP backward on the
  stored values;
* shapes the fused launch does not take (small, or F not a multiple of 256
  for the backward) run the separate kernels inside the library; a ragged
  token count and an F that is not a multiple of the 128 gate/up pairs of a
  tile exercise the edge tiles;
* the 1.7B-shaped block's step with and without the fusion: same bits.

Sampled-row bound for a: a = bf16(fp32 silu(g) * u) on the stored bf16 g, u,
so |a - a_ref| <= 2^-8 |a_ref| (one bf16 rounding) plus the fp32 evaluation,
a few units of 2^-24 relative (exp, reciprocal, two products); 2^-8 + 2^-16
relative covers both.  d up likewise.  d gate = d a * up * sigma(g) *
(1 + g (1 - sigma(g))) cancels inside the bracket near g = -1.278, so its
fp32 evaluation error is bounded against the size of the terms instead:
2^-20 |d a| |up| (1 + |g|) on top of the bf16 rounding."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, to_dev_bf16
from oracle import block as ob
from oracle import lmst

pytestmark = pytest.mark.gpu

RTOL = 2.0 ** -8 + 2.0 ** -16


def _bits(t):
    import torch
    return t.view(torch.int16)


def _gateup(catq, M, F, K, seed):
    import torch
    xb = sg.normal_bf16(seed, "X", (M, K))
    wb = sg.normal_bf16(seed, "W", (2 * F, K), std=0.05)
    X, W = to_dev_bf16(xb), to_dev_bf16(wb)
    gu_f = torch.full((M, 2 * F), float("nan"), dtype=torch.bfloat16, device="cuda")
    a_f = torch.full((M, F), float("nan"), dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_gateup_swiglu_fwd(X, W, gu_f, a_f, M, F, K)
    gu_s = torch.empty_like(gu_f)
    a_s = torch.empty_like(a_f)
    catq.catq_fakeq_linear_fwd(X, W, gu_s, M, 2 * F, K)
    catq.catq_aux_swiglu_fwd(gu_s, a_s)
    torch.cuda.synchronize()
    return xb, wb, gu_f, a_f, gu_s, a_s


@pytest.mark.parametrize("M,F,K", [(2048, 4096, 512),     # fused
                                   (2085, 4104, 256),     # fused, ragged M, partial pair tile
                                   (300, 384, 256),       # separate kernels
                                   (1, 8, 64)])
def test_gateup_swiglu_fused(catq, M, F, K):
    xb, wb, gu_f, a_f, gu_s, a_s = _gateup(catq, M, F, K, 1)
    import torch
    assert torch.equal(_bits(gu_f), _bits(gu_s))
    assert torch.equal(_bits(a_f), _bits(a_s))
    rows = np.unique(np.r_[0, M - 1, np.random.default_rng(M).integers(0, M, 14)])
    ref = f64(xb[rows]) @ f64(wb).T
    gu = host(gu_f)[rows]
    assert max_norm_err(gu, ref) <= 4e-3
    a_ref = ob.silu(gu[:, :F]) * gu[:, F:]
    err = np.abs(host(a_f)[rows] - a_ref)
    assert np.all(err <= RTOL * np.abs(a_ref) + 1e-30), float(err.max())


def _down(catq, M, N, F, seed):
    import torch
    dyb = sg.normal_bf16(seed, "Y", (M, N))
    wb = sg.normal_bf16(seed, "W", (N, F), std=0.05)
    gub = sg.normal_bf16(seed, "X", (M, 2 * F))
    dY, W, gu = to_dev_bf16(dyb), to_dev_bf16(wb), to_dev_bf16(gub)
    dgu_f = torch.full((M, 2 * F), float("nan"), dtype=torch.bfloat16, device="cuda")
    da = torch.empty(M, F, dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_down_swiglu_bwd(dY, W, gu, dgu_f, M, N, F, da=da)
    da_s = torch.empty_like(da)
    dgu_s = torch.empty_like(dgu_f)
    p = catq.lmst_params(mode=lmst.SOFT, s=15.0)
    catq.catq_fakeq_linear_bwd(dY, da, W, M, N, F, W, None, None, None, None, p,
                               None, None, None, None, dX=da_s)
    catq.catq_aux_swiglu_bwd(gu, da_s, dgu_s)
    torch.cuda.synchronize()
    return dyb, wb, gub, dgu_f, dgu_s, da_s


@pytest.mark.parametrize("M,N,F", [(4096, 512, 4096),      # fused
                                   (4141, 256, 4096),      # fused, ragged M
                                   (2048, 256, 10240),     # fused, 1.25 rounds of tiles
                                   (4096, 256, 4104),      # separate (F % 256)
                                   (512, 256, 384)])       # separate (small)
def test_down_swiglu_bwd_fused(catq, M, N, F):
    import torch
    dyb, wb, gub, dgu_f, dgu_s, da_s = _down(catq, M, N, F, 2)
    assert torch.equal(_bits(dgu_f), _bits(dgu_s))
    rows = np.unique(np.r_[0, M - 1, np.random.default_rng(M).integers(0, M, 14)])
    da_ref = f64(dyb[rows]) @ f64(wb)
    da = host(da_s)[rows]
    assert max_norm_err(da, da_ref) <= 4e-3
    gu = f64(gub[rows])
    # the oracle's MLP backward from d a (as stored) to d gate, d up
    c = {"gt": gu[:, :F], "up": gu[:, F:]}
    dgt = da * c["up"] * ob.silu_grad(c["gt"])
    dup = da * ob.silu(c["gt"])
    got = host(dgu_f)[rows]
    terms = 2.0 ** -20 * np.abs(da) * np.abs(c["up"]) * (1 + np.abs(c["gt"]))
    for g_, r_, t_ in ((got[:, :F], dgt, terms), (got[:, F:], dup, 0.0)):
        err = np.abs(g_ - r_)
        assert np.all(err <= RTOL * np.abs(r_) + t_ + 1e-30), float(err.max())


def test_down_swiglu_bwd_needs_scratch_when_not_fused(catq):
    import torch
    M, N, F = 512, 256, 384
    z = torch.zeros(M, max(N, 2 * F), dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(N, F, dtype=torch.bfloat16, device="cuda")
    dgu = torch.zeros(M, 2 * F, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(catq.CatqError, match="scratch"):
        catq.catq_fakeq_down_swiglu_bwd(z[:, :N].contiguous(), W, dgu.clone(), dgu, M, N, F)


def test_full_size_block_fused_equals_separate(catq):
    """The 1.7B-shaped block (4 x 2048 tokens, F = 6144): both fused launches
    are taken, and the step's loss, input gradient and every factor
    gradient are the same bits as with the separate SwiGLU kernels."""
    import torch
    from paper_2606_26650_amd.block import DenseBlock
    cfg = sg.QWEN3_1P7B
    blk = DenseBlock(cfg, sg.block_weights(cfg, 0))
    for i, L in enumerate(blk.lin.values()):
        L.set_factors(*sg.perturbed_factors(5, L.n_groups, extra=(i,)))
    x = to_dev_bf16(sg.activations(cfg, 0))
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    out = []
    for fuse in (False, True):
        blk.fuse_swiglu = fuse
        l = blk.step(x, y_fp, mode=lmst.SOFT, s=15.0).clone()
        torch.cuda.synchronize()
        out.append((l, blk.dx.clone(), blk.a.clone(),
                    [t.clone() for L in blk.lin.values() for t in (L.g_mu, L.g_alpha, L.g_delta)]))
    a, b = out
    assert torch.isfinite(a[0]).all() and a[0].item() > 0
    assert torch.equal(a[0], b[0])
    assert torch.equal(_bits(a[1]), _bits(b[1]))
    assert torch.equal(_bits(a[2]), _bits(b[2]))
    for u, v in zip(a[3], b[3]):
        assert torch.equal(u, v)
