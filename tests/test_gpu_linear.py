"""GPU parity of the fake-ternary linear layer (forward GEMM, dX and dW GEMMs,
factor gradients) against the oracle, at sizes that span several tiles with
ragged tails, for routed experts with uneven (and empty) groups, and at the
full size of the 1.7B-shaped block on sampled outputs."""
import numpy as np
import pytest

import synthgen as sg
from helpers import f64, host, max_norm_err, to_dev_bf16, to_dev_f32
from oracle import lmst

pytestmark = pytest.mark.gpu


def _xw(seed, M, N, K, wstd=0.02):
    xb = sg.normal_bf16(seed, "X", (M, K))
    wb = sg.normal_bf16(seed, "W", (N, K), std=wstd)
    return xb, wb


@pytest.mark.parametrize("M,N,K", [(1, 8, 8), (77, 136, 200), (300, 256, 64), (513, 520, 1024),
                                   (1024, 1280, 384)])
def test_fwd_gemm(catq, M, N, K):
    import torch
    xb, wb = _xw(1, M, N, K)
    X, W = to_dev_bf16(xb), to_dev_bf16(wb)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K)
    torch.cuda.synchronize()
    ref = f64(xb) @ f64(wb).T
    assert max_norm_err(host(Y), ref) <= 4e-3


def test_fwd_gemm_residual(catq):
    import torch
    M, N, K = 200, 264, 136
    xb, wb = _xw(2, M, N, K)
    rb = sg.normal_bf16(3, "Y", (M, N))
    X, W, R = to_dev_bf16(xb), to_dev_bf16(wb), to_dev_bf16(rb)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K, residual=R)
    torch.cuda.synchronize()
    ref = f64(xb) @ f64(wb).T + f64(rb)
    assert max_norm_err(host(Y), ref) <= 4e-3


def _bwd_case(catq, M, N, K, mode, s=15.0, seed=4):
    import torch
    xb = sg.normal_bf16(seed, "X", (M, K))
    wb = sg.normal_bf16(seed, "W", (N, K), std=0.02)
    dyb = sg.normal_bf16(seed, "Y", (M, N), std=1e-3)
    ng = N * K // 128
    fac = sg.perturbed_factors(seed, ng)
    W = to_dev_bf16(wb)
    dm, da, dd = (to_dev_f32(f) for f in fac)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(N, K, dtype=torch.bfloat16, device="cuda")
    p = catq.lmst_params(mode=mode, s=s, s_bwd=30.0)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    X, dY = to_dev_bf16(xb), to_dev_bf16(dyb)
    dX = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dW = torch.empty(N, K, dtype=torch.float32, device="cuda")
    g = [torch.empty(ng, dtype=torch.float32, device="cuda") for _ in range(3)]
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K), dtype=torch.uint8, device="cuda")
    catq.catq_fakeq_linear_bwd(dY, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws, dX=dX,
                               dW_fake=dW)
    torch.cuda.synchronize()
    Wo = f64(wb)
    wf_ref = lmst.modulate_ternarize(Wo, 128, *fac, mode, s=s)["W_fake"]
    G = f64(dyb).T @ f64(xb)
    assert max_norm_err(host(dW), G) <= 1e-4
    assert max_norm_err(host(dX), f64(dyb) @ wf_ref) <= 2e-2
    ref = lmst.factor_grads(G, Wo, 128, *fac, mode, s=s, s_bwd=30.0)
    for a, b in zip(g, ref):
        assert max_norm_err(host(a), b) <= 2e-2


@pytest.mark.parametrize("M,N,K", [(96, 256, 384), (4096, 256, 256), (1000, 384, 640),
                                   (640, 136, 256), (2048, 1024, 512)])
def test_bwd_soft(catq, M, N, K):
    _bwd_case(catq, M, N, K, catq.SOFT)


def test_bwd_hard_and_identity(catq):
    _bwd_case(catq, 300, 256, 256, catq.HARD)
    _bwd_case(catq, 300, 256, 256, catq.IDENTITY)


@pytest.mark.parametrize("E,N,K,counts", [
    (5, 256, 384, [130, 0, 7, 300, 64]),
    # extents that the direct-to-LDS kernels take for all three products
    # (rows by expert, and the contraction by expert with ragged ends)
    (4, 512, 768, [300, 0, 77, 650]),
    (3, 256, 256, [1, 513, 64])])
def test_grouped_experts(catq, E, N, K, counts):
    """Routed experts with uneven row counts, one expert empty."""
    import torch
    counts = np.array(counts)
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    M = int(off[-1])
    xb = sg.normal_bf16(5, "X", (M, K))
    wb = sg.normal_bf16(5, "W", (E, N, K), std=0.02)
    dyb = sg.normal_bf16(5, "Y", (M, N), std=1e-3)
    X, W, dY = to_dev_bf16(xb), to_dev_bf16(wb), to_dev_bf16(dyb)
    offs = torch.from_numpy(off).cuda()
    Y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    catq.catq_trace_enable(64)
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K, n_experts=E, row_offsets=offs)
    ng = E * N * K // 128
    fac = sg.perturbed_factors(6, ng)
    dm, da, dd = (to_dev_f32(f) for f in fac)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty_like(W)
    p = catq.lmst_params(mode=catq.SOFT, s=7.0)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    dX = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    dW = torch.empty(E, N, K, dtype=torch.float32, device="cuda")
    g = [torch.empty(ng, dtype=torch.float32, device="cuda") for _ in range(3)]
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K, E), dtype=torch.uint8, device="cuda")
    catq.catq_fakeq_linear_bwd(dY, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws, dX=dX,
                               dW_fake=dW, n_experts=E, row_offsets=offs)
    torch.cuda.synchronize()
    recs = [r for r in catq.trace_records() if r["tag"].startswith("gemm")]
    catq.catq_trace_disable()
    # forward, dX and G of the routed experts: each is 2 M N K flops in total
    # over the experts (the rows, or the contraction, split among them)
    assert len(recs) == 3
    for r in recs:
        assert r["flops"] == 2.0 * M * N * K, r
    Xo, Wo, dYo = f64(xb), f64(wb), f64(dyb)
    wfo = lmst.modulate_ternarize(Wo.reshape(E * N, K), 128, *fac, lmst.SOFT,
                                  s=7.0)["W_fake"].reshape(E, N, K)
    Yref = np.zeros((M, N))
    dXref = np.zeros((M, K))
    Gref = np.zeros((E, N, K))
    for e in range(E):
        r0, r1 = off[e], off[e + 1]
        Yref[r0:r1] = Xo[r0:r1] @ Wo[e].T
        dXref[r0:r1] = dYo[r0:r1] @ wfo[e]
        Gref[e] = dYo[r0:r1].T @ Xo[r0:r1]
    assert max_norm_err(host(Y), Yref) <= 4e-3
    assert max_norm_err(host(dX), dXref) <= 2e-2
    assert max_norm_err(host(dW), Gref) <= 1e-4
    for e in np.flatnonzero(counts == 0):       # an empty expert
        assert np.all(host(dW)[e] == 0)
    ref = lmst.factor_grads(Gref.reshape(E * N, K), Wo.reshape(E * N, K), 128, *fac, lmst.SOFT,
                            s=7.0)
    for a, b in zip(g, ref):
        assert max_norm_err(host(a), b) <= 2e-2


@pytest.mark.parametrize("mode,s_bwd,strides", [
    (lmst.SOFT, 30.0, (1, 1, 1)), (lmst.HARD, 30.0, (1, 1, 1)), (lmst.HARD, 0.0, (1, 1, 1)),
    (lmst.SOFT, 30.0, (1, 1, 0))])
def test_grouped_factor_epilogue(catq, mode, s_bwd, strides):
    """Routed experts whose weight gradients are reduced to factor gradients
    in the GEMM epilogue (no dW_fake requested, 128-weight groups, extents
    that are multiples of 256): against the oracle, and against the separate
    factor-gradient kernel on the materialised G (requested through
    dW_fake), which sums the same terms in another order."""
    import torch
    E, N, K = 3, 512, 256
    counts = np.array([300, 0, 177])
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    M = int(off[-1])
    xb = sg.normal_bf16(8, "X", (M, K))
    wb = sg.normal_bf16(8, "W", (E, N, K), std=0.02)
    dyb = sg.normal_bf16(8, "Y", (M, N), std=1e-3)
    X, W, dY = to_dev_bf16(xb), to_dev_bf16(wb), to_dev_bf16(dyb)
    offs = torch.from_numpy(off).cuda()
    ng = E * N * K // 128
    fac = list(sg.perturbed_factors(9, ng))
    if strides[2] == 0:
        fac[2] = fac[2][:1]
    dm, da, dd = (to_dev_f32(f) for f in fac)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty_like(W)
    p = catq.lmst_params(mode=mode, s=7.0, s_bwd=s_bwd, strides=strides)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K, E), dtype=torch.uint8, device="cuda")

    def run(with_dw):
        g = [torch.full((ng if st else 1,), float("nan"), dtype=torch.float32, device="cuda")
             for st in strides]
        dW = torch.empty(E, N, K, dtype=torch.float32, device="cuda") if with_dw else None
        catq.catq_fakeq_linear_bwd(dY, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws,
                                   dW_fake=dW, n_experts=E, row_offsets=offs)
        return g

    torch.cuda.synchronize()
    catq.catq_trace_enable(64)
    fused = run(False)
    torch.cuda.synchronize()
    tags = [r["tag"] for r in catq.trace_records()]
    catq.catq_trace_disable()
    assert any("factor_grads" in t for t in tags) and not any(t.startswith("lmst_bwd") for t in tags)
    sep = run(True)
    torch.cuda.synchronize()
    Xo, Wo, dYo = f64(xb), f64(wb), f64(dyb)
    Gref = np.zeros((E, N, K))
    for e in range(E):
        Gref[e] = dYo[off[e]:off[e + 1]].T @ Xo[off[e]:off[e + 1]]
    ref = lmst.factor_grads(Gref.reshape(E * N, K), Wo.reshape(E * N, K), 128, *fac, mode, s=7.0,
                            s_bwd=s_bwd, strides=strides)
    for a, b, r in zip(fused, sep, ref):
        assert torch.isfinite(a).all()
        assert max_norm_err(host(a), r) <= 2e-2
        assert max_norm_err(host(a), host(b)) <= 1e-4



@pytest.mark.parametrize("M,N,K,fused", [(1984, 512, 768, True),     # unsplit: epilogue
                                         (1000, 512, 768, False),    # tokens % 64: two passes
                                         (8192, 256, 256, False)])   # split: two passes
@pytest.mark.parametrize("mode,s_bwd,strides", [
    (lmst.SOFT, 30.0, (1, 1, 1)), (lmst.HARD, 30.0, (1, 1, 1)), (lmst.HARD, 0.0, (1, 1, 1)),
    (lmst.SOFT, 30.0, (0, 1, 0)), (lmst.IDENTITY, 0.0, (1, 1, 1))])
def test_dense_factor_epilogue(catq, M, N, K, fused, mode, s_bwd, strides):
    """A dense weight gradient whose token contraction is not split has its
    factor gradients reduced in the GEMM epilogue (bf16, 128-weight groups,
    no dW_fake requested); other shapes take the two-pass path.  Both against
    the oracle and against the separate factor-gradient kernel on the
    materialised G (requested through dW_fake)."""
    _dense_factor_case(catq, M, N, K, fused, mode, s_bwd, strides)


@pytest.mark.parametrize("mode,s_bwd,strides", [
    (lmst.SOFT, 30.0, (1, 1, 1)), (lmst.HARD, 30.0, (1, 1, 1)), (lmst.SOFT, 30.0, (0, 1, 0))])
def test_dense_factor_epilogue_partial_round(catq, mode, s_bwd, strides):
    """A 2048 x 10240 gradient is 320 tiles of 256 x 256, a quarter of a
    second round: its last 2048 columns run as a 128 x 128 factor-epilogue
    launch of their own (weights, group arrays and outputs from that column
    on), the rest on 256 x 256 tiles.  Oracle parity as above, shared factors
    included."""
    tags = _dense_factor_case(catq, 256, 2048, 10240, True, mode, s_bwd, strides)
    assert any(t.startswith("gemm_dma_kernel<128, 128") and "factor_grads" in t for t in tags), tags
    assert any(t.startswith("gemm_dma_kernel<256, 256") and "factor_grads" in t for t in tags), tags


def _dense_factor_case(catq, M, N, K, fused, mode, s_bwd, strides):
    import torch
    xb = sg.normal_bf16(11, "X", (M, K))
    wb = sg.normal_bf16(11, "W", (N, K), std=0.02)
    dyb = sg.normal_bf16(11, "Y", (M, N), std=1e-3)
    X, W, dY = to_dev_bf16(xb), to_dev_bf16(wb), to_dev_bf16(dyb)
    ng = N * K // 128
    fac = list(sg.perturbed_factors(12, ng))
    for i, st in enumerate(strides):
        if st == 0:
            fac[i] = fac[i][:1]
    dm, da, dd = (to_dev_f32(f) for f in fac)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty_like(W)
    p = catq.lmst_params(mode=mode, s=7.0, s_bwd=s_bwd, strides=strides)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K, 1), dtype=torch.uint8, device="cuda")

    def run(with_dw):
        g = [torch.full((ng if st else 1,), float("nan"), dtype=torch.float32, device="cuda")
             for st in strides]
        dW = torch.empty(N, K, dtype=torch.float32, device="cuda") if with_dw else None
        catq.catq_fakeq_linear_bwd(dY, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws,
                                   dW_fake=dW)
        return g, dW

    torch.cuda.synchronize()
    catq.catq_trace_enable(64)
    first, _ = run(False)
    torch.cuda.synchronize()
    tags = [r["tag"] for r in catq.trace_records()]
    catq.catq_trace_disable()
    assert any("factor_grads" in t for t in tags) == fused, tags
    assert any(t.startswith("lmst_bwd") for t in tags) != fused, tags
    sep, dW = run(True)
    torch.cuda.synchronize()
    Gref = f64(dyb).T @ f64(xb)
    assert max_norm_err(host(dW), Gref) <= 1e-5
    ref = lmst.factor_grads(Gref, f64(wb), 128, *fac, mode, s=7.0, s_bwd=s_bwd, strides=strides)
    for a, b, r in zip(first, sep, ref):
        assert torch.isfinite(a).all()
        assert max_norm_err(host(a), r) <= 2e-2
        assert max_norm_err(host(a), host(b)) <= 1e-4
    return tags


def test_fp32_linear(catq):
    import torch
    W, X = sg.single_linear_case(0)
    M, K = X.shape
    N = W.shape[0]
    Wd, Xd = to_dev_f32(W), to_dev_f32(X)
    Y = torch.empty(M, N, dtype=torch.float32, device="cuda")
    catq.catq_fakeq_linear_fwd(Xd, Wd, Y, M, N, K)
    torch.cuda.synchronize()
    ref = X.astype(np.float64) @ W.astype(np.float64).T
    assert max_norm_err(host(Y), ref) <= 1e-5


def test_full_size_qkv_gemm_sampled(catq):
    """Fused q|k|v projection of the 1.7B-shaped block (M=8192, N=4096,
    K=2048): 4096 sampled outputs against float64 dot products."""
    import torch
    M, N, K = 8192, 4096, 2048
    xb, wb = _xw(7, M, N, K)
    X, W = to_dev_bf16(xb), to_dev_bf16(wb)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K)
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    mi = rng.integers(0, M, 4096)
    ni = rng.integers(0, N, 4096)
    Xo, Wo = f64(xb), f64(wb)
    ref = np.einsum("ij,ij->i", Xo[mi], Wo[ni])
    got = host(Y)[mi, ni]
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-3 * np.abs(ref).max())


def test_streamed_weight_fwd_sampled(catq):
    """Forward product whose weight exceeds 128 MB (the down projection of
    the 14B-shaped block, ragged in both output extents: 2011 x 5080 over
    17408 inputs), fp32 output with an fp32 residual: sampled outputs, the
    last row and column included, against float64 dot products."""
    import torch
    M, N, K = 2011, 5080, 17408
    xb, wb = _xw(11, M, N, K)
    r = sg.bf16_bits_to_f32(sg.normal_bf16(12, "Y", (M, N)))
    X, W, R = to_dev_bf16(xb), to_dev_bf16(wb), to_dev_f32(r)
    Y = torch.empty(M, N, dtype=torch.float32, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K, residual=R)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    mi = np.concatenate([rng.integers(0, M, 4096), [M - 1] * 64, np.arange(64)])
    ni = np.concatenate([rng.integers(0, N, 4096), np.arange(64), [N - 1] * 64])
    Xo, Wo = f64(xb[mi]), f64(wb[ni])
    ref = np.einsum("ij,ij->i", Xo, Wo) + r[mi, ni]
    mag = np.einsum("ij,ij->i", np.abs(Xo), np.abs(Wo))
    got = host(Y)[mi, ni]
    # fp32 accumulation of exact bf16 products over 17408 terms
    assert np.all(np.abs(got - ref) <= 2.0 ** -14 * mag + 2.0 ** -20 * np.abs(ref))


@pytest.mark.parametrize("M,N,out_f32", [(8192, 5120, False), (8192, 5120, True),
                                         (8092, 5080, True)])   # ragged rows and tail
def test_partial_last_round_split(catq, M, N, out_f32):
    """8192 x 5120 outputs are 640 tiles of 256 x 256, 2.5 rounds of the 256
    compute units: the columns past the second round run as a 128 x 128
    launch of their own (for 8092 x 5080, with ragged rows and a ragged last
    tile column).  The whole output against float64 (with a residual in the
    fp32 case), and the split-off columns bit for bit against the same
    columns from an unsplit launch (the weight's rows 1024.., whole rounds)."""
    import torch
    K = 192
    xb, wb = _xw(13, M, N, K)
    X, W = to_dev_bf16(xb), to_dev_bf16(wb)
    dt = torch.float32 if out_f32 else torch.bfloat16
    rb = sg.normal_bf16(14, "Y", (M, N)) if out_f32 else None
    R = to_dev_bf16(rb) if out_f32 else None
    Y = torch.empty(M, N, dtype=dt, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K, residual=R)
    Y2 = torch.empty(M, N - 1024, dtype=dt, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W[1024:].contiguous(), Y2, M, N - 1024, K,
                               residual=R[:, 1024:].contiguous() if out_f32 else None)
    torch.cuda.synchronize()
    assert torch.equal(Y[:, 4096:], Y2[:, 3072:])
    ref = f64(xb) @ f64(wb).T
    if out_f32:
        ref += f64(rb)
    assert max_norm_err(host(Y), ref) <= (1e-5 if out_f32 else 4e-3)


def test_partial_last_round_split_dx(catq):
    """The input gradient of a 256 -> 5120 linear over 8192 tokens (8192 x
    5120 outputs, K-major weight): split as the forward above."""
    _bwd_case(catq, 8192, 256, 5120, catq.SOFT)


def test_full_size_dw_gemm_sampled(catq):
    """Weight gradient of the down projection at full size (G = dY^T X over
    8192 tokens, N=2048, K=6144) on sampled entries; exercises split-K."""
    import torch
    M, N, K = 8192, 2048, 6144
    xb = sg.normal_bf16(8, "X", (M, K))
    wb = sg.normal_bf16(8, "W", (N, K), std=0.02)
    dyb = sg.normal_bf16(8, "Y", (M, N), std=1e-3)
    ng = N * K // 128
    fac = sg.perturbed_factors(8, ng)
    W, X, dY = to_dev_bf16(wb), to_dev_bf16(xb), to_dev_bf16(dyb)
    dm, da, dd = (to_dev_f32(f) for f in fac)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(N, K, dtype=torch.bfloat16, device="cuda")
    p = catq.lmst_params(mode=catq.SOFT, s=15.0)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    dW = torch.empty(N, K, dtype=torch.float32, device="cuda")
    g = [torch.empty(ng, dtype=torch.float32, device="cuda") for _ in range(3)]
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K), dtype=torch.uint8, device="cuda")
    catq.catq_fakeq_linear_bwd(dY, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws, dW_fake=dW)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    ni = rng.integers(0, N, 2048)
    ki = rng.integers(0, K, 2048)
    dYo, Xo = f64(dyb), f64(xb)
    ref = np.einsum("mi,mi->i", dYo[:, ni], Xo[:, ki])
    got = host(dW)[ni, ki]
    assert np.all(np.abs(got - ref) <= 1e-4 * np.abs(ref).max() + 1e-5 * np.abs(ref))
    # factor gradients of 64 sampled rows from the full G of those rows
    rows = rng.choice(N, 64, replace=False)
    Grows = dYo[:, rows].T @ Xo
    Wo = f64(wb)
    gpu = [host(a).reshape(N, K // 128)[rows] for a in g]
    facr = [f.reshape(N, K // 128)[rows].reshape(-1) for f in fac]
    ref = lmst.factor_grads(Grows, Wo[rows], 128, *facr, lmst.SOFT, s=15.0)
    for a, b in zip(gpu, ref):
        assert max_norm_err(a.reshape(-1), b) <= 2e-2


def test_determinism(catq):
    import torch
    M, N, K = 2048, 512, 1024
    xb, wb = _xw(9, M, N, K)
    X, W = to_dev_bf16(xb), to_dev_bf16(wb)
    outs = []
    for _ in range(2):
        Y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        catq.catq_fakeq_linear_fwd(X, W, Y, M, N, K)
        outs.append(Y)
    torch.cuda.synchronize()
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
