"""GPU parity of the LM+ST entry points against the oracle (bit-exact stats,
codes and packed bytes; fp32 fake weights within 1e-5 relative)."""
import numpy as np
import pytest

import synthgen as sg
from helpers import elem_rel_ok, f64, host, max_norm_err, to_dev_bf16, to_dev_f32
from oracle import lmst

pytestmark = pytest.mark.gpu


def _case(seed, rows, d_in, g, wdtype="bf16", spread=0.3, shared=(1, 1, 1)):
    if wdtype == "bf16":
        bits = sg.normal_bf16(seed, "W", (rows, d_in), std=0.02)
        Wo = f64(bits)
        Wd = to_dev_bf16(bits)
    else:
        Wo = sg.rng(seed, "W").standard_normal((rows, d_in)).astype(np.float32) * np.float32(0.02)
        Wd = to_dev_f32(Wo)
        Wo = Wo.astype(np.float64)
    ng = rows * d_in // g
    fac = sg.perturbed_factors(seed, ng, spread)
    fac = [f if st else f[:1].copy() for f, st in zip(fac, shared)]
    return Wo, Wd, fac


@pytest.mark.parametrize("g", [16, 64, 128, 256, 512])
@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_stats_bit_exact(catq, g, wdtype):
    import torch
    rows, d_in = 37, 1024            # ragged against the 2048-element blocks
    Wo, Wd, fac = _case(1, rows, d_in, g, wdtype)
    ng = rows * d_in // g
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(rows, d_in, dtype=torch.float32, device="cuda")
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.IDENTITY)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, W_fake=wf)
    torch.cuda.synchronize()
    mu0, al0 = lmst.group_stats(Wo, g)
    st = stats.cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(st[:, 0], mu0)
    np.testing.assert_array_equal(st[:, 1], al0)
    np.testing.assert_array_equal(host(wf), Wo)        # identity branch: W itself


@pytest.mark.parametrize("s", [0.625, 3.75, 15.0, 30.0])
@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_soft_fp32_within_1e5(catq, s, wdtype):
    import torch
    rows, d_in, g = 53, 768, 128
    Wo, Wd, fac = _case(2, rows, d_in, g, wdtype)
    ng = rows * d_in // g
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(rows, d_in, dtype=torch.float32, device="cuda")
    alpha = torch.empty(ng, dtype=torch.float32, device="cuda")
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.SOFT, s=s)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, W_fake=wf, alpha_out=alpha)
    torch.cuda.synchronize()
    ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.SOFT, s=s)
    ok, worst = elem_rel_ok(host(wf), ref["W_fake"], 1e-5)
    assert ok, worst
    np.testing.assert_array_equal(alpha.cpu().numpy().astype(np.float64), ref["alpha"])


def test_soft_bf16_output_and_cached_stats(catq):
    import torch
    rows, d_in, g = 64, 512, 128
    Wo, Wd, fac = _case(3, rows, d_in, g)
    ng = rows * d_in // g
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(rows, d_in, dtype=torch.bfloat16, device="cuda")
    wf2 = torch.empty_like(wf)
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.SOFT, s=15.0)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, W_fake=wf)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 1, W_fake=wf2)
    torch.cuda.synchronize()
    assert torch.equal(wf.view(torch.int16), wf2.view(torch.int16))
    ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.SOFT, s=15.0)["W_fake"]
    got = host(wf)
    # one bf16 rounding of a value accurate to ~1e-6
    assert np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-30)


@pytest.mark.parametrize("g", [32, 64, 128, 256, 512])
@pytest.mark.parametrize("wdtype,odtype", [("bf16", "bf16"), ("bf16", "f32"), ("f32", "bf16"),
                                           ("f32", "f32")])
def test_soft_cached_stats_kernel(catq, g, wdtype, odtype):
    """The soft step with cached statistics (its own kernel: 32 weights per
    lane) writes the same bits as the soft branch that computes the
    statistics, for every group size it takes, a ragged row count and a
    shared threshold factor; fp32 outputs within 1e-5 of the oracle."""
    import torch
    rows, d_in = 45, 1536
    for s, shared in ((15.0, (1, 1, 1)), (0.625, (1, 1, 0)), (30.0, (0, 1, 1))):
        Wo, Wd, fac = _case(5, rows, d_in, g, wdtype, shared=shared)
        ng = rows * d_in // g
        dt = torch.bfloat16 if odtype == "bf16" else torch.float32
        stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
        wf = torch.empty(rows, d_in, dtype=dt, device="cuda")
        wf2 = torch.empty_like(wf)
        al, al2 = (torch.empty(ng, dtype=torch.float32, device="cuda") for _ in range(2))
        dm, da, dd = (to_dev_f32(f) for f in fac)
        p = catq.lmst_params(group_size=g, mode=catq.SOFT, s=s, strides=shared)
        catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, W_fake=wf, alpha_out=al)
        catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 1, W_fake=wf2, alpha_out=al2)
        torch.cuda.synchronize()
        bits = torch.int16 if odtype == "bf16" else torch.int32
        assert torch.equal(wf.view(bits), wf2.view(bits)), (g, s, shared)
        assert torch.equal(al, al2)
        if odtype == "f32":
            ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.SOFT, s=s, strides=shared)
            ok, worst = elem_rel_ok(host(wf2), ref["W_fake"], 1e-5)
            assert ok, (g, s, worst)


@pytest.mark.parametrize("shared", [(1, 1, 1), (1, 1, 0), (0, 0, 0)])
@pytest.mark.parametrize("wdtype", ["bf16", "f32"])
def test_hard_codes_bit_exact(catq, shared, wdtype):
    import torch
    rows, d_in, g = 41, 640, 128
    Wo, Wd, fac = _case(4, rows, d_in, g, wdtype, shared=shared)
    ng = rows * d_in // g
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    wf = torch.empty(rows, d_in, dtype=torch.float32, device="cuda")
    codes = torch.empty(rows, d_in, dtype=torch.int8, device="cuda")
    alpha = torch.empty(ng, dtype=torch.float32, device="cuda")
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.HARD, strides=shared)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, W_fake=wf, codes=codes,
                                 alpha_out=alpha)
    torch.cuda.synchronize()
    ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.HARD, strides=shared)
    np.testing.assert_array_equal(codes.cpu().numpy(), ref["codes"])
    np.testing.assert_array_equal(host(wf), ref["W_fake"])
    np.testing.assert_array_equal(alpha.cpu().numpy().astype(np.float64), ref["alpha"])


def test_hard_ties_and_constant_groups(catq):
    import torch
    # hand-built groups: exact ties at |W_hat| = Delta give 0; a constant group gives 0
    base = np.tile([3.0, 1.0, -1.0, -3.0], 32) * 2.0 ** -6
    W = np.stack([base, base + 0.5, np.full(128, 0.25), -base]).astype(np.float32)
    bits = sg.f32_to_bf16_bits(W)
    Wd = to_dev_bf16(bits)
    ng = 4
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    codes = torch.empty(4, 128, dtype=torch.int8, device="cuda")
    one = torch.ones(ng, dtype=torch.float32, device="cuda")
    zero = torch.zeros(ng, dtype=torch.float32, device="cuda")
    p = catq.lmst_params(group_size=128, mode=catq.HARD)
    catq.catq_modulate_ternarize(Wd, zero, one, one, p, stats, 0, codes=codes)
    torch.cuda.synchronize()
    ref = lmst.modulate_ternarize(f64(bits), 128, 0.0, 1.0, 1.0, lmst.HARD)["codes"]
    got = codes.cpu().numpy()
    np.testing.assert_array_equal(got, ref)
    np.testing.assert_array_equal(got[0, :4], [1, 0, 0, -1])
    assert np.all(got[2] == 0)


def test_full_size_qwen3_block_weights(catq):
    """All seven weights of the 1.7B-shaped block (50.3M weights): stats and
    hard codes bit-exact, soft fake weights (fp32) within 1e-5."""
    import torch
    cfg = sg.QWEN3_1P7B
    W = sg.block_weights(cfg, 0)
    for name in ("Wq", "Wd"):
        bits = W[name]
        rows, d_in = bits.shape
        ng = rows * d_in // 128
        fac = sg.perturbed_factors(5, ng)
        Wd = to_dev_bf16(bits)
        stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
        wf = torch.empty(rows, d_in, dtype=torch.float32, device="cuda")
        codes = torch.empty(rows, d_in, dtype=torch.int8, device="cuda")
        dm, da, dd = (to_dev_f32(f) for f in fac)
        catq.catq_modulate_ternarize(Wd, dm, da, dd, catq.lmst_params(mode=catq.SOFT, s=15.0),
                                     stats, 0, W_fake=wf)
        torch.cuda.synchronize()
        Wo = f64(bits)
        ref = lmst.modulate_ternarize(Wo, 128, *fac, lmst.SOFT, s=15.0)
        st = stats.cpu().numpy().astype(np.float64)
        np.testing.assert_array_equal(st[:, 0], ref["mu0"])
        np.testing.assert_array_equal(st[:, 1], ref["alpha0"])
        ok, worst = elem_rel_ok(host(wf), ref["W_fake"], 1e-5)
        assert ok, (name, worst)
        catq.catq_modulate_ternarize(Wd, dm, da, dd, catq.lmst_params(mode=catq.HARD), stats, 1,
                                     W_fake=None, codes=codes)
        torch.cuda.synchronize()
        rh = lmst.modulate_ternarize(Wo, 128, *fac, lmst.HARD)
        np.testing.assert_array_equal(codes.cpu().numpy(), rh["codes"])


def test_pack_bit_exact(catq):
    import torch
    rng = np.random.default_rng(0)
    for shape in [(1, 4), (3, 12), (37, 1000), (64, 4096)]:
        c = rng.integers(-1, 2, size=shape).astype(np.int8)
        cd = torch.from_numpy(c).cuda()
        pk = torch.empty(shape[0], shape[1] // 4, dtype=torch.uint8, device="cuda")
        catq.catq_pack_ternary(cd, pk)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(pk.cpu().numpy(), lmst.pack_ternary(c))
    one = torch.tensor([[1, 0, -1, 0]], dtype=torch.int8, device="cuda")
    pk = torch.zeros(1, 1, dtype=torch.uint8, device="cuda")
    catq.catq_pack_ternary(one, pk)
    assert int(pk.item()) == 0x46


@pytest.mark.parametrize("rows,d_in,g,wdtype,shared,stats_mode", [
    (41, 640, 128, "bf16", (1, 1, 1), 0), (41, 640, 128, "f32", (1, 1, 1), 0),
    (7, 96, 16, "bf16", (0, 1, 0), 0), (300, 1024, 512, "bf16", (1, 1, 1), 1),
    (1, 128, 128, "bf16", (1, 1, 1), 0)])
def test_ternarize_pack_bit_exact(catq, rows, d_in, g, wdtype, shared, stats_mode):
    """The fused hard ternarisation + packing: packed bytes equal the oracle's
    packing of the oracle's hard codes, scales (and computed statistics) bit
    for bit, and the same bytes as the two-launch path (codes, then pack)."""
    import torch
    Wo, Wd, fac = _case(9, rows, d_in, g, wdtype, shared=shared)
    ng = rows * d_in // g
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.HARD, strides=shared)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    if stats_mode == 1:  # statistics from an earlier soft call on the same W
        wf = torch.empty(rows, d_in, dtype=torch.bfloat16, device="cuda")
        catq.catq_modulate_ternarize(Wd, dm, da, dd, catq.lmst_params(group_size=g, mode=catq.SOFT,
                                                                      s=5.0, strides=shared),
                                     stats, 0, W_fake=wf)
    packed = torch.full((rows, d_in // 4), 0xAB, dtype=torch.uint8, device="cuda")
    alpha = torch.full((ng,), float("nan"), dtype=torch.float32, device="cuda")
    catq.catq_ternarize_pack(Wd, dm, da, dd, p, stats, stats_mode, packed, alpha_out=alpha)
    stats2 = stats.clone()
    codes = torch.empty(rows, d_in, dtype=torch.int8, device="cuda")
    packed2 = torch.empty_like(packed)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats2, 1, codes=codes)
    catq.catq_pack_ternary(codes, packed2)
    torch.cuda.synchronize()
    ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.HARD, strides=shared)
    np.testing.assert_array_equal(packed.cpu().numpy(), lmst.pack_ternary(ref["codes"]))
    assert torch.equal(packed, packed2)
    np.testing.assert_array_equal(alpha.cpu().numpy().astype(np.float64), ref["alpha"])
    st = stats.cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(st[:, 0], ref["mu0"])
    np.testing.assert_array_equal(st[:, 1], ref["alpha0"])


def test_hard_codes_near_threshold(catq):
    """Thresholds placed within a few float32 ulps of |W - mu| of one weight
    per group (so the float32 screen defers to the exact float64 decision),
    plus zero, negative, NaN and huge thresholds: codes bit-exact against the
    oracle, through both the codes path and the one-pass packing."""
    import torch
    rows, d_in, g = 64, 256, 128
    bits = sg.normal_bf16(21, "W", (rows, d_in), std=0.02)
    Wo = f64(bits)
    ng = rows * d_in // g
    rng = np.random.default_rng(21)
    d_mu = (rng.standard_normal(ng) * 0.1).astype(np.float32)
    d_alpha = (1.0 + rng.standard_normal(ng) * 0.1).astype(np.float32)
    mu0, alpha0 = lmst.group_stats(Wo, g)
    mu, alpha, _ = lmst.modulation(mu0, alpha0, d_mu, d_alpha, np.ones(ng, np.float32))
    r = np.abs(Wo.reshape(ng, g)[np.arange(ng), rng.integers(0, g, ng)] - mu)
    base = (r / lmst.safe_alpha(alpha) / 0.5).astype(np.float32)
    ulps = rng.integers(-3, 4, ng).astype(np.int32)
    d_delta = (base.view(np.int32) + ulps).view(np.float32)
    d_delta[:4] = [0.0, -0.5, np.nan, 1e30]
    fac = [d_mu, d_alpha, d_delta]
    dm, da, dd = (to_dev_f32(f) for f in fac)
    p = catq.lmst_params(group_size=g, mode=catq.HARD)
    stats = torch.zeros(ng, 2, dtype=torch.float32, device="cuda")
    codes = torch.empty(rows, d_in, dtype=torch.int8, device="cuda")
    packed = torch.empty(rows, d_in // 4, dtype=torch.uint8, device="cuda")
    Wd = to_dev_bf16(bits)
    catq.catq_modulate_ternarize(Wd, dm, da, dd, p, stats, 0, codes=codes)
    catq.catq_ternarize_pack(Wd, dm, da, dd, p, stats, 1, packed)
    torch.cuda.synchronize()
    ref = lmst.modulate_ternarize(Wo, g, *fac, lmst.HARD)["codes"]
    np.testing.assert_array_equal(codes.cpu().numpy(), ref)
    np.testing.assert_array_equal(packed.cpu().numpy(), lmst.pack_ternary(ref))
    # the placed weights decide both ways across the groups
    placed = ref.reshape(ng, g)
    assert (placed != 0).any() and (placed == 0).any()


def test_loss_parity(catq):
    import torch
    for n, dtype in [(8, "bf16"), (4096 * 3 + 8, "bf16"), (1 << 21, "bf16"), (40000, "f32")]:
        a = sg.rng(0, "Y", n).standard_normal(n)
        b = a + 0.1 * sg.rng(1, "Y", n).standard_normal(n)
        if dtype == "bf16":
            ab, bb = sg.to_bf16_bits(a), sg.to_bf16_bits(b)
            A, B = to_dev_bf16(ab), to_dev_bf16(bb)
            ao, bo = f64(ab), f64(bb)
        else:
            ao, bo = a.astype(np.float32).astype(np.float64), b.astype(np.float32).astype(np.float64)
            A, B = to_dev_f32(ao), to_dev_f32(bo)
        loss = torch.zeros(1, dtype=torch.float32, device="cuda")
        dy = torch.empty_like(A)
        ws = torch.empty(catq.catq_workspace_size(1, n, 1, 1), dtype=torch.uint8, device="cuda")
        catq.catq_block_recon_loss(A, B, loss, dy, ws)
        torch.cuda.synchronize()
        from oracle import block
        rl, rdy = block.recon_loss(ao, bo)
        assert abs(loss.item() - rl) <= 1e-5 * rl, (n, loss.item(), rl)
        tol = 2.0 ** -8 if dtype == "bf16" else 1e-6
        assert np.all(np.abs(host(dy) - rdy) <= tol * np.abs(rdy) + 1e-30)


def test_loss_identity_is_zero(catq):
    import torch
    bits = sg.normal_bf16(0, "Y", (64, 256))
    A = to_dev_bf16(bits)
    loss = torch.ones(1, dtype=torch.float32, device="cuda")
    dy = torch.ones_like(A)
    ws = torch.empty(catq.catq_workspace_size(1, A.numel(), 1, 1), dtype=torch.uint8,
                     device="cuda")
    catq.catq_block_recon_loss(A, A.clone(), loss, dy, ws)
    torch.cuda.synchronize()
    assert loss.item() == 0.0 and torch.count_nonzero(dy).item() == 0


def test_adamw_parity(catq):
    import torch
    from oracle import calib
    n = 1000
    p = sg.rng(0, "dmu").uniform(-0.5, 0.5, n).astype(np.float32)
    g = sg.rng(0, "G").standard_normal(n).astype(np.float32)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    P, Gd, Md, Vd = (to_dev_f32(a) for a in (p, g, m, v))
    pr, mr, vr = p.astype(np.float64), m.astype(np.float64), v.astype(np.float64)
    for step in (1, 2, 3):
        catq.catq_aux_adamw(P, Gd, Md, Vd, step, 1e-3, lo=-1 + 1e-4, hi=1 - 1e-4)
        pr, mr, vr = calib.adamw_step(pr, g, mr, vr, step, 1e-3, kind="mu")
    torch.cuda.synchronize()
    assert np.all(np.abs(host(P) - pr) <= 1e-5 * np.abs(pr) + 1e-7)
