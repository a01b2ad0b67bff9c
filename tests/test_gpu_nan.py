"""NaN in the data is not an error and propagates (the C ABI's contract): one
NaN weight, or one NaN factor, in group j of row r of a bf16 linear.

* LM+ST: the fake weights of group j are NaN and every other group's are
  exactly the clean run's;
* forward: output column r is NaN for every token, every other column equals
  the clean run's bit for bit (the GEMM reads the NaN group only for r);
* loss: NaN;
* backward: the factor gradients of row r's groups are NaN, every other
  row's are finite (G = dY^T X mixes only column r of dY into row r);
* the final hard ternarisation: codes stay in {-1, 0, +1} everywhere (a
  comparison with NaN is false, so the group's codes are 0), the other
  groups' codes, packed bytes and scales equal the clean run's.
"""
import numpy as np
import pytest

import synthgen as sg
from helpers import to_dev_bf16

pytestmark = pytest.mark.gpu

M, N, K, G = 128, 64, 256, 128
ROW, GCOL = 37, 1                 # the poisoned group: row 37, columns 128..255
GROUP = ROW * (K // G) + GCOL


def _run(catq, Wb, fac, mode=1):
    import torch
    W = to_dev_bf16(Wb)
    X = to_dev_bf16(sg.normal_bf16(0, "X", (M, K)))
    dm, da, dd = (torch.from_numpy(np.ascontiguousarray(f, np.float32)).cuda() for f in fac)
    ng = N * K // G
    stats = torch.empty(ng, 2, device="cuda")
    wf = torch.empty(N, K, dtype=torch.bfloat16, device="cuda")
    p = catq.lmst_params(mode=mode, s=15.0, s_bwd=30.0)
    catq.catq_modulate_ternarize(W, dm, da, dd, p, stats, 0, W_fake=wf)
    y_fp = torch.empty(M, N, dtype=torch.float32, device="cuda")
    y = torch.empty(M, N, dtype=torch.float32, device="cuda")
    catq.catq_fakeq_linear_fwd(X, W, y_fp, M, N, K)
    catq.catq_fakeq_linear_fwd(X, wf, y, M, N, K)
    loss = torch.zeros(1, device="cuda")
    dy = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    lws = torch.empty(catq.catq_workspace_size(1, M * N, 1, 1), dtype=torch.uint8, device="cuda")
    catq.catq_block_recon_loss(y, y_fp, loss, dy, lws)
    g = [torch.empty(ng, device="cuda") for _ in range(3)]
    ws = torch.empty(catq.catq_workspace_size(0, M, N, K), dtype=torch.uint8, device="cuda")
    dx = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
    catq.catq_fakeq_linear_bwd(dy, X, wf, M, N, K, W, stats, dm, da, dd, p, *g, ws, dX=dx)
    codes = torch.empty(N, K, dtype=torch.int8, device="cuda")
    alpha = torch.empty(ng, device="cuda")
    catq.catq_modulate_ternarize(W, dm, da, dd, catq.lmst_params(mode=catq.HARD), stats, 1,
                                 codes=codes, alpha_out=alpha)
    packed = torch.empty(N, K // 4, dtype=torch.uint8, device="cuda")
    catq.catq_pack_ternary(codes, packed)
    torch.cuda.synchronize()
    cpu = lambda t: t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()
    return dict(wf=cpu(wf), y=cpu(y), loss=loss.item(), g=[cpu(t) for t in g], dx=cpu(dx),
                codes=cpu(codes), alpha=cpu(alpha), packed=cpu(packed))


@pytest.mark.parametrize("where", ["weight", "d_mu", "d_alpha", "d_delta"])
def test_nan_propagates_and_codes_stay_defined(catq, where):
    Wb = sg.normal_bf16(0, "W", (N, K), std=0.02)
    ng = N * K // G
    fac = [np.zeros(ng), np.ones(ng), np.ones(ng)]
    clean = _run(catq, Wb, fac)
    if where == "weight":
        Wb = Wb.copy()
        Wb[ROW, GCOL * G + 5] = 0x7FC0          # bf16 quiet NaN
    else:
        fac = [f.copy() for f in fac]
        fac[["d_mu", "d_alpha", "d_delta"].index(where)][GROUP] = np.nan
    bad = _run(catq, Wb, fac)
    grp = np.zeros((N, K), bool)
    grp[ROW, GCOL * G:(GCOL + 1) * G] = True
    assert np.isnan(bad["wf"][grp]).all()
    np.testing.assert_array_equal(bad["wf"][~grp], clean["wf"][~grp])
    assert np.isnan(bad["y"][:, ROW]).all()
    others = np.arange(N) != ROW
    np.testing.assert_array_equal(bad["y"][:, others], clean["y"][:, others])
    assert np.isnan(bad["loss"])
    row_groups = np.zeros(ng, bool)
    row_groups[ROW * (K // G):(ROW + 1) * (K // G)] = True
    for a in bad["g"]:
        assert np.isnan(a[row_groups]).all()
        assert np.isfinite(a[~row_groups]).all()
    assert np.isnan(bad["dx"]).all()            # dX = dY . W_fake mixes column ROW everywhere
    assert set(np.unique(bad["codes"]).tolist()) <= {-1, 0, 1}
    assert (bad["codes"][grp] == 0).all()
    np.testing.assert_array_equal(bad["codes"][~grp], clean["codes"][~grp])
    keep = np.ones(ng, bool)
    keep[GROUP] = False
    np.testing.assert_array_equal(bad["alpha"][keep], clean["alpha"][keep])
    rows = np.arange(N) != ROW
    np.testing.assert_array_equal(bad["packed"][rows], clean["packed"][rows])
    print(f"[nan] {where}: loss {bad['loss']}, group codes all 0", flush=True)
