"""The allocation-free loss entry point against the one that takes a
workspace: same kernels and reduction order, so the loss and its gradient
agree bit for bit.  Called through the C ABI twice in a row on the same GPU
(the library's scratch keeps the last call's partials), the second time on a
smaller input, then once more on the first size with a bf16 gradient."""
import ctypes as C

import numpy as np
import pytest

import synthgen as sg
from helpers import to_dev_bf16, to_dev_f32

pytestmark = pytest.mark.gpu


def _pair(catq, yq, yfp, dy_dtype):
    import torch
    n = yq.numel()
    L = catq.lib
    dt = catq.BF16 if yq.dtype == torch.bfloat16 else catq.F32
    out = []
    for noalloc in (False, True):
        loss = torch.full((1,), float("nan"), dtype=torch.float32, device="cuda")
        dy = torch.full((n,), float("nan"), dtype=dy_dtype, device="cuda")
        ddt = catq.BF16 if dy_dtype == torch.bfloat16 else catq.F32
        stream = torch.cuda.current_stream().cuda_stream
        if noalloc:
            st = L.catq_block_recon_loss_noalloc(yq.data_ptr(), yfp.data_ptr(), dt, n,
                                                 loss.data_ptr(), dy.data_ptr(), ddt, stream)
        else:
            ws = torch.empty(catq.catq_workspace_size(catq.WS_LOSS, n, 1, 1), dtype=torch.uint8,
                             device="cuda")
            st = L.catq_block_recon_loss(yq.data_ptr(), yfp.data_ptr(), dt, n, loss.data_ptr(),
                                         dy.data_ptr(), ddt, ws.data_ptr(), ws.numel(), stream)
        assert st == 0, L.catq_last_error_message().decode()
        torch.cuda.synchronize()
        out.append((loss.clone(), dy.clone()))
    return out


def test_noalloc_loss_matches_workspace_loss(catq):
    import torch
    print("[no-alloc] first call: 8192 x 2048 fp32 outputs", flush=True)
    a = to_dev_f32(sg.uniform_f32(0, "Y", (8192 * 2048,), extra=(1,)))
    b = to_dev_f32(sg.uniform_f32(0, "Y", (8192 * 2048,), extra=(2,)))
    (l1, d1), (l2, d2) = _pair(catq, a, b, torch.float32)
    assert torch.equal(l1, l2) and torch.isfinite(l1).all()
    assert torch.equal(d1.view(torch.int32), d2.view(torch.int32))
    ref = float(np.mean((a.double() - b.double()).cpu().numpy() ** 2))
    assert abs(l2.item() - ref) <= 1e-6 * ref
    print("[no-alloc] second call: 1000 bf16 outputs (fewer partials)", flush=True)
    c = to_dev_bf16(sg.normal_bf16(1, "Y", (1000,), extra=(1,)))
    d = to_dev_bf16(sg.normal_bf16(1, "Y", (1000,), extra=(2,)))
    (l1, d1), (l2, d2) = _pair(catq, c, d, torch.bfloat16)
    assert torch.equal(l1, l2) and torch.isfinite(l1).all()
    assert torch.equal(d1.view(torch.int16), d2.view(torch.int16))
    print("[no-alloc] third call: the first size again, bf16 gradient", flush=True)
    (l1, d1), (l2, d2) = _pair(catq, a, b, torch.bfloat16)
    assert torch.equal(l1, l2)
    assert torch.equal(d1.view(torch.int16), d2.view(torch.int16))
