"""The calibration step captured as a HIP graph (one stream, or both) and replayed:
every replay equals the eager step bit for bit, also after other eager work
has reused the same buffers in between (the captured kernels must not depend
on state that only the capture saw)."""
import pytest

import synthgen as sg
from helpers import to_dev_bf16
from oracle import lmst

pytestmark = pytest.mark.gpu


def _outputs(blk, fin):
    import torch
    return ([blk.loss.clone(), blk.dx.clone().view(torch.int16)] +
            [t.clone() for L in blk.lin.values() for t in (L.g_mu, L.g_alpha, L.g_delta)] +
            [fin["_flat"]["packed"].clone(), fin["_flat"]["alpha"].clone()])


@pytest.mark.parametrize("kind,overlap", [("dense", False), ("dense", True), ("moe", True)])
def test_graph_replays_match_eager(catq, kind, overlap):
    import torch
    from paper_2606_26650_amd.block import DenseBlock, MoEBlock, StepGraph
    if kind == "dense":
        cfg = sg.small_dense(batch=2, seq=128, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
        blk = DenseBlock(cfg, sg.block_weights(cfg, 0))
    else:
        cfg = sg.small_moe(batch=1, seq=96, hidden=256, n_q=4, n_kv=2, head_dim=64, n_experts=8,
                           top_k=2, expert_ffn=128, router_bias_std=1.0)
        blk = MoEBlock(cfg, sg.block_weights(cfg, 0), sg.router_logits(cfg, 0))
    for i, L in enumerate(blk.lin.values()):
        L.set_factors(*sg.perturbed_factors(2, L.n_groups, extra=(i,)))
    x = to_dev_bf16(sg.activations(cfg, 0))
    y_fp = blk.new_output()
    blk.target(x, y_fp)
    fin = blk.finalize_buffers()
    kw = dict(mode=lmst.SOFT, s=15.0, s_bwd=30.0, recompute_stats=True, finalize=fin,
              overlap=overlap)
    blk.step(x, y_fp, **kw)
    torch.cuda.synchronize()
    ref = _outputs(blk, fin)
    g = StepGraph(blk, x, y_fp, **kw)
    for r in range(3):
        # other eager work on the same buffers between replays
        blk.step(x, y_fp, mode=lmst.HARD, s_bwd=30.0, overlap=overlap)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _outputs(blk, fin)
        for a, b in zip(ref, got):
            assert torch.equal(a, b), r


def test_graph_replay_of_a_window(catq):
    import torch
    from paper_2606_26650_amd.block import DenseBlock, StepGraph
    from paper_2606_26650_amd.window import Window
    cfg = sg.small_dense(batch=2, seq=64, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=384)
    win = Window([DenseBlock(cfg, sg.block_weights(cfg, i)) for i in range(2)])
    x = to_dev_bf16(sg.activations(cfg, 0))
    y_fp = win.new_output()
    win.target(x, y_fp)
    kw = dict(mode=lmst.SOFT, s=7.5, s_bwd=30.0, overlap=True)
    win.step(x, y_fp, **kw)
    torch.cuda.synchronize()
    ref = [win.loss.clone(), win.dx.clone().view(torch.int16)] + \
        [L.g_delta.clone() for b in win.blocks for L in b.lin.values()]
    g = StepGraph(win, x, y_fp, **kw)
    for _ in range(3):
        win.step(x, y_fp, mode=lmst.SOFT, s=30.0, s_bwd=30.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [win.loss.clone(), win.dx.clone().view(torch.int16)] + \
            [L.g_delta.clone() for b in win.blocks for L in b.lin.values()]
        for a, b in zip(ref, got):
            assert torch.equal(a, b)
