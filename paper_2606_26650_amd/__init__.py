"""CAT-Q calibration hot path on AMD Instinct MI355X (gfx950).

Python face of libcatq.so: the functions below carry the C ABI's names and do
argument marshalling only (torch tensors supply device memory and the current
HIP stream); every step of the path runs in the library's HIP kernels.
"""
from __future__ import annotations

import ctypes as C

from . import _lib
from ._lib import (BF16, F32, HARD, IDENTITY, SOFT, WS_LINEAR_BWD, WS_LOSS, AttnDesc, CatqError,
                   LmstParams)

__all__ = [
    "catq_modulate_ternarize", "catq_fakeq_linear_fwd", "catq_fakeq_linear_bwd",
    "catq_block_recon_loss", "catq_block_recon_loss_noalloc", "catq_pack_ternary", "catq_ternarize_pack",
    "catq_fakeq_gateup_swiglu_fwd",
    "catq_fakeq_down_swiglu_bwd", "catq_ternary_linear", "catq_workspace_size",
    "catq_aux_act_quant", "catq_aux_rmsnorm_fwd", "catq_aux_rmsnorm_bwd", "catq_aux_attention_fwd",
    "catq_aux_attention_bwd", "catq_attn_saved_bytes", "catq_attn_bwd_workspace_bytes",
    "catq_aux_swiglu_fwd", "catq_aux_swiglu_bwd", "catq_aux_moe_route",
    "catq_aux_moe_route_workspace_bytes", "catq_aux_moe_gather", "catq_aux_moe_combine",
    "catq_aux_moe_combine_bwd", "catq_aux_moe_scatter_add", "catq_aux_adamw", "catq_aux_add",
    "lmst_params", "attn_desc", "IDENTITY", "SOFT", "HARD", "F32", "BF16", "CatqError",
    "LmstParams", "AttnDesc", "lib", "catq_trace_enable", "catq_trace_pause",
    "catq_trace_reset", "catq_trace_count", "catq_trace_get", "catq_trace_disable",
    "trace_records",
]

lib = _lib.load()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _dt(t):
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def lmst_params(group_size=128, mode=SOFT, delta0=0.5, s=15.0, s_bwd=30.0, strides=(1, 1, 1)):
    p = LmstParams()
    p.group_size = group_size
    p.mode = mode
    p.delta0 = delta0
    p.s = s
    p.s_bwd = s_bwd
    for i in range(3):
        p.factor_stride[i] = strides[i]
    return p


def attn_desc(batch, seq, n_q, n_kv, head_dim, qk_norm, rope_theta, eps=1e-6, act_quant=False):
    a = AttnDesc()
    a.batch, a.seq, a.n_q, a.n_kv, a.head_dim = batch, seq, n_q, n_kv, head_dim
    a.qk_norm = int(bool(qk_norm))
    a.rope_theta = rope_theta
    a.eps = eps
    a.act_quant = int(bool(act_quant))
    return a


def catq_modulate_ternarize(W, d_mu, d_alpha, d_delta, params, stats, stats_mode, W_fake=None,
                            codes=None, alpha_out=None, stream=None):
    d_out, d_in = W.shape[-2], W.shape[-1]
    rows = W.numel() // d_in
    wf_dt = _dt(W_fake) if W_fake is not None else BF16
    st = lib.catq_modulate_ternarize(_ptr(W), _dt(W), rows, d_in, _ptr(d_mu), _ptr(d_alpha),
                                     _ptr(d_delta), C.byref(params), _ptr(stats), stats_mode,
                                     _ptr(W_fake), wf_dt, _ptr(codes), _ptr(alpha_out),
                                     _stream(stream))
    _lib.check("catq_modulate_ternarize", st)


def catq_fakeq_linear_fwd(X, W_fake, Y, M, N, K, n_experts=1, row_offsets=None, residual=None,
                          stream=None):
    r_dt = _dt(residual) if residual is not None else _dt(Y)
    st = lib.catq_fakeq_linear_fwd(_ptr(X), _ptr(W_fake), _dt(X), _ptr(Y), _dt(Y), M, N, K,
                                   n_experts, _ptr(row_offsets), _ptr(residual), r_dt,
                                   _stream(stream))
    _lib.check("catq_fakeq_linear_fwd", st)


def catq_fakeq_linear_bwd(dY, X, W_fake, M, N, K, W, stats, d_mu, d_alpha, d_delta, params,
                          g_d_mu, g_d_alpha, g_d_delta, workspace, dX=None, dW_fake=None,
                          n_experts=1, row_offsets=None, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = lib.catq_fakeq_linear_bwd(_ptr(dY), _ptr(X), _ptr(W_fake), _dt(X), M, N, K, n_experts,
                                   _ptr(row_offsets), _ptr(W), _dt(W), _ptr(stats), _ptr(d_mu),
                                   _ptr(d_alpha), _ptr(d_delta), C.byref(params), _ptr(dX),
                                   _ptr(g_d_mu), _ptr(g_d_alpha), _ptr(g_d_delta), _ptr(dW_fake),
                                   _ptr(workspace), ws_bytes, _stream(stream))
    _lib.check("catq_fakeq_linear_bwd", st)


def catq_block_recon_loss(Y_q, Y_fp, loss, dY_q, workspace, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size()
    dy_dt = _dt(dY_q) if dY_q is not None else BF16
    st = lib.catq_block_recon_loss(_ptr(Y_q), _ptr(Y_fp), _dt(Y_q), Y_q.numel(), _ptr(loss),
                                   _ptr(dY_q), dy_dt, _ptr(workspace), ws_bytes, _stream(stream))
    _lib.check("catq_block_recon_loss", st)


def catq_block_recon_loss_noalloc(Y_q, Y_fp, loss, dY_q, stream=None):
    """catq_block_recon_loss with the library's own scratch (no workspace,
    no allocation); calls that overlap on one GPU race on that scratch."""
    dy_dt = _dt(dY_q) if dY_q is not None else BF16
    st = lib.catq_block_recon_loss_noalloc(_ptr(Y_q), _ptr(Y_fp), _dt(Y_q), Y_q.numel(),
                                           _ptr(loss), _ptr(dY_q), dy_dt, _stream(stream))
    _lib.check("catq_block_recon_loss_noalloc", st)


def catq_ternarize_pack(W, d_mu, d_alpha, d_delta, params, stats, stats_mode, packed,
                        alpha_out=None, stream=None):
    d_in = W.shape[-1]
    rows = W.numel() // d_in
    st = lib.catq_ternarize_pack(_ptr(W), _dt(W), rows, d_in, _ptr(d_mu), _ptr(d_alpha),
                                 _ptr(d_delta), C.byref(params), _ptr(stats), stats_mode,
                                 _ptr(packed), _ptr(alpha_out), _stream(stream))
    _lib.check("catq_ternarize_pack", st)


def catq_pack_ternary(codes, packed, stream=None):
    d_in = codes.shape[-1]
    rows = codes.numel() // d_in
    st = lib.catq_pack_ternary(_ptr(codes), rows, d_in, _ptr(packed), _stream(stream))
    _lib.check("catq_pack_ternary", st)


def catq_ternary_linear(X, packed, alpha, Y, g=128, stream=None):
    """Y = X (alpha * T)^T from the 2-bit storage: X bf16 [M][d_in] (rows may
    be strided), packed uint8 [d_out][d_in/4], alpha fp32 [d_out][d_in/g],
    Y fp32 or bf16 [M][d_out] (rows may be strided)."""
    d_out, d_in = packed.shape[0], packed.shape[1] * 4
    M = X.shape[0]
    st = lib.catq_ternary_linear(_ptr(X), M, X.stride(0) if M else d_in, _ptr(packed),
                                 _ptr(alpha), d_out, d_in, g, _ptr(Y), _dt(Y),
                                 Y.stride(0) if M else d_out, _stream(stream))
    _lib.check("catq_ternary_linear", st)


def catq_fakeq_gateup_swiglu_fwd(X, W_fake, gu, a, M, F, K, stream=None):
    st = lib.catq_fakeq_gateup_swiglu_fwd(_ptr(X), _ptr(W_fake), M, F, K, _ptr(gu), _ptr(a),
                                          _stream(stream))
    _lib.check("catq_fakeq_gateup_swiglu_fwd", st)


def catq_fakeq_down_swiglu_bwd(dY, W_fake, gu, dgu, M, N, F, da=None, stream=None):
    st = lib.catq_fakeq_down_swiglu_bwd(_ptr(dY), _ptr(W_fake), M, N, F, _ptr(gu), _ptr(dgu),
                                        _ptr(da), _stream(stream))
    _lib.check("catq_fakeq_down_swiglu_bwd", st)


def catq_workspace_size(which, M, N, K, n_experts=1):
    return int(lib.catq_workspace_size(which, M, N, K, n_experts))


def catq_aux_act_quant(x, y, group=None, stream=None):
    """8-bit absmax fake quantization of each group of `group` consecutive
    values of every row of x (default: the whole row) into bf16 y (may be x)."""
    n = x.shape[-1]
    st = lib.catq_aux_act_quant(_ptr(x), _dt(x), x.numel() // n if n else 0, n,
                                group or n, _ptr(y), _stream(stream))
    _lib.check("catq_aux_act_quant", st)


def catq_aux_rmsnorm_fwd(x, y, rstd, eps=1e-6, stream=None):
    n = x.shape[-1]
    st = lib.catq_aux_rmsnorm_fwd(_ptr(x), _dt(x), x.numel() // n, n, eps, _ptr(y), _ptr(rstd),
                                  _stream(stream))
    _lib.check("catq_aux_rmsnorm_fwd", st)


def catq_aux_rmsnorm_bwd(x, rstd, dy, dx, dres=None, stream=None):
    n = x.shape[-1]
    st = lib.catq_aux_rmsnorm_bwd(_ptr(x), _dt(x), _ptr(rstd), _ptr(dy), _ptr(dres),
                                  x.numel() // n, n, _ptr(dx), _stream(stream))
    _lib.check("catq_aux_rmsnorm_bwd", st)


def catq_attn_saved_bytes(desc):
    return int(lib.catq_attn_saved_bytes(C.byref(desc)))


def catq_attn_bwd_workspace_bytes(desc):
    return int(lib.catq_attn_bwd_workspace_bytes(C.byref(desc)))


def catq_aux_attention_fwd(desc, qkv, o, saved, stream=None):
    st = lib.catq_aux_attention_fwd(C.byref(desc), _ptr(qkv), _ptr(o), _ptr(saved),
                                    saved.numel() * saved.element_size(), _stream(stream))
    _lib.check("catq_aux_attention_fwd", st)


def catq_aux_attention_bwd(desc, qkv, o, saved, d_o, dqkv, workspace, stream=None):
    st = lib.catq_aux_attention_bwd(C.byref(desc), _ptr(qkv), _ptr(o), _ptr(saved), _ptr(d_o),
                                    _ptr(dqkv), _ptr(workspace),
                                    workspace.numel() * workspace.element_size(), _stream(stream))
    _lib.check("catq_aux_attention_bwd", st)


def catq_aux_swiglu_fwd(gu, a, stream=None):
    F = a.shape[-1]
    st = lib.catq_aux_swiglu_fwd(_ptr(gu), a.numel() // F, F, _ptr(a), _stream(stream))
    _lib.check("catq_aux_swiglu_fwd", st)


def catq_aux_swiglu_bwd(gu, da, dgu, stream=None):
    F = da.shape[-1]
    st = lib.catq_aux_swiglu_bwd(_ptr(gu), _ptr(da), da.numel() // F, F, _ptr(dgu),
                                 _stream(stream))
    _lib.check("catq_aux_swiglu_bwd", st)


def catq_aux_moe_route_workspace_bytes(T, E, k):
    return int(lib.catq_aux_moe_route_workspace_bytes(T, E, k))


def catq_aux_moe_route(logits, k, expert_ids, weights, perm_row, row_offsets, workspace,
                       stream=None):
    T, E = logits.shape
    st = lib.catq_aux_moe_route(_ptr(logits), T, E, k, _ptr(expert_ids), _ptr(weights),
                                _ptr(perm_row), _ptr(row_offsets), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(stream))
    _lib.check("catq_aux_moe_route", st)


def catq_aux_moe_gather(x, perm_row, k, xg, stream=None):
    T, h = x.shape
    st = lib.catq_aux_moe_gather(_ptr(x), _ptr(perm_row), T, k, h, _ptr(xg), _stream(stream))
    _lib.check("catq_aux_moe_gather", st)


def catq_aux_moe_combine(yg, perm_row, weights, res, y, k, stream=None):
    T, h = y.shape
    st = lib.catq_aux_moe_combine(_ptr(yg), _ptr(perm_row), _ptr(weights), _ptr(res), T, k, h,
                                  _ptr(y), _dt(y), _stream(stream))
    _lib.check("catq_aux_moe_combine", st)


def catq_aux_moe_combine_bwd(dy, perm_row, weights, dyg, k, stream=None):
    T, h = dy.shape
    st = lib.catq_aux_moe_combine_bwd(_ptr(dy), _ptr(perm_row), _ptr(weights), T, k, h,
                                      _ptr(dyg), _stream(stream))
    _lib.check("catq_aux_moe_combine_bwd", st)


def catq_aux_moe_scatter_add(dxg, perm_row, dx, k, stream=None):
    T, h = dx.shape
    st = lib.catq_aux_moe_scatter_add(_ptr(dxg), _ptr(perm_row), T, k, h, _ptr(dx),
                                      _stream(stream))
    _lib.check("catq_aux_moe_scatter_add", st)


def catq_aux_adamw(p, grad, m, v, step, lr, beta1=0.9, beta2=0.999, eps=1e-8, lo=-1e30, hi=1e30,
                   stream=None):
    st = lib.catq_aux_adamw(_ptr(p), _ptr(grad), _ptr(m), _ptr(v), p.numel(), step, lr, beta1,
                            beta2, eps, lo, hi, _stream(stream))
    _lib.check("catq_aux_adamw", st)


def catq_aux_add(a, b, y, stream=None):
    st = lib.catq_aux_add(_ptr(a), _ptr(b), _ptr(y), _dt(a), a.numel(), _stream(stream))
    _lib.check("catq_aux_add", st)


def catq_trace_enable(capacity):
    _lib.check("catq_trace_enable", lib.catq_trace_enable(capacity))


def catq_trace_pause(paused=True):
    lib.catq_trace_pause(int(bool(paused)))


def catq_trace_reset():
    lib.catq_trace_reset()


def catq_trace_count():
    return int(lib.catq_trace_count())


def catq_trace_get(i):
    r = _lib.TraceRec()
    _lib.check("catq_trace_get", lib.catq_trace_get(i, C.byref(r)))
    return dict(tag=r.tag.decode(), flops=r.flops, bytes=r.bytes, M=r.M, N=r.N, K=r.K, ms=r.ms)


def catq_trace_disable():
    lib.catq_trace_disable()


def trace_records():
    """Every record since the last reset, with its event-measured duration."""
    return [catq_trace_get(i) for i in range(catq_trace_count())]
