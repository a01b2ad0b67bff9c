"""C ABI checks that need no GPU: the library loads, exports every function
that include/catq.h declares, and rejects bad arguments before launching
anything.  Every call below fails validation, so no kernel is ever enqueued
(the fake device addresses are never dereferenced)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "catq.h")
LIB = os.path.join(ROOT, "paper_2606_26650_amd", "libcatq.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libcatq.so not built")

FAKE = 0x100000  # 16-byte aligned, never dereferenced (validation fails first)


def declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(catq_[a-z0-9_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def cq():
    import paper_2606_26650_amd as pkg
    return pkg


def test_every_declared_symbol_is_exported(cq):
    names = declared()
    assert len(names) >= 24
    lib = C.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), n
    # and the binding re-exports the same names
    for n in names:
        if n in ("catq_status_string", "catq_last_error_message"):
            continue
        assert hasattr(cq, n), n


def test_status_strings(cq):
    for code, name in cq._lib.STATUS.items():
        assert cq.lib.catq_status_string(code).decode() == name


def _mt(cq, p, W=FAKE, dmu=FAKE, dal=FAKE, dde=FAKE, stats=FAKE, stats_mode=0, wf=FAKE,
        codes=None, d_out=4, d_in=128, w_dt=1, wf_dt=1):
    return cq.lib.catq_modulate_ternarize(W, w_dt, d_out, d_in, dmu, dal, dde,
                                          C.byref(p) if p is not None else None, stats,
                                          stats_mode, wf, wf_dt, codes, None, None)


def test_modulate_validation(cq):
    ok = cq.lmst_params(mode=cq.SOFT, s=10.0)
    assert _mt(cq, ok, W=None) == 1
    assert _mt(cq, ok, stats=None) == 1
    assert _mt(cq, None) == 1
    assert _mt(cq, ok, d_out=0) == 2
    assert _mt(cq, ok, d_in=96) == 2                       # not a multiple of g
    assert _mt(cq, cq.lmst_params(group_size=96)) == 4     # not 8 * power of two
    assert _mt(cq, cq.lmst_params(group_size=1024)) == 4
    assert _mt(cq, cq.lmst_params(mode=cq.SOFT, s=0.0)) == 4
    assert _mt(cq, cq.lmst_params(mode=cq.SOFT, s=float("nan"))) == 4
    assert _mt(cq, cq.lmst_params(mode=cq.SOFT, s=float("inf"))) == 4
    assert _mt(cq, cq.lmst_params(delta0=0.0)) == 4
    assert _mt(cq, cq.lmst_params(s_bwd=-1.0)) == 4
    assert _mt(cq, cq.lmst_params(mode=7)) == 4
    assert _mt(cq, cq.lmst_params(strides=(2, 1, 1))) == 4
    assert _mt(cq, ok, w_dt=5) == 3
    assert _mt(cq, ok, stats_mode=2) == 4
    assert _mt(cq, ok, wf=None) == 1                        # SOFT needs W_fake
    assert _mt(cq, ok, codes=FAKE) == 4                     # codes only in HARD
    assert _mt(cq, ok, W=FAKE + 8) == 5
    msg = cq.lib.catq_last_error_message().decode()
    assert "aligned" in msg


def test_ternarize_pack_validation(cq):
    """The fused hard ternarisation + packing rejects everything before any
    launch: NULL pointers, a mode other than HARD, shapes, dtypes, alignment."""
    L = cq.lib
    hard = cq.lmst_params(mode=cq.HARD)

    def tp(p, W=FAKE, w_dt=1, d_out=4, d_in=256, stats=FAKE, mode_st=1, packed=FAKE):
        return L.catq_ternarize_pack(W, w_dt, d_out, d_in, FAKE, FAKE, FAKE,
                                     None if p is None else C.byref(p), stats, mode_st, packed,
                                     None, None)

    assert tp(hard, W=None) == 1
    assert tp(hard, packed=None) == 1
    assert tp(hard, stats=None) == 1
    assert tp(None) == 1
    assert tp(cq.lmst_params(mode=cq.SOFT, s=10.0)) == 4
    assert tp(cq.lmst_params(mode=cq.IDENTITY)) == 4
    assert tp(hard, d_out=0) == 2
    assert tp(hard, d_in=96) == 2
    assert tp(hard, w_dt=5) == 3
    assert tp(hard, mode_st=2) == 4
    assert tp(hard, packed=FAKE + 2) == 5
    assert "aligned" in L.catq_last_error_message().decode()


def test_linear_and_loss_validation(cq):
    L = cq.lib
    fwd = L.catq_fakeq_linear_fwd
    assert fwd(FAKE, FAKE, 1, FAKE, 1, 0, 8, 8, 1, None, None, 1, None) == 2
    assert fwd(FAKE, FAKE, 1, FAKE, 1, 8, 8, 12, 1, None, None, 1, None) == 2
    assert fwd(None, FAKE, 1, FAKE, 1, 8, 8, 8, 1, None, None, 1, None) == 1
    assert fwd(FAKE, FAKE, 1, FAKE, 1, 8, 8, 8, 4, None, None, 1, None) == 1
    assert fwd(FAKE, FAKE, 9, FAKE, 1, 8, 8, 8, 1, None, None, 1, None) == 3
    assert fwd(FAKE, FAKE, 0, FAKE, 0, 8, 8, 8, 4, FAKE, None, 0, None) == 3
    assert fwd(FAKE, FAKE, 1, FAKE, 1, 8, 8, 8, 4, FAKE, FAKE, 1, None) == 4
    assert fwd(FAKE, FAKE, 0, FAKE, 1, 8, 8, 8, 1, None, None, 0, None) == 3   # f32 in, bf16 out
    assert fwd(FAKE, FAKE, 1, FAKE, 1, 8, 8, 8, 1, None, FAKE, 0, None) == 3   # bf16 out, f32 res
    assert fwd(FAKE + 2, FAKE, 1, FAKE, 1, 8, 8, 8, 1, None, None, 1, None) == 5
    p = cq.lmst_params()
    args = [FAKE, FAKE, FAKE, 1, 64, 256, 128, 1, None, FAKE, 1, FAKE, FAKE, FAKE, FAKE,
            C.byref(p), FAKE, FAKE, FAKE, FAKE, None, FAKE, 16, None]
    assert L.catq_fakeq_linear_bwd(*args) == 6                 # workspace too small
    a2 = list(args)
    a2[12] = None
    assert L.catq_fakeq_linear_bwd(*a2) == 1                   # missing factor
    a3 = list(args)
    a3[5] = 252
    assert L.catq_fakeq_linear_bwd(*a3) == 2                   # N % 8
    a4 = list(args)
    a4[17] = None
    assert L.catq_fakeq_linear_bwd(*a4) == 1                   # one factor gradient missing
    a5 = list(args)
    a5[16:20] = [None, None, None, None]
    assert L.catq_fakeq_linear_bwd(*a5) == 1                   # neither dX nor gradients
    a6 = list(args)
    a6[17:20] = [None, None, None]
    a6[16] = FAKE + 2
    assert L.catq_fakeq_linear_bwd(*a6) == 5                   # dX-only path: alignment
    need = L.catq_workspace_size(0, 64, 256, 128, 1)
    assert need >= 256 * 128 * 4
    assert L.catq_block_recon_loss(FAKE, FAKE, 1, 12, FAKE, None, 1, FAKE, 1 << 20, None) == 2
    assert L.catq_block_recon_loss(FAKE, FAKE, 1, 16, FAKE, None, 1, FAKE, 8, None) == 6
    assert L.catq_block_recon_loss(FAKE, None, 1, 16, FAKE, None, 1, FAKE, 1 << 20, None) == 1
    assert L.catq_block_recon_loss(FAKE, FAKE, 0, 16, FAKE, FAKE, 4, FAKE, 1 << 20, None) == 3
    nl = L.catq_block_recon_loss_noalloc                       # rejected before any HIP call
    assert nl(FAKE, FAKE, 1, 12, FAKE, None, 1, None) == 2
    assert nl(FAKE, None, 1, 16, FAKE, None, 1, None) == 1
    assert nl(FAKE, FAKE, 0, 16, FAKE, FAKE, 4, None) == 3
    assert nl(FAKE, FAKE, 7, 16, FAKE, FAKE, 1, None) == 3
    assert nl(FAKE + 2, FAKE, 1, 16, FAKE, None, 1, None) == 5
    assert L.catq_pack_ternary(FAKE, 4, 6, FAKE, None) == 2
    assert L.catq_pack_ternary(None, 4, 8, FAKE, None) == 1


def test_aux_validation(cq):
    L = cq.lib
    assert L.catq_aux_rmsnorm_fwd(FAKE, 1, 4, 12, 1e-6, FAKE, None, None) == 2
    assert L.catq_aux_rmsnorm_fwd(FAKE, 3, 4, 16, 1e-6, FAKE, None, None) == 3
    assert L.catq_aux_swiglu_fwd(FAKE, 4, 12, FAKE, None) == 2
    assert L.catq_fakeq_gateup_swiglu_fwd(FAKE, FAKE, 4, 12, 64, FAKE, FAKE, None) == 2
    assert L.catq_fakeq_gateup_swiglu_fwd(FAKE, None, 4, 16, 64, FAKE, FAKE, None) == 1
    assert L.catq_fakeq_gateup_swiglu_fwd(FAKE, FAKE, 4, 16, 64, FAKE, FAKE + 2, None) == 5
    assert L.catq_fakeq_down_swiglu_bwd(FAKE, FAKE, 4, 64, 12, FAKE, FAKE, FAKE, None) == 2
    assert L.catq_fakeq_down_swiglu_bwd(FAKE, FAKE, 4, 64, 16, None, FAKE, FAKE, None) == 1
    d = cq.attn_desc(1, 16, 3, 2, 64, True, 1e6)          # n_q not a multiple of n_kv
    assert L.catq_aux_attention_fwd(C.byref(d), FAKE, FAKE, FAKE, 1 << 30, None) == 2
    d = cq.attn_desc(1, 16, 2, 1, 96, True, 1e6)          # head_dim
    assert L.catq_aux_attention_fwd(C.byref(d), FAKE, FAKE, FAKE, 1 << 30, None) == 2
    d = cq.attn_desc(1, 16, 2, 1, 64, True, 1e6)
    assert L.catq_aux_attention_fwd(C.byref(d), FAKE, FAKE, FAKE, 16, None) == 6
    assert L.catq_attn_saved_bytes(C.byref(d)) > 16 * 16 * 2 * 2
    assert L.catq_aux_moe_route(FAKE, 8, 4, 5, FAKE, FAKE, FAKE, FAKE, FAKE, 4096, None) == 2
    assert L.catq_aux_adamw(FAKE, FAKE, FAKE, FAKE, 4, 0, 1e-3, 0.9, 0.999, 1e-8, -1, 1,
                            None) == 2
    assert L.catq_aux_adamw(FAKE, FAKE, FAKE, FAKE, 4, 1, 1e-3, 1.5, 0.999, 1e-8, -1, 1,
                            None) == 4


def test_workspace_sizes_monotone(cq):
    a = cq.catq_workspace_size(0, 8192, 4096, 2048)
    b = cq.catq_workspace_size(0, 8192, 4096, 4096)
    assert 0 < a < b
    assert cq.catq_workspace_size(1, 1 << 20, 1, 1) > 0
    assert cq.catq_workspace_size(0, 0, 4, 4) == 0


def test_ternary_linear_validation(cq):
    """Packed-ternary linear: shape, group size, dtype and alignment checks
    fail before any launch; M = 0 is a no-op that touches nothing."""
    L = cq.lib
    # (X, M, ldx, packed, alpha, d_out, d_in, g, Y, y_dtype, ldy, stream)
    ok = dict(X=FAKE, M=4, ldx=256, P=FAKE, A=FAKE, d_out=32, d_in=256, g=128, Y=FAKE, dt=0,
              ldy=32)

    def call(**kw):
        a = dict(ok, **kw)
        return L.catq_ternary_linear(a["X"], a["M"], a["ldx"], a["P"], a["A"], a["d_out"],
                                     a["d_in"], a["g"], a["Y"], a["dt"], a["ldy"], None)

    assert call(M=0, X=None, P=None) == 0          # no-op
    assert call(M=-1) == 2
    assert call(X=None) == 1 and call(P=None) == 1 and call(A=None) == 1 and call(Y=None) == 1
    assert call(d_in=192) == 2                      # not a multiple of g
    assert call(g=64) == 4 and call(g=0) == 4       # g must be 128 * 2^j
    assert call(g=384, d_in=768, ldx=768) == 4
    assert call(g=256, d_in=384) == 2
    assert call(d_in=128 * 513, ldx=128 * 513) == 2  # longer than the staged scales
    assert call(ldx=200) == 2 and call(ldx=260) == 2
    assert call(ldy=16) == 2
    assert call(dt=3) == 3
    assert call(X=FAKE + 8) == 5 and call(A=FAKE + 4) == 5 and call(P=FAKE + 4) == 5
    assert call(Y=FAKE + 2) == 5
    assert call(d_out=0) == 2


def test_act_quant_validation(cq):
    L = cq.lib
    # (x, dtype, rows, n, group, y, stream)
    assert L.catq_aux_act_quant(None, 1, 0, 64, 64, None, None) == 0      # rows = 0: no-op
    assert L.catq_aux_act_quant(FAKE, 1, 4, 64, 24, FAKE, None) == 2      # group does not divide n
    assert L.catq_aux_act_quant(FAKE, 1, 4, 60, 60, FAKE, None) == 2      # group % 8
    assert L.catq_aux_act_quant(FAKE, 3, 4, 64, 64, FAKE, None) == 3
    assert L.catq_aux_act_quant(FAKE + 8, 1, 4, 64, 64, FAKE, None) == 5
    assert L.catq_aux_act_quant(FAKE, 0, 4, 64, 64, FAKE, None) == 4      # fp32 in place
    assert L.catq_aux_act_quant(None, 1, 4, 64, 64, FAKE, None) == 1
    d = cq.attn_desc(1, 16, 2, 1, 256, True, 1e6, act_quant=True)       # needs fused attention
    assert L.catq_aux_attention_fwd(C.byref(d), FAKE, FAKE, FAKE, 1 << 30, None) == 4
    d = cq.attn_desc(1, 16, 2, 1, 64, True, 1e6)
    d.act_quant = 2
    assert L.catq_aux_attention_fwd(C.byref(d), FAKE, FAKE, FAKE, 1 << 30, None) == 4
