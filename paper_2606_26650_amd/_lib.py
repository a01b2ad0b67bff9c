"""ctypes view of libcatq.so (the C ABI declared in include/catq.h).

Loading fails loudly when the library has not been built: there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libcatq.so")

IDENTITY, SOFT, HARD = 0, 1, 2
F32, BF16 = 0, 1
WS_LINEAR_BWD, WS_LOSS = 0, 1

STATUS = {0: "CATQ_OK", 1: "CATQ_ERR_NULL", 2: "CATQ_ERR_SHAPE", 3: "CATQ_ERR_DTYPE",
          4: "CATQ_ERR_VALUE", 5: "CATQ_ERR_ALIGN", 6: "CATQ_ERR_WORKSPACE", 7: "CATQ_ERR_HIP"}


class LmstParams(C.Structure):
    _fields_ = [("group_size", C.c_int32), ("mode", C.c_int32), ("delta0", C.c_float),
                ("s", C.c_float), ("s_bwd", C.c_float), ("factor_stride", C.c_int64 * 3)]


class AttnDesc(C.Structure):
    _fields_ = [("batch", C.c_int32), ("seq", C.c_int32), ("n_q", C.c_int32),
                ("n_kv", C.c_int32), ("head_dim", C.c_int32), ("qk_norm", C.c_int32),
                ("rope_theta", C.c_float), ("eps", C.c_float), ("act_quant", C.c_int32)]


class TraceRec(C.Structure):
    _fields_ = [("tag", C.c_char * 96), ("flops", C.c_double), ("bytes", C.c_double),
                ("M", C.c_int64), ("N", C.c_int64), ("K", C.c_int64), ("ms", C.c_float)]


class CatqError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: {STATUS.get(status, status)}: {msg}")
        self.status = status


P, I64, I32, F, SZ = C.c_void_p, C.c_int64, C.c_int32, C.c_float, C.c_size_t
PP = C.POINTER(LmstParams)
PA = C.POINTER(AttnDesc)

SIGNATURES = {
    "catq_modulate_ternarize": [P, I32, I64, I64, P, P, P, PP, P, I32, P, I32, P, P, P],
    "catq_fakeq_linear_fwd": [P, P, I32, P, I32, I64, I64, I64, I32, P, P, I32, P],
    "catq_fakeq_linear_bwd": [P, P, P, I32, I64, I64, I64, I32, P, P, I32, P, P, P, P, PP, P, P,
                              P, P, P, P, SZ, P],
    "catq_block_recon_loss": [P, P, I32, I64, P, P, I32, P, SZ, P],
    "catq_block_recon_loss_noalloc": [P, P, I32, I64, P, P, I32, P],
    "catq_pack_ternary": [P, I64, I64, P, P],
    "catq_ternarize_pack": [P, I32, I64, I64, P, P, P, PP, P, I32, P, P, P],
    "catq_fakeq_gateup_swiglu_fwd": [P, P, I64, I64, I64, P, P, P],
    "catq_fakeq_down_swiglu_bwd": [P, P, I64, I64, I64, P, P, P, P],
    "catq_ternary_linear": [P, I64, I64, P, P, I64, I64, I32, P, I32, I64, P],
    "catq_workspace_size": [I32, I64, I64, I64, I32],
    "catq_status_string": [I32],
    "catq_last_error_message": [],
    "catq_aux_act_quant": [P, I32, I64, I64, I64, P, P],
    "catq_aux_rmsnorm_fwd": [P, I32, I64, I64, F, P, P, P],
    "catq_aux_rmsnorm_bwd": [P, I32, P, P, P, I64, I64, P, P],
    "catq_attn_saved_bytes": [PA],
    "catq_attn_bwd_workspace_bytes": [PA],
    "catq_aux_attention_fwd": [PA, P, P, P, SZ, P],
    "catq_aux_attention_bwd": [PA, P, P, P, P, P, P, SZ, P],
    "catq_aux_swiglu_fwd": [P, I64, I64, P, P],
    "catq_aux_swiglu_bwd": [P, P, I64, I64, P, P],
    "catq_aux_moe_route": [P, I64, I32, I32, P, P, P, P, P, SZ, P],
    "catq_aux_moe_route_workspace_bytes": [I64, I32, I32],
    "catq_aux_moe_gather": [P, P, I64, I32, I64, P, P],
    "catq_aux_moe_combine": [P, P, P, P, I64, I32, I64, P, I32, P],
    "catq_aux_moe_combine_bwd": [P, P, P, I64, I32, I64, P, P],
    "catq_aux_moe_scatter_add": [P, P, I64, I32, I64, P, P],
    "catq_aux_adamw": [P, P, P, P, I64, I64, F, C.c_double, C.c_double, C.c_double, F, F, P],
    "catq_aux_add": [P, P, P, I32, I64, P],
    "catq_trace_enable": [I32],
    "catq_trace_pause": [I32],
    "catq_trace_reset": [],
    "catq_trace_count": [],
    "catq_trace_get": [I32, C.POINTER(TraceRec)],
    "catq_trace_disable": [],
}
RESTYPES = {"catq_workspace_size": SZ, "catq_status_string": C.c_char_p,
            "catq_last_error_message": C.c_char_p, "catq_attn_saved_bytes": SZ,
            "catq_attn_bwd_workspace_bytes": SZ, "catq_aux_moe_route_workspace_bytes": SZ,
            "catq_trace_pause": None, "catq_trace_reset": None, "catq_trace_disable": None}

_lib = None


def load(path: str = LIB_PATH):
    """Open libcatq.so and attach the signatures; raises if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with paper_2606_26650_amd/build.py "
                          "(hipcc, gfx950); there is no fallback path")
    lib = C.CDLL(path)
    for name, args in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = RESTYPES.get(name, C.c_int)
    _lib = lib
    return lib


def check(fn_name: str, status: int):
    if status != 0:
        msg = _lib.catq_last_error_message().decode()
        raise CatqError(fn_name, status, msg)
