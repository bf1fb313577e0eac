"""ctypes binding of libmoe_quant.so (the C ABI declared in include/moe_quant.h).

Argument marshalling only: every step of the hot path runs in the library's
gfx950 kernels.  Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe_quant.so")

OK, ERR_ARG, ERR_BITS, ERR_ALIGN, ERR_WORKSPACE, ERR_SLOT, ERR_RANGE, ERR_HIP = (
    0, -1, -2, -3, -4, -5, -6, -7)
KIND_GATE, KIND_UP, KIND_DOWN = 0, 1, 2
MAX_EXPERTS = 256
MAX_TOPK = 16
NOALLOC_SCRATCH_BYTES = 64 << 20

EXPORTS = (
    "moe_quant_pack", "moe_code_row_words", "moe_route_permute", "moe_route_workspace_bytes",
    "moe_ffn_plan",
    "moe_expert_ffn_mixed", "moe_expert_ffn_mixed_ev", "moe_expert_ffn_mixed_noalloc",
    "moe_set_channel_switch",
    "moe_requant_channels", "moe_unpermute_combine", "moe_status_str",
    "moe_expert_significance", "moe_allocate_bits",
)


class KindDesc(C.Structure):
    _fields_ = [
        ("codes", C.c_void_p), ("sz", C.c_void_p), ("code_off", C.c_void_p),
        ("sz_off", C.c_void_p), ("code_off_host", C.c_void_p),
        ("n_slots", C.c_int32), ("reserved0", C.c_int32),
        ("copy_codes", C.c_void_p), ("copy_sz", C.c_void_p), ("copy_hdr", C.c_void_p),
        ("copy_hdr_host", C.c_void_p), ("row_slot", C.c_void_p),
    ]


class LayerDesc(C.Structure):
    _fields_ = [
        ("n_experts", C.c_int32), ("n_shared", C.c_int32), ("d_model", C.c_int32),
        ("d_ff", C.c_int32), ("d_ff_shared", C.c_int32), ("group", C.c_int32),
        ("bits_host", C.c_void_p), ("bits", C.c_void_p), ("kind", KindDesc * 3),
        ("order_gu", C.c_void_p), ("order_dn", C.c_void_p), ("class_cnt", C.c_void_p),
        ("staging", C.c_void_p),
    ]


class MoEError(RuntimeError):
    pass


_lib = None


def load() -> C.CDLL:
    """Load the in-tree library; raises if it is missing (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise MoEError("libmoe_quant.so is not built (run __graft_entry__.build() or "
                       "python paper_2503_21135_amd/build.py); there is no CPU fallback")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, sz_t = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "moe_quant_pack": (C.c_int, [vp, i64, i32, i32, i32, i32, vp, i32, vp, i64, vp, i64, i64, vp, vp]),
        "moe_route_permute": (C.c_int, [vp, i32, i32, vp, vp, i32, i32, i32, vp, vp, vp, vp, vp, vp,
                                        vp, sz_t, vp]),
        "moe_route_workspace_bytes": (sz_t, [i32, i32, i32, i32]),
        "moe_code_row_words": (i64, [i32, i32]),
        "moe_ffn_plan": (C.c_int, [C.POINTER(LayerDesc), i32, i32, C.POINTER(i32), C.POINTER(sz_t)]),
        "moe_expert_ffn_mixed": (C.c_int, [C.POINTER(LayerDesc), vp, i32, i32, vp, vp, vp, vp,
                                           sz_t, vp, vp]),
        "moe_expert_ffn_mixed_ev": (C.c_int, [C.POINTER(LayerDesc), vp, i32, i32, vp, vp, vp, vp,
                                              sz_t, vp, vp, vp, i32]),
        "moe_expert_ffn_mixed_noalloc": (C.c_int, [C.POINTER(LayerDesc), vp, i32, i32, vp, vp, vp,
                                                   vp, vp]),
        "moe_set_channel_switch": (C.c_int, [C.POINTER(LayerDesc), i32, vp, i32, vp]),
        "moe_requant_channels": (C.c_int, [C.POINTER(LayerDesc), i32, vp, i64, vp, vp, vp]),
        "moe_unpermute_combine": (C.c_int, [vp, i32, i64, vp, vp, i32, i32, i32, i32, vp, vp]),
        "moe_status_str": (C.c_char_p, [C.c_int]),
        "moe_expert_significance": (C.c_int, [vp, vp, i32, i32, i32, vp, vp]),
        "moe_allocate_bits": (C.c_int, [vp, vp, i32, vp, i32, C.c_double, C.c_double, i32,
                                        C.c_double, vp, vp, vp, C.POINTER(i32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def check(status: int, what: str) -> None:
    if status != OK:
        msg = load().moe_status_str(status).decode()
        raise MoEError("%s failed: %s (%d)" % (what, msg, status))
