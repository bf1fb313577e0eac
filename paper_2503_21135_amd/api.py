"""Python names of the C ABI (include/moe_quant.h), taking torch tensors.

torch supplies device memory and the stream only; each function marshals its
arguments into the matching ``extern "C"`` entry point of libmoe_quant.so and
raises MoEError on a non-zero status.  Integer bit patterns (packed codes,
{scale, zero} words) live in int32 tensors; bf16 activations in bfloat16
tensors.
"""
from __future__ import annotations

import ctypes as C
from typing import Optional, Tuple

import numpy as np
import torch

from ._lib import LayerDesc, MoEError, check, load


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _s(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _need_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise MoEError("expected a device tensor")


def moe_quant_pack(w: torch.Tensor, bits: int, group: int, codes: torch.Tensor,
                   sz: torch.Tensor, n: Optional[int] = None,
                   rows: Optional[torch.Tensor] = None, ld_codes: Optional[int] = None,
                   sz_row_stride: Optional[int] = None, sz_group_stride: int = 1,
                   status: Optional[torch.Tensor] = None, stream=None) -> None:
    """Quantize rows of fp32 w [R][K] at `bits` and pack them (Sec. IV-A, V-B)."""
    _need_cuda(w, codes, sz, rows, status)
    R, K = w.shape
    n = (R if rows is None else rows.numel()) if n is None else n
    ld = K * bits // 32 if ld_codes is None else ld_codes
    srs = K // group if sz_row_stride is None else sz_row_stride
    st = load().moe_quant_pack(_p(w), w.stride(0), R, K, bits, group, _p(rows), n,
                               _p(codes), ld, _p(sz), srs, sz_group_stride, _p(status),
                               _s(stream))
    check(st, "moe_quant_pack")


def moe_code_row_words(K: int, bits: int) -> int:
    """Row stride (32-bit words) of packed code matrices read by the FFN."""
    n = int(load().moe_code_row_words(K, bits))
    if n <= 0:
        raise MoEError("moe_code_row_words: bad K=%d or bits=%d" % (K, bits))
    return n


def moe_route_workspace_bytes(T: int, E: int, k: int, S: int) -> int:
    return int(load().moe_route_workspace_bytes(T, E, k, S))


def moe_route_permute(x: torch.Tensor, w_router: torch.Tensor, bias: Optional[torch.Tensor],
                      k: int, S: int, topk_ids: torch.Tensor, topk_w: torch.Tensor,
                      offsets: torch.Tensor, perm_token: torch.Tensor, inv_perm: torch.Tensor,
                      ws: torch.Tensor, x_perm: Optional[torch.Tensor] = None,
                      stream=None) -> None:
    """Router, top-k and permutation into per-expert segments (Sec. II-A)."""
    _need_cuda(x, w_router, bias, topk_ids, topk_w, offsets, perm_token, inv_perm, ws, x_perm)
    T, d = x.shape
    E = w_router.shape[0]
    st = load().moe_route_permute(_p(x), T, d, _p(w_router), _p(bias), E, k, S, _p(topk_ids),
                                  _p(topk_w), _p(offsets), _p(perm_token), _p(inv_perm),
                                  _p(x_perm), _p(ws), ws.numel() * ws.element_size(), _s(stream))
    check(st, "moe_route_permute")


def moe_ffn_plan(desc: LayerDesc, T: int, k: int) -> Tuple[int, int]:
    ns = C.c_int32(0)
    wb = C.c_size_t(0)
    check(load().moe_ffn_plan(C.byref(desc), T, k, C.byref(ns), C.byref(wb)), "moe_ffn_plan")
    return int(ns.value), int(wb.value)


def moe_expert_ffn_mixed(desc: LayerDesc, x: torch.Tensor, k: int, offsets: torch.Tensor,
                         perm_token: torch.Tensor, o: torch.Tensor, ws: torch.Tensor,
                         status: Optional[torch.Tensor] = None, stream=None) -> None:
    """Grouped mixed-precision SiLU-GLU expert FFN (Sec. IV-A, IV-B, V-B).
    `status` (device int32, optional) receives MOE_ERR_RANGE when the fp16
    operand path meets a value beyond fp16's range."""
    _need_cuda(x, offsets, perm_token, o, ws, status)
    T = x.shape[0]
    st = load().moe_expert_ffn_mixed(C.byref(desc), _p(x), T, k, _p(offsets), _p(perm_token),
                                     _p(o), _p(ws), ws.numel() * ws.element_size(), _p(status),
                                     _s(stream))
    check(st, "moe_expert_ffn_mixed")


def moe_expert_ffn_mixed_ev(desc: LayerDesc, x: torch.Tensor, k: int, offsets: torch.Tensor,
                            perm_token: torch.Tensor, o: torch.Tensor, ws: torch.Tensor,
                            events, status: Optional[torch.Tensor] = None, stream=None) -> None:
    """moe_expert_ffn_mixed recording caller-created hipEvent_t handles
    (a ctypes c_void_p array) at its stage boundaries."""
    _need_cuda(x, offsets, perm_token, o, ws, status)
    T = x.shape[0]
    st = load().moe_expert_ffn_mixed_ev(C.byref(desc), _p(x), T, k, _p(offsets), _p(perm_token),
                                        _p(o), _p(ws), ws.numel() * ws.element_size(), _p(status),
                                        _s(stream), C.cast(events, C.c_void_p), len(events))
    check(st, "moe_expert_ffn_mixed_ev")


def moe_expert_ffn_mixed_noalloc(desc: LayerDesc, x: torch.Tensor, k: int, offsets: torch.Tensor,
                                 perm_token: torch.Tensor, o: torch.Tensor,
                                 status: Optional[torch.Tensor] = None, stream=None) -> None:
    """moe_expert_ffn_mixed with the library's fixed per-GPU workspace
    (no workspace argument, no allocation)."""
    _need_cuda(x, offsets, perm_token, o, status)
    T = x.shape[0]
    st = load().moe_expert_ffn_mixed_noalloc(C.byref(desc), _p(x), T, k, _p(offsets),
                                             _p(perm_token), _p(o), _p(status), _s(stream))
    check(st, "moe_expert_ffn_mixed_noalloc")


def moe_set_channel_switch(desc: LayerDesc, kind: int, slots_on: Optional[np.ndarray],
                           stream=None) -> None:
    """Install cached copies by (expert, row) header (Sec. IV-B, V-A)."""
    if slots_on is None or len(slots_on) == 0:
        arr, ptr, n = None, None, 0
    else:
        arr = np.ascontiguousarray(slots_on, dtype=np.int32)
        ptr, n = arr.ctypes.data_as(C.c_void_p), int(arr.size)
    st = load().moe_set_channel_switch(C.byref(desc), kind, ptr, n, _s(stream))
    check(st, "moe_set_channel_switch")


def moe_requant_channels(desc: LayerDesc, kind: int, cache: torch.Tensor,
                         expert_bits: np.ndarray, status: Optional[torch.Tensor] = None,
                         stream=None) -> None:
    """Requantize the cached 16-bit channels of one kind into its copy slots at
    each expert's new precision (Sec. IV-B, requantization for new datasets).

    cache        device float16 [n_slots][K] (row s = original channel of slot s)
    expert_bits  int [n_experts], 0 = leave that expert's slots as they are
    """
    _need_cuda(cache, status)
    if cache.dtype != torch.float16 or cache.dim() != 2 or cache.stride(1) != 1:
        raise MoEError("cache must be a row-major float16 matrix")
    eb = np.ascontiguousarray(expert_bits, dtype=np.int32)
    if eb.size != desc.n_experts:
        raise MoEError("expert_bits needs one entry per routed expert")
    st = load().moe_requant_channels(C.byref(desc), kind, _p(cache), cache.stride(0),
                                     eb.ctypes.data_as(C.c_void_p), _p(status), _s(stream))
    check(st, "moe_requant_channels")


def moe_unpermute_combine(o: torch.Tensor, n_split: int, inv_perm: torch.Tensor,
                          topk_w: torch.Tensor, k: int, S: int, y: torch.Tensor,
                          stream=None) -> None:
    """y[t] = sum_j w[t][j] o[inv[t][j]] + sum_s o[inv[t][k+s]]."""
    _need_cuda(o, inv_perm, topk_w, y)
    T, d = y.shape
    split_stride = o.stride(0) if o.dim() == 3 else o.numel()
    st = load().moe_unpermute_combine(_p(o), n_split, split_stride, _p(inv_perm), _p(topk_w),
                                      T, k, S, d, _p(y), _s(stream))
    check(st, "moe_unpermute_combine")


# ---------------------------------------------------------------------------
# offline bit allocation (host only)
# ---------------------------------------------------------------------------
def _np_ptr(a: np.ndarray) -> C.c_void_p:
    return a.ctypes.data_as(C.c_void_p)


def moe_expert_significance(sig: np.ndarray, topk_ids: np.ndarray, n_experts: int):
    """Eq. (1): (s_exp float64 [E], token share float64 [E]) of one dataset."""
    sig = np.ascontiguousarray(sig, np.float32)
    ids = np.ascontiguousarray(topk_ids, np.int32)
    if ids.ndim != 2 or ids.shape[0] != sig.shape[0]:
        raise MoEError("topk_ids must be [T][k] with T = len(sig)")
    s = np.empty(n_experts, np.float64)
    sh = np.empty(n_experts, np.float64)
    st = load().moe_expert_significance(_np_ptr(sig), _np_ptr(ids), ids.shape[0], ids.shape[1],
                                        n_experts, _np_ptr(s), _np_ptr(sh))
    check(st, "moe_expert_significance")
    return s, sh


def moe_allocate_bits(x: np.ndarray, share: np.ndarray, levels=(8, 4, 3, 2), m: float = 2.0,
                      eps: float = 1e-9, max_iter: int = 300, alpha: float = 0.3) -> dict:
    """Alg. 1 + cluster precision + low-precision-first -> per-expert bits."""
    x = np.ascontiguousarray(x, np.float64)
    share = np.ascontiguousarray(share, np.float64)
    lv = np.ascontiguousarray(levels, np.int32)
    n, c = x.shape[0], lv.shape[0]
    bits = np.empty(n, np.int32)
    V = np.empty(c, np.float64)
    U = np.empty((n, c), np.float64)
    rounds = C.c_int32(0)
    st = load().moe_allocate_bits(_np_ptr(x), _np_ptr(share), n, _np_ptr(lv), c, m, eps,
                                  max_iter, alpha, _np_ptr(bits), _np_ptr(V), _np_ptr(U),
                                  C.byref(rounds))
    check(st, "moe_allocate_bits")
    return dict(bits=bits, V=V, U=U, rounds=int(rounds.value))
