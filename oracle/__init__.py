"""CPU oracle of the mixed-precision MoE expert-FFN hot path (DynaMo,
arXiv 2503.21135).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; the product path never imports it.
It shares no code with the GPU library: ``oracle.c`` is compiled by gcc alone
and this module only marshals numpy arrays into it.

The arithmetic lives in ``oracle.c``; ``layer_forward`` below strings its
steps together in the paper's order: route (Sec. II-A), quantize each expert at
its precision (Sec. IV-A), replace switched rows by their cached copies
(Sec. IV-B, Sec. V-A) -- either the 8-bit copies made from the original rows
or the cached 16-bit channels requantized at their expert's precision for a
new dataset (``requant_channels``, Sec. IV-B) -- expert FFN, combine.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, ERR_ARG, ERR_BITS, ERR_SLOT, ERR_RANGE = 0, -1, -2, -5, -6


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (no HIP) into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-fopenmp", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = C.CDLL(_LIB_PATH)
        vp, i32, i64 = C.c_void_p, C.c_int, C.c_int64
        sig = {
            "oracle_fp16_value": (C.c_double, [C.c_uint16]),
            "oracle_fp16_round_up": (C.c_uint16, [C.c_double]),
            "oracle_bf16_value": (C.c_double, [C.c_uint16]),
            "oracle_bf16_round": (C.c_uint16, [C.c_double]),
            "oracle_quantize": (i32, [vp, i64, i32, i32, i32, i32, vp, vp, vp]),
            "oracle_dequant": (None, [vp, vp, vp, i32, i32, i32, vp]),
            "oracle_pack": (i32, [vp, i32, i32, i32, vp]),
            "oracle_unpack": (i32, [vp, i32, i32, i32, vp]),
            "oracle_cexp": (C.c_float, [C.c_float]),
            "oracle_route": (i32, [vp, i32, i32, vp, vp, i32, i32, vp, vp, vp]),
            "oracle_permute": (i32, [vp, i32, i32, i32, i32, vp, vp, vp]),
            "oracle_switch": (i32, [vp, i32, i32, i32, vp, i32, vp]),
            "oracle_expert_ffn": (None, [vp, vp, vp, i32, i32, vp, vp, i32, i32, vp]),
            "oracle_combine": (None, [vp, vp, vp, i32, i32, i32, i32, vp]),
            "oracle_bf16_weights": (None, [vp, i64, vp]),
            "oracle_num_threads": (i32, []),
            "oracle_set_num_threads": (None, [i32]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def num_threads() -> int:
    return int(lib().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's later OpenMP loops (timing only)."""
    lib().oracle_set_num_threads(int(n))


# ---------------------------------------------------------------------------
# scalar helpers
# ---------------------------------------------------------------------------
def fp16_value(h: int) -> float:
    return lib().oracle_fp16_value(h)


def fp16_round_up(s: float) -> int:
    return lib().oracle_fp16_round_up(s)


def bf16_round(v: float) -> int:
    return lib().oracle_bf16_round(v)


def cexp(x: float) -> float:
    return lib().oracle_cexp(x)


def cexp_many(x: np.ndarray) -> np.ndarray:
    f = lib().oracle_cexp
    return np.array([f(float(v)) for v in np.asarray(x, np.float32).ravel()],
                    dtype=np.float32).reshape(np.shape(x))


# ---------------------------------------------------------------------------
# quantization and packing
# ---------------------------------------------------------------------------
def quantize(w: np.ndarray, bits: int, group: int):
    """Returns (status, q uint8 [R][K], s16 uint16 [R][K/g], z16 uint16 [R][K/g])."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    R, K = w.shape
    q = np.empty((R, K), np.uint8)
    G = K // group if group > 0 else 0
    s16 = np.empty((R, max(G, 1)), np.uint16)
    z16 = np.empty((R, max(G, 1)), np.uint16)
    st = lib().oracle_quantize(_ptr(w), K, R, K, bits, group, _ptr(q), _ptr(s16), _ptr(z16))
    return st, q, s16[:, :G], z16[:, :G]


def dequant(q: np.ndarray, s16: np.ndarray, z16: np.ndarray, group: int) -> np.ndarray:
    q = np.ascontiguousarray(q, np.uint8)
    R, K = q.shape
    out = np.empty((R, K), np.float64)
    lib().oracle_dequant(_ptr(q), _ptr(np.ascontiguousarray(s16)),
                         _ptr(np.ascontiguousarray(z16)), R, K, group, _ptr(out))
    return out


def pack(q: np.ndarray, bits: int) -> np.ndarray:
    q = np.ascontiguousarray(q, np.uint8)
    R, K = q.shape
    out = np.empty((R, K * bits // 32), np.uint32)
    st = lib().oracle_pack(_ptr(q), R, K, bits, _ptr(out))
    if st != OK:
        raise ValueError("oracle_pack: status %d" % st)
    return out


def unpack(words: np.ndarray, K: int, bits: int) -> np.ndarray:
    words = np.ascontiguousarray(words, np.uint32)
    R = words.shape[0]
    out = np.empty((R, K), np.uint8)
    st = lib().oracle_unpack(_ptr(words), R, K, bits, _ptr(out))
    if st != OK:
        raise ValueError("oracle_unpack: status %d" % st)
    return out


def sz_words(s16: np.ndarray, z16: np.ndarray) -> np.ndarray:
    """{s16, z} per (row, group) as the 32-bit word the library stores."""
    return s16.astype(np.uint32) | (z16.astype(np.uint32) << 16)


# ---------------------------------------------------------------------------
# routing
# ---------------------------------------------------------------------------
def route(x_bits: np.ndarray, w_router: np.ndarray, k: int,
          bias: Optional[np.ndarray] = None):
    """Returns (logits fp32 [T][E], topk_ids int32 [T][k], topk_w fp32 [T][k])."""
    x_bits = np.ascontiguousarray(x_bits, np.uint16)
    w_router = np.ascontiguousarray(w_router, np.float32)
    T, d = x_bits.shape
    E = w_router.shape[0]
    logits = np.empty((T, E), np.float32)
    ids = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    st = lib().oracle_route(_ptr(x_bits), T, d, _ptr(w_router), _ptr(b), E, k,
                            _ptr(logits), _ptr(ids), _ptr(w))
    if st != OK:
        raise ValueError("oracle_route: status %d" % st)
    return logits, ids, w


def permute(ids: np.ndarray, E: int, S: int):
    """Returns (offsets [E+S+1], perm_token [T*(k+S)], inv_perm [T][k+S])."""
    ids = np.ascontiguousarray(ids, np.int32)
    T, k = ids.shape
    offsets = np.empty(E + S + 1, np.int32)
    perm = np.empty(T * (k + S), np.int32)
    inv = np.empty((T, k + S), np.int32)
    st = lib().oracle_permute(_ptr(ids), T, E, k, S, _ptr(offsets), _ptr(perm), _ptr(inv))
    if st != OK:
        raise ValueError("oracle_permute: status %d" % st)
    return offsets, perm, inv


# ---------------------------------------------------------------------------
# switch
# ---------------------------------------------------------------------------
def switch(hdr: np.ndarray, E: int, R: int, slots_on: Sequence[int]):
    """Returns (status, row_slot int32 [E][R])."""
    hdr = np.ascontiguousarray(hdr, np.int32).reshape(-1, 2)
    on = np.ascontiguousarray(np.asarray(slots_on, np.int32))
    row_slot = np.empty((E, R), np.int32)
    st = lib().oracle_switch(_ptr(hdr), hdr.shape[0], E, R, _ptr(on), len(on), _ptr(row_slot))
    return st, row_slot


def switch_state(layer, epoch: int = 0, kinds=(0, 1, 2)) -> Dict[int, np.ndarray]:
    """row_slot tables {kind: [E][R]} of a layer's mask epoch."""
    cfg = layer.cfg
    out = {}
    for kind in kinds:
        st, rs = switch(layer.copy_headers(kind), cfg.n_experts, cfg.rows(kind, 0),
                        layer.slots_on(kind, epoch))
        if st != OK:
            raise ValueError("oracle switch: status %d" % st)
        out[kind] = rs
    return out


def fp16_values(h: np.ndarray) -> np.ndarray:
    """binary16 bit patterns -> float32 values (exact)."""
    return np.ascontiguousarray(h, np.uint16).view(np.float16).astype(np.float32)


def requant_channels(cache16: np.ndarray, hdr: np.ndarray, expert_bits: np.ndarray,
                     group: int):
    """Requantization of cached 16-bit channels for a new dataset (Sec. IV-B):
    every cached channel whose expert has a new precision b = expert_bits[e] > 0
    is quantized afresh at b bits from its binary16 values, with the same
    group-wise quantizer as the experts themselves (Sec. IV-A).

    cache16  uint16 binary16 patterns [n][K], row s = channel of header hdr[s]
    Returns (status, touched bool [n], q uint8 [n][K], s16, z16 uint16 [n][K/g]);
    rows not touched hold zeros.
    """
    cache16 = np.ascontiguousarray(cache16, np.uint16)
    hdr = np.ascontiguousarray(hdr, np.int32).reshape(-1, 2)
    n, K = cache16.shape
    G = K // group
    eb = np.asarray(expert_bits, np.int32)
    bits_of = eb[hdr[:, 0]]
    q = np.zeros((n, K), np.uint8)
    s16 = np.zeros((n, G), np.uint16)
    z16 = np.zeros((n, G), np.uint16)
    status = OK
    for b in np.unique(bits_of):
        if b == 0:
            continue
        sl = np.nonzero(bits_of == b)[0]
        st, qb, sb, zb = quantize(fp16_values(cache16[sl]), int(b), group)
        status = min(status, st)
        q[sl], s16[sl], z16[sl] = qb, sb, zb
    return status, bits_of > 0, q, s16, z16


# ---------------------------------------------------------------------------
# FFN and combine
# ---------------------------------------------------------------------------
def expert_ffn(Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray, x_bits: np.ndarray,
               rows: np.ndarray, round_h: bool = True) -> np.ndarray:
    Wg = np.ascontiguousarray(Wg, np.float64)
    Wu = np.ascontiguousarray(Wu, np.float64)
    Wd = np.ascontiguousarray(Wd, np.float64)
    f, d = Wg.shape
    assert Wu.shape == (f, d) and Wd.shape == (d, f)
    x_bits = np.ascontiguousarray(x_bits, np.uint16)
    rows = np.ascontiguousarray(rows, np.int32)
    out = np.empty((len(rows), d), np.float64)
    if len(rows):
        lib().oracle_expert_ffn(_ptr(Wg), _ptr(Wu), _ptr(Wd), f, d, _ptr(x_bits),
                                _ptr(rows), len(rows), 1 if round_h else 0, _ptr(out))
    return out


def combine(o: np.ndarray, inv: np.ndarray, w: np.ndarray, k: int, S: int) -> np.ndarray:
    o = np.ascontiguousarray(o, np.float64)
    inv = np.ascontiguousarray(inv, np.int32)
    w = np.ascontiguousarray(w, np.float32)
    T = inv.shape[0]
    d = o.shape[1]
    y = np.empty((T, d), np.float64)
    lib().oracle_combine(_ptr(o), _ptr(inv), _ptr(w), T, k, S, d, _ptr(y))
    return y


def bf16_weights(w: np.ndarray) -> np.ndarray:
    """The unquantized 16-bit weights: each fp32 weight rounded to the nearest
    bfloat16 (ties to even), as float64."""
    w = np.ascontiguousarray(w, np.float32)
    out = np.empty(w.shape, np.float64)
    lib().oracle_bf16_weights(_ptr(w), w.size, _ptr(out))
    return out


def effective_weight(w_fp32: np.ndarray, bits: int, group: int,
                     switched_rows: Optional[np.ndarray] = None,
                     copy_bits: int = 0, copy_src16: Optional[np.ndarray] = None) -> np.ndarray:
    """Dequantized expert matrix as the FFN sees it: base codes at `bits`,
    except the switched rows, which read their cached copy (Sec. IV-B: the
    cache keeps the original channels).  With copy_bits == 0 the copy is the
    8-bit quantization of the original fp32 row; with copy_bits = b > 0 it is
    the b-bit requantization of the cached binary16 channel copy_src16[i] of
    switched row i (requantization for a new dataset, Sec. IV-B).  bits == 16
    is the unquantized reference: the bf16 values of the fp32 weights (no
    channel copies)."""
    if bits == 16:
        if switched_rows is not None and len(switched_rows):
            raise ValueError("an unquantized expert has no channel copies")
        return bf16_weights(w_fp32)
    st, q, s, z = quantize(w_fp32, bits, group)
    if st != OK:
        raise ValueError("oracle quantize: status %d" % st)
    W = dequant(q, s, z, group)
    if switched_rows is not None and len(switched_rows):
        rows = np.asarray(switched_rows, np.int64)
        if copy_bits:
            src, b = fp16_values(copy_src16), copy_bits
        else:
            src, b = w_fp32[rows], 8
        st, q8, s8, z8 = quantize(src, b, group)
        if st != OK:
            raise ValueError("oracle quantize: status %d" % st)
        W[rows] = dequant(q8, s8, z8, group)
    return W


class LayerWeights:
    """The dequantized weights of a layer, built once, for checking many
    batches and switch masks (the 8-bit-copy mode of ``effective_weight``).

    Per (expert, kind): the dequantized base codes at the expert's precision
    (Sec. IV-A) and the dequantized 8-bit copies of every row a copy header
    names (Sec. IV-B, V-A).  ``effective(e, kind, switched)`` returns the
    matrix the FFN sees when `switched` rows read their copies.  The copy of
    a row is the quantization of that row alone, so quantizing every cached
    row at once gives each row the codes ``effective_weight`` gives it.
    """

    def __init__(self, layer, experts=None):
        cfg = layer.cfg
        self.group = cfg.group
        self.base = {}
        self.copy_rows = {}
        self.copy = {}
        hdr = {kind: np.asarray(layer.copy_headers(kind), np.int64).reshape(-1, 2) for kind in (0, 1, 2)}
        for e in (range(cfg.n_experts + cfg.n_shared) if experts is None else experts):
            for kind in (0, 1, 2):
                w = layer.weight(e, kind)
                self.base[(e, kind)] = effective_weight(w, int(layer.bits[e]), cfg.group)
                rows = np.unique(hdr[kind][hdr[kind][:, 0] == e, 1]) if e < cfg.n_experts else \
                    np.zeros(0, np.int64)
                self.copy_rows[(e, kind)] = rows
                if len(rows):
                    st, q8, s8, z8 = quantize(w[rows], 8, cfg.group)
                    if st != OK:
                        raise ValueError("oracle quantize: status %d" % st)
                    self.copy[(e, kind)] = dequant(q8, s8, z8, cfg.group)

    def effective(self, e: int, kind: int, switched: Optional[np.ndarray]) -> np.ndarray:
        W = self.base[(e, kind)]
        if switched is None or len(switched) == 0:
            return W
        rows = self.copy_rows[(e, kind)]
        idx = np.searchsorted(rows, switched)
        if np.any(idx >= len(rows)) or np.any(rows[np.minimum(idx, len(rows) - 1)] != switched):
            raise ValueError("a switched row of expert %d, kind %d has no cached copy" % (e, kind))
        W = W.copy()
        W[switched] = self.copy[(e, kind)][idx]
        return W


def layer_forward(layer, x_bits: np.ndarray, bias: Optional[np.ndarray] = None,
                  row_slot: Optional[Dict[int, np.ndarray]] = None,
                  round_h: bool = True, tokens: Optional[np.ndarray] = None,
                  weight_cache: Optional[dict] = None,
                  copy_bits: Optional[Dict[int, np.ndarray]] = None,
                  weights: Optional[LayerWeights] = None):
    """One MoE layer on the CPU.

    layer     moe_inputs.LayerInputs (weights are drawn from it)
    row_slot  {kind: int32 [E][R]} switch state (-1 = base), or None
    copy_bits {kind: int32 [E]} precision of each expert's cached copies: 0 =
              8-bit copies of the fp32 rows, b > 0 = b-bit requantization of
              the cached 16-bit channels (layer.channel_cache), or None
    tokens    optional subset of token indices whose outputs are computed
              (routing is always done for all tokens)
    weights   optional LayerWeights of the same layer (8-bit-copy mode only):
              its dequantized matrices are used instead of quantizing afresh
    Returns dict with logits, topk_ids, topk_w, offsets, perm, inv, y (y rows
    for `tokens`, float64), o_rows (the permuted rows whose expert output was
    computed, ascending) and o (those rows' expert outputs, float64).
    """
    cfg = layer.cfg
    E, S, k = cfg.n_experts, cfg.n_shared, cfg.top_k
    logits, ids, w = route(x_bits, layer.router, k, bias)
    offsets, perm, inv = permute(ids, E, S)
    T = x_bits.shape[0]
    sel = np.arange(T) if tokens is None else np.asarray(tokens)
    need = np.zeros(T * (k + S), bool)
    need[inv[sel].ravel()] = True
    o = np.zeros((T * (k + S), cfg.d_model), np.float64)
    for e in range(E + S):
        lo, hi = offsets[e], offsets[e + 1]
        rows_p = np.arange(lo, hi)[need[lo:hi]]
        if len(rows_p) == 0:
            continue
        Ws = []
        for kind in (0, 1, 2):
            key = (e, kind)
            if weight_cache is not None and key in weight_cache:
                Ws.append(weight_cache[key])
                continue
            sw, cb, src = None, 0, None
            if row_slot is not None and e < E:
                sw = np.nonzero(row_slot[kind][e] >= 0)[0]
                if copy_bits is not None and kind in copy_bits:
                    cb = int(copy_bits[kind][e])
                if cb and len(sw):
                    src = layer.channel_cache(kind)[row_slot[kind][e][sw]]
            if weights is not None and cb == 0:
                W = weights.effective(e, kind, sw)
            else:
                W = effective_weight(layer.weight(e, kind), int(layer.bits[e]), cfg.group, sw,
                                     cb, src)
            if weight_cache is not None:
                weight_cache[key] = W
            Ws.append(W)
        o[rows_p] = expert_ffn(Ws[0], Ws[1], Ws[2], x_bits, perm[rows_p], round_h)
    y = combine(o, inv[sel], w[sel], k, S)
    o_rows = np.nonzero(need)[0]
    return dict(logits=logits, topk_ids=ids, topk_w=w, offsets=offsets,
                perm=perm, inv=inv, y=y, tokens=sel, o_rows=o_rows, o=o[o_rows])
