"""The C-ABI library loads on a host without a GPU, exports every entry point
include/moe_quant.h declares, and rejects bad arguments on the host before
any device work (no compute call is made here)."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2503_21135_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2503_21135_amd import build
        build.build()
    return _lib.load()


def declared_functions():
    src = open(os.path.join(ROOT, "include", "moe_quant.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 8
    for n in names:
        assert hasattr(lib, n), n
    from paper_2503_21135_amd import _lib
    assert sorted(_lib.EXPORTS) == names


def test_status_strings(lib):
    for st in (0, -1, -2, -3, -4, -5, -6, -7):
        assert lib.moe_status_str(st)
    assert lib.moe_status_str(-99) == b"unknown status"


FAKE = C.c_void_p(1 << 20)       # non-NULL, 16-byte aligned, never dereferenced
MISALIGNED = C.c_void_p((1 << 20) + 4)


def test_pack_validation(lib):
    f = lib.moe_quant_pack
    ok = dict(w=FAKE, ld=256, R=8, K=256, b=4, g=64, rows=None, n=8, codes=FAKE, ldc=32,
              sz=FAKE, srs=4, sgs=1)

    def call(**kw):
        a = dict(ok, **kw)
        return f(a["w"], a["ld"], a["R"], a["K"], a["b"], a["g"], a["rows"], a["n"], a["codes"],
                 a["ldc"], a["sz"], a["srs"], a["sgs"], None, None)
    assert call(b=5) == -2
    assert call(b=1) == -2
    assert call(g=32) == -1
    assert call(K=200) == -1
    assert call(b=3, g=64) == -1
    assert call(b=6, g=64) == -1
    assert call(b=7) == -2
    assert call(b=6, g=128, ldc=47) == -1    # 6-bit rows of K = 256 need 48 words
    assert call(w=None) == -1
    assert call(ldc=8) == -1
    assert call(n=9) == -1
    assert call(codes=MISALIGNED) == -3
    assert call(ldc=33) == -3
    assert call(n=0) == 0           # nothing to do, no device call
    assert call(b=16, ldc=127) == -1  # unquantized rows of K = 256 need 128 words
    assert call(b=16, ldc=128, n=0) == 0


def test_route_validation(lib):
    f = lib.moe_route_permute
    ws_need = lib.moe_route_workspace_bytes(100, 8, 2, 1)
    assert ws_need > 0

    def call(T=100, d=256, E=8, k=2, S=1, ws=FAKE, wsb=ws_need, xp=None, x=FAKE):
        return f(x, T, d, FAKE, None, E, k, S, FAKE, FAKE, FAKE, FAKE, FAKE, xp, ws, wsb, None)
    assert call(d=100) == -1
    assert call(k=9) == -1
    assert call(k=0) == -1
    assert call(k=17, E=32) == -1
    assert call(E=250, S=20) == -1
    assert call(ws=None) == -4
    assert call(wsb=ws_need - 1) == -4
    assert call(xp=MISALIGNED) == -3


def test_combine_validation(lib):
    f = lib.moe_unpermute_combine
    assert f(FAKE, 1, 0, FAKE, FAKE, 4, 2, 0, 6, FAKE, None) == -1      # d % 4
    assert f(FAKE, 0, 0, FAKE, FAKE, 4, 2, 0, 8, FAKE, None) == -1      # n_split
    assert f(FAKE, 2, 10, FAKE, FAKE, 4, 2, 0, 8, FAKE, None) == -1     # split stride
    assert f(MISALIGNED, 1, 0, FAKE, FAKE, 4, 2, 0, 8, FAKE, None) == -3
    assert f(FAKE, 1, 0, FAKE, FAKE, 0, 2, 0, 8, FAKE, None) == 0        # T == 0


def _fake_layer(n_slots=4, hdr=None):
    from paper_2503_21135_amd._lib import LayerDesc
    L = LayerDesc()
    L.n_experts, L.n_shared, L.d_model, L.d_ff, L.d_ff_shared, L.group = 4, 0, 256, 512, 0, 64
    bits = np.array([8, 4, 3, 2], np.int32)
    L.bits_host = bits.ctypes.data
    L.bits = FAKE.value
    keep = [bits]
    if hdr is None:
        hdr = np.array([[0, 1], [0, 2], [1, 1], [1, 1]], np.int32)
    hdr = np.ascontiguousarray(hdr, np.int32)
    off = np.zeros(4, np.int64)
    keep += [hdr, off]
    for kd in range(3):
        K = L.kind[kd]
        K.codes = K.sz = K.code_off = K.sz_off = FAKE.value
        K.code_off_host = off.ctypes.data
        K.n_slots = n_slots
        K.copy_codes = K.copy_sz = K.copy_hdr = FAKE.value
        K.copy_hdr_host = hdr.ctypes.data
        K.row_slot = FAKE.value
    L.order_gu = L.order_dn = L.class_cnt = L.staging = FAKE.value
    return L, keep


def test_switch_and_ffn_validation(lib):
    L, keep = _fake_layer()
    sw = lib.moe_set_channel_switch

    def slots(*s):
        a = np.array(s, np.int32)
        keep.append(a)
        return a.ctypes.data_as(C.c_void_p), len(s)
    p, n = slots(0, 4)
    assert sw(C.byref(L), 0, p, n, None) == -5          # slot out of range
    p, n = slots(1, 1)
    assert sw(C.byref(L), 0, p, n, None) == -5          # duplicate slot
    p, n = slots(2, 3)
    assert sw(C.byref(L), 0, p, n, None) == -5          # two slots, same (expert, row)
    p, n = slots(0, 1, 2, 3, 0)
    assert sw(C.byref(L), 0, p, n, None) == -5          # more than n_slots
    assert sw(C.byref(L), 3, None, 0, None) == -1       # bad kind
    assert sw(C.byref(L), -1, p, 1, None) == -1         # reset with a list
    bad_hdr, keep2 = _fake_layer(hdr=[[4, 0], [0, 0], [0, 1], [0, 2]])
    p, n = slots(0)
    assert sw(C.byref(bad_hdr), 0, p, n, None) == -5    # header expert out of range
    # FFN plan / entry validation
    ns, wb = C.c_int32(0), C.c_size_t(0)
    assert lib.moe_ffn_plan(C.byref(L), 16, 2, C.byref(ns), C.byref(wb)) == -1   # 3-bit, group 64
    L.group = 128
    assert lib.moe_ffn_plan(C.byref(L), 16, 2, C.byref(ns), C.byref(wb)) == 0
    assert ns.value >= 1 and wb.value > 0
    assert lib.moe_ffn_plan(C.byref(L), 16, 5, C.byref(ns), C.byref(wb)) == -1   # k > E
    f = lib.moe_expert_ffn_mixed
    assert f(C.byref(L), FAKE, 16, 2, FAKE, FAKE, FAKE, FAKE, wb.value - 1, None, None) == -4
    assert f(C.byref(L), MISALIGNED, 16, 2, FAKE, FAKE, FAKE, FAKE, wb.value, None, None) == -3
    L.d_ff = 500
    assert f(C.byref(L), FAKE, 16, 2, FAKE, FAKE, FAKE, FAKE, wb.value, None, None) == -1
    L.d_ff = 512
    # an empty batch: OK without touching any buffer (null activations, no workspace)
    assert f(C.byref(L), None, 0, 2, None, None, None, None, 0, None, None) == 0
    assert f(C.byref(L), None, -1, 2, None, None, None, None, 0, None, None) == -1
    # the no-allocation variant: an empty batch needs nothing; a batch whose
    # workspace exceeds the fixed per-GPU array is refused before any device work
    na = lib.moe_expert_ffn_mixed_noalloc
    assert na(C.byref(L), None, 0, 2, None, None, None, None, None) == 0
    assert na(C.byref(L), None, -1, 2, None, None, None, None, None) == -1
    from paper_2503_21135_amd import _lib
    T = 16
    while True:
        assert lib.moe_ffn_plan(C.byref(L), T, 2, C.byref(ns), C.byref(wb)) == 0
        if wb.value > _lib.NOALLOC_SCRATCH_BYTES:
            break
        T *= 2
    assert na(C.byref(L), FAKE, T, 2, FAKE, FAKE, FAKE, None, None) == -4
    b16 = np.array([8, 4, 16, 2], np.int32)   # an unquantized expert needs group 64
    keep.append(b16)
    L.bits_host = b16.ctypes.data
    assert f(C.byref(L), FAKE, 16, 2, FAKE, FAKE, FAKE, FAKE, wb.value, None, None) == -1
    bits = np.array([8, 4, 5, 2], np.int32)
    keep.append(bits)
    L.bits_host = bits.ctypes.data
    assert f(C.byref(L), FAKE, 16, 2, FAKE, FAKE, FAKE, FAKE, wb.value, None, None) == -2
    assert na(C.byref(L), FAKE, 16, 2, FAKE, FAKE, FAKE, None, None) == -2


def test_requant_validation(lib):
    L, keep = _fake_layer()
    rq = lib.moe_requant_channels

    def eb(*b):
        a = np.array(b, np.int32)
        keep.append(a)
        return a.ctypes.data_as(C.c_void_p)
    ok = eb(8, 0, 4, 2)
    assert rq(C.byref(L), 3, FAKE, 256, ok, None, None) == -1        # bad kind
    assert rq(C.byref(L), 0, FAKE, 256, None, None, None) == -1      # no bit list
    assert rq(C.byref(L), 0, FAKE, 256, eb(8, 5, 4, 2), None, None) == -2   # 5 bits
    assert rq(C.byref(L), 0, FAKE, 200, ok, None, None) == -1        # ld_cache < K
    assert rq(C.byref(L), 2, FAKE, 256, ok, None, None) == -1        # down: K = d_ff = 512
    assert rq(C.byref(L), 0, FAKE, 257, ok, None, None) == -1        # odd row stride
    assert rq(C.byref(L), 0, C.c_void_p(FAKE.value + 2), 256, ok, None, None) == -1
    assert rq(C.byref(L), 0, None, 256, ok, None, None) == -1        # no cache
    bad_hdr, keep2 = _fake_layer(hdr=[[4, 0], [0, 0], [0, 1], [0, 2]])
    assert rq(C.byref(bad_hdr), 0, FAKE, 256, ok, None, None) == -5  # header expert
    empty, keep3 = _fake_layer(n_slots=0)
    assert rq(C.byref(empty), 0, None, 0, ok, None, None) == 0       # nothing cached


def test_code_row_words(lib):
    # K*bits/32 words of codes plus 16 (32 at 8 bits) words of padding
    assert lib.moe_code_row_words(4096, 4) == 4096 * 4 // 32 + 16
    assert lib.moe_code_row_words(4096, 8) == 4096 // 4 + 32
    assert lib.moe_code_row_words(1408, 3) == 1408 * 3 // 32 + 16
    assert lib.moe_code_row_words(128, 2) == 8 + 16
    assert lib.moe_code_row_words(4096, 6) == 4096 * 6 // 32 + 16
    assert lib.moe_code_row_words(1408, 6) == 1408 * 6 // 32 + 16
    assert lib.moe_code_row_words(4096, 16) == 4096 // 2 + 32   # unquantized bf16 rows
    for K, b in ((4096, 5), (100, 4), (0, 4), (-128, 8), (4096, 12)):
        assert lib.moe_code_row_words(K, b) == 0
