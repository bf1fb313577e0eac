"""Pins of the oracle's expert FFN, combine and switch (CPU only).

  F1  lossless (grid) weights: the oracle's expert FFN equals the textbook
      SiLU-GLU built from torch's F.linear / F.silu in fp64, and the whole
      layer equals a textbook top-k MoE (torch.topk, torch.softmax)
  F2  the bf16 rounding of h is torch's bf16 rounding; the oracle's bf16
      rounding agrees with torch on fp32 inputs bit for bit
  F3  8-bit everywhere: interval propagation from |w - w_hat| <= s16/2
      contains both the quantized oracle output and the unquantized textbook
      output
  F4  bit convergence: error vs the unquantized FFN shrinks with bit-width,
      roughly in proportion to 1/(2^b - 1)
  C1  combine with k = 1 and unit weight is a row gather
  W1  switch-all (every row on its 8-bit copy) == 8-bit everywhere, bitwise
  W2  switch-none == base; switching rows of an 8-bit expert is a no-op
  W3  switch table semantics and its error cases
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import moe_inputs as mi
from _layers import BitsOverride, GridLayer

TINY = mi.TINY


def _t(a):
    return torch.tensor(np.asarray(a, np.float64))


def _torch_ffn(Wg, Wu, Wd, x, round_h):
    h = F.silu(F.linear(x, _t(Wg))) * F.linear(x, _t(Wu))
    if round_h:
        h = h.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    return F.linear(h, _t(Wd))


def test_f1_expert_ffn_grid_weights(orc):
    layer = GridLayer(TINY)
    x = mi.make_x(TINY, 16)
    xt = _t(mi.bf16_values(x))
    rows = np.arange(16, dtype=np.int32)
    for e in (0, 2, 6):
        b = int(layer.bits[e])
        Ws = [orc.effective_weight(layer.weight(e, kd), b, TINY.group) for kd in range(3)]
        for kd in range(3):
            assert np.array_equal(Ws[kd], layer.weight(e, kd).astype(np.float64))
        got = orc.expert_ffn(*Ws, x, rows, round_h=False)
        ref = _torch_ffn(*Ws, xt, False).numpy()
        assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()
        got_r = orc.expert_ffn(*Ws, x, rows, round_h=True)
        ref_r = _torch_ffn(*Ws, xt, True).numpy()
        assert np.linalg.norm(got_r - ref_r) <= 1e-6 * np.linalg.norm(ref_r)
        assert np.linalg.norm(got_r - got) > 0


def test_f1_layer_is_textbook_moe(orc):
    layer = GridLayer(TINY)
    x = mi.make_x(TINY, 16)
    res = orc.layer_forward(layer, x, round_h=False)
    xt = _t(mi.bf16_values(x))
    logits = xt @ _t(layer.router).T
    topv, topi = torch.topk(logits, TINY.top_k, dim=1)
    assert np.array_equal(topi.numpy(), res["topk_ids"])
    wts = torch.softmax(topv, dim=1)
    y = torch.zeros(16, TINY.d_model, dtype=torch.float64)
    for e in range(TINY.n_experts):
        Ws = [layer.weight(e, kd) for kd in range(3)]
        out = _torch_ffn(*Ws, xt, False)
        for j in range(TINY.top_k):
            m = topi[:, j] == e
            y[m] += wts[m, j:j + 1] * out[m]
    y = y.numpy()
    assert np.linalg.norm(res["y"] - y) <= 1e-6 * np.linalg.norm(y)


def test_f2_bf16_rounding_matches_torch(orc):
    rng = np.random.default_rng(4)
    v = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.uniform(-6, 6, 20000),
                        [1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 0.0]])
    v = v.astype(np.float32)
    ref = torch.tensor(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([orc.bf16_round(float(a)) for a in v], np.uint16)
    assert np.array_equal(got, ref)


def _silu(g):
    return g / (1.0 + np.exp(-g))


def _silu_interval(a, b):
    gstar = -1.2784645427610738
    sa, sb = _silu(a), _silu(b)
    lo = np.where(b <= gstar, sb, np.where(a >= gstar, sa, _silu(gstar)))
    hi = np.where(b <= gstar, sa, np.where(a >= gstar, sb, np.maximum(sa, sb)))
    return lo, hi


def _imul(alo, ahi, blo, bhi):
    c = np.stack([alo * blo, alo * bhi, ahi * blo, ahi * bhi])
    return c.min(0), c.max(0)


def test_f3_int8_interval_bound(orc):
    layer = BitsOverride(mi.LayerInputs(TINY), 8)
    x = mi.make_x(TINY, 16)
    xf = mi.bf16_values(x).astype(np.float64)
    g = TINY.group
    slack = 1e-9
    for e in (0, 3, 7):
        Wt = [layer.weight(e, kd).astype(np.float64) for kd in range(3)]
        rad = []
        Wq = []
        for kd in range(3):
            st, q, s16, z16 = orc.quantize(Wt[kd], 8, g)
            Wq.append(orc.dequant(q, s16, z16, g))
            rad.append(np.repeat(s16.view(np.float16).astype(np.float64), g, 1) / 2)
        assert all(np.all(np.abs(Wq[i] - Wt[i]) <= rad[i]) for i in range(3))
        got = orc.expert_ffn(*Wq, x, np.arange(16, dtype=np.int32), round_h=False)
        gt, ut = xf @ Wt[0].T, xf @ Wt[1].T
        true = (_silu(gt) * ut) @ Wt[2].T
        rg, ru = np.abs(xf) @ rad[0].T, np.abs(xf) @ rad[1].T
        slo, shi = _silu_interval(gt - rg - slack, gt + rg + slack)
        hlo, hhi = _imul(slo, shi, ut - ru - slack, ut + ru + slack)
        # sum_i [Wd - r, Wd + r] * [hlo, hhi]
        Wlo, Whi = Wt[2] - rad[2], Wt[2] + rad[2]
        lo = np.zeros_like(true)
        hi = np.zeros_like(true)
        for t in range(16):
            a, b = _imul(Wlo, Whi, hlo[t][None, :], hhi[t][None, :])
            lo[t], hi[t] = a.sum(1), b.sum(1)
        tol = 1e-9 * np.abs(true).max()
        assert np.all(got >= lo - tol) and np.all(got <= hi + tol)
        assert np.all(true >= lo - tol) and np.all(true <= hi + tol)
        # the worst-case interval is wide; the FFN's structure itself is
        # pinned by the lossless-grid and bit-convergence tests
        assert np.all(hi - lo > 0)


def test_f4_bit_convergence(orc):
    base = mi.LayerInputs(TINY)
    x = mi.make_x(TINY, 16)
    xt = _t(mi.bf16_values(x))
    rows = np.arange(16, dtype=np.int32)
    errs = {}
    for b in (2, 4, 8):
        num = den = 0.0
        for e in range(4):
            Wt = [base.weight(e, kd) for kd in range(3)]
            Wq = [orc.effective_weight(w, b, TINY.group) for w in Wt]
            got = orc.expert_ffn(*Wq, x, rows, round_h=False)
            ref = _torch_ffn(*Wt, xt, False).numpy()
            num += np.sum((got - ref) ** 2)
            den += np.sum(ref ** 2)
        errs[b] = np.sqrt(num / den)
    assert errs[2] > errs[4] > errs[8] > 0
    r84 = errs[4] / errs[8]
    r42 = errs[2] / errs[4]
    assert 0.6 * 255 / 15 < r84 < 1.6 * 255 / 15, r84
    assert 0.6 * 15 / 3 < r42 < 1.6 * 15 / 3, r42


def test_c1_combine_gather(orc):
    rng = np.random.default_rng(2)
    o = rng.standard_normal((10, 8))
    inv = rng.permutation(10).astype(np.int32).reshape(10, 1)
    w = np.ones((10, 1), np.float32)
    y = orc.combine(o, inv, w, 1, 0)
    assert np.array_equal(y, np.take(o, inv[:, 0], axis=0))
    # shared rows are added with weight 1 on top of the routed rows
    inv2 = np.stack([inv[:, 0], (inv[:, 0] + 3) % 10], 1).astype(np.int32)
    y2 = orc.combine(o, inv2, w, 1, 1)
    assert np.allclose(y2, np.take(o, inv2[:, 0], 0) + np.take(o, inv2[:, 1], 0), rtol=0, atol=1e-15)


def _row_slots(orc, layer, slots=None):
    cfg = layer.cfg
    out = {}
    for kd in range(3):
        hdr = layer.copy_headers(kd)
        on = layer.slots_on(kd) if slots is None else slots(kd, hdr)
        st, rs = orc.switch(hdr, cfg.n_experts, cfg.rows(kd, 0), on)
        assert st == 0
        out[kd] = rs
    return out


def test_w1_switch_all_equals_int8_everywhere(orc):
    layer = mi.LayerInputs(TINY)
    x = mi.make_x(TINY, 16)
    rs_all = _row_slots(orc, layer, lambda kd, hdr: np.arange(len(hdr), dtype=np.int32))
    y_all = orc.layer_forward(layer, x, row_slot=rs_all)["y"]
    y_8 = orc.layer_forward(BitsOverride(layer, 8), x)["y"]
    assert np.array_equal(y_all, y_8)


def test_w2_switch_none_and_int8_noop(orc):
    layer = mi.LayerInputs(TINY)
    x = mi.make_x(TINY, 16)
    rs_none = _row_slots(orc, layer, lambda kd, hdr: np.zeros(0, np.int32))
    y0 = orc.layer_forward(layer, x)["y"]
    assert np.array_equal(orc.layer_forward(layer, x, row_slot=rs_none)["y"], y0)
    # experts 0 and 1 are 8-bit: switching only their rows changes nothing
    def only_int8(kd, hdr):
        return np.nonzero(hdr[:, 0] <= 1)[0].astype(np.int32)
    rs8 = _row_slots(orc, layer, only_int8)
    assert np.array_equal(orc.layer_forward(layer, x, row_slot=rs8)["y"], y0)
    # while the default 10 % mask does change the output
    rs = _row_slots(orc, layer)
    assert not np.array_equal(orc.layer_forward(layer, x, row_slot=rs)["y"], y0)


def test_w3_switch_table(orc):
    layer = mi.LayerInputs(TINY)
    hdr = layer.copy_headers(0)
    on = layer.slots_on(0)
    st, rs = orc.switch(hdr, 8, 512, on)
    assert st == 0
    want = -np.ones((8, 512), np.int32)
    for s in on:
        want[hdr[s, 0], hdr[s, 1]] = s
    assert np.array_equal(rs, want)
    assert orc.switch(hdr, 8, 512, [len(hdr)])[0] == orc.ERR_SLOT
    assert orc.switch(hdr, 8, 512, [3, 3])[0] == orc.ERR_SLOT
    dup = np.concatenate([hdr, hdr[:1]], 0)
    assert orc.switch(dup, 8, 512, [0, len(dup) - 1])[0] == orc.ERR_SLOT
    # set(M) -> set(M') -> set(M) gives the same table
    st2, _ = orc.switch(hdr, 8, 512, layer.slots_on(0)[:5])
    st3, rs3 = orc.switch(hdr, 8, 512, on)
    assert np.array_equal(rs3, rs)


def test_layer_weights_cache_matches_fresh_quantization(orc):
    # the cached dequantized weights (used to check many steps) give each
    # (expert, kind) exactly the matrix the oracle quantizes afresh, for
    # several switch masks, and the same layer output bit for bit
    wk = mi.WORKLOADS["tiny"]
    inp = mi.LayerInputs(wk.layer)
    lw = orc.LayerWeights(inp)
    x = mi.make_x(wk.layer, 12, stream=321)
    for epoch, slots in ((0, None), (0, "all")):
        if slots is None:
            rs = orc.switch_state(inp, epoch)
        else:
            rs = {}
            for kd in range(3):
                st, rs[kd] = orc.switch(inp.copy_headers(kd), wk.layer.n_experts,
                                        wk.layer.rows(kd, 0),
                                        np.arange(len(inp.copy_headers(kd)), dtype=np.int32))
                assert st == 0
        for e in range(wk.layer.n_experts):
            for kd in range(3):
                sw = np.nonzero(rs[kd][e] >= 0)[0]
                ref = orc.effective_weight(inp.weight(e, kd), int(inp.bits[e]), wk.layer.group, sw)
                assert np.array_equal(lw.effective(e, kd, sw), ref)
        a = orc.layer_forward(inp, x, row_slot=rs)
        b = orc.layer_forward(inp, x, row_slot=rs, weights=lw)
        assert np.array_equal(a["y"], b["y"]) and np.array_equal(a["o"], b["o"])
        assert np.array_equal(a["o_rows"], np.arange(12 * wk.layer.top_k))
    # a row without a cached copy cannot be switched
    with pytest.raises(ValueError):
        lw.effective(0, 0, np.array([wk.layer.d_ff + 5]))


def test_bf16_reference_weights(orc):
    # the unquantized 16-bit weights are the fp32 weights rounded to nearest
    # bfloat16 with ties to even: torch's conversion, on random values and on
    # hand-built ties (both directions) and magnitudes across the range
    rng = np.random.default_rng(3)
    w = (rng.standard_normal(50000) * 10.0 ** rng.uniform(-30, 30, 50000)).astype(np.float32)
    ties = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 2.0 ** -130 * 1.5,
                     0.0, -0.0, 3.4e38], np.float32)
    w = np.concatenate([w, ties])
    ref = torch.from_numpy(w).to(torch.bfloat16).double().numpy()
    got = orc.bf16_weights(w)
    assert np.array_equal(got, ref)
    assert got[len(w) - 7] == 1.0 and got[len(w) - 6] == 1.0 + 2.0 ** -6   # ties to even
    # an unquantized layer's effective weights are these values; no copies
    cfg = mi.unquantized(mi.TINY)
    inp = mi.LayerInputs(cfg)
    assert list(inp.bits) == [16] * cfg.n_experts and len(inp.copy_headers(0)) == 0
    W = orc.effective_weight(inp.weight(1, 0), 16, cfg.group)
    assert np.array_equal(W, torch.from_numpy(inp.weight(1, 0)).to(torch.bfloat16).double().numpy())
    with pytest.raises(ValueError):
        orc.effective_weight(inp.weight(1, 0), 16, cfg.group, np.array([3]))
