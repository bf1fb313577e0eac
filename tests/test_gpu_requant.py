"""GPU parity of moe_requant_channels -- requantization of the cached 16-bit
channels at each expert's new precision when the dataset changes (Sec. IV-B)
-- against the oracle: codes and {scale, zero} words bit for bit, slots of
experts left out unchanged, and the layer output after the switch within the
FFN tolerance of the other parity tests (relative L2 <= 2e-3)."""
import numpy as np
import pytest
import torch

import moe_inputs as mi
from gpu_util import oracle_row_slots, rel_l2, routing_matches, to_dev_bf16

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _layer(name):
    import paper_2503_21135_amd as P
    wk = mi.WORKLOADS[name]
    inp = mi.LayerInputs(wk.layer)
    return wk, inp, P.MoELayer(inp)


def _check_copies(orc, inp, layer, kind, eb, before):
    """GPU copies of one kind after a requantization at eb == oracle's."""
    codes, sz = layer.packed_copies(kind)
    st, touched, q, s16, z16 = orc.requant_channels(
        inp.channel_cache(kind), inp.copy_headers(kind), eb, inp.cfg.group)
    assert st == orc.OK
    want_codes, want_sz = before[0].copy(), before[1].copy()
    if touched.any():
        want_codes[touched] = orc.pack(q[touched], 8)
        want_sz[touched] = orc.sz_words(s16[touched], z16[touched])
    assert np.array_equal(codes, want_codes), "copy codes differ (kind %d)" % kind
    assert np.array_equal(sz, want_sz), "copy scale/zero words differ (kind %d)" % kind
    return int(touched.sum())


def _requant_and_check(orc, inp, layer, eb, kinds=(0, 1, 2)):
    for kind in kinds:
        before = layer.packed_copies(kind)
        layer.requant(kind, eb)
        torch.cuda.synchronize()
        n = _check_copies(orc, inp, layer, kind, eb, before)
        print(inp.cfg.name, "kind", kind, "requantized", n, "of",
              len(inp.copy_headers(kind)), "slots", flush=True)
    assert int(layer.status.item()) == 0


def test_requant_tiny_bitexact_and_ffn(orc):
    # group 64, every row cached: higher and lower new precisions, an expert
    # left out, then a second dataset on top of the first
    wk, inp, layer = _layer("tiny")
    x = mi.make_x(wk.layer, wk.tokens)
    for dataset, drop in ((0, ()), (1, (2, 5))):
        eb = inp.dataset_bits(dataset)
        eb[list(drop)] = 0
        _requant_and_check(orc, inp, layer, eb)
        layer.set_epoch(0)
        rs = oracle_row_slots(orc, inp)
        xd = to_dev_bf16(x)
        y = layer.forward(xd)
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        res = orc.layer_forward(inp, x, row_slot=rs, copy_bits=layer.copy_bits)
        routing_matches(layer, res, layer.buffers(wk.tokens))
        err = rel_l2(y, res["y"])
        print("tiny dataset", dataset, "copy bits", layer.copy_bits[0], "rel_l2", err, flush=True)
        assert err <= TOL and err <= 2e-4


def test_requant_deepseek_bitexact_and_ffn(orc):
    # 64 routed experts, K = 2048 (gate/up) and 1408 (down), group 128
    wk, inp, layer = _layer("deepseek-decode")
    eb = inp.dataset_bits(0)
    eb[::7] = 0
    _requant_and_check(orc, inp, layer, eb)
    layer.set_epoch(0)
    rs = oracle_row_slots(orc, inp)
    batch = mi.make_batch(wk, inp)
    y = layer.forward(to_dev_bf16(batch.x))
    torch.cuda.synchronize()
    y = y.cpu().numpy()
    toks = np.sort(np.random.default_rng(5).choice(wk.tokens, 32, replace=False))
    res = orc.layer_forward(inp, batch.x, row_slot=rs, tokens=toks,
                            copy_bits=layer.copy_bits)
    routing_matches(layer, res, layer.buffers(wk.tokens))
    err = rel_l2(y[toks], res["y"])
    print("deepseek after requant rel_l2", err, flush=True)
    assert err <= TOL


def test_requant_mixtral_long_rows_bitexact(orc):
    # down rows of 14336 values (112 groups), gate rows of 4096
    wk, inp, layer = _layer("mixtral-decode")
    eb = inp.dataset_bits(0)
    _requant_and_check(orc, inp, layer, eb, kinds=(2, 0))
