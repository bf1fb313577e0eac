"""The unquantized 16-bit reference layer run through the library's own
kernels: every expert at bits = 16, i.e. the bf16 values of the same seeded
fp32 weights as the quantized layers (the "FP16 model" that the paper's
inference speedup is measured against, Sec. VI-C, kept in bf16 like the
activations), no channel copies, group 64.

Packing is checked bit for bit against the oracle's bf16 rounding; the layer
output against oracle.layer_forward on those weights: the streaming kernel
multiplies the bf16 weights as stored (diagnostic bound 5e-4, as for exact
quantized weights), the tile kernel converts them to fp16 exactly (normal
range) and multiplies fp16 activations, so the same bound applies.
"""
import numpy as np
import pytest
import torch

import moe_inputs as mi
from gpu_util import dev, rel_l2, routing_matches, to_dev_bf16
from test_gpu_ffn import TOL, check_segments, gpu_o_rows, segment_sample

pytestmark = pytest.mark.gpu

DIAG = 5e-4


def _layer(cfg):
    import paper_2503_21135_amd as P
    inp = mi.LayerInputs(mi.unquantized(cfg))
    layer = P.MoELayer(inp)
    layer.set_epoch(0)
    return inp, layer


def test_unquantized_pack_bitexact(orc):
    inp, layer = _layer(mi.TINY)
    for kind in range(3):
        for e in (0, 5, 7):
            codes, sz = layer.packed_expert(kind, e)
            w = inp.weight(e, kind)
            want = orc.bf16_weights(w).astype(np.float32).view(np.uint32) >> 16
            got = np.stack([codes & 0xFFFF, codes >> 16], -1).reshape(w.shape)
            assert np.array_equal(got, want), (kind, e)
            assert np.all(sz == 0x3C00)   # scale 1.0, zero 0


@pytest.mark.parametrize("T", [16, 512])
def test_unquantized_tiny_layer(orc, T):
    # 16 tokens stream every expert; 512 tokens (128 per expert) tile them
    inp, layer = _layer(mi.TINY)
    x = mi.make_x(inp.cfg, T, stream=1300 + T)
    y = layer.forward(to_dev_bf16(x)).cpu().numpy()
    b = layer.buffers(T)
    res = orc.layer_forward(inp, x)
    routing_matches(layer, res, b)
    err = rel_l2(y, res["y"])
    print("unquantized tiny T", T, "rel_l2", err, flush=True)
    assert err <= TOL and err <= DIAG


@pytest.mark.parametrize("name", ["mixtral-decode", "deepseek-decode", "mixtral-prefill"])
def test_unquantized_full_size(orc, name):
    wk = mi.WORKLOADS[name]
    inp, layer = _layer(wk.layer)
    q = mi.LayerInputs(wk.layer)   # the quantized layer's batch (same x, same router bias)
    batch = mi.make_batch(wk, q)
    x = to_dev_bf16(batch.x)
    bias = None if batch.bias is None else torch.from_numpy(batch.bias).to(dev())
    y = layer.forward(x, bias).cpu().numpy()
    b = layer.buffers(wk.tokens)
    _, ids, _ = orc.route(batch.x, inp.router, wk.layer.top_k, batch.bias)
    off, perm, _ = orc.permute(ids, wk.layer.n_experts, wk.layer.n_shared)
    toks = segment_sample(off, perm, wk.tokens, 8, 11)
    res = orc.layer_forward(inp, batch.x, bias=batch.bias, tokens=toks)
    routing_matches(layer, res, b)
    seg = check_segments(res, gpu_o_rows(b, res["o_rows"]))
    err = rel_l2(y[toks], res["y"])
    print("unquantized", name, "rel_l2", err, "worst expert segment", seg, flush=True)
    assert err <= TOL and err <= DIAG
