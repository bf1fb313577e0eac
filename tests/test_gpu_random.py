"""Seeded random small layers through every path of the expert FFN.

Each case draws a layer shape (experts, shared experts, top-k, d_model,
d_ff, group size), per-expert bit-widths from every width the group allows,
a copy recipe and switch state (none, the masked rows, or every cached row
switched) and a token count from 1 to 700, so the cases between them reach
the streaming kernel at one and two 16-token tiles, the 32-token tile sets
with split K, the tile kernel with full and partial token tiles and with
items that mix source classes, and tiled shared experts beside streaming
routed ones.  Routing is compared bit for bit with the oracle and the layer
output within the 2e-3 relative L2 gate; the FFN's status word stays clear.
The shapes are drawn from a fixed seed, so every run checks the same cases.
"""
import dataclasses

import numpy as np
import pytest

import moe_inputs as mi
from gpu_util import oracle_row_slots, rel_l2, routing_matches, to_dev_bf16

pytestmark = pytest.mark.gpu

TOL = 2e-3
N_CASES = 24


def _case(i):
    rng = np.random.default_rng([20261202, i])
    E = int(rng.choice([4, 6, 8, 12, 16]))
    S = int(rng.choice([0, 0, 1, 2]))
    k = int(rng.integers(1, min(E, 6) + 1))
    group = int(rng.choice([64, 128]))
    d = int(rng.choice([256, 384, 512]))
    f = int(rng.choice([256, 512, 768, 1024]))
    fs = int(rng.choice([256, 512, 1024])) if S else 0
    widths = [2, 4, 8] + ([3, 6] if group == 128 else [])
    bits = tuple(int(b) for b in rng.choice(widths, E))
    copies = str(rng.choice(["all", "mask", "none"]))
    mask_frac = float(rng.choice([0.03, 0.1, 0.3]))
    T = int(rng.choice([1, 7, 16, 33, 64, 130, 300, 520, 700]))
    mode = "none" if copies == "none" else str(rng.choice(["mask", "all"] if copies == "all" else ["mask"]))
    cfg = mi.LayerConfig(name="random-%d" % i, cfg_id=200 + i, d_model=d, n_experts=E, n_shared=S, top_k=k,
                         d_ff=f, d_ff_shared=fs, group=group, bits_literal=bits, copies=copies,
                         mask_frac=mask_frac, outliers=2)
    return cfg, T, mode


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_layer(orc, i):
    import torch
    import paper_2503_21135_amd as P
    from paper_2503_21135_amd import api
    cfg, T, mode = _case(i)
    inp = mi.LayerInputs(cfg)
    layer = P.MoELayer(inp)
    n_split, _ = api.moe_ffn_plan(layer.desc, T, cfg.top_k)
    if mode == "none":
        layer.reset_switch()
        rs = None
    elif mode == "mask":
        layer.set_epoch(0)
        rs = oracle_row_slots(orc, inp)
    else:
        slots = {kd: np.arange(len(inp.copy_headers(kd)), dtype=np.int32) for kd in range(3)}
        for kd in range(3):
            layer.set_switch(kd, slots[kd])
        rs = oracle_row_slots(orc, inp, slots=slots)
    x = mi.make_x(cfg, T, stream=5000 + i)
    layer.clear_ffn_status()
    y = layer.forward(to_dev_bf16(x)).cpu().numpy()
    torch.cuda.synchronize()
    b = layer.buffers(T)
    res = orc.layer_forward(inp, x, row_slot=rs)
    routing_matches(layer, res, b)
    err = rel_l2(y, res["y"])
    print("case %d: E=%d S=%d k=%d d=%d f=%d fs=%d g=%d bits=%s copies=%s/%s T=%d n_split=%d rel_l2 %.3g"
          % (i, cfg.n_experts, cfg.n_shared, cfg.top_k, cfg.d_model, cfg.d_ff, cfg.d_ff_shared, cfg.group,
             list(cfg.bits_literal), cfg.copies, mode, T, n_split, err), flush=True)
    assert layer.ffn_status_value() == 0
    assert err <= TOL


def test_cases_reach_every_path():
    # the drawn cases cover small and large batches, both group sizes, shared
    # experts and every switch mode (CPU-side check of the draws only)
    cases = [_case(i) for i in range(N_CASES)]
    assert {c.group for c, _, _ in cases} == {64, 128}
    assert {m for _, _, m in cases} == {"none", "mask", "all"}
    assert any(c.n_shared > 0 for c, _, _ in cases)
    assert min(T * c.top_k / c.n_experts for c, T, _ in cases) <= 12      # one 16-token tile
    assert max(T * c.top_k / c.n_experts for c, T, _ in cases) > 96       # the tile kernel
