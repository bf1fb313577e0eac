"""The runtime-switch stress workload verified at every step: the
Qwen1.5-MoE-A2.7B-shaped layer (60 routed experts of d_ff 1408 at top-4, one
8-bit shared FFN of d_ff 5632), 512 fresh tokens per step for 200 steps, the
copy mask redrawn every 10 steps with 2-10 % of each expert's rows switched
(Sec. IV-B: channels replaced by cached copies at run time).

Every step: the switch tables and the whole routing (ids, weights as bits,
offsets, permutation, inverse) of all 512 tokens bit-exact against the
oracle, and the layer output of 8 tokens per step within the 2e-3 relative L2
gate (and the streaming kernel's 5e-4 diagnostic bound: ~34 tokens per
routed expert and 512 on the shared one all stream).

The oracle's work is batched per mask epoch: the sampled tokens of the
epoch's ten steps are one oracle batch, with the layer's dequantized weights
built once (oracle.LayerWeights).  A token's output depends only on its own
routing and the weights, so this is the per-step check.
"""
import numpy as np
import pytest

import moe_inputs as mi
from gpu_util import oracle_row_slots, rel_l2, routing_matches, to_dev_bf16

pytestmark = pytest.mark.gpu

TOL = 2e-3
DIAG_STREAM = 5e-4
PER_STEP = 8
PARTS = 4


@pytest.fixture(scope="module")
def stress(orc):
    import paper_2503_21135_amd as P
    wk = mi.WORKLOADS["qwen-stress"]
    inp = mi.LayerInputs(wk.layer)
    layer = P.MoELayer(inp)
    print("building the oracle's dequantized weights", flush=True)
    weights = orc.LayerWeights(inp)
    return wk, inp, layer, weights, {}


@pytest.mark.parametrize("part", range(PARTS))
def test_qwen_stress_every_step(orc, stress, part):
    wk, inp, layer, weights, worst = stress
    cfg = wk.layer
    per = wk.steps // PARTS
    assert wk.steps == 200 and per % wk.redraw_every == 0
    for ep0 in range(part * per, (part + 1) * per, wk.redraw_every):
        epoch = ep0 // wk.redraw_every
        layer.set_epoch(epoch)
        rs = oracle_row_slots(orc, inp, epoch=epoch)
        for kd in range(3):
            assert np.array_equal(layer.row_slot(kd), rs[kd])
        xs, samples, ys = [], [], []
        for step in range(ep0, ep0 + wk.redraw_every):
            batch = mi.make_batch(wk, inp, step=step)
            x = to_dev_bf16(batch.x)
            y = layer.forward(x).cpu().numpy()
            b = layer.buffers(wk.tokens)
            # routing of every token of the step, bit for bit
            _, ids, w = orc.route(batch.x, inp.router, cfg.top_k)
            off, perm, inv = orc.permute(ids, cfg.n_experts, cfg.n_shared)
            routing_matches(layer, dict(topk_ids=ids, topk_w=w, offsets=off, perm=perm, inv=inv), b)
            toks = np.sort(np.random.default_rng([part, step]).choice(wk.tokens, PER_STEP, replace=False))
            xs.append(batch.x)
            samples.append(toks)
            ys.append(y[toks])
        # one oracle batch for the epoch's sampled tokens
        X = np.concatenate(xs)
        sel = np.concatenate([t + i * wk.tokens for i, t in enumerate(samples)])
        res = orc.layer_forward(inp, X, row_slot=rs, tokens=sel, weights=weights)
        for i in range(wk.redraw_every):
            err = rel_l2(ys[i], res["y"][i * PER_STEP:(i + 1) * PER_STEP])
            worst[ep0 + i] = err
            assert err <= TOL, "step %d: rel L2 %.3g" % (ep0 + i, err)
            assert err <= DIAG_STREAM, "step %d: rel L2 %.3g" % (ep0 + i, err)
        print("epoch %d (%d%% switched): steps %d-%d worst rel L2 %.3g"
              % (epoch, inp.switch_percent(epoch), ep0, ep0 + wk.redraw_every - 1,
                 max(worst[ep0 + i] for i in range(wk.redraw_every))), flush=True)
    if len(worst) == wk.steps:
        print("all %d steps verified; worst rel L2 %.3g" % (wk.steps, max(worst.values())), flush=True)
