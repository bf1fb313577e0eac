"""Helpers shared by the GPU parity tests (marshalling and comparison only)."""
import numpy as np
import torch

import moe_inputs as mi


def dev():
    return torch.device("cuda:0")


def to_dev_bf16(x_bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to(dev()).view(torch.bfloat16)


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def routing_matches(layer, res, b):
    """Bitwise comparison of the GPU routing buffers with the oracle's."""
    T = res["topk_ids"].shape[0]
    E, S = layer.E, layer.S
    ids = b.topk_ids.cpu().numpy()
    w = b.topk_w.cpu().numpy()
    assert np.array_equal(ids, res["topk_ids"]), "topk_ids differ"
    assert np.array_equal(w.view(np.uint32), res["topk_w"].view(np.uint32)), "topk_w differ"
    assert np.array_equal(b.offsets.cpu().numpy(), res["offsets"]), "offsets differ"
    n = T * (layer.k + S)
    assert np.array_equal(b.perm.cpu().numpy()[:n], res["perm"]), "perm differs"
    assert np.array_equal(b.inv.cpu().numpy(), res["inv"]), "inv differs"


def oracle_row_slots(orc, inputs, epoch=0, kinds=(0, 1, 2), slots=None):
    cfg = inputs.cfg
    out = {}
    for kind in kinds:
        hdr = inputs.copy_headers(kind)
        on = inputs.slots_on(kind, epoch) if slots is None else slots[kind]
        st, rs = orc.switch(hdr, cfg.n_experts, cfg.rows(kind, 0), on)
        assert st == 0
        out[kind] = rs
    return out
