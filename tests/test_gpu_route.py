"""GPU parity of moe_route_permute against the oracle: top-k ids, combine
weights, segment offsets, permutation and inverse permutation must be
identical bit for bit (Sec. II-A top-k routing)."""
import numpy as np
import pytest
import torch

import moe_inputs as mi
from gpu_util import dev, to_dev_bf16

pytestmark = pytest.mark.gpu


def gpu_route(x_bits, router, bias, k, S, want_xperm=False, misalign=False):
    import paper_2503_21135_amd as P
    T, d = x_bits.shape
    E = router.shape[0]
    D = dev()
    ids = torch.full((T, k), -7, dtype=torch.int32, device=D)
    w = torch.zeros((T, k), dtype=torch.float32, device=D)
    off = torch.zeros(E + S + 1, dtype=torch.int32, device=D)
    perm = torch.full((max(T * (k + S), 1),), -7, dtype=torch.int32, device=D)
    inv = torch.full((T, k + S), -7, dtype=torch.int32, device=D)
    ws = torch.empty(max(P.moe_route_workspace_bytes(T, E, k, S), 256), dtype=torch.uint8, device=D)
    x = to_dev_bf16(x_bits)
    if misalign:   # rows start 2 bytes past a 16-byte boundary
        buf = torch.empty(T * d + 1, dtype=torch.bfloat16, device=D)
        buf[1:] = x.reshape(-1)
        x = buf[1:].view(T, d)
    xp = torch.empty((max(T * (k + S), 1), d), dtype=torch.bfloat16, device=D) if want_xperm else None
    P.moe_route_permute(x, torch.from_numpy(router).to(D),
                        None if bias is None else torch.from_numpy(bias).to(D),
                        k, S, ids, w, off, perm, inv, ws, x_perm=xp)
    torch.cuda.synchronize()
    out = dict(ids=ids.cpu().numpy(), w=w.cpu().numpy(), off=off.cpu().numpy(),
               perm=perm.cpu().numpy()[:T * (k + S)], inv=inv.cpu().numpy())
    if want_xperm:
        out["xp"] = xp.view(torch.int16).cpu().numpy().view(np.uint16)[:T * (k + S)]
    return out


def check_route(orc, x_bits, router, bias, k, S):
    g = gpu_route(x_bits, router, bias, k, S, want_xperm=True)
    lg, ids, w = orc.route(x_bits, router, k, bias)
    off, perm, inv = orc.permute(ids, router.shape[0], S)
    assert np.array_equal(g["ids"], ids)
    assert np.array_equal(g["w"].view(np.uint32), w.view(np.uint32))
    assert np.array_equal(g["off"], off)
    assert np.array_equal(g["perm"], perm)
    assert np.array_equal(g["inv"], inv)
    assert np.array_equal(g["xp"], x_bits[perm])
    return g


@pytest.mark.parametrize("name", ["tiny", "mixtral-decode", "deepseek-decode", "qwen-stress",
                                  "mixtral-prefill", "deepseek-prefill"])
def test_route_workloads(orc, name):
    wk = mi.WORKLOADS[name]
    inp = mi.LayerInputs(wk.layer)
    batch = mi.make_batch(wk, inp)
    print("route parity", name, "T", wk.tokens, flush=True)
    g = check_route(orc, batch.x, inp.router, batch.bias, wk.layer.top_k, wk.layer.n_shared)
    if wk.zipf_s is not None:
        loads = np.diff(g["off"][:wk.layer.n_experts + 1]) / (wk.tokens * wk.layer.top_k)
        tgt = mi.zipf_targets(wk.layer.n_experts, wk.zipf_s)
        assert np.all(np.abs(loads - tgt) < 0.02), (loads, tgt)


@pytest.mark.parametrize("T,E,k,S,d", [(1, 8, 2, 0, 256), (65, 8, 8, 0, 256), (130, 64, 6, 2, 128),
                                       (7, 256, 16, 0, 64), (200, 3, 1, 1, 192),
                                       (1024, 255, 16, 1, 64), (1025, 60, 4, 1, 128),
                                       (300, 20, 3, 1, 320), (257, 5, 2, 0, 192), (520, 9, 2, 0, 576),
                                       (100, 20, 3, 1, 320), (33, 16, 16, 0, 2112)])
def test_route_edges(orc, T, E, k, S, d):
    rng = np.random.default_rng(T + E)
    x = mi.bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    router = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    check_route(orc, x, router, None, k, S)


@pytest.mark.parametrize("T", [300, 100])
def test_route_misaligned_rows(orc, T):
    # token rows off a 16-byte boundary take the routers that read a column
    # per lane; the results are the same bits
    E, k, S, d = 20, 3, 1, 320
    rng = np.random.default_rng(77)
    x = mi.bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    router = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    g = gpu_route(x, router, None, k, S, misalign=True)
    lg, ids, w = orc.route(x, router, k, None)
    assert np.array_equal(g["ids"], ids)
    assert np.array_equal(g["w"].view(np.uint32), w.view(np.uint32))


@pytest.mark.parametrize("T,E,k,n_nan", [(20, 8, 2, 1), (20, 8, 4, 6), (300, 8, 4, 6), (40, 20, 4, 18),
                                         (300, 20, 3, 2)])
def test_route_nan_logits_rank_as_minus_inf(orc, T, E, k, n_nan):
    # experts whose router rows are NaN have NaN logits for every token; they
    # rank as -inf on every router form (one workgroup per token, staged
    # logits with the rank selection), so the ids stay valid experts and match
    # the oracle, and a NaN pick gets weight 0
    rng = np.random.default_rng(T + E + n_nan)
    d = 256
    x = mi.bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    router = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    router[:n_nan] = np.nan
    g = check_route(orc, x, router, None, k, 1)
    assert np.all((g["ids"] >= 0) & (g["ids"] < E))


def test_route_ties_and_empty_experts(orc):
    rng = np.random.default_rng(3)
    d, E = 256, 16
    x = mi.bf16_bits(rng.standard_normal((50, d)).astype(np.float32))
    router = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    router[9] = router[4]          # identical logits -> lower index first
    router[12] = router[4]
    bias = np.zeros(E, np.float32)
    bias[13:] = -1e4               # experts 13..15 never chosen: empty segments
    g = check_route(orc, x, router, bias, 4, 1)
    assert np.all(np.diff(g["off"])[13:16] == 0)


def test_route_run_to_run(orc):
    wk = mi.WORKLOADS["deepseek-decode"]
    inp = mi.LayerInputs(wk.layer)
    batch = mi.make_batch(wk, inp)
    a = gpu_route(batch.x, inp.router, None, 6, 2)
    b = gpu_route(batch.x, inp.router, None, 6, 2)
    for key in a:
        assert np.array_equal(a[key], b[key])


def test_route_empty_batch():
    # no tokens: every segment (routed and shared) is empty, nothing is read
    rng = np.random.default_rng(5)
    d, E, k, S = 256, 8, 2, 1
    x = np.zeros((0, d), np.uint16)
    router = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    g = gpu_route(x, router, None, k, S)
    assert np.array_equal(g["off"], np.zeros(E + S + 1, np.int32))
