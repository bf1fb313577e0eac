"""Pins of the oracle's router and permutation (CPU only).

Router (Sec. II-A: a fixed number k of experts per token):
  R1  cexp is within 2 ulp of the binary64 exponential on [-80, 0]
  R2  logits are the fp64 dot product within the classical summation bound
  R3  top-k equals a full lexicographic sort (logit desc, index asc)
  R4  weights are the softmax over the selected logits (fp64 reference),
      non-negative, summing to 1 within 2k ulp; ties go to the lower index
  R5  a NaN logit ranks as -inf: never picked while k numbers are left, and
      the picks are always k distinct experts
Permutation (one-to-many token -> expert mapping as per-expert segments):
  P1  segments partition the T*k assignments, offsets are the expert counts,
      tokens ascend within a segment, inv_perm inverts perm_token, and the
      routed part equals numpy's stable argsort by expert
"""
import math

import numpy as np
import pytest

import moe_inputs as mi


def test_r1_cexp_accuracy(orc):
    rng = np.random.default_rng(0)
    xs = np.concatenate([
        -rng.uniform(0, 80, 200000),
        -(10.0 ** rng.uniform(-30, 0, 20000)),
        -np.arange(0, 116) * math.log(2.0),
        [0.0, -1e-45, -80.0, -79.99999, -0.5 * math.log(2.0)],
    ]).astype(np.float32)
    got = orc.cexp_many(xs).astype(np.float64)
    ref = np.exp(xs.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(got - ref) / ulp
    assert err.max() <= 2.0, float(err.max())
    assert orc.cexp(0.0) == 1.0
    assert orc.cexp(-80.5) == 0.0
    s = np.sort(xs)
    v = orc.cexp_many(s)
    assert np.all(np.diff(v.astype(np.float64)) >= 0)   # monotone on the sample


def _route_case(T=40, d=256, E=8, k=2, seed=1, bias=False):
    rng = np.random.default_rng(seed)
    x = mi.bf16_bits(rng.standard_normal((T, d)).astype(np.float32))
    Wr = (rng.standard_normal((E, d)) * 0.02).astype(np.float32)
    b = (rng.standard_normal(E) * 0.5).astype(np.float32) if bias else None
    return x, Wr, b


@pytest.mark.parametrize("E,k,bias", [(8, 2, False), (8, 2, True), (64, 6, False),
                                      (60, 4, True), (1, 1, False), (5, 5, False)])
def test_r2_r3_r4_router(orc, E, k, bias):
    x, Wr, b = _route_case(E=E, k=k, bias=bias, seed=E * 10 + k)
    lg, ids, w = orc.route(x, Wr, k, b)
    xf = mi.bf16_values(x).astype(np.float64)
    dot = xf @ Wr.astype(np.float64).T
    if b is not None:
        dot = dot + b.astype(np.float64)
    # R2: fixed-order fp32 sum is within gamma_n * sum|x w| (+ the bias add)
    n = x.shape[1] // 64 + 6 + 1
    u = 2.0 ** -24
    gamma = n * u / (1 - n * u)
    bound = gamma * (np.abs(xf) @ np.abs(Wr.astype(np.float64)).T)
    if b is not None:
        bound = bound + u * np.abs(dot) + u * np.abs(b)
    assert np.all(np.abs(lg.astype(np.float64) - dot) <= bound + 1e-30)
    # R3: top-k is the head of a full (logit desc, index asc) sort
    for t in range(x.shape[0]):
        order = np.lexsort((np.arange(E), -lg[t].astype(np.float64)))
        assert list(ids[t]) == list(order[:k])
    # R4: weights
    sel = np.take_along_axis(lg.astype(np.float64), ids.astype(np.int64), 1)
    ref = np.exp(sel - sel[:, :1])
    ref = ref / ref.sum(1, keepdims=True)
    assert np.all(w >= 0)
    assert np.allclose(w, ref, rtol=2e-6, atol=1e-30)
    assert np.all(np.abs(w.astype(np.float64).sum(1) - 1.0) <= 2 * k * u)


def test_r4_ties_go_to_lower_index(orc):
    x, Wr, _ = _route_case(T=16, E=8, k=3, seed=5)
    Wr[5] = Wr[2]
    Wr[7] = Wr[2]
    Wr[2] = Wr[2] * 0 + np.abs(Wr[2]) * 0  # expert 2 all zero
    Wr[4] = Wr[6]
    lg, ids, w = orc.route(x, Wr, 3)
    for t in range(16):
        order = sorted(range(8), key=lambda e: (-float(lg[t, e]), e))
        assert list(ids[t]) == order[:3]
        assert lg[t, 4] == lg[t, 6] and lg[t, 5] == lg[t, 7]
        if 4 in ids[t] and 6 in ids[t]:
            assert list(ids[t]).index(4) < list(ids[t]).index(6)


@pytest.mark.parametrize("nan_rows,k", [((3,), 2), ((0, 1, 2, 3, 4, 5), 4)])
def test_r5_nan_logits_rank_as_minus_inf(orc, nan_rows, k):
    x, Wr, _ = _route_case(T=16, E=8, k=k, seed=9)
    Wr[list(nan_rows)] = np.nan           # those experts' logits are NaN for every token
    lg, ids, w = orc.route(x, Wr, k)
    finite = [e for e in range(8) if e not in nan_rows]
    for t in range(16):
        assert np.all(np.isnan(lg[t, list(nan_rows)]))
        key = lambda e: (math.inf, e) if e in nan_rows else (-float(lg[t, e]), e)   # NaN after every number
        assert list(ids[t]) == sorted(range(8), key=key)[:k]
        assert len(set(ids[t])) == k and all(0 <= e < 8 for e in ids[t])
        # the picked NaN experts enter the softmax as -inf: weight 0, and the
        # finite picks' weights are the softmax over the finite logits alone
        picked = [e for e in ids[t] if e in finite]
        ref = np.exp(np.float64(lg[t, picked]) - np.float64(lg[t, picked]).max())
        ref /= ref.sum()
        got = np.array([w[t, j] for j in range(k) if ids[t, j] in finite], np.float64)
        assert np.allclose(got, ref, rtol=2e-6)
        assert all(w[t, j] == 0.0 for j in range(k) if ids[t, j] in nan_rows)


@pytest.mark.parametrize("T,E,k,S", [(64, 8, 2, 0), (50, 64, 6, 2), (33, 60, 4, 1),
                                     (0, 8, 2, 1), (7, 4, 4, 0), (9, 1, 1, 0)])
def test_p1_permutation(orc, T, E, k, S):
    rng = np.random.default_rng(T * 100 + E)
    ids = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) \
        if T else np.zeros((0, k), np.int32)
    offsets, perm, inv = orc.permute(ids, E, S)
    cnt = np.bincount(ids.ravel(), minlength=E)
    assert offsets[0] == 0
    assert np.array_equal(np.diff(offsets[:E + 1]), cnt)
    assert offsets[E] == T * k and offsets[E + S] == T * (k + S)
    assert np.array_equal(perm[:T * k], np.argsort(ids.ravel(), kind="stable") // k)
    for e in range(E + S):
        seg = perm[offsets[e]:offsets[e + 1]]
        assert np.all(np.diff(seg) > 0)
    for t in range(T):
        for j in range(k):
            p = inv[t, j]
            assert perm[p] == t
            assert offsets[ids[t, j]] <= p < offsets[ids[t, j] + 1]
        for s in range(S):
            assert inv[t, k + s] == offsets[E + s] + t and perm[inv[t, k + s]] == t
    assert sorted(inv.ravel().tolist()) == list(range(T * (k + S)))


def test_p1_rejects_bad_ids(orc):
    with pytest.raises(ValueError):
        orc.permute(np.array([[1, 1]], np.int32), 4, 0)
    with pytest.raises(ValueError):
        orc.permute(np.array([[0, 4]], np.int32), 4, 0)
