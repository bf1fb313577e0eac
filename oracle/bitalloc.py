"""CPU oracle of the offline expert-level bit allocation (DynaMo, Sec. III-B
and Sec. IV-A).  TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``.

Steps, in the paper's order:
  1. expert significance of one dataset, Eq. (1)
  2. fuzzy c-means over the experts' significance, Alg. 1 (c = 4 clusters,
     fuzzifier m > 1, tolerance eps)
  3. one precision per cluster: the most significant cluster gets the highest
     bit-width, the least significant the lowest (Sec. IV-A)
  4. low-precision-first for experts in the overlap of clusters (Sec. IV-A,
     "Quantization for Expert Located in Clustering Boundary")

Readings (the printed text is garbled or silent here):
  - Eq. (1): s[i] is the significance of token i's combined top-K channel
    output (one non-negative scalar per token, an input); the numerator sums
    s[i] over the tokens routed to expert j, the denominator over all T
    tokens.  So S_exp[j] lies in [0, 1] and the S_exp of all experts add up
    to K.
  - Alg. 1 initial U: experts sorted by significance (ties by index) are cut
    into c consecutive runs of about equal token share -- token share p_i
    being the proportion of the dataset's tokens routed to expert i -- and
    u_ik = 1 for the run k that holds the midpoint of expert i's share.
    (A uniform U would leave every center equal and the iteration stuck.)
  - stopping rule ||U_new - U_old|| < eps with the Frobenius norm, and at
    most max_iter rounds; a point that coincides with centers gets its
    membership split equally among them.
  - cluster order: by center v_k, the membership-weighted significance of
    the cluster's experts; ties by cluster index.
  - overlap: expert i is in cluster k's region when u_ik >= alpha; an expert
    in several regions takes the lowest precision among them; an expert in
    none takes its largest-membership cluster.
parity: pinned in tests/test_oracle_bitalloc.py (hand cases, textbook FCM
properties: memberships sum to one, the FCM objective never rises, tight
separated groups give their means as centers).
"""
from __future__ import annotations

from typing import Dict, Sequence

import numpy as np


def expert_significance(sig: np.ndarray, topk_ids: np.ndarray, n_experts: int) -> np.ndarray:
    """Eq. (1).  sig float [T] (>= 0), topk_ids int [T][K] -> float64 [E]."""
    sig = np.asarray(sig, np.float64)
    ids = np.asarray(topk_ids, np.int64)
    T = sig.shape[0]
    total = 0.0
    for i in range(T):
        total += sig[i]
    out = np.zeros(n_experts, np.float64)
    for j in range(n_experts):
        num = 0.0
        for i in range(T):
            if (ids[i] == j).any():
                num += sig[i]
        out[j] = num / total if total > 0 else 0.0
    return out


def token_share(topk_ids: np.ndarray, n_experts: int) -> np.ndarray:
    """Proportion of the dataset's T tokens routed to each expert."""
    ids = np.asarray(topk_ids, np.int64)
    T = ids.shape[0]
    out = np.zeros(n_experts, np.float64)
    for j in range(n_experts):
        out[j] = float((ids == j).any(axis=1).sum()) / T if T else 0.0
    return out


def initial_u(x: np.ndarray, share: np.ndarray, c: int) -> np.ndarray:
    n = len(x)
    order = sorted(range(n), key=lambda i: (x[i], i))
    tot = float(np.sum(share))
    U = np.zeros((n, c), np.float64)
    run = 0.0
    for i in order:
        mid = (run + share[i] / 2.0) / tot if tot > 0 else (order.index(i) + 0.5) / n
        k = min(int(mid * c), c - 1)
        U[i, k] = 1.0
        run += share[i]
    return U


def fcm(x: np.ndarray, U0: np.ndarray, m: float, eps: float, max_iter: int):
    """Alg. 1 on 1-D data.  Returns (V [c], U [n][c], rounds, objective
    history J_m after each round's center update)."""
    x = np.asarray(x, np.float64)
    U = np.array(U0, np.float64)
    n, c = U.shape
    V = np.zeros(c)
    hist = []
    rounds = 0
    while True:
        rounds += 1
        for k in range(c):
            w = U[:, k] ** m
            den = w.sum()
            V[k] = (w * x).sum() / den if den > 0 else 0.0
        hist.append(float(((U ** m) * (x[:, None] - V[None, :]) ** 2).sum()))
        Un = np.zeros_like(U)
        for i in range(n):
            d = np.abs(x[i] - V)
            zero = d == 0.0
            if zero.any():
                Un[i, zero] = 1.0 / zero.sum()
                continue
            for k in range(c):
                Un[i, k] = 1.0 / np.sum((d[k] / d) ** (2.0 / (m - 1.0)))
        delta = np.sqrt(((Un - U) ** 2).sum())
        U = Un
        if delta < eps or rounds >= max_iter:
            break
    return V, U, rounds, hist


def cluster_levels(V: np.ndarray, levels: Sequence[int]) -> np.ndarray:
    """Bit-width of each cluster: levels[0] (highest) to the largest center."""
    c = len(V)
    rank = sorted(range(c), key=lambda k: (-V[k], k))
    out = np.zeros(c, np.int32)
    for r, k in enumerate(rank):
        out[k] = levels[r]
    return out


def assign_bits(U: np.ndarray, cl_bits: np.ndarray, alpha: float) -> np.ndarray:
    n, c = U.shape
    bits = np.zeros(n, np.int32)
    for i in range(n):
        inside = [k for k in range(c) if U[i, k] >= alpha]
        if inside:
            bits[i] = min(int(cl_bits[k]) for k in inside)
        else:
            bits[i] = int(cl_bits[int(np.argmax(U[i]))])
    return bits


def allocate_bits(x: np.ndarray, share: np.ndarray, levels: Sequence[int], m: float = 2.0,
                  eps: float = 1e-9, max_iter: int = 300, alpha: float = 0.3) -> Dict:
    """Steps 2-4 for the experts' significance x and token share."""
    c = len(levels)
    U0 = initial_u(np.asarray(x, np.float64), np.asarray(share, np.float64), c)
    V, U, rounds, hist = fcm(x, U0, m, eps, max_iter)
    cl = cluster_levels(V, levels)
    return dict(bits=assign_bits(U, cl, alpha), V=V, U=U, rounds=rounds, hist=hist,
                cluster_bits=cl, U0=U0)
