"""Seeded synthetic inputs for the MoE-layer workloads.

This module holds no arithmetic of the method: it draws random numbers and
does the bookkeeping of shapes, bit-width assignment, copy pools and switch
masks.  Both the GPU library (through its Python binding) and the CPU oracle
consume the arrays it returns; neither is imported here.

Every draw comes from ``numpy.random.default_rng([seed, cfg_id, stream])``
with a fixed stream number per array, so any single expert matrix, mask or
activation batch can be regenerated on its own.

Stream numbers:
    0                      router weights
    1                      permutation assigning bit-widths to experts
    2                      activations (x) of the default batch
    3                      outlier input columns
    100 + 3*e + kind       expert e's weight matrix of that kind (row chunk c
                           of 256 rows draws from [seed, cfg_id, stream, c])
    1000 + 3*e + kind      copy pool / switch mask rows of (e, kind)
    3000 + epoch           switched fraction of a mask epoch (pool mode)
    4000 + 1000*epoch + 3*e + kind   rows of (e, kind) switched in that epoch
    5000 + step            activations of step `step` (stress workload)
    6000 + dataset         permutation assigning bit-widths for a new dataset
    7000 + dataset         per-token significance and activations of a
                           dataset's calibration batch
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
from concurrent.futures import ThreadPoolExecutor

CHUNK = 256
KIND_GATE, KIND_UP, KIND_DOWN = 0, 1, 2
KINDS = (KIND_GATE, KIND_UP, KIND_DOWN)


@dataclass(frozen=True)
class LayerConfig:
    """Shapes and quantization recipe of one synthetic MoE layer."""

    name: str
    cfg_id: int                 # seed stream id of the layer's weights
    d_model: int
    n_experts: int              # routed experts E
    n_shared: int               # shared experts S (8-bit, never switched)
    top_k: int
    d_ff: int
    d_ff_shared: int
    group: int
    bits_literal: Optional[Tuple[int, ...]] = None   # per routed expert
    bit_shares: Optional[Tuple[Tuple[int, float], ...]] = None
    copies: str = "mask"        # 'all' | 'mask' | 'pool' | 'none'
    mask_frac: float = 0.05     # switched fraction ('all', 'mask')
    pool_frac: float = 0.10     # copy-pool fraction ('pool')
    outliers: int = 0           # input columns scaled x20
    weight_std: float = 0.02
    shared_bits: int = 8        # bit-width of the shared experts

    def rows(self, kind: int, expert: int) -> int:
        f = self.d_ff if expert < self.n_experts else self.d_ff_shared
        return self.d_model if kind == KIND_DOWN else f

    def cols(self, kind: int, expert: int) -> int:
        f = self.d_ff if expert < self.n_experts else self.d_ff_shared
        return f if kind == KIND_DOWN else self.d_model


@dataclass(frozen=True)
class Workload:
    """A batch shape on a layer: T tokens, optional Zipf-skewed router."""

    name: str
    layer: LayerConfig
    tokens: int
    zipf_s: Optional[float] = None
    steps: int = 1              # stress workload: steps per run
    redraw_every: int = 0       # stress workload: steps per mask epoch


TINY = LayerConfig(
    name="tiny", cfg_id=0, d_model=256, n_experts=8, n_shared=0, top_k=2,
    d_ff=512, d_ff_shared=0, group=64, bits_literal=(8, 8, 4, 4, 4, 4, 2, 2),
    copies="all", mask_frac=0.10, outliers=4)

# The small layer again with group 128 and every bit-width of the paper's
# precision set (INT2/4/6/8) plus 3-bit.
TINY6 = LayerConfig(
    name="tiny-int6", cfg_id=5, d_model=256, n_experts=8, n_shared=1, top_k=2,
    d_ff=512, d_ff_shared=256, group=128, bits_literal=(8, 6, 6, 4, 6, 3, 2, 6),
    copies="all", mask_frac=0.10, outliers=4)

MIXTRAL = LayerConfig(
    name="mixtral-8x7b", cfg_id=1, d_model=4096, n_experts=8, n_shared=0,
    top_k=2, d_ff=14336, d_ff_shared=0, group=128,
    bit_shares=((8, 0.25), (4, 0.50), (2, 0.25)), copies="mask",
    mask_frac=0.05, outliers=41)

DEEPSEEK = LayerConfig(
    name="deepseekmoe-16b", cfg_id=3, d_model=2048, n_experts=64, n_shared=2,
    top_k=6, d_ff=1408, d_ff_shared=1408, group=128,
    bit_shares=((8, 0.20), (4, 0.50), (3, 0.15), (2, 0.15)), copies="mask",
    mask_frac=0.05, outliers=20)

# Bits and group of this layer are not given by the workload description; the
# DeepSeekMoE-shaped layer's distribution and group 128 are used.
QWEN = LayerConfig(
    name="qwen1.5-moe-a2.7b", cfg_id=4, d_model=2048, n_experts=60,
    n_shared=1, top_k=4, d_ff=1408, d_ff_shared=5632, group=128,
    bit_shares=((8, 0.20), (4, 0.50), (3, 0.15), (2, 0.15)), copies="pool",
    pool_frac=0.10, outliers=20)

def unquantized(cfg: LayerConfig) -> LayerConfig:
    """The same layer (same seeded fp32 weights, router and activations)
    with every expert, routed and shared, kept at 16 bits: the bf16 values of
    the fp32 weights, no channel copies.  The reference for the speedup of
    the packed low-bit weights over a 16-bit model (Sec. VI-C).  Group 64:
    the library runs 16-bit experts in its group-64 kernels."""
    import dataclasses
    return dataclasses.replace(cfg, name=cfg.name + "-bf16", group=64, copies="none",
                               bits_literal=(16,) * cfg.n_experts, bit_shares=None,
                               shared_bits=16)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", TINY, 16),
    "tiny-int6": Workload("tiny-int6", TINY6, 16),
    "mixtral-decode": Workload("mixtral-decode", MIXTRAL, 64),
    "mixtral-prefill": Workload("mixtral-prefill", MIXTRAL, 4096, zipf_s=1.1),
    "deepseek-decode": Workload("deepseek-decode", DEEPSEEK, 128),
    "deepseek-prefill": Workload("deepseek-prefill", DEEPSEEK, 8192),
    "qwen-stress": Workload("qwen-stress", QWEN, 512, steps=200,
                            redraw_every=10),
}


def rng(seed: int, cfg_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([seed, cfg_id, stream])


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_values(b: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> fp32 values (exact)."""
    return (b.astype(np.uint32) << 16).view(np.float32)


def bit_counts(shares: Sequence[Tuple[int, float]], n: int) -> Dict[int, int]:
    """Largest-remainder rounding of share*n per bit-width; equal remainders
    go to the lower bit-width first."""
    raw = {b: p * n for b, p in shares}
    cnt = {b: int(np.floor(v + 1e-9)) for b, v in raw.items()}
    left = n - sum(cnt.values())
    order = sorted(raw, key=lambda b: (-(round(raw[b] - cnt[b], 9)), b))
    for b in order[:left]:
        cnt[b] += 1
    return cnt


class LayerInputs:
    """Weights, bit-widths, copy pools and masks of one synthetic layer."""

    def __init__(self, cfg: LayerConfig, seed: int = 0):
        self.cfg = cfg
        self.seed = seed
        E, S = cfg.n_experts, cfg.n_shared
        if cfg.bits_literal is not None:
            routed = np.asarray(cfg.bits_literal, dtype=np.int32)
        else:
            routed = self._assign_bits(1)
        self.bits = np.concatenate([routed, np.full(S, cfg.shared_bits, np.int32)])
        self.router = (rng(seed, cfg.cfg_id, 0)
                       .standard_normal((E, cfg.d_model), dtype=np.float32)
                       * np.float32(cfg.weight_std))
        self._pool: Dict[int, np.ndarray] = {}
        for kind in KINDS:
            self._pool[kind] = self._make_pool(kind)
        self._cache16: Dict[int, np.ndarray] = {}

    def _assign_bits(self, stream: int) -> np.ndarray:
        cfg = self.cfg
        E = cfg.n_experts
        cnt = bit_counts(cfg.bit_shares, E)
        seq: List[int] = []
        for b in sorted(cnt, reverse=True):
            seq += [b] * cnt[b]
        perm = rng(self.seed, cfg.cfg_id, stream).permutation(E)
        out = np.empty(E, dtype=np.int32)
        out[perm] = np.asarray(seq, dtype=np.int32)
        return out

    def dataset_bits(self, dataset: int) -> np.ndarray:
        """Per-routed-expert bit-widths for a new dataset: the same shares of
        bit-widths as the layer's own assignment, handed to a fresh seeded
        permutation of the experts (a stand-in for the clustering of the new
        dataset's expert significance).  Layers with a literal assignment
        rotate it by dataset + 1 positions."""
        cfg = self.cfg
        if cfg.bits_literal is not None:
            lit = np.asarray(cfg.bits_literal, dtype=np.int32)
            return np.roll(lit, dataset + 1)
        return self._assign_bits(6000 + dataset)

    # ---- weights -------------------------------------------------------
    def weight(self, expert: int, kind: int) -> np.ndarray:
        """fp32 [R][K] ~ N(0, weight_std^2), drawn in 256-row chunks."""
        c = self.cfg
        R, K = c.rows(kind, expert), c.cols(kind, expert)
        out = np.empty((R, K), np.float32)
        stream = 100 + 3 * expert + kind

        def draw(ci: int) -> None:
            g = np.random.default_rng([self.seed, c.cfg_id, stream, ci])
            g.standard_normal(out=out[ci * CHUNK:(ci + 1) * CHUNK], dtype=np.float32)

        n = (R + CHUNK - 1) // CHUNK
        if n > 1:
            with ThreadPoolExecutor(min(8, n)) as ex:
                list(ex.map(draw, range(n)))
        else:
            draw(0)
        out *= np.float32(c.weight_std)
        return out

    # ---- copy pools and masks ------------------------------------------
    def _rows_drawn(self, kind: int, e: int, frac: float) -> np.ndarray:
        R = self.cfg.rows(kind, e)
        n = int(round(frac * R))
        g = rng(self.seed, self.cfg.cfg_id, 1000 + 3 * e + kind)
        return np.sort(g.choice(R, size=n, replace=False)).astype(np.int32)

    def _make_pool(self, kind: int) -> np.ndarray:
        """Copy headers (expert, row) of one kind, expert-major, rows ascending."""
        c = self.cfg
        hdr = []
        for e in range(c.n_experts if c.copies != "none" else 0):
            R = c.rows(kind, e)
            if c.copies == "all":
                rows = np.arange(R, dtype=np.int32)
            elif c.copies == "mask":
                rows = self._rows_drawn(kind, e, c.mask_frac)
            else:
                rows = self._rows_drawn(kind, e, c.pool_frac)
            hdr.append(np.stack([np.full(len(rows), e, np.int32), rows], 1))
        if not hdr:
            return np.zeros((0, 2), np.int32)
        return np.ascontiguousarray(np.concatenate(hdr, 0).astype(np.int32))

    def copy_headers(self, kind: int) -> np.ndarray:
        return self._pool[kind]

    def channel_cache(self, kind: int) -> np.ndarray:
        """The retained original 16-bit channels of the copy pool of one kind,
        in slot order: binary16 bit patterns uint16 [n_slots][K].  The fp32
        weights stand in for a checkpoint; their binary16 values (round to
        nearest even) stand in for its 16-bit channels."""
        if kind in self._cache16:
            return self._cache16[kind]
        hdr = self._pool[kind]
        K = self.cfg.cols(kind, 0)
        out = np.empty((len(hdr), K), np.float16)
        for e in np.unique(hdr[:, 0]):
            sl = np.nonzero(hdr[:, 0] == e)[0]
            out[sl] = self.weight(int(e), kind)[hdr[sl, 1]].astype(np.float16)
        self._cache16[kind] = out.view(np.uint16)
        return self._cache16[kind]

    def slots_on(self, kind: int, epoch: int = 0) -> np.ndarray:
        """Slots of the copy pool switched on in a mask epoch."""
        c = self.cfg
        hdr = self._pool[kind]
        if c.copies in ("mask", "none"):
            return np.arange(len(hdr), dtype=np.int32)
        if c.copies == "all":
            out = []
            base = 0
            for e in range(c.n_experts):
                R = c.rows(kind, e)
                rows = self._rows_drawn(kind, e, c.mask_frac)
                out.append(base + rows)
                base += R
            return np.concatenate(out).astype(np.int32)
        pct = int(rng(self.seed, c.cfg_id, 3000 + epoch).integers(2, 11))
        out = []
        base = 0
        for e in range(c.n_experts):
            n_pool = int(np.sum(hdr[:, 0] == e))
            R = c.rows(kind, e)
            n = min(n_pool, int(round(pct / 100.0 * R)))
            g = rng(self.seed, c.cfg_id, 4000 + 1000 * epoch + 3 * e + kind)
            out.append(base + np.sort(g.choice(n_pool, size=n, replace=False)))
            base += n_pool
        return np.concatenate(out).astype(np.int32)

    def switch_percent(self, epoch: int) -> int:
        if self.cfg.copies == "none":
            return 0
        if self.cfg.copies != "pool":
            return int(round(self.cfg.mask_frac * 100))
        return int(rng(self.seed, self.cfg.cfg_id, 3000 + epoch).integers(2, 11))


def calibration_batch(cfg: LayerConfig, dataset: int, T: int = 1024, seed: int = 0):
    """A dataset's calibration batch: bf16 activations [T][d_model] and a
    per-token significance (exponential, mean 1) standing in for the channel
    significance a trained model would give on real text."""
    x = make_x(cfg, T, seed, 7000 + dataset)
    sig = rng(seed, cfg.cfg_id, 7500 + dataset).exponential(size=T).astype(np.float32)
    return x, sig


def make_x(cfg: LayerConfig, T: int, seed: int = 0, stream: int = 2) -> np.ndarray:
    """Activations: N(0,1) fp32, a seeded set of outlier columns x20, rounded
    to bfloat16.  Returns bf16 bit patterns [T][d_model]."""
    x = rng(seed, cfg.cfg_id, stream).standard_normal((T, cfg.d_model),
                                                      dtype=np.float32)
    if cfg.outliers:
        cols = rng(seed, cfg.cfg_id, 3).choice(cfg.d_model, size=cfg.outliers,
                                               replace=False)
        x[:, cols] *= np.float32(20.0)
    return bf16_bits(x)


def zipf_targets(E: int, s: float) -> np.ndarray:
    w = (np.arange(E) + 1.0) ** (-s)
    return w / w.sum()


def zipf_router_bias(router: np.ndarray, x_bits: np.ndarray, k: int, s: float,
                     iters: int = 20) -> np.ndarray:
    """Router bias that skews expert loads toward Zipf(s) over expert index.

    Input shaping only: loads are estimated with a float64 top-k of x W^T + b,
    and b_e is moved by log(target_e / load_e) for a fixed number of rounds.
    The realised loads are whatever the router under test computes.
    """
    E = router.shape[0]
    xf = bf16_values(x_bits).astype(np.float64)
    base = xf @ router.astype(np.float64).T
    tgt = zipf_targets(E, s)
    b = np.zeros(E)
    for _ in range(iters):
        lg = base + b
        top = np.argsort(-lg, axis=1, kind="stable")[:, :k]
        load = np.bincount(top.ravel(), minlength=E) / top.size
        b = b + np.log(tgt / np.maximum(load, 1e-6))
    return b.astype(np.float32)


@dataclass
class Batch:
    x: np.ndarray                 # bf16 bits [T][d]
    bias: Optional[np.ndarray]    # fp32 [E] or None


def make_batch(work: Workload, layer: LayerInputs, step: Optional[int] = None) -> Batch:
    cfg = work.layer
    stream = 2 if step is None else 5000 + step
    x = make_x(cfg, work.tokens, layer.seed, stream)
    bias = None
    if work.zipf_s is not None:
        bias = zipf_router_bias(layer.router, x, cfg.top_k, work.zipf_s)
    return Batch(x=x, bias=bias)
