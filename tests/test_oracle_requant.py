"""Pins of the oracle's requantization of cached channels for a new dataset
(Sec. IV-B "Channel Weights Requantization for New Datasets"), CPU only.

  R1  exact recovery: cached binary16 channels built on a b-bit grid with a
      power-of-two scale come back with exactly the planted codes, scale and
      zero when their expert's new precision is b; experts given 0 are left
      out, and each slot's bit-width follows the expert column of its header
  R2  closed-form bound |fp16(w) - w_hat| <= s16/2 at every new precision,
      and a higher new precision never has a larger worst error per group than
      a lower one on the same channels -- the precision may move either way
  R3  forward wiring: on a layer whose weights are binary16-exact grids,
      switching rows to copies requantized at their own expert's bit-width
      gives bit for bit the unswitched layer output, while 8-bit copies of the
      same cache rows do not (the copy precision and the slot-to-cache-row
      mapping are both used)
  R4  channel_cache holds the binary16 values of the header-named rows
"""
import numpy as np
import pytest

import moe_inputs as mi
from _layers import Pow2GridLayer


def _grid_rows(rng, n, K, group, bits):
    qmax = (1 << bits) - 1
    G = K // group
    s = 2.0 ** rng.integers(-10, -4, (n, G))
    z = rng.integers(0, qmax + 1, (n, G))
    q = rng.integers(0, qmax + 1, (n, G, group))
    q[:, :, 0] = 0
    q[:, :, 1] = qmax
    w = s[:, :, None] * (q - z[:, :, None])
    return (w.reshape(n, K).astype(np.float16).view(np.uint16),
            q.reshape(n, K).astype(np.uint8), s, z)


@pytest.mark.parametrize("group", (64, 128))
def test_r1_exact_recovery_per_expert(orc, group):
    rng = np.random.default_rng(11)
    K = 256
    # experts 0, 1, 2 -> new precisions 4, 0 (left out), 2; expert 3 -> 8
    eb = np.array([4, 0, 2, 8], np.int32)
    hdr = np.array([[0, 5], [0, 9], [1, 3], [2, 0], [2, 7], [3, 1], [0, 2]], np.int32)
    n = len(hdr)
    cache = np.zeros((n, K), np.uint16)
    want_q = np.zeros((n, K), np.uint8)
    want_s = np.zeros((n, K // group))
    want_z = np.zeros((n, K // group), np.int64)
    for i, (e, _) in enumerate(hdr):
        b = int(eb[e]) or 3  # the left-out row is on some other grid
        c, q, s, z = _grid_rows(rng, 1, K, group, b)
        cache[i], want_q[i], want_s[i], want_z[i] = c[0], q[0], s[0], z[0]
    st, touched, q, s16, z16 = orc.requant_channels(cache, hdr, eb, group)
    assert st == orc.OK
    np.testing.assert_array_equal(touched, eb[hdr[:, 0]] > 0)
    t = touched
    np.testing.assert_array_equal(q[t], want_q[t])
    np.testing.assert_array_equal(s16[t].view(np.float16).astype(np.float64), want_s[t])
    np.testing.assert_array_equal(z16[t].view(np.float16).astype(np.int64), want_z[t])
    assert not q[~t].any() and not s16[~t].any()
    # a header read by its row column instead of its expert column would pick
    # other precisions for these slots
    assert (eb[hdr[:, 1] % len(eb)] != eb[hdr[:, 0]]).any()


def test_r2_error_bound_both_directions(orc):
    rng = np.random.default_rng(12)
    K, group, n = 512, 128, 40
    w = (rng.standard_normal((n, K)) * 0.02).astype(np.float16)
    cache = w.view(np.uint16)
    hdr = np.stack([np.zeros(n, np.int32), np.arange(n, dtype=np.int32)], 1)
    wf = w.astype(np.float64).reshape(n, K // group, group)
    worst = {}
    for b in (2, 3, 4, 8):
        st, touched, q, s16, z16 = orc.requant_channels(cache, hdr, np.array([b]), group)
        assert st == orc.OK and touched.all()
        what = orc.dequant(q, s16, z16, group).reshape(n, K // group, group)
        s = s16.view(np.float16).astype(np.float64)[:, :, None]
        err = np.abs(wf - what)
        assert (err <= s / 2 * (1 + 1e-12)).all(), b
        worst[b] = err.max(axis=2)
    for lo, hi in ((2, 3), (3, 4), (4, 8)):
        assert (worst[hi] <= worst[lo] + 1e-12).all(), (lo, hi)
        assert worst[hi].mean() < 0.6 * worst[lo].mean()


def _tiny_grid():
    return Pow2GridLayer(mi.TINY, seed=3)


def test_r4_channel_cache_rows(orc):
    L = mi.LayerInputs(mi.TINY, seed=1)
    for kind in mi.KINDS:
        hdr = L.copy_headers(kind)
        cache = L.channel_cache(kind)
        assert cache.shape == (len(hdr), mi.TINY.cols(kind, 0)) and cache.dtype == np.uint16
        for s in (0, len(hdr) // 2, len(hdr) - 1):
            e, r = hdr[s]
            want = L.weight(int(e), kind)[r].astype(np.float16).view(np.uint16)
            np.testing.assert_array_equal(cache[s], want)


def test_r3_forward_reads_requantized_cache(orc):
    L = _tiny_grid()
    x = mi.make_x(L.cfg, 16, seed=3)
    base = orc.layer_forward(L, x)
    rs = orc.switch_state(L)
    assert any((rs[k] >= 0).any() for k in rs)
    own = {k: L.bits[:L.cfg.n_experts].copy() for k in mi.KINDS}
    same = orc.layer_forward(L, x, row_slot=rs, copy_bits=own)
    np.testing.assert_array_equal(same["y"], base["y"])
    eight = {k: np.full(L.cfg.n_experts, 8, np.int32) for k in mi.KINDS}
    other = orc.layer_forward(L, x, row_slot=rs, copy_bits=eight)
    assert np.abs(other["y"] - base["y"]).max() > 0
    # 8-bit copies of the 16-bit cache are not the 8-bit copies of the fp32
    # rows only where rounding to binary16 moved a weight; on this layer the
    # weights are binary16-exact, so the two copy sources agree
    orig = orc.layer_forward(L, x, row_slot=rs)
    np.testing.assert_array_equal(other["y"], orig["y"])
