"""Pins of the oracle's quantizer and packer (CPU only).

Quantizer (Sec. IV-A, uniform quantization at the expert's precision):
  Q0  the fp16 scale is the smallest binary16 >= s, checked against numpy's
      own float16 conversion stepped with nextafter (a different mechanism)
  Q1  closed-form bound |w - w_hat| <= s16/2 for every element, clamped or not
  Q2  exact recovery of groups built on a quantization grid
  Q3  consistency: rint(w_hat/s16) + z gives the code back
  Q4  b = 8, group = K is textbook per-channel asymmetric round-to-nearest
      int8, written independently in numpy
  Q5  degenerate group (all zero) -> scale 1, zero 0, codes 0; overflow status
Packer (Sec. V-B, codes packed into 32-bit words):
  P1  hand-worked words for each bit-width (6-bit: the two planes checked
      against the hand-worked 4-bit and 2-bit words)
  P2  unpack(pack(q)) == q and pack(unpack(w)) == w (bijection), sizes
"""
import numpy as np
import pytest

BITS = (2, 3, 4, 6, 8)


def np_fp16_round_up(s: float) -> np.float16:
    h = np.float16(s)
    if float(h) < s:
        h = np.nextafter(h, np.float16(np.inf))
    return h


def test_fp16_round_up_matches_numpy(orc):
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        10.0 ** rng.uniform(-9, 4.8, 20000),
        rng.uniform(0, 1e-4, 2000),            # subnormal binary16 range
        [2.0 ** -24, 2.0 ** -14, 1.0, 65504.0, 0.1, 1.0 / 3, 6.1e-5, 5.96e-8],
    ])
    for s in vals:
        want = np_fp16_round_up(float(s)).view(np.uint16)
        got = orc.fp16_round_up(float(s))
        assert got == int(want), (s, hex(got), hex(int(want)))
        assert orc.fp16_value(got) >= s
    assert orc.fp16_round_up(65504.5) == 0x7C00


def _groups(rng, n, g):
    """Value distributions with the edge cases of a quantizer."""
    out = [
        rng.standard_normal((n, g)) * 0.02,
        rng.uniform(0.1, 2.0, (n, g)),           # all positive: mn = 0
        -rng.uniform(0.1, 2.0, (n, g)),          # all negative: mx = 0
        rng.standard_normal((n, g)) * 1e-9,      # tiny: subnormal fp16 scales
        np.where(rng.random((n, g)) < 0.01, 50.0, 1.0) * rng.standard_normal((n, g)),
        np.full((n, g), 0.37),                   # constant group
        np.zeros((n, g)),
    ]
    return np.concatenate(out, 0).astype(np.float32)


@pytest.mark.parametrize("bits", BITS)
@pytest.mark.parametrize("group", (64, 128))
def test_q1_error_bound(orc, bits, group):
    if bits == 3 and group == 64:
        pytest.skip("3-bit is defined with group 128")
    rng = np.random.default_rng(bits * 1000 + group)
    w = _groups(rng, 40, group).reshape(-1, 2 * group)
    st, q, s16, z16 = orc.quantize(w, bits, group)
    assert st == 0
    qmax = (1 << bits) - 1
    assert q.max() <= qmax
    sf = s16.view(np.float16).astype(np.float64)
    zf = z16.view(np.float16).astype(np.float64)
    assert np.all(zf == np.rint(zf)) and zf.min() >= 0 and zf.max() <= qmax
    w_hat = orc.dequant(q, s16, z16, group)
    bound = np.repeat(sf, group, axis=1) / 2
    err = np.abs(w.astype(np.float64) - w_hat)
    assert np.all(err <= bound), float((err / bound).max())
    # exact zeros stay exact (the range always contains 0)
    zero = w == 0
    assert np.all(w_hat[zero] == 0)


@pytest.mark.parametrize("bits", BITS)
def test_q2_exact_recovery(orc, bits):
    rng = np.random.default_rng(7 + bits)
    group, R = 128, 64
    qmax = (1 << bits) - 1
    s = np.array([np_fp16_round_up(v) for v in 10.0 ** rng.uniform(-4, -1, R)],
                 dtype=np.float16)
    z = rng.integers(0, qmax + 1, R)
    q = rng.integers(0, qmax + 1, (R, group))
    q[:, 0] = 0
    q[:, 1] = qmax
    w = (s.astype(np.float64)[:, None] * (q - z[:, None])).astype(np.float32)
    assert np.all(w.astype(np.float64) == s.astype(np.float64)[:, None] * (q - z[:, None]))
    st, q2, s2, z2 = orc.quantize(w, bits, group)
    assert st == 0
    assert np.array_equal(q2, q)
    assert np.array_equal(s2[:, 0], s.view(np.uint16))
    assert np.array_equal(z2[:, 0].view(np.float16).astype(np.int64), z)


@pytest.mark.parametrize("bits", BITS)
def test_q3_code_consistency(orc, bits):
    rng = np.random.default_rng(11 + bits)
    w = (rng.standard_normal((32, 512)) * 0.02).astype(np.float32)
    st, q, s16, z16 = orc.quantize(w, bits, 128)
    w_hat = orc.dequant(q, s16, z16, 128)
    sf = np.repeat(s16.view(np.float16).astype(np.float64), 128, 1)
    zf = np.repeat(z16.view(np.float16).astype(np.float64), 128, 1)
    assert np.array_equal(np.rint(w_hat / sf) + zf, q.astype(np.float64))


def test_q4_per_channel_int8_is_textbook_rtn(orc):
    rng = np.random.default_rng(3)
    K = 256
    w = (rng.standard_normal((20, K)) * 0.05).astype(np.float32)
    w[3] = np.abs(w[3])
    st, q, s16, z16 = orc.quantize(w, 8, K)
    assert st == 0
    for r in range(w.shape[0]):
        x = w[r].astype(np.float64)
        lo, hi = min(0.0, x.min()), max(0.0, x.max())
        scale = np_fp16_round_up((hi - lo) / 255.0)
        zp = np.rint(-lo / float(scale))
        ref = np.clip(np.rint(x / float(scale)) + zp, 0, 255)
        assert s16[r, 0] == scale.view(np.uint16)
        assert float(z16[r:r + 1, 0].view(np.float16)[0]) == zp
        assert np.array_equal(q[r], ref.astype(np.uint8))


def test_q5_degenerate_and_overflow(orc):
    w = np.zeros((2, 128), np.float32)
    st, q, s16, z16 = orc.quantize(w, 4, 128)
    assert st == 0 and np.all(q == 0) and np.all(s16 == 0x3C00) and np.all(z16 == 0)
    w = np.zeros((1, 128), np.float32)
    w[0, 0] = 1e9
    st, *_ = orc.quantize(w, 2, 128)
    assert st == orc.ERR_RANGE
    st, *_ = orc.quantize(w, 5, 128)
    assert st == orc.ERR_BITS
    st, *_ = orc.quantize(w, 7, 128)
    assert st == orc.ERR_BITS


# ---------------------------------------------------------------------------
# packing
# ---------------------------------------------------------------------------
def test_p1_hand_worked_words(orc):
    # 4-bit: codes 0..7 -> even codes 0,2,4,6 in the low half, odd 1,3,5,7 high
    q = np.zeros((1, 32), np.uint8)
    q[0, :8] = np.arange(8)
    w = orc.pack(q, 4)
    assert w[0, 0] == 0x75316420 and np.all(w[0, 1:] == 0)
    # 2-bit: codes i % 4 for i = 0..15 -> low half fields 0,2,0,2,.. high 1,3,1,3,..
    q = (np.arange(32) % 4).astype(np.uint8).reshape(1, 32)
    w = orc.pack(q, 2)
    assert w[0, 0] == 0xDDDD8888
    # 8-bit: codes 10,20,30,40 -> bytes (c0, c2, c1, c3)
    q = np.zeros((1, 32), np.uint8)
    q[0, :4] = [10, 20, 30, 40]
    assert orc.pack(q, 8)[0, 0] == 0x28141E0A
    # 3-bit: code 5 = 7 (low bits 3 at field 2 of the high half of word 0,
    # bit 2 at bit 16+2 of word 2); code 20 = 6 (low bits 2 at field 2 of the
    # low half of word 1, bit 2 at bit 10 of word 2)
    q = np.zeros((1, 32), np.uint8)
    q[0, 5] = 7
    q[0, 20] = 6
    assert list(orc.pack(q, 3)[0]) == [0x00300000, 0x00000020, 0x00040400]
    # 6-bit: low four bits i % 8 and high two bits 0 (codes 0..15) or 3
    # (codes 16..31) -> four copies of the 4-bit word above, then 0 and all ones
    q = ((np.arange(32) % 8) + 48 * (np.arange(32) >= 16)).astype(np.uint8).reshape(1, 32)
    assert list(orc.pack(q, 6)[0]) == [0x75316420] * 4 + [0, 0xFFFFFFFF]
    # high two bits i % 4 -> both 2-bit words as in the 2-bit case above
    q = (16 * (np.arange(32) % 4)).astype(np.uint8).reshape(1, 32)
    assert list(orc.pack(q, 6)[0]) == [0] * 4 + [0xDDDD8888] * 2


@pytest.mark.parametrize("bits", BITS)
@pytest.mark.parametrize("K", (256, 1408, 2048, 4096))
def test_p2_round_trip(orc, bits, K):
    rng = np.random.default_rng(bits * K)
    qmax = (1 << bits) - 1
    q = rng.integers(0, qmax + 1, (5, K)).astype(np.uint8)
    q[0, :2] = (0, qmax)
    words = orc.pack(q, bits)
    assert words.shape == (5, K * bits // 32)
    assert words.nbytes == 5 * K * bits // 8
    assert np.array_equal(orc.unpack(words, K, bits), q)
    rw = rng.integers(0, 2 ** 32, (3, K * bits // 32), dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(orc.pack(orc.unpack(rw, K, bits), bits), rw)
