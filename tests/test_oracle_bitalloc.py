"""Pins of the oracle's offline bit allocation (Eq. (1), Alg. 1, cluster
precision and the low-precision-first boundary rule), CPU only.

  B1  Eq. (1) on a hand-worked routing (values computed by hand), and the
      invariant that the experts' significance adds up to K
  B2  token share and the initial U of a hand-worked case
  B3  textbook FCM properties: every membership row sums to one, the FCM
      objective never rises from round to round, a single cluster's center is
      numpy's mean, a crisp start gives numpy's per-group means as the first
      centers, tight separated groups converge to their means (m = 2)
  B4  hand case: four separated groups of experts get 8, 4, 3, 2 bits from
      the most to the least significant group, whatever the expert order
  B5  low-precision-first: an expert between two groups whose membership
      reaches alpha in both takes the lower precision; without the rule
      (alpha above every membership) it takes its larger membership
"""
import numpy as np
import pytest

from oracle import bitalloc as ba


def test_b1_eq1_hand_case():
    sig = np.array([1.0, 2.0, 3.0, 4.0])
    ids = np.array([[0, 1], [1, 2], [0, 2], [0, 1]])
    s = ba.expert_significance(sig, ids, 3)
    # expert 0: tokens 0, 2, 3 -> 8/10; expert 1: tokens 0, 1, 3 -> 7/10;
    # expert 2: tokens 1, 2 -> 5/10
    np.testing.assert_allclose(s, [0.8, 0.7, 0.5], rtol=0, atol=1e-15)
    rng = np.random.default_rng(0)
    T, E, K = 300, 16, 4
    ids = np.stack([rng.choice(E, K, replace=False) for _ in range(T)])
    sig = rng.exponential(size=T)
    s = ba.expert_significance(sig, ids, E)
    assert abs(s.sum() - K) < 1e-12
    assert (s >= 0).all() and (s <= 1).all()


def test_b2_share_and_initial_u():
    ids = np.array([[0, 1], [1, 2], [0, 2], [0, 1]])
    np.testing.assert_allclose(ba.token_share(ids, 3), [0.75, 0.75, 0.5])
    x = np.array([0.1, 0.9, 0.5, 0.3])
    U0 = ba.initial_u(x, np.full(4, 0.25), 4)
    # sorted by significance: experts 0, 3, 2, 1 take runs 0, 1, 2, 3
    np.testing.assert_array_equal(np.argmax(U0, 1), [0, 3, 2, 1])
    np.testing.assert_array_equal(U0.sum(1), np.ones(4))
    # a heavy expert spans the middle of the token share
    U0 = ba.initial_u(np.array([0.1, 0.2, 0.3]), np.array([0.1, 0.8, 0.1]), 4)
    np.testing.assert_array_equal(np.argmax(U0, 1), [0, 2, 3])


def _groups(rng, centers, per, spread):
    return np.concatenate([c + spread * rng.standard_normal(per) for c in centers])


@pytest.mark.parametrize("m", (1.5, 2.0, 3.0))
def test_b3_fcm_textbook(m):
    rng = np.random.default_rng(1)
    x = rng.random(40)
    U0 = ba.initial_u(x, rng.random(40) + 0.1, 4)
    V, U, rounds, hist = ba.fcm(x, U0, m, 1e-10, 500)
    np.testing.assert_allclose(U.sum(1), np.ones(40), atol=1e-12)
    assert (np.diff(hist) <= 1e-12 * max(hist[0], 1e-300)).all()
    # one round from a crisp start: centers are the per-group means
    V1, _, _, _ = ba.fcm(x, U0, m, 1e300, 1)
    for k in range(4):
        np.testing.assert_allclose(V1[k], np.mean(x[U0[:, k] == 1]), rtol=1e-13)
    # a single cluster: the plain mean
    V1c, U1c, _, _ = ba.fcm(x, np.ones((40, 1)), m, 1e-12, 50)
    np.testing.assert_allclose(V1c[0], np.mean(x), rtol=1e-13)
    np.testing.assert_array_equal(U1c, np.ones((40, 1)))


def test_b3_tight_groups_converge_to_means():
    rng = np.random.default_rng(2)
    cs = (0.05, 0.3, 0.6, 0.9)
    x = _groups(rng, cs, 10, 1e-3)
    res = ba.allocate_bits(x, np.full(40, 0.1), (8, 4, 3, 2))
    got = np.sort(res["V"])
    want = [np.mean(x[i * 10:(i + 1) * 10]) for i in range(4)]
    np.testing.assert_allclose(got, want, atol=2e-4)
    assert (res["U"].max(1) > 0.99).all()


def test_b4_hand_bits():
    x = np.array([0.60, 0.05, 0.90, 0.31, 0.62, 0.88, 0.06, 0.30])
    res = ba.allocate_bits(x, np.full(8, 0.25), (8, 4, 3, 2))
    np.testing.assert_array_equal(res["bits"], [4, 2, 8, 3, 4, 8, 2, 3])
    res = ba.allocate_bits(x, np.full(8, 0.25), (8, 6, 4, 2))
    np.testing.assert_array_equal(res["bits"], [6, 2, 8, 4, 6, 8, 2, 4])


def test_b5_low_precision_first():
    x = np.array([0.60, 0.05, 0.90, 0.31, 0.62, 0.88, 0.06, 0.30, 0.47])
    share = np.full(9, 0.2)
    res = ba.allocate_bits(x, share, (8, 4, 3, 2), alpha=0.3)
    u = res["U"][8]
    top2 = np.sort(u)[-2:]
    assert top2[0] >= 0.3, u            # in the region of both neighbours
    assert res["bits"][8] == 3          # the lower of 4 and 3 bits
    res = ba.allocate_bits(x, share, (8, 4, 3, 2), alpha=1.01)
    assert res["bits"][8] == 4          # its larger membership: the 0.6 group
    np.testing.assert_array_equal(res["bits"][:8], [4, 2, 8, 3, 4, 8, 2, 3])
