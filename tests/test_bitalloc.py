"""The library's offline bit allocation (host C++: Eq. (1), Alg. 1, cluster
precision, low-precision-first) against the oracle, on the CPU.

Eq. (1) adds each expert's tokens in the same ascending order on both sides,
so the significance and token share agree bit for bit.  The fuzzy c-means
sums run in a different order (numpy's pairwise sums in the oracle), so
centers and memberships agree to 1e-9 and the bit-widths exactly; the inputs
keep every expert's memberships at least 1e-6 away from alpha.
"""
import numpy as np
import pytest

from oracle import bitalloc as ba


@pytest.fixture(scope="module")
def api():
    from paper_2503_21135_amd import _lib, api as A
    import os
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2503_21135_amd import build
        build.build()
    return A


def _routing(rng, T, E, k, zipf):
    w = (np.arange(E) + 1.0) ** (-zipf)
    w = w[rng.permutation(E)]
    w /= w.sum()
    ids = np.stack([rng.choice(E, k, replace=False, p=w) for _ in range(T)]).astype(np.int32)
    sig = rng.exponential(size=T).astype(np.float32)
    return sig, ids


@pytest.mark.parametrize("T,E,k", [(1, 4, 1), (512, 8, 2), (2048, 64, 6), (1024, 60, 4),
                                   (4096, 256, 8)])
def test_significance_bitexact(api, T, E, k):
    rng = np.random.default_rng(T + E)
    sig, ids = _routing(rng, T, E, k, 1.0)
    s, sh = api.moe_expert_significance(sig, ids, E)
    np.testing.assert_array_equal(s, ba.expert_significance(sig, ids, E))
    np.testing.assert_array_equal(sh, ba.token_share(ids, E))


def test_significance_validation(api):
    from paper_2503_21135_amd._lib import MoEError
    ids = np.array([[0, 1], [1, 2]], np.int32)
    with pytest.raises(MoEError):
        api.moe_expert_significance(np.array([1.0, -1.0]), ids, 3)
    with pytest.raises(MoEError):
        api.moe_expert_significance(np.array([1.0, 1.0]), ids, 2)   # id 2 >= E
    s, sh = api.moe_expert_significance(np.zeros(0, np.float32), np.zeros((0, 2), np.int32), 3)
    assert not s.any() and not sh.any()


def _compare(api, x, share, levels, m, alpha):
    got = api.moe_allocate_bits(x, share, levels, m=m, alpha=alpha)
    want = ba.allocate_bits(x, share, levels, m=m, alpha=alpha)
    np.testing.assert_allclose(got["V"], want["V"], rtol=0, atol=1e-9)
    np.testing.assert_allclose(got["U"], want["U"], rtol=0, atol=1e-9)
    assert abs(got["rounds"] - want["rounds"]) <= 1
    assert np.abs(want["U"] - alpha).min() > 1e-6
    np.testing.assert_array_equal(got["bits"], want["bits"])
    return got


@pytest.mark.parametrize("E,k,m,levels", [(8, 2, 2.0, (8, 4, 3, 2)), (64, 6, 2.0, (8, 4, 3, 2)),
                                          (60, 4, 1.7, (8, 6, 4, 2)), (256, 8, 2.5, (8, 4, 3, 2))])
def test_allocate_bits_matches_oracle(api, E, k, m, levels):
    rng = np.random.default_rng(E)
    sig, ids = _routing(rng, 4 * E * 8, E, k, 1.1)
    s, sh = api.moe_expert_significance(sig, ids, E)
    got = _compare(api, s, sh, levels, m, 0.3)
    print(E, "experts, bits", np.bincount(got["bits"], minlength=9)[[2, 3, 4, 6, 8]],
          "rounds", got["rounds"])


def test_allocate_bits_hand_cases(api):
    x = np.array([0.60, 0.05, 0.90, 0.31, 0.62, 0.88, 0.06, 0.30, 0.47])
    sh = np.full(9, 0.2)
    np.testing.assert_array_equal(api.moe_allocate_bits(x, sh, alpha=0.3)["bits"],
                                  [4, 2, 8, 3, 4, 8, 2, 3, 3])
    np.testing.assert_array_equal(api.moe_allocate_bits(x, sh, alpha=1.01)["bits"],
                                  [4, 2, 8, 3, 4, 8, 2, 3, 4])
    # coinciding experts and a zero token share everywhere
    x = np.array([0.2, 0.2, 0.2, 0.8])
    got = api.moe_allocate_bits(x, np.zeros(4), (8, 2), m=2.0)
    want = ba.allocate_bits(x, np.zeros(4), (8, 2), m=2.0)
    np.testing.assert_array_equal(got["bits"], want["bits"])
    np.testing.assert_array_equal(got["bits"], [2, 2, 2, 8])


def test_allocate_bits_validation(api):
    from paper_2503_21135_amd._lib import MoEError
    x, sh = np.array([0.1, 0.2]), np.array([0.5, 0.5])
    for kw in (dict(m=1.0), dict(eps=0.0), dict(max_iter=0), dict(levels=(8, 9))):
        with pytest.raises(MoEError):
            api.moe_allocate_bits(x, sh, **kw)
    with pytest.raises(MoEError):
        api.moe_allocate_bits(x, np.array([0.5, -0.1]))
