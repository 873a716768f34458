"""Pins of the oracle router: brute-force ranking, exact ties, softmax special cases."""
import itertools

import numpy as np
import pytest
from scipy.special import softmax

from oracle import router


def _brute_topk(z, k):
    return sorted(range(len(z)), key=lambda e: (-z[e], e))[:k]


def test_topk_matches_brute_force_on_random_logits():
    rng = np.random.default_rng(0)
    for trial in range(300):
        E = int(rng.integers(2, 20))
        k = int(rng.integers(1, E + 1))
        # few distinct values -> many exact ties
        z = rng.integers(-3, 4, size=(5, E)).astype(np.float64) * 0.5
        idx, w, gap = router.topk(z, k)
        for t in range(5):
            assert list(idx[t]) == _brute_topk(list(z[t]), k)
            assert abs(w[t].sum() - 1) < 1e-14


def test_hand_ties():
    z = np.array([[1.0, 3.0, 3.0, 2.0]])
    assert list(router.topk(z, 2)[0][0]) == [1, 2]
    assert list(router.topk(z, 1)[0][0]) == [1]
    assert list(router.topk(z, 3)[0][0]) == [1, 2, 3]
    assert router.topk(z, 2)[2][0] == 1.0     # gap between 3 (2nd) and 2 (3rd)
    assert router.topk(z, 1)[2][0] == 0.0     # exact tie at the boundary


def test_k_equals_all_is_full_softmax():
    rng = np.random.default_rng(1)
    z = rng.standard_normal((4, 9)) * 3
    idx, w, gap = router.topk(z, 9)
    for t in range(4):
        full = softmax(z[t])
        np.testing.assert_allclose(w[t], full[idx[t]], rtol=1e-14, atol=1e-16)
        assert np.isinf(gap[t])


def test_k1_weight_is_one_and_renormalisation():
    rng = np.random.default_rng(2)
    z = rng.standard_normal((6, 12))
    idx, w, _ = router.topk(z, 1)
    np.testing.assert_array_equal(w, 1.0)
    idx, w, _ = router.topk(z, 4)
    for t in range(6):
        p = softmax(z[t])
        np.testing.assert_allclose(w[t], p[idx[t]] / p[idx[t]].sum(), rtol=1e-13)


def test_logits_exact_on_integer_inputs():
    rng = np.random.default_rng(3)
    x = rng.integers(-50, 50, size=(3, 16)).astype(np.float32)
    wr = rng.integers(-50, 50, size=(16, 5)).astype(np.float32)
    z = router.logits(x, wr)
    for t, e in itertools.product(range(3), range(5)):
        assert z[t, e] == sum(int(x[t, i]) * int(wr[i, e]) for i in range(16))


@pytest.mark.parametrize("E,k", [(16, 2), (128, 8)])
def test_weights_order_descending(E, k):
    rng = np.random.default_rng(E)
    z = rng.standard_normal((10, E))
    idx, w, gap = router.topk(z, k)
    assert np.all(np.diff(w, axis=1) <= 0)
    assert np.all(gap >= 0)
