"""Oracle pins for the product-key search and softmax (CPU only)."""
import numpy as np
import pytest

import oracle
from tests import oracle_pins as pins


@pytest.mark.parametrize("seed", range(40))
def test_search_equals_brute_force_integer_ties(seed):
    # small integer entries: many exact ties at both levels
    rng = np.random.default_rng(seed)
    q, K, k = pins.rand_search_case(rng, integer=True)
    pins.check_search_vs_brute_force(oracle.search, oracle.brute_force_search, q, K, k)


@pytest.mark.parametrize("seed", range(20))
def test_search_equals_brute_force_float(seed):
    rng = np.random.default_rng(100 + seed)
    q, K, k = pins.rand_search_case(rng, integer=False)
    pins.check_search_vs_brute_force(oracle.search, oracle.brute_force_search, q, K, k)


def test_search_equals_brute_force_wider():
    rng = np.random.default_rng(7)
    q, K, k = pins.rand_search_case(rng, integer=True, S=12, d=6, H=2, k=9, T=6, lo=-4, hi=4)
    pins.check_search_vs_brute_force(oracle.search, oracle.brute_force_search, q, K, k)


def test_all_equal_subkeys_give_lowest_indices():
    pins.check_all_equal_subkeys(oracle.search)


def test_k1_is_argmax():
    pins.check_k1_argmax(oracle.search, np.random.default_rng(3))


def test_hand_example():
    pins.check_hand_example(oracle.search, oracle.bag_forward, oracle.bag_backward)


def test_softmax_pins():
    pins.check_softmax(oracle.softmax, np.random.default_rng(5))


def test_search_outputs_consistent():
    # idx and half_idx agree: idx = i1 * S + i2 with i1 among half 0's top-k,
    # i2 among half 1's; scores are the sums of the half scores.
    rng = np.random.default_rng(11)
    q, K, k = pins.rand_search_case(rng, integer=False, S=7, d=3, H=2, k=5, T=4)
    out = oracle.search(q, K, k)
    S = K.shape[2]
    for t in range(q.shape[0]):
        for h in range(q.shape[1]):
            for j in range(k):
                i1, i2 = divmod(int(out["idx"][t, h, j]), S)
                a = list(out["half_idx"][t, h, 0]).index(i1)
                b = list(out["half_idx"][t, h, 1]).index(i2)
                assert out["score"][t, h, j] == out["half_score"][t, h, 0, a] + out["half_score"][t, h, 1, b]
    assert np.all(np.diff(out["score"], axis=-1) <= 0)
    np.testing.assert_allclose(out["w"].sum(-1), 1.0, atol=1e-15)


@pytest.mark.parametrize("seed", range(3))
def test_search_backward_pins(seed):
    pins.check_search_backward(oracle.search, oracle.search_backward, np.random.default_rng(60 + seed))
