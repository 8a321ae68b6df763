"""Oracle pins for the weighted EmbeddingBag forward and backward (CPU only)."""
import numpy as np
import pytest

import oracle
from tests import oracle_pins as pins


@pytest.mark.parametrize("seed", range(3))
def test_bag_forward_vs_torch_embedding_bag(seed):
    pins.check_bag_forward(oracle.bag_forward, np.random.default_rng(seed))


@pytest.mark.parametrize("seed", range(3))
def test_bag_backward_vs_autograd(seed):
    pins.check_bag_backward(oracle.bag_backward, np.random.default_rng(10 + seed))


def test_bag_backward_finite_differences():
    pins.check_bag_backward_fd(oracle.bag_forward, oracle.bag_backward, np.random.default_rng(21))


def test_grad_values_accumulate():
    pins.check_accumulate(oracle.bag_backward, np.random.default_rng(31))


def test_rows_form_matches_dense():
    V, idx, z, w, dy = pins.random_bag_case(np.random.default_rng(41))
    T, H, k = idx.shape
    dense = oracle.bag_backward(dy, V, idx, w, H, k)["grad_values"]
    rows = oracle.bag_backward_rows(dy, V, idx, w, H, k)
    assert list(rows["rows"]) == sorted(set(idx.ravel().tolist()))
    np.testing.assert_array_equal(dense[rows["rows"]], rows["grad_rows"])
    untouched = np.setdiff1d(np.arange(V.shape[0]), rows["rows"])
    assert np.all(dense[untouched] == 0)


def test_invert_index_invariants():
    rng = np.random.default_rng(51)
    idx = rng.integers(0, 20, size=300)
    inv = oracle.invert_index(idx)
    assert inv["row_ptr"][-1] == idx.size
    assert np.all(np.diff(inv["rows"]) > 0)
    pairs = []
    for u, r in enumerate(inv["rows"]):
        seg = inv["lookups"][inv["row_ptr"][u]:inv["row_ptr"][u + 1]]
        assert len(seg) > 0 and np.all(np.diff(seg) > 0)
        assert np.all(idx[seg] == r)
        pairs += [(int(r), int(l)) for l in seg]
    assert sorted(pairs) == sorted((int(r), l) for l, r in enumerate(idx))
