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
    pins.check_rows_form(oracle.bag_backward, oracle.bag_backward_rows, np.random.default_rng(41))


def test_invert_index_invariants():
    pins.check_invert_index(oracle.invert_index, np.random.default_rng(51))
