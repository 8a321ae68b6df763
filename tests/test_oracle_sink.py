"""Oracle pins for the fixed (sink) key-value pair beside the selection
(Sec. 5.4): its key scored like any key, its value a row of the table."""
import numpy as np

import oracle
from tests import oracle_pins as pins


def test_search_sink_pins():
    for s in range(3):
        pins.check_search_sink(oracle.search_sink, oracle.search_extra, np.random.default_rng(150 + s))


def test_search_backward_sink_pins():
    for s in range(3):
        pins.check_search_backward_sink(oracle.search_sink, oracle.search_backward_sink,
                                        np.random.default_rng(160 + s))


def test_sink_value_row_through_the_plain_bag():
    """The sink's value is a table row: the bag forward adds w_sink * V[row]
    and the bag backward adds w_sink * dy into that row (dense A.T @ dy)."""
    rng = np.random.default_rng(170)
    T, H, S, d, k, D = 6, 2, 4, 2, 2, 5
    q = rng.standard_normal((T, H, 2 * d))
    K = rng.standard_normal((H, 2, S, d))
    ks = rng.standard_normal((H, 2 * d))
    N = S * S + H
    V = rng.standard_normal((N, D))
    out = oracle.search_sink(q, K, k, np.zeros((T, H, 0), dtype=np.int64), ks, S * S)
    kk = k + 1
    y = oracle.bag_forward(V, out["idx"].reshape(T, -1), out["w"].reshape(T, -1))
    A = np.zeros((T, N))
    for t in range(T):
        for h in range(H):
            for j in range(kk):
                A[t, out["idx"][t, h, j]] += out["w"][t, h, j]
    np.testing.assert_allclose(y, A @ V, rtol=1e-12)
    dy = rng.standard_normal((T, D))
    b = oracle.bag_backward(dy, V, out["idx"], out["w"], H, kk)
    np.testing.assert_allclose(b["grad_values"], A.T @ dy, rtol=1e-12, atol=1e-14)
