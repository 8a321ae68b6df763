"""Oracle pins for the Memory+ gating (Sec. 3.1.4): out = y * silu(x^T W1)."""
import numpy as np

import oracle
from tests import oracle_pins as pins


def test_gated_output_pins():
    pins.check_gated_output(oracle.gated_output, oracle.silu, np.random.default_rng(71))


def test_gated_backward_pins():
    pins.check_gated_backward(oracle.gated_backward, np.random.default_rng(72))


def test_gated_chain_through_the_bag():
    """The gated output's dy feeds the bag backward: the value gradient of
    L = sum(d_out * gated(bag(V))) equals bag_backward(dy = gated_backward.dy)
    (central differences in one value entry)."""
    rng = np.random.default_rng(73)
    N, D, T, H, k = 9, 5, 3, 2, 2
    V = rng.standard_normal((N, D))
    idx = rng.integers(0, N, size=(T, H, k))
    w = rng.random((T, H, k))
    g = rng.standard_normal((T, D))
    d = rng.standard_normal((T, D))
    y = oracle.bag_forward(V, idx.reshape(T, -1), w.reshape(T, -1))
    dy = oracle.gated_backward(d, y, g)["dy"]
    gv = oracle.bag_backward(dy, V, idx, w, H, k)["grad_values"]
    h = 1e-6
    for (r, e) in [(int(idx[0, 0, 0]), 1), (int(idx[2, 1, 1]), 4)]:
        Vp = V.copy(); Vp[r, e] += h
        Vm = V.copy(); Vm[r, e] -= h
        L = lambda VV: float((d * oracle.gated_output(  # noqa: E731
            oracle.bag_forward(VV, idx.reshape(T, -1), w.reshape(T, -1)), g)).sum())
        assert abs((L(Vp) - L(Vm)) / (2 * h) - gv[r, e]) < 1e-7
