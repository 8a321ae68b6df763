"""Oracle pins for extra key-value pairs beside the top-k (Sec. 5.4): scored
like any full key and joined to the softmax."""
import numpy as np

import oracle
from tests import oracle_pins as pins


def test_search_extra_pins():
    for s in range(5):
        pins.check_search_extra(oracle.search_extra, oracle.search, oracle.brute_force_search,
                                np.random.default_rng(120 + s))


def test_extra_slots_carry_gradients_through_the_plain_backwards():
    """The bag and search backwards need nothing new: with k' = k + r slots
    the softmax backward runs over all of them and the search backward sends
    each extra slot's gradient to its sub-keys (central differences in q)."""
    rng = np.random.default_rng(131)
    T, H, S, d, k, r = 3, 2, 5, 2, 3, 2
    q = rng.standard_normal((T, H, 2 * d))
    K = rng.standard_normal((H, 2, S, d))
    ex = rng.integers(0, S * S, size=(T, H, r))
    out = oracle.search_extra(q, K, k, ex)
    gz = rng.standard_normal((T, H, k + r))
    g = oracle.search_backward(q, K, out["idx"], gz)
    h = 1e-6
    for (t, hh, e) in [(0, 0, 1), (2, 1, 3)]:
        qp = q.copy(); qp[t, hh, e] += h
        qm = q.copy(); qm[t, hh, e] -= h
        L = lambda qq: float((pins.selected_scores(qq, K, out["idx"]) * gz).sum())  # noqa: E731
        assert abs((L(qp) - L(qm)) / (2 * h) - g["grad_q"][t, hh, e]) < 1e-7
