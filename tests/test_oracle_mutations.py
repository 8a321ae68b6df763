"""The pins must catch plausible mistakes: each test plants one mistake in a
copy of the oracle (on the CPU) and asserts that some pin rejects it."""
import numpy as np
import pytest

import oracle
from oracle import pkm_oracle as po
from tests import oracle_pins as pins


def _search_pins_fail(search_fn, monkeypatch=None):
    rng = np.random.default_rng(0)
    failures = 0
    checks = [
        lambda: pins.check_all_equal_subkeys(search_fn),
        lambda: pins.check_k1_argmax(search_fn, np.random.default_rng(3)),
        lambda: pins.check_hand_example(search_fn, oracle.bag_forward, oracle.bag_backward),
    ]
    for s in range(30):
        q, K, k = pins.rand_search_case(np.random.default_rng(s), integer=True)
        checks.append(lambda q=q, K=K, k=k: pins.check_search_vs_brute_force(
            search_fn, oracle.brute_force_search, q, K, k))
    for c in checks:
        try:
            c()
        except (AssertionError, ValueError, IndexError):
            failures += 1
    return failures


def test_real_oracle_passes_all_search_pins():
    assert _search_pins_fail(oracle.search) == 0


def test_catches_swapped_halves():
    assert _search_pins_fail(lambda q, K, k: oracle.search(q, K[:, ::-1], k)) > 0


def test_catches_transposed_composed_index():
    def mutant(q, K, k):
        out = oracle.search(q, K, k)
        S = K.shape[2]
        out["idx"] = (out["idx"] % S) * S + out["idx"] // S
        return out
    assert _search_pins_fail(mutant) > 0


def test_catches_reversed_tie_break(monkeypatch):
    monkeypatch.setattr(po, "rank_order", lambda s, ids: np.lexsort((-np.asarray(ids), -np.asarray(s))))
    assert _search_pins_fail(po.search) > 0


def test_catches_per_half_off_by_one(monkeypatch):
    # per-half selection that starts one rank too late (skips the best)
    monkeypatch.setattr(po, "topk_desc", lambda s, k: np.roll(po.order_desc(s), -1)[:k])
    assert _search_pins_fail(po.search) > 0


def test_catches_per_half_ascending(monkeypatch):
    monkeypatch.setattr(po, "topk_desc", lambda s, k: po.order_desc(-np.asarray(s))[:k])
    assert _search_pins_fail(po.search) > 0


def test_catches_half_score_dropped():
    def mutant(q, K, k):
        K2 = K.copy()
        K2[:, 1] = 0.0          # second half's score ignored
        out = oracle.search(q, K2, k)
        return out
    assert _search_pins_fail(mutant) > 0


def test_catches_unnormalised_softmax(monkeypatch):
    monkeypatch.setattr(po, "softmax", lambda z: np.exp(np.asarray(z) - np.max(z)))
    with pytest.raises(AssertionError):
        pins.check_softmax(po.softmax, np.random.default_rng(5))
    assert _search_pins_fail(po.search) > 0


def _bag_fails(fwd=oracle.bag_forward, bwd=oracle.bag_backward):
    fails = 0
    for c in (lambda: pins.check_bag_forward(fwd, np.random.default_rng(1)),
              lambda: pins.check_bag_backward(bwd, np.random.default_rng(2)),
              lambda: pins.check_bag_backward_fd(fwd, bwd, np.random.default_rng(3)),
              lambda: pins.check_accumulate(bwd, np.random.default_rng(4)),
              lambda: pins.check_hand_example(oracle.search, fwd, bwd)):
        try:
            c()
        except (AssertionError, ValueError, IndexError):
            fails += 1
    return fails


def test_real_oracle_passes_all_bag_pins():
    assert _bag_fails() == 0


def test_catches_heads_averaged():
    def fwd(V, idx, w):
        H = idx.shape[1] if np.asarray(idx).ndim == 3 else 1
        return oracle.bag_forward(V, idx, w) / H
    assert _bag_fails(fwd=fwd) > 0


def test_catches_softmax_backward_sign():
    def bwd(dy, V, idx, w, H, k, grad_values_in=None):
        out = oracle.bag_backward(dy, V, idx, w, H, k, grad_values_in)
        out["grad_z"] = -out["grad_z"]
        return out
    assert _bag_fails(bwd=bwd) > 0


def test_catches_softmax_backward_missing_inner_term():
    def bwd(dy, V, idx, w, H, k, grad_values_in=None):
        out = oracle.bag_backward(dy, V, idx, w, H, k, grad_values_in)
        out["grad_z"] = np.asarray(w).reshape(out["grad_w"].shape) * out["grad_w"]
        return out
    assert _bag_fails(bwd=bwd) > 0


def test_catches_overwrite_instead_of_sum_for_repeated_rows():
    def bwd(dy, V, idx, w, H, k, grad_values_in=None):
        out = oracle.bag_backward(dy, V, idx, w, H, k, grad_values_in)
        T = dy.shape[0]
        gv = np.zeros_like(out["grad_values"]) if grad_values_in is None else np.array(grad_values_in, dtype=float)
        ww = np.asarray(w).reshape(T, -1)
        ii = np.asarray(idx).reshape(T, -1)
        for t in range(T):
            for j in range(ii.shape[1]):
                gv[ii[t, j]] = ww[t, j] * np.asarray(dy[t], dtype=float)   # '=' not '+='
        out["grad_values"] = gv
        return out
    assert _bag_fails(bwd=bwd) > 0


def test_catches_grad_values_not_accumulated():
    def bwd(dy, V, idx, w, H, k, grad_values_in=None):
        return oracle.bag_backward(dy, V, idx, w, H, k, None)
    assert _bag_fails(bwd=bwd) > 0


def test_catches_weighted_grad_w():
    def bwd(dy, V, idx, w, H, k, grad_values_in=None):
        out = oracle.bag_backward(dy, V, idx, w, H, k, grad_values_in)
        out["grad_w"] = out["grad_w"] * np.asarray(w).reshape(out["grad_w"].shape)
        return out
    assert _bag_fails(bwd=bwd) > 0


def _sbwd_fails(bwd):
    try:
        pins.check_search_backward(oracle.search, bwd, np.random.default_rng(61))
    except (AssertionError, ValueError, IndexError):
        return True
    return False


def test_real_search_backward_passes():
    assert not _sbwd_fails(oracle.search_backward)


def test_catches_search_backward_halves_swapped():
    def bwd(q, K, idx, gz, base=None):
        out = oracle.search_backward(q, K[:, ::-1], idx, gz, None if base is None else base[:, ::-1])
        out["grad_K"] = out["grad_K"][:, ::-1]
        return out
    assert _sbwd_fails(bwd)


def test_catches_search_backward_index_transposed():
    def bwd(q, K, idx, gz, base=None):
        S = K.shape[2]
        return oracle.search_backward(q, K, (idx % S) * S + idx // S, gz, base)
    assert _sbwd_fails(bwd)


def test_catches_search_backward_key_grad_not_accumulated():
    def bwd(q, K, idx, gz, base=None):
        return oracle.search_backward(q, K, idx, gz, None)
    assert _sbwd_fails(bwd)


def test_catches_search_backward_repeated_subkey_counted_once():
    # a sub-key chosen by several ranks of one (token, head) must receive every
    # rank's gradient; this mutant keeps only the first rank of each sub-key
    def bwd(q, K, idx, gz, base=None):
        S = K.shape[2]
        gz = np.array(gz, dtype=np.float64, copy=True)
        idx = np.asarray(idx)
        T, H, k = idx.shape
        for t in range(T):
            for h in range(H):
                seen = set()
                for j in range(k):
                    i1 = int(idx[t, h, j]) // S
                    if i1 in seen:
                        gz[t, h, j] = 0.0
                    seen.add(i1)
        return oracle.search_backward(q, K, idx, gz, base)
    assert _sbwd_fails(bwd)


def _gating_fails(out_fn=None, bwd_fn=None):
    fails = 0
    try:
        pins.check_gated_output(out_fn or oracle.gated_output, oracle.silu, np.random.default_rng(81))
    except (AssertionError, ValueError):
        fails += 1
    try:
        pins.check_gated_backward(bwd_fn or oracle.gated_backward, np.random.default_rng(82))
    except (AssertionError, ValueError):
        fails += 1
    return fails


def _sig(x):
    return 1.0 / (1.0 + np.exp(-np.asarray(x, dtype=np.float64)))


def test_real_gating_passes():
    assert _gating_fails() == 0


def test_catches_sigmoid_gate_instead_of_silu():
    assert _gating_fails(out_fn=lambda y, g: np.asarray(y) * _sig(g)) > 0


def test_catches_gate_derivative_missing_factor():
    def bwd(d, y, g):
        out = oracle.gated_backward(d, y, g)
        out["dg"] = np.asarray(d) * np.asarray(y) * _sig(g)
        return out
    assert _gating_fails(bwd_fn=bwd) > 0


def test_catches_ungated_value_gradient():
    def bwd(d, y, g):
        out = oracle.gated_backward(d, y, g)
        out["dy"] = np.asarray(d, dtype=np.float64)
        return out
    assert _gating_fails(bwd_fn=bwd) > 0


def test_catches_gate_gradient_with_silu_not_its_derivative():
    def bwd(d, y, g):
        out = oracle.gated_backward(d, y, g)
        out["dg"] = np.asarray(d) * np.asarray(y) * oracle.silu(g)
        return out
    assert _gating_fails(bwd_fn=bwd) > 0
