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


# ----------------------------------------------------- query normalisation ----
def _qnorm_fails(ln=None, rnd=None, sq=None, bwd=None):
    ln = ln or oracle.query_layernorm
    rnd = rnd or oracle.round_bf16
    sq = sq or oracle.search_qnorm
    bwd = bwd or oracle.search_backward_qnorm
    checks = [
        lambda: pins.check_query_layernorm(ln, np.random.default_rng(101)),
        lambda: pins.check_round_bf16(rnd, np.random.default_rng(102)),
        lambda: pins.check_search_qnorm_exact(sq, oracle.search, oracle.brute_force_search,
                                              np.random.default_rng(103)),
        lambda: pins.check_search_qnorm_rounding(sq, np.random.default_rng(104)),
        lambda: pins.check_search_backward_qnorm(sq, bwd, np.random.default_rng(105)),
    ]
    failures = 0
    for c in checks:
        try:
            c()
        except (AssertionError, ValueError, IndexError):
            failures += 1
    return failures


def _ln(q, eps, ddof=0, eps_outside=False, halves=False):
    x = np.asarray(q, dtype=np.float64)
    if halves:
        d = x.shape[-1] // 2
        a, b = _ln(x[..., :d], eps), _ln(x[..., d:], eps)
        return dict(qhat=np.concatenate([a["qhat"], b["qhat"]], -1), mean=a["mean"], rstd=a["rstd"])
    mu = x.mean(-1)
    xc = x - mu[..., None]
    var = (xc * xc).sum(-1) / (x.shape[-1] - ddof)
    rstd = 1.0 / (np.sqrt(var) + eps) if eps_outside else 1.0 / np.sqrt(var + eps)
    return dict(qhat=xc * rstd[..., None], mean=mu, rstd=rstd)


def _sq_with(ln):
    def sq(q, K, k, eps, dtype="fp64"):
        r = ln(q, eps)
        qs = po.round_to(r["qhat"], dtype)
        out = oracle.search(qs, K, k)
        out.update(qhat=qs, mean=r["mean"], rstd=r["rstd"])
        return out
    return sq


def test_real_qnorm_passes():
    assert _qnorm_fails() == 0


def test_catches_unbiased_variance():
    ln = lambda q, eps: _ln(q, eps, ddof=1)  # noqa: E731
    assert _qnorm_fails(ln=ln, sq=_sq_with(ln)) > 0


def test_catches_eps_outside_the_root():
    ln = lambda q, eps: _ln(q, eps, eps_outside=True)  # noqa: E731
    assert _qnorm_fails(ln=ln, sq=_sq_with(ln)) > 0


def test_catches_per_half_normalisation():
    ln = lambda q, eps: _ln(q, eps, halves=True)  # noqa: E731
    assert _qnorm_fails(ln=ln, sq=_sq_with(ln)) > 0


def test_catches_bf16_truncation():
    def trunc(x):
        b = np.asarray(x, dtype=np.float64).astype(np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
        return b.view(np.float32).astype(np.float64)
    assert _qnorm_fails(rnd=trunc) > 0


def test_catches_unrounded_scoring():
    def sq(q, K, k, eps, dtype="fp64"):
        return oracle.search_qnorm(q, K, k, eps, "fp64")
    assert _qnorm_fails(sq=sq) > 0


def _bwd_variant(drop_mean=False, drop_proj=False, rounded_xhat=False, unrounded_dk=False):
    def bwd(q, K, idx, gz, eps, dtype="fp64", base=None):
        ln = oracle.query_layernorm(q, eps)
        qs = po.round_to(ln["qhat"], dtype)
        r = oracle.search_backward(ln["qhat"] if unrounded_dk else qs, K, idx, gz, base)
        g = oracle.search_backward(qs, K, idx, gz)["grad_q"]
        xh = qs if rounded_xhat else ln["qhat"]
        out = g.copy()
        if not drop_mean:
            out -= g.mean(-1, keepdims=True)
        if not drop_proj:
            out -= xh * (g * xh).mean(-1, keepdims=True)
        return dict(grad_q=ln["rstd"][..., None] * out, grad_K=r["grad_K"])
    return bwd


def test_qnorm_backward_variant_helper_is_faithful():
    assert _qnorm_fails(bwd=_bwd_variant()) == 0


def test_catches_qnorm_backward_without_mean_term():
    assert _qnorm_fails(bwd=_bwd_variant(drop_mean=True)) > 0


def test_catches_qnorm_backward_without_projection_term():
    assert _qnorm_fails(bwd=_bwd_variant(drop_proj=True)) > 0


def test_catches_qnorm_backward_with_rounded_xhat():
    assert _qnorm_fails(bwd=_bwd_variant(rounded_xhat=True)) > 0


def test_catches_qnorm_key_gradient_from_unrounded_query():
    assert _qnorm_fails(bwd=_bwd_variant(unrounded_dk=True)) > 0


# ------------------------------------------------------ extra key-value pairs ----
def _extra_fails(fn):
    failures = 0
    for s in range(3):
        try:
            pins.check_search_extra(fn, oracle.search, oracle.brute_force_search,
                                    np.random.default_rng(140 + s))
        except (AssertionError, ValueError, IndexError, KeyError):
            failures += 1
    return failures


def test_real_extra_passes():
    assert _extra_fails(oracle.search_extra) == 0


def test_catches_extra_halves_swapped():
    def mutant(q, K, k, ex):
        S = K.shape[2]
        ex = np.asarray(ex)
        return oracle.search_extra(q, K, k, (ex % S) * S + ex // S)
    assert _extra_fails(mutant) > 0


def test_catches_extras_left_out_of_the_softmax():
    def mutant(q, K, k, ex):
        out = oracle.search_extra(q, K, k, ex)
        out["w"][..., :k] = oracle.search(q, K, k)["w"]
        out["w"][..., k:] = 0.0
        return out
    assert _extra_fails(mutant) > 0


def test_catches_extra_scored_with_one_half_only():
    def mutant(q, K, k, ex):
        out = oracle.search_extra(q, K, k, ex)
        S = K.shape[2]
        d = q.shape[2] // 2
        T, H, r = np.asarray(ex).shape
        for t in range(T):
            for h in range(H):
                for e in range(r):
                    i1 = int(ex[t, h, e]) // S
                    out["score"][t, h, k + e] = np.asarray(q, float)[t, h, :d] @ np.asarray(K, float)[h, 0, i1]
                z = out["score"][t, h]
                out["w"][t, h] = np.exp(z - z.max()) / np.exp(z - z.max()).sum()
        return out
    assert _extra_fails(mutant) > 0


# ------------------------------------------------------------ sink pair ----
def _sink_fails(fn=None, bwd=None):
    failures = 0
    for s in range(2):
        try:
            pins.check_search_sink(fn or oracle.search_sink, oracle.search_extra,
                                   np.random.default_rng(180 + s))
        except (AssertionError, ValueError, IndexError):
            failures += 1
        try:
            pins.check_search_backward_sink(fn or oracle.search_sink, bwd or oracle.search_backward_sink,
                                            np.random.default_rng(190 + s))
        except (AssertionError, ValueError, IndexError):
            failures += 1
    return failures


def test_real_sink_passes():
    assert _sink_fails() == 0


def test_catches_sink_outside_the_softmax():
    def mutant(q, K, k, ex, ks, row0):
        out = oracle.search_sink(q, K, k, ex, ks, row0)
        base = oracle.search_extra(q, K, k, ex)
        out["w"][..., :-1] = base["w"]
        out["w"][..., -1] = 0.0
        return out
    assert _sink_fails(fn=mutant) > 0


def test_catches_sink_scored_on_one_half():
    def mutant(q, K, k, ex, ks, row0):
        ks = np.asarray(ks, float).copy()
        ks[:, ks.shape[1] // 2:] = 0.0
        return oracle.search_sink(q, K, k, ex, ks, row0)
    assert _sink_fails(fn=mutant) > 0


def test_catches_sink_key_gradient_not_accumulated():
    def bwd(q, K, idx, gz, ks, gK=None, gs=None):
        return oracle.search_backward_sink(q, K, idx, gz, ks, gK, None)
    assert _sink_fails(bwd=bwd) > 0


def test_catches_sink_query_gradient_dropped():
    def bwd(q, K, idx, gz, ks, gK=None, gs=None):
        out = oracle.search_backward_sink(q, K, idx, gz, ks, gK, gs)
        r = oracle.search_backward(q, K, np.asarray(idx)[..., :-1], np.asarray(gz)[..., :-1], gK)
        out["grad_q"] = r["grad_q"]
        return out
    assert _sink_fails(bwd=bwd) > 0


# ------------------------------------------------- rows form, inversion ----
def _rows_fails(rows_fn):
    fails = 0
    for s in range(2):
        try:
            pins.check_rows_form(oracle.bag_backward, rows_fn, np.random.default_rng(200 + s))
        except AssertionError:
            fails += 1
    return fails


def _inv_fails(inv_fn):
    fails = 0
    for s in range(2):
        try:
            pins.check_invert_index(inv_fn, np.random.default_rng(210 + s))
        except (AssertionError, IndexError):
            fails += 1
    return fails


def test_real_rows_form_and_inversion_pass():
    assert _rows_fails(oracle.bag_backward_rows) == 0
    assert _inv_fails(oracle.invert_index) == 0


def test_catches_rows_descending():
    def mutant(dy, V, idx, w, H, k):
        r = oracle.bag_backward_rows(dy, V, idx, w, H, k)
        return dict(r, rows=r["rows"][::-1], grad_rows=r["grad_rows"][::-1])
    assert _rows_fails(mutant) > 0


def test_catches_rows_overwrite_on_repeats():
    def mutant(dy, V, idx, w, H, k):
        r = oracle.bag_backward_rows(dy, V, idx, w, H, k)
        T = dy.shape[0]
        flat, wf = np.asarray(idx).reshape(T, -1), np.asarray(w, float).reshape(T, -1)
        g = r["grad_rows"].copy()
        for u, row in enumerate(r["rows"]):   # keep only the last lookup's term
            t, j = [(t, j) for t in range(T) for j in range(flat.shape[1]) if flat[t, j] == row][-1]
            g[u] = wf[t, j] * np.asarray(dy, float)[t]
        return dict(r, grad_rows=g)
    assert _rows_fails(mutant) > 0


def test_catches_inversion_lookups_reversed_within_a_row():
    def mutant(idx):
        inv = oracle.invert_index(idx)
        lk = inv["lookups"].copy()
        for u in range(len(inv["rows"])):
            a, b = inv["row_ptr"][u], inv["row_ptr"][u + 1]
            lk[a:b] = lk[a:b][::-1]
        return dict(inv, lookups=lk)
    assert _inv_fails(mutant) > 0


def test_catches_inversion_offsets_shifted():
    def mutant(idx):
        inv = oracle.invert_index(idx)
        rp = inv["row_ptr"].copy()
        rp[1:-1] += 1
        return dict(inv, row_ptr=rp)
    assert _inv_fails(mutant) > 0
