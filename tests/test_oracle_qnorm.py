"""Oracle pins for the query normalisation fused in front of the search
(qk-normalisation, Sec. 3.1.4): LayerNorm without affine of each query."""
import numpy as np

import oracle
from tests import oracle_pins as pins


def test_query_layernorm_pins():
    pins.check_query_layernorm(oracle.query_layernorm, np.random.default_rng(91))


def test_round_bf16_pins():
    pins.check_round_bf16(oracle.round_bf16, np.random.default_rng(92))


def test_search_qnorm_exact_rows():
    for s in range(4):
        pins.check_search_qnorm_exact(oracle.search_qnorm, oracle.search, oracle.brute_force_search,
                                      np.random.default_rng(93 + s))


def test_search_qnorm_rounding():
    pins.check_search_qnorm_rounding(oracle.search_qnorm, np.random.default_rng(96))


def test_search_backward_qnorm_pins():
    pins.check_search_backward_qnorm(oracle.search_qnorm, oracle.search_backward_qnorm,
                                     np.random.default_rng(97))


def test_qnorm_backward_accumulates_and_matches_plain_on_normalised_rows():
    """With eps = 0 on exactly normalisable rows the sub-key gradient equals
    the plain search backward at x / 2, and it accumulates."""
    rng = np.random.default_rng(98)
    q, half = pins.exact_norm_rows(rng, 4, 2, 16)
    K = rng.integers(-2, 3, size=(2, 2, 6, 8)).astype(np.float64)
    idx = oracle.search_qnorm(q, K, 3, 0.0, "bf16")["idx"]
    gz = rng.standard_normal(idx.shape)
    base = rng.standard_normal(K.shape)
    a = oracle.search_backward_qnorm(q, K, idx, gz, 0.0, "bf16", base)
    b = oracle.search_backward(half, K, idx, gz)
    np.testing.assert_allclose(a["grad_K"], base + b["grad_K"], rtol=1e-14, atol=1e-15)
