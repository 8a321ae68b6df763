"""Checks that pin the oracle to facts outside itself.

Each check takes the implementation under test as arguments, so the same
check runs against the real oracle (tests/test_oracle_*.py) and against
copies with a planted mistake (tests/test_oracle_mutations.py), which must
fail at least one check.  Not collected by pytest (no test_ prefix).

What pins what:
  search        - Eq. (1) with the full key set instantiated (brute force):
                  the product-key result must equal it exactly on small
                  integer-valued inputs, ties included (Sec. 3.1.1 claims the
                  product-key lookup finds the top-k of the full set);
                - all-equal sub-keys: every full score ties, so the result is
                  the k smallest composed indices 0..k-1;
                - k = 1: the arg-max of the full scores;
                - the hand-worked fixture tests/golden/hand_example.json.
  softmax       - closed form for two entries, sum to one, order, shift.
  bag forward   - torch.nn.functional.embedding_bag (sum mode, per-sample
                  weights) in fp64 on the CPU; dense A @ V.
  bag backward  - torch autograd of that embedding_bag and of softmax in
                  fp64; central finite differences; dense A.T @ dy;
                  the score gradients of one (token, head) sum to zero.
  search bwd    - central finite differences of the selected scores at a
                  fixed selection; torch autograd of the gathered scores;
                  the bilinear identities sum(grad_q q) = sum(grad_z z) =
                  sum(grad_K K); accumulation onto an existing key gradient.
  query norm    - torch.nn.functional.layer_norm in fp64; the closed form
                  for [1, 2, 3, 4]; zero mean, mean square var / (var + eps),
                  shift and scale invariance; bf16 rounding against torch's
                  conversion and hand-worked ties; with eps = 0, rows built to
                  normalise exactly give the plain search (and brute force) of
                  x / 2; the backward by central differences and torch
                  autograd through layer_norm.
  extra pairs   - r = 0 gives the plain search; each extra slot's score is
                  its key's brute-force full score (integer inputs, exact); a
                  repeated selected index repeats its score; closed-form
                  softmax over the k + r scores.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def rand_search_case(rng, integer: bool, S=None, d=None, H=None, k=None, T=None, lo=-2, hi=2):
    S = S or int(rng.integers(2, 9))
    d = d or int(rng.integers(1, 5))
    H = H or int(rng.integers(1, 4))
    k = k or int(rng.integers(1, S + 1))
    T = T or int(rng.integers(1, 6))
    if integer:
        q = rng.integers(lo, hi + 1, size=(T, H, 2 * d)).astype(np.float64)
        K = rng.integers(lo, hi + 1, size=(H, 2, S, d)).astype(np.float64)
    else:
        q = rng.standard_normal((T, H, 2 * d))
        K = rng.standard_normal((H, 2, S, d))
    return q, K, k


def check_search_vs_brute_force(search_fn, brute_fn, q, K, k):
    out = search_fn(q, K, k)
    ref = brute_fn(q, K, k)
    np.testing.assert_array_equal(out["idx"], ref["idx"])
    np.testing.assert_allclose(out["score"], ref["score"], rtol=0, atol=1e-12)


def check_all_equal_subkeys(search_fn, S=5, d=3, H=2, k=4, T=3):
    q = np.ones((T, H, 2 * d))
    K = np.full((H, 2, S, d), 0.5)
    out = search_fn(q, K, k)
    want = np.broadcast_to(np.arange(k), (T, H, k))
    np.testing.assert_array_equal(out["idx"], want)
    np.testing.assert_allclose(out["w"], 1.0 / k, rtol=0, atol=1e-15)


def check_k1_argmax(search_fn, rng, S=6, d=3, H=2, T=4):
    q = rng.standard_normal((T, H, 2 * d))
    K = rng.standard_normal((H, 2, S, d))
    out = search_fn(q, K, 1)
    for t in range(T):
        for h in range(H):
            full = np.array([q[t, h, :d] @ K[h, 0, i // S] + q[t, h, d:] @ K[h, 1, i % S]
                             for i in range(S * S)])
            assert out["idx"][t, h, 0] == int(np.argmax(full))
            assert out["w"][t, h, 0] == 1.0


def load_hand_example():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        return json.load(f)


def _eval(expr: str) -> float:
    return float(eval(expr, {"__builtins__": {}}, {"e": math.e, "exp": math.exp}))


def check_hand_example(search_fn, bag_fwd_fn, bag_bwd_fn):
    ex = load_hand_example()
    q = np.array(ex["q"], dtype=np.float64)
    K = np.array(ex["subkeys"], dtype=np.float64)
    k = ex["k"]
    out = search_fn(q, K, k)
    np.testing.assert_array_equal(out["half_idx"], np.array(ex["half_idx"]))
    np.testing.assert_array_equal(out["idx"], np.array(ex["idx"]))
    np.testing.assert_array_equal(out["score"], np.array(ex["score"], dtype=np.float64))
    w_want = np.array([[[_eval(e) for e in row] for row in tok] for tok in ex["w"]])
    np.testing.assert_allclose(out["w"], w_want, rtol=1e-15, atol=0)
    V = np.array(ex["values"], dtype=np.float64)
    y = bag_fwd_fn(V, out["idx"], out["w"])
    y_want = np.array([[_eval(e) for e in row] for row in ex["y"]])
    np.testing.assert_allclose(y, y_want, rtol=1e-14, atol=1e-14)
    dy = np.array(ex["dy"], dtype=np.float64)
    T, H, _ = q.shape
    g = bag_bwd_fn(dy, V, out["idx"], out["w"], H, k)
    np.testing.assert_allclose(g["grad_w"], np.array(ex["grad_w"], dtype=np.float64), rtol=0, atol=1e-14)
    gz_want = np.array([[[_eval(e) for e in row] for row in tok] for tok in ex["grad_z"]])
    np.testing.assert_allclose(g["grad_z"], gz_want, rtol=1e-13, atol=1e-14)
    gv_want = np.zeros_like(V)
    for r, row in ex["grad_values"].items():
        gv_want[int(r)] = [_eval(e) for e in row]
    np.testing.assert_allclose(g["grad_values"], gv_want, rtol=1e-14, atol=1e-15)


def check_softmax(softmax_fn, rng):
    a, b = 1.25, -0.5
    np.testing.assert_allclose(softmax_fn(np.array([a, b])),
                               [1 / (1 + math.exp(b - a)), 1 / (1 + math.exp(a - b))], rtol=1e-15)
    z = np.sort(rng.standard_normal(9))[::-1] * 3
    w = softmax_fn(z)
    assert abs(w.sum() - 1) < 1e-15 and np.all(w > 0)
    assert np.all(np.diff(w) <= 0)
    np.testing.assert_allclose(softmax_fn(z + 100.0), w, rtol=1e-13)
    assert softmax_fn(np.array([3.7]))[0] == 1.0


def _torch_bag(V, idx, w):
    T = idx.shape[0]
    Vt = torch.tensor(V, dtype=torch.float64, requires_grad=True)
    wt = torch.tensor(np.asarray(w, dtype=np.float64).reshape(T, -1), requires_grad=True)
    it = torch.tensor(np.asarray(idx).reshape(T, -1), dtype=torch.int64)
    y = torch.nn.functional.embedding_bag(it, Vt, mode="sum", per_sample_weights=wt)
    return Vt, wt, y


def random_bag_case(rng, T=7, H=2, k=3, N=11, D=5):
    V = rng.standard_normal((N, D))
    idx = rng.integers(0, N, size=(T, H, k))
    idx[0, 1, :] = idx[0, 0, :]          # a row chosen by two heads of one token
    z = rng.standard_normal((T, H, k))
    w = np.exp(z - z.max(-1, keepdims=True))
    w /= w.sum(-1, keepdims=True)
    dy = rng.standard_normal((T, D))
    return V, idx, z, w, dy


def check_bag_forward(bag_fwd_fn, rng):
    V, idx, z, w, dy = random_bag_case(rng)
    T, H, k = idx.shape
    y = bag_fwd_fn(V, idx, w)
    _, _, yt = _torch_bag(V, idx, w)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-13, atol=1e-15)
    A = np.zeros((T, V.shape[0]))
    for t in range(T):
        for j, r in enumerate(idx[t].ravel()):
            A[t, r] += w[t].ravel()[j]
    np.testing.assert_allclose(y, A @ V, rtol=1e-13, atol=1e-15)
    # one-hot weights copy a row exactly
    w1 = np.zeros_like(w)
    w1[:, 0, 0] = 1.0
    np.testing.assert_array_equal(bag_fwd_fn(V, idx, w1), V[idx[:, 0, 0]])


def check_bag_backward(bag_bwd_fn, rng):
    V, idx, z, w, dy = random_bag_case(rng)
    T, H, k = idx.shape
    g = bag_bwd_fn(dy, V, idx, w, H, k)
    # torch autograd through embedding_bag and softmax, fp64
    Vt = torch.tensor(V, requires_grad=True)
    zt = torch.tensor(z, requires_grad=True)
    wt = torch.softmax(zt, dim=-1)
    y = torch.nn.functional.embedding_bag(torch.tensor(idx.reshape(T, -1)), Vt, mode="sum",
                                          per_sample_weights=wt.reshape(T, -1))
    wt.retain_grad()
    (y * torch.tensor(dy)).sum().backward()
    np.testing.assert_allclose(g["grad_values"], Vt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(g["grad_w"], wt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(g["grad_z"], zt.grad.numpy(), rtol=1e-11, atol=1e-14)
    # dense transpose
    A = np.zeros((T, V.shape[0]))
    for t in range(T):
        for j, r in enumerate(idx[t].ravel()):
            A[t, r] += w[t].ravel()[j]
    np.testing.assert_allclose(g["grad_values"], A.T @ dy, rtol=1e-12, atol=1e-14)
    # score gradients of one (token, head) sum to zero (softmax is shift invariant)
    np.testing.assert_allclose(g["grad_z"].sum(-1), 0.0, atol=1e-13)


def check_bag_backward_fd(bag_fwd_fn, bag_bwd_fn, rng, h=1e-6):
    """Central differences of L = sum_t dy[t] . y[t] in V and in the scores z."""
    V, idx, z, w, dy = random_bag_case(rng, T=3, H=2, k=3, N=6, D=4)
    T, H, k = idx.shape
    g = bag_bwd_fn(dy, V, idx, w, H, k)

    def sm(zz):
        e = np.exp(zz - zz.max(-1, keepdims=True))
        return e / e.sum(-1, keepdims=True)

    def loss(VV, zz):
        return float((bag_fwd_fn(VV, idx, sm(zz)) * dy).sum())

    for (r, c) in [(int(idx[0, 0, 0]), 0), (int(idx[2, 1, 2]), 3), (int(idx[1, 0, 1]), 2)]:
        Vp = V.copy(); Vp[r, c] += h
        Vm = V.copy(); Vm[r, c] -= h
        fd = (loss(Vp, z) - loss(Vm, z)) / (2 * h)
        assert abs(fd - g["grad_values"][r, c]) < 1e-7, (r, c, fd, g["grad_values"][r, c])
    for (t, hh, j) in [(0, 0, 0), (1, 1, 2), (2, 0, 1)]:
        zp = z.copy(); zp[t, hh, j] += h
        zm = z.copy(); zm[t, hh, j] -= h
        fd = (loss(V, zp) - loss(V, zm)) / (2 * h)
        assert abs(fd - g["grad_z"][t, hh, j]) < 1e-7, (t, hh, j, fd, g["grad_z"][t, hh, j])


def check_accumulate(bag_bwd_fn, rng):
    V, idx, z, w, dy = random_bag_case(rng)
    T, H, k = idx.shape
    base = rng.standard_normal(V.shape)
    g0 = bag_bwd_fn(dy, V, idx, w, H, k)
    g1 = bag_bwd_fn(dy, V, idx, w, H, k, grad_values_in=base)
    np.testing.assert_allclose(g1["grad_values"], base + g0["grad_values"], rtol=1e-14, atol=1e-15)


def selected_scores(q, K, idx):
    """z[t,h,j] for a fixed selection (used only as the function that the
    finite differences and autograd differentiate)."""
    T, H, n = q.shape
    d = n // 2
    S = K.shape[2]
    k = idx.shape[2]
    z = np.zeros((T, H, k))
    for t in range(T):
        for h in range(H):
            for j in range(k):
                i1, i2 = divmod(int(idx[t, h, j]), S)
                z[t, h, j] = q[t, h, :d] @ K[h, 0, i1] + q[t, h, d:] @ K[h, 1, i2]
    return z


def check_search_backward(search_fn, bwd_fn, rng, T=4, H=2, S=5, d=3, k=4, h=1e-6):
    q = rng.standard_normal((T, H, 2 * d))
    K = rng.standard_normal((H, 2, S, d))
    idx = search_fn(q, K, k)["idx"]
    gz = rng.standard_normal((T, H, k))
    g = bwd_fn(q, K, idx, gz)
    L = lambda qq, KK: float((selected_scores(qq, KK, idx) * gz).sum())  # noqa: E731
    # central differences at the fixed selection (the score is bilinear, so
    # the difference quotient is exact up to rounding)
    for (t, hh, e) in [(0, 0, 0), (1, 1, 4), (3, 0, 2), (2, 1, 5)]:
        qp = q.copy(); qp[t, hh, e] += h
        qm = q.copy(); qm[t, hh, e] -= h
        fd = (L(qp, K) - L(qm, K)) / (2 * h)
        assert abs(fd - g["grad_q"][t, hh, e]) < 1e-7, (t, hh, e, fd, g["grad_q"][t, hh, e])
    for (hh, p, i, e) in [(0, 0, int(idx[0, 0, 0]) // S, 1), (1, 1, int(idx[2, 1, 1]) % S, 2), (0, 1, 4, 0)]:
        Kp = K.copy(); Kp[hh, p, i, e] += h
        Km = K.copy(); Km[hh, p, i, e] -= h
        fd = (L(q, Kp) - L(q, Km)) / (2 * h)
        assert abs(fd - g["grad_K"][hh, p, i, e]) < 1e-7, (hh, p, i, e, fd, g["grad_K"][hh, p, i, e])
    # torch autograd of the gathered scores
    qt = torch.tensor(q, requires_grad=True)
    Kt = torch.tensor(K, requires_grad=True)
    it = torch.tensor(idx)
    i1, i2 = it // S, it % S
    hh_ = torch.arange(H).view(1, H, 1).expand_as(it)
    z = (qt[..., :d].unsqueeze(2) * Kt[hh_, 0, i1]).sum(-1) + (qt[..., d:].unsqueeze(2) * Kt[hh_, 1, i2]).sum(-1)
    (z * torch.tensor(gz)).sum().backward()
    np.testing.assert_allclose(g["grad_q"], qt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(g["grad_K"], Kt.grad.numpy(), rtol=1e-12, atol=1e-14)
    # bilinearity: sum(grad_q . q) = sum(grad_z . z) = sum(grad_K . K)
    zz = selected_scores(q, K, idx)
    lhs = float((g["grad_q"] * q).sum())
    mid = float((gz * zz).sum())
    rhs = float((g["grad_K"] * K).sum())
    assert abs(lhs - mid) < 1e-10 * max(1.0, abs(mid)) and abs(rhs - mid) < 1e-10 * max(1.0, abs(mid))
    # accumulation onto an existing sub-key gradient
    base = rng.standard_normal(K.shape)
    g2 = bwd_fn(q, K, idx, gz, base)
    np.testing.assert_allclose(g2["grad_K"], base + g["grad_K"], rtol=1e-14, atol=1e-15)


# ---------------------------------------------------------------- Memory+ ----
def check_gated_output(gated_fn, silu_fn, rng, T=5, D=7):
    """out = y * silu(g): torch's silu (fp64, CPU) as the library routine, and
    closed forms at points where the sigmoid is rational."""
    y = rng.standard_normal((T, D))
    g = 3.0 * rng.standard_normal((T, D))
    ref = torch.tensor(y) * torch.nn.functional.silu(torch.tensor(g))
    np.testing.assert_allclose(gated_fn(y, g), ref.numpy(), rtol=1e-13, atol=1e-15)
    # sigmoid(0) = 1/2, sigmoid(ln 3) = 3/4, sigmoid(-ln 3) = 1/4
    pts = np.array([0.0, np.log(3.0), -np.log(3.0)])
    np.testing.assert_allclose(silu_fn(pts), [0.0, 0.75 * np.log(3.0), -0.25 * np.log(3.0)],
                               rtol=1e-15, atol=0.0)
    # limits: silu(x) -> x for large x, -> 0 for very negative x
    assert math.isclose(silu_fn(np.array([40.0]))[0], 40.0, rel_tol=1e-15)
    assert abs(silu_fn(np.array([-40.0]))[0]) < 1e-15
    assert np.isfinite(silu_fn(np.array([-1000.0, 1000.0]))).all()
    # y = 1 everywhere returns silu(g) itself
    np.testing.assert_allclose(gated_fn(np.ones_like(g), g), silu_fn(g), rtol=0, atol=0)


def check_gated_backward(bwd_fn, rng, T=4, D=6, h=1e-6):
    """dy, dg of out = y * silu(g): torch autograd (fp64), central differences,
    closed form at g = 0 (silu(0) = 0, silu'(0) = 1/2)."""
    y = rng.standard_normal((T, D))
    g = 2.0 * rng.standard_normal((T, D))
    d = rng.standard_normal((T, D))
    out = bwd_fn(d, y, g)
    yt = torch.tensor(y, requires_grad=True)
    gt = torch.tensor(g, requires_grad=True)
    (yt * torch.nn.functional.silu(gt) * torch.tensor(d)).sum().backward()
    np.testing.assert_allclose(out["dy"], yt.grad.numpy(), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["dg"], gt.grad.numpy(), rtol=1e-12, atol=1e-14)
    # central differences of L = sum(d * y * silu(g)) in g, with silu written out here
    silu = lambda x: x / (1.0 + np.exp(-x))  # noqa: E731
    for (t, e) in [(0, 0), (1, 3), (3, 5)]:
        gp = g.copy(); gp[t, e] += h
        gm = g.copy(); gm[t, e] -= h
        fd = (float((d * y * silu(gp)).sum()) - float((d * y * silu(gm)).sum())) / (2 * h)
        assert abs(fd - out["dg"][t, e]) < 1e-7, (t, e, fd, out["dg"][t, e])
    z = bwd_fn(d, y, np.zeros_like(g))
    np.testing.assert_allclose(z["dy"], 0.0, atol=0)
    np.testing.assert_allclose(z["dg"], 0.5 * d * y, rtol=1e-15, atol=0)
    zero = bwd_fn(np.zeros_like(d), y, g)
    assert not zero["dy"].any() and not zero["dg"].any()


# ---------------------------------------------------- query normalisation ----
def check_query_layernorm(ln_fn, rng, T=5, H=3, n=12):
    """LayerNorm without affine: torch.nn.functional.layer_norm (fp64, CPU) as
    the library routine; the closed form for [1, 2, 3, 4]; zero mean and mean
    square var / (var + eps); invariance to a shift, and (eps = 0) to a
    positive scale; a constant query with eps = 0 gives zeros."""
    q = 3.0 * rng.standard_normal((T, H, n)) + 1.5
    for eps in (1e-5, 0.5):
        out = ln_fn(q, eps)
        ref = torch.nn.functional.layer_norm(torch.tensor(q), (n,), eps=eps)
        np.testing.assert_allclose(out["qhat"], ref.numpy(), rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(out["qhat"].mean(-1), 0.0, atol=1e-14)
        var = ((q - q.mean(-1, keepdims=True)) ** 2).mean(-1)
        np.testing.assert_allclose((out["qhat"] ** 2).mean(-1), var / (var + eps), rtol=1e-13)
        np.testing.assert_allclose(out["qhat"], ln_fn(q + 7.25, eps)["qhat"], rtol=1e-11, atol=1e-12)
    # mean 5/2, variance 5/4: (x - 5/2) / sqrt(5/4) = (2x - 5) / sqrt(5)
    x = np.array([[[1.0, 2.0, 3.0, 4.0]]])
    c = ln_fn(x, 0.0)
    np.testing.assert_allclose(c["qhat"][0, 0], np.array([-3.0, -1.0, 1.0, 3.0]) / math.sqrt(5.0),
                               rtol=1e-15, atol=0)
    assert math.isclose(float(c["mean"][0, 0]), 2.5, rel_tol=0, abs_tol=0)
    assert math.isclose(float(c["rstd"][0, 0]), 2.0 / math.sqrt(5.0), rel_tol=1e-15)
    np.testing.assert_allclose(ln_fn(4.0 * q, 0.0)["qhat"], ln_fn(q, 0.0)["qhat"], rtol=1e-12, atol=1e-13)
    z = ln_fn(np.full((1, 1, 6), 2.5), 0.0)
    assert not z["qhat"].any() and float(z["rstd"][0, 0]) == 0.0


def check_round_bf16(round_fn, rng):
    """Against torch's bfloat16 conversion of fp32 values (for a value that is
    exact in fp32 the single and the fp32-first roundings coincide), and hand
    ties: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 and goes to the even 1;
    1 + 3 * 2^-8 lies halfway between 1 + 2^-7 and 1 + 2^-6 and goes to 1 + 2^-6."""
    x = (rng.standard_normal(4000) * np.exp2(rng.integers(-20, 20, 4000))).astype(np.float32)
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(round_fn(x.astype(np.float64)), ref)
    ties = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), 255.5, 0.0, 0.75])
    np.testing.assert_array_equal(round_fn(ties), [1.0, 1 + 2.0 ** -6, -1.0, 256.0, 0.0, 0.75])


def exact_norm_rows(rng, T, H, n, shift=True):
    """Queries whose LayerNorm (eps = 0) is exact in binary arithmetic: each
    (t, h) row is c + 2^m * x with x a permutation of 3n/16 entries of each of
    +3 and -3 and 5n/16 of each of +1 and -1 (mean 0, variance 4), c an
    integer and m in {-1, 0, 1, 2}; its normalised form is x / 2.  Returns
    (q, x / 2).  n must be a multiple of 16."""
    assert n % 16 == 0
    a, b = 5 * n // 16, 3 * n // 16
    base = np.array([3.0] * b + [-3.0] * b + [1.0] * a + [-1.0] * a)
    xs = np.stack([rng.permutation(base) for _ in range(T * H)]).reshape(T, H, n)
    c = rng.integers(-4, 5, size=(T, H, 1)).astype(np.float64) if shift else 0.0
    m = np.exp2(rng.integers(-1, 3, size=(T, H, 1)).astype(np.float64)) if shift else 1.0
    return c + m * xs, xs / 2.0


def check_search_qnorm_exact(search_qnorm_fn, search_fn, brute_fn, rng, T=6, H=2, n=32, S=7, k=5):
    """eps = 0 on exactly normalisable rows: the normalised search equals the
    plain search, and brute force, on x / 2, ties included (integer sub-keys),
    and reports mean c and rstd 1 / (2 * 2^m)."""
    q, half = exact_norm_rows(rng, T, H, n)
    K = rng.integers(-2, 3, size=(H, 2, S, n // 2)).astype(np.float64)
    for dt in ("fp64", "bf16"):
        out = search_qnorm_fn(q, K, k, 0.0, dt)
        np.testing.assert_array_equal(out["qhat"], half)
        ref = search_fn(half, K, k)
        np.testing.assert_array_equal(out["idx"], ref["idx"])
        np.testing.assert_array_equal(out["idx"], brute_fn(half, K, k)["idx"])
        np.testing.assert_array_equal(out["score"], ref["score"])
        np.testing.assert_allclose(out["w"], ref["w"], rtol=1e-15, atol=0)
    np.testing.assert_allclose(out["mean"], q.mean(-1), rtol=0, atol=0)
    spread = (q - q.mean(-1, keepdims=True))[..., :1] / (2.0 * half[..., :1])
    np.testing.assert_allclose(out["rstd"], 1.0 / (2.0 * spread[..., 0]), rtol=1e-15)


def check_search_backward_qnorm(search_qnorm_fn, bwd_fn, rng, T=3, H=2, S=5, d=4, k=3, h=1e-6):
    """Gradient through the normalisation at a fixed selection: central
    differences in the raw queries and sub-keys of L = sum(gz * z(LN(q))), and
    torch autograd through layer_norm (fp64).  Storage rounding off (fp64)."""
    n = 2 * d
    q = 2.0 * rng.standard_normal((T, H, n)) + 0.7
    K = rng.standard_normal((H, 2, S, d))
    for eps in (1e-5, 0.25):
        idx = search_qnorm_fn(q, K, k, eps, "fp64")["idx"]
        gz = rng.standard_normal((T, H, k))
        g = bwd_fn(q, K, idx, gz, eps, "fp64")

        def L(qq, KK):
            mu = qq.mean(-1, keepdims=True)
            xc = qq - mu
            qh = xc / np.sqrt((xc * xc).mean(-1, keepdims=True) + eps)
            return float((selected_scores(qh, KK, idx) * gz).sum())

        for (t, hh, e) in [(0, 0, 0), (1, 1, 5), (2, 0, 7), (0, 1, 3)]:
            qp = q.copy(); qp[t, hh, e] += h
            qm = q.copy(); qm[t, hh, e] -= h
            fd = (L(qp, K) - L(qm, K)) / (2 * h)
            assert abs(fd - g["grad_q"][t, hh, e]) < 2e-7, (eps, t, hh, e, fd, g["grad_q"][t, hh, e])
        i1 = int(idx[0, 0, 0]) // S
        Kp = K.copy(); Kp[0, 0, i1, 1] += h
        Km = K.copy(); Km[0, 0, i1, 1] -= h
        fd = (L(q, Kp) - L(q, Km)) / (2 * h)
        assert abs(fd - g["grad_K"][0, 0, i1, 1]) < 2e-7
        qt = torch.tensor(q, requires_grad=True)
        Kt = torch.tensor(K, requires_grad=True)
        qh = torch.nn.functional.layer_norm(qt, (n,), eps=eps)
        it = torch.tensor(idx)
        j1, j2 = it // S, it % S
        hh_ = torch.arange(H).view(1, H, 1).expand_as(it)
        z = (qh[..., :d].unsqueeze(2) * Kt[hh_, 0, j1]).sum(-1) + (qh[..., d:].unsqueeze(2) * Kt[hh_, 1, j2]).sum(-1)
        (z * torch.tensor(gz)).sum().backward()
        np.testing.assert_allclose(g["grad_q"], qt.grad.numpy(), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(g["grad_K"], Kt.grad.numpy(), rtol=1e-10, atol=1e-12)
        # a LayerNorm gradient is orthogonal to the constant direction
        np.testing.assert_allclose(g["grad_q"].sum(-1), 0.0, atol=1e-10)
    # bf16 storage: the scores (and so grad_K) use the rounded query, and the
    # rounding passes the gradient unchanged into the LayerNorm backward
    eps = 1e-5
    idx = search_qnorm_fn(q, K, k, eps, "bf16")["idx"]
    gz = rng.standard_normal((T, H, k))
    g = bwd_fn(q, K, idx, gz, eps, "bf16")
    qt = torch.tensor(q, requires_grad=True)
    Kt = torch.tensor(K, requires_grad=True)
    qh = torch.nn.functional.layer_norm(qt, (n,), eps=eps)
    qs = qh + (qh.detach().float().to(torch.bfloat16).double() - qh.detach())
    it = torch.tensor(idx)
    j1, j2 = it // S, it % S
    hh_ = torch.arange(H).view(1, H, 1).expand_as(it)
    z = (qs[..., :d].unsqueeze(2) * Kt[hh_, 0, j1]).sum(-1) + (qs[..., d:].unsqueeze(2) * Kt[hh_, 1, j2]).sum(-1)
    (z * torch.tensor(gz)).sum().backward()
    np.testing.assert_allclose(g["grad_q"], qt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(g["grad_K"], Kt.grad.numpy(), rtol=1e-10, atol=1e-12)


def check_search_qnorm_rounding(search_qnorm_fn, rng, T=4, H=2, n=48, S=6, k=3):
    """The normalised queries as scored: torch's layer_norm (fp64) rounded by
    torch to fp32, and to bf16 via fp32 (seeded random values, where the two
    bf16 roundings coincide)."""
    q = 1.7 * rng.standard_normal((T, H, n)) - 0.4
    K = rng.standard_normal((H, 2, S, n // 2))
    ref = torch.nn.functional.layer_norm(torch.tensor(q), (n,), eps=1e-5)
    out = search_qnorm_fn(q, K, k, 1e-5, "fp32")
    np.testing.assert_array_equal(out["qhat"], ref.float().double().numpy())
    out = search_qnorm_fn(q, K, k, 1e-5, "bf16")
    np.testing.assert_array_equal(out["qhat"], ref.float().to(torch.bfloat16).double().numpy())


# ------------------------------------------------------ extra key-value pairs ----
def check_search_extra(extra_fn, search_fn, brute_fn, rng, T=5, H=2, S=6, d=3, k=4, r=3):
    """Extra pairs: r = 0 is the plain search; every extra slot's score is the
    full-key score of its index from the instantiated key set (brute force
    over all S^2 keys, integer inputs: exact); a repeated selected index
    repeats its score; the weights are exp(z) / sum exp(z) over the k + r
    scores (closed form, written here without max subtraction)."""
    q = rng.integers(-2, 3, size=(T, H, 2 * d)).astype(np.float64)
    K = rng.integers(-2, 3, size=(H, 2, S, d)).astype(np.float64)
    base = search_fn(q, K, k)
    out0 = extra_fn(q, K, k, np.zeros((T, H, 0), dtype=np.int64))
    np.testing.assert_array_equal(out0["idx"], base["idx"])
    np.testing.assert_allclose(out0["w"], base["w"], rtol=1e-15, atol=0)
    ex = rng.integers(0, S * S, size=(T, H, r))
    ex[0, 0, 0] = base["idx"][0, 0, 2]          # repeat of a selected key
    out = extra_fn(q, K, k, ex)
    assert out["idx"].shape == (T, H, k + r)
    np.testing.assert_array_equal(out["idx"][..., :k], base["idx"])
    np.testing.assert_array_equal(out["idx"][..., k:], ex)
    full = brute_fn(q, K, S * S)                # every key, rank order
    for t in range(T):
        for h in range(H):
            score_of = dict(zip(full["idx"][t, h].tolist(), full["score"][t, h].tolist()))
            for e in range(r):
                assert out["score"][t, h, k + e] == score_of[int(ex[t, h, e])]
    assert out["score"][0, 0, k] == out["score"][0, 0, 2]
    z = out["score"]
    np.testing.assert_allclose(out["w"], np.exp(z) / np.exp(z).sum(-1, keepdims=True), rtol=1e-12)
    np.testing.assert_allclose(out["w"].sum(-1), 1.0, rtol=1e-14)


# ------------------------------------------------------------ sink pair ----
def check_search_sink(sink_fn, extra_fn, rng, T=4, H=2, S=6, d=3, k=3, r=2):
    """Sink pair: with a zero key the sink's logit is 0 and the weights are
    exp(z_j) / (1 + sum exp(z)) over the other slots (closed form); the other
    slots are exactly `search_extra`'s; a sink key that scores far above every
    key takes the whole weight; the sink slot carries row sink_row0 + h."""
    n = 2 * d
    q = rng.standard_normal((T, H, n))
    K = rng.standard_normal((H, 2, S, d))
    ex = rng.integers(0, S * S, size=(T, H, r))
    base = extra_fn(q, K, k, ex)
    out = sink_fn(q, K, k, ex, np.zeros((H, n)), 1000)
    np.testing.assert_array_equal(out["idx"][..., :-1], base["idx"])
    np.testing.assert_array_equal(out["idx"][..., -1], 1000 + np.arange(H)[None, :].repeat(T, 0))
    np.testing.assert_allclose(out["score"][..., :-1], base["score"], rtol=0, atol=0)
    assert not out["score"][..., -1].any()
    e = np.exp(base["score"])
    np.testing.assert_allclose(out["w"][..., :-1], e / (1.0 + e.sum(-1, keepdims=True)), rtol=1e-12)
    np.testing.assert_allclose(out["w"][..., -1], 1.0 / (1.0 + e.sum(-1)), rtol=1e-12)
    # a sink key equal to a real key (its two sub-keys concatenated), also
    # passed as the last extra index: the two slots must score alike
    ij = rng.integers(0, S, size=(H, 2))
    ks_real = np.stack([np.concatenate([K[h, 0, ij[h, 0]], K[h, 1, ij[h, 1]]]) for h in range(H)])
    ex2 = ex.copy()
    ex2[..., -1] = (ij[:, 0] * S + ij[:, 1])[None, :]
    same = sink_fn(q, K, k, ex2, ks_real, 0)
    np.testing.assert_allclose(same["score"][..., -1], same["score"][..., -2], rtol=1e-12, atol=1e-12)
    ks = np.stack([1e3 * q[:, h].sum(0) / np.linalg.norm(q[:, h].sum(0)) for h in range(H)])
    hot = sink_fn(q, K, k, ex, ks, 7)
    z = hot["score"]
    dominant = (z[..., -1] > z[..., :-1].max(-1) + 60.0)
    assert dominant.any()
    np.testing.assert_allclose(hot["w"][..., -1][dominant], 1.0, rtol=1e-12)


def check_search_backward_sink(sink_fn, bwd_fn, rng, T=3, H=2, S=5, d=2, k=2, r=1, h=1e-6):
    """Sink gradients at a fixed selection: central differences in q and in the
    sink keys of L = sum(gz * z), torch autograd (fp64), accumulation."""
    n = 2 * d
    q = rng.standard_normal((T, H, n))
    K = rng.standard_normal((H, 2, S, d))
    ks = rng.standard_normal((H, n))
    ex = rng.integers(0, S * S, size=(T, H, r))
    sel = sink_fn(q, K, k, ex, ks, S * S)
    idx = sel["idx"]
    gz = rng.standard_normal(idx.shape)
    g = bwd_fn(q, K, idx, gz, ks)

    def L(qq, kk):
        z = selected_scores(qq, K, idx[..., :-1])
        zs = np.einsum("thn,hn->th", qq, kk)
        return float((z * gz[..., :-1]).sum() + (zs * gz[..., -1]).sum())

    for (t, hh, e) in [(0, 0, 0), (2, 1, 3), (1, 0, 2)]:
        qp = q.copy(); qp[t, hh, e] += h
        qm = q.copy(); qm[t, hh, e] -= h
        assert abs((L(qp, ks) - L(qm, ks)) / (2 * h) - g["grad_q"][t, hh, e]) < 1e-7
    for (hh, e) in [(0, 1), (1, 3)]:
        kp = ks.copy(); kp[hh, e] += h
        km = ks.copy(); km[hh, e] -= h
        assert abs((L(q, kp) - L(q, km)) / (2 * h) - g["grad_sink"][hh, e]) < 1e-7
    qt = torch.tensor(q, requires_grad=True)
    kt = torch.tensor(ks, requires_grad=True)
    zs = (qt * kt[None]).sum(-1)
    (zs * torch.tensor(gz[..., -1])).sum().backward()
    np.testing.assert_allclose(g["grad_sink"], kt.grad.numpy(), rtol=1e-12, atol=1e-14)
    base = rng.standard_normal(ks.shape)
    g2 = bwd_fn(q, K, idx, gz, ks, None, base)
    np.testing.assert_allclose(g2["grad_sink"], base + g["grad_sink"], rtol=1e-14, atol=1e-15)


# ------------------------------------------------- rows form, inversion ----
def check_rows_form(dense_fn, rows_fn, rng):
    """The touched-rows form of the value gradient: ascending distinct rows,
    each equal to the dense gradient's row exactly (same sums in the same
    order); every untouched dense row is zero."""
    V, idx, z, w, dy = random_bag_case(rng)
    T, H, k = idx.shape
    dense = dense_fn(dy, V, idx, w, H, k)["grad_values"]
    rows = rows_fn(dy, V, idx, w, H, k)
    assert list(rows["rows"]) == sorted(set(idx.ravel().tolist()))
    np.testing.assert_array_equal(dense[rows["rows"]], rows["grad_rows"])
    untouched = np.setdiff1d(np.arange(V.shape[0]), rows["rows"])
    assert np.all(dense[untouched] == 0)


def check_invert_index(inv_fn, rng):
    """CSR inversion of lookup -> row: offsets end at L, rows strictly
    ascending, every segment non-empty with ascending lookup ids that map back
    to its row, and the (row, lookup) pairs are exactly the input's."""
    idx = rng.integers(0, 20, size=300)
    inv = inv_fn(idx)
    assert inv["row_ptr"][0] == 0 and inv["row_ptr"][-1] == idx.size
    assert np.all(np.diff(inv["rows"]) > 0)
    pairs = []
    for u, r in enumerate(inv["rows"]):
        seg = inv["lookups"][inv["row_ptr"][u]:inv["row_ptr"][u + 1]]
        assert len(seg) > 0 and np.all(np.diff(seg) > 0)
        assert np.all(idx[seg] == r)
        pairs += [(int(r), int(l)) for l in seg]
    assert sorted(pairs) == sorted((int(r), l) for l, r in enumerate(idx))
