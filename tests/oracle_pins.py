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
