"""GPU parity over seeded random shapes within the documented limits: search
(S from 1 to 700, tiles of 64 sub-keys and of 256 tokens left ragged), bag
forward, bag backward in both modes, search backward — each against the fp64
oracle.  Integer-valued queries and sub-keys make every score exact, so the
selection and the scores must match bit for bit; everything else within 1e-5
(2e-2 for bf16 outputs), normwise."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from tests.test_gpu_parity import TOL_BF16, TOL_F32, h64, int_tensor, normwise

pytestmark = pytest.mark.gpu


def random_shape(seed):
    rng = np.random.default_rng(seed)
    f32 = rng.random() < 0.3
    S = int(rng.integers(1, 701))
    H = int(rng.integers(1, 9))
    d = int(rng.choice([4, 8, 12, 16, 32, 64])) if f32 else int(8 * rng.integers(1, 33))
    k = int(rng.integers(1, min(S, 64) + 1))
    T = int(rng.integers(1, 601))
    T = max(1, min(T, 12000 // (H * k)))  # keep the oracle's per-lookup loops short
    D = int(8 * rng.integers(1, 65))
    D = max(8, min(D, (1 << 24) // (S * S) // 8 * 8))  # the dense value gradient stays small
    return dict(S=S, H=H, n=2 * d, k=k, T=T, D=D, dt=torch.float32 if f32 else torch.bfloat16)


SEEDS = list(range(1000, 1024))


@pytest.mark.parametrize("seed", SEEDS)
def test_random_shape_full_path(gpu_lib, seed):
    c = random_shape(seed)
    S, H, n, k, T, D, dt = c["S"], c["H"], c["n"], c["k"], c["T"], c["D"], c["dt"]
    print(f"[random] seed {seed}: {c}", flush=True)
    N = S * S
    q = int_tensor((T, H, n), seed + 1, dt)
    K = int_tensor((H, 2, S, n // 2), seed + 2, dt)
    g = torch.Generator().manual_seed(seed + 3)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt)
    dy = torch.randn((T, D), generator=g).to(dt)
    idx, w, score, hidx = pk.mem_search(q.cuda(), K.cuda(), k, want_half=True)
    torch.cuda.synchronize()
    ref = oracle.search(h64(q), h64(K), k)
    np.testing.assert_array_equal(hidx.cpu().numpy(), ref["half_idx"])
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32

    tol_v = TOL_BF16 if dt == torch.bfloat16 else TOL_F32
    y = pk.mem_bag_forward(V.cuda(), idx.view(T, -1), w.view(T, -1))
    b = oracle.bag_backward(h64(dy), h64(V), ref["idx"], ref["w"], H, k)
    outs = {}
    for mode in ("sorted", "atomic"):
        outs[mode] = pk.mem_bag_backward(dy.cuda(), V.cuda(), idx, w, mode=mode)
    torch.cuda.synchronize()
    yref = oracle.bag_forward(h64(V), ref["idx"].reshape(T, -1), ref["w"].reshape(T, -1))
    assert normwise(h64(y), yref) <= tol_v
    for mode, (gv, gw, gz) in outs.items():
        assert normwise(h64(gv), b["grad_values"]) <= TOL_F32, mode
        assert normwise(h64(gw), b["grad_w"]) <= TOL_F32, mode
        assert normwise(h64(gz), b["grad_z"]) <= TOL_F32, mode

    gq, gK = pk.mem_search_backward(q.cuda(), K.cuda(), idx, outs["sorted"][2])
    torch.cuda.synchronize()
    s = oracle.search_backward(h64(q), h64(K), ref["idx"], b["grad_z"])
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32


@pytest.mark.parametrize("seed", list(range(2000, 2012)))
def test_random_shape_extra_and_sink(gpu_lib, seed):
    """Extra pairs (r random, possibly 0) and the sink pair over random shapes:
    search exact, then the bag over k + r + 1 slots (the sink values in rows
    S*S .. S*S + H - 1) and the sink search backward, against the oracle."""
    c = random_shape(seed)
    S, H, n, T, D, dt = c["S"], c["H"], c["n"], c["T"], c["D"], c["dt"]
    rng = np.random.default_rng(seed)
    k = min(c["k"], 48)
    r = int(rng.integers(0, 64 - k))  # k + r + 1 <= 64
    T = max(1, min(T, 12000 // (H * (k + r + 1))))
    print(f"[random sink] seed {seed}: S={S} H={H} n={n} k={k} r={r} T={T} D={D} {dt}", flush=True)
    N = S * S + H
    q = int_tensor((T, H, n), seed + 1, dt)
    K = int_tensor((H, 2, S, n // 2), seed + 2, dt)
    ks = int_tensor((H, n), seed + 4, dt, -1, 1)
    g = torch.Generator().manual_seed(seed + 3)
    ex = torch.randint(0, S * S, (T, H, r), generator=g, dtype=torch.int64)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt)
    dy = torch.randn((T, D), generator=g).to(dt)
    idx, w, score, _ = pk.mem_search_sink(q.cuda(), K.cuda(), k, ks.cuda(), S * S, ex.cuda())
    torch.cuda.synchronize()
    ref = oracle.search_sink(h64(q), h64(K), k, ex.numpy(), h64(ks), S * S)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32
    kk = k + r + 1
    gv, gw, gz = pk.mem_bag_backward(dy.cuda(), V.cuda(), idx, w, mode="sorted")
    gq, gK, gs = pk.mem_search_backward_sink(q.cuda(), K.cuda(), idx, gz, ks.cuda())
    torch.cuda.synchronize()
    b = oracle.bag_backward(h64(dy), h64(V), ref["idx"], ref["w"], H, kk)
    assert normwise(h64(gv), b["grad_values"]) <= TOL_F32
    assert normwise(h64(gz), b["grad_z"]) <= TOL_F32
    s = oracle.search_backward_sink(h64(q), h64(K), ref["idx"], b["grad_z"], h64(ks))
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32
    # the sink's weight can be negligible (peaked softmax over integer scores):
    # its score gradient then underflows in fp32, so the error is measured
    # against one token's contribution to a key gradient as well
    scale = max(np.abs(s["grad_sink"]).max(), np.abs(b["grad_z"]).max() * np.abs(h64(q)).max())
    assert np.abs(h64(gs) - s["grad_sink"]).max() <= TOL_F32 * scale


@pytest.mark.parametrize("seed", list(range(3000, 3012)))
def test_random_large_S_search_and_backward(gpu_lib, seed):
    """Search and search backward at random S from 1500 to 8192 (every first
    sweep split: a half, a quarter or an eighth of the chunks, ragged last
    chunks), random k <= 64, H, d and dtype: integer inputs in [-32, 32]
    (scores exact in fp32), selection bit for bit and gradients within 1e-5
    against the oracle."""
    rng = np.random.default_rng(seed)
    f32 = rng.random() < 0.3
    S = int(rng.integers(1500, 8193))
    H = int(rng.integers(1, 5))
    d = int(rng.choice([8, 16, 32])) if f32 else int(8 * rng.integers(1, 17))
    k = int(rng.integers(1, 65))
    T = int(rng.integers(1, 40))
    dt = torch.float32 if f32 else torch.bfloat16
    n = 2 * d
    print(f"[random large S] seed {seed}: S={S} H={H} n={n} k={k} T={T} {dt}", flush=True)
    q = int_tensor((T, H, n), seed + 1, dt, -32, 32)
    K = int_tensor((H, 2, S, d), seed + 2, dt, -32, 32)
    idx, w, score, hidx = pk.mem_search(q.cuda(), K.cuda(), k, want_half=True)
    torch.cuda.synchronize()
    ref = oracle.search(h64(q), h64(K), k)
    np.testing.assert_array_equal(hidx.cpu().numpy(), ref["half_idx"])
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32
    g = torch.Generator().manual_seed(seed + 3)
    gz = torch.randn((T, H, k), generator=g)
    gq, gK = pk.mem_search_backward(q.cuda(), K.cuda(), idx, gz.cuda())
    torch.cuda.synchronize()
    s = oracle.search_backward(h64(q), h64(K), ref["idx"], gz.double().numpy())
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32
