"""GPU parity of mem_search_extra (extra key-value pairs beside the top-k,
scored as full keys and joined to the softmax) against the fp64 oracle, and
of the unchanged bag and search backwards run with k + r slots.  Integer
inputs make every score exact, so indices and scores must match bit for bit;
weights within 1e-5."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_queries, gen_subkeys
from tests.test_gpu_parity import TOL_BF16, TOL_F32, _certify_near_ties, h64, int_tensor, normwise

pytestmark = pytest.mark.gpu

CASES = [
    # (name, S, H, n, k, r, T, dtype)
    ("bf16_S1024_H4_k32_r32_ragged", 1024, 4, 512, 32, 32, 200, torch.bfloat16),
    ("bf16_S100_k16_r8", 100, 2, 64, 16, 8, 130, torch.bfloat16),
    ("bf16_k1_r1", 512, 1, 16, 1, 1, 300, torch.bfloat16),
    ("bf16_k63_r1", 256, 2, 128, 63, 1, 70, torch.bfloat16),
    ("f32_S200_d64_r5", 200, 2, 128, 20, 5, 99, torch.float32),
    ("bf16_S8192_r16", 8192, 1, 512, 16, 16, 40, torch.bfloat16),
]


def extra_indices(T, H, r, S, seed, dup_from=None):
    g = torch.Generator().manual_seed(seed)
    ex = torch.randint(0, S * S, (T, H, r), generator=g, dtype=torch.int64)
    if dup_from is not None:  # some extras repeat a selected key
        ex[::3, :, 0] = dup_from[::3, :, 0]
    return ex


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_search_extra_integer_inputs(gpu_lib, case):
    name, S, H, n, k, r, T, dt = case
    print(f"[extra] {name}", flush=True)
    q = int_tensor((T, H, n), 51, dt)
    K = int_tensor((H, 2, S, n // 2), 52, dt)
    sel = oracle.search(h64(q), h64(K), k)["idx"]
    ex = extra_indices(T, H, r, S, 53, torch.from_numpy(sel))
    idx, w, score, hidx = pk.mem_search_extra(q.cuda(), K.cuda(), k, ex.cuda(), want_half=True)
    torch.cuda.synchronize()
    ref = oracle.search_extra(h64(q), h64(K), k, ex.numpy())
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    np.testing.assert_array_equal(hidx.cpu().numpy(), ref["half_idx"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32
    np.testing.assert_allclose(h64(w).sum(-1), 1.0, rtol=1e-5)


def test_search_extra_without_extras_is_the_plain_search(gpu_lib):
    S, H, n, k, T = 1024, 4, 512, 32, 300
    q = torch.randn((T, H, n), generator=torch.Generator().manual_seed(5)).to(torch.bfloat16).cuda()
    K = (torch.randn((H, 2, S, n // 2), generator=torch.Generator().manual_seed(6)) / 16).to(torch.bfloat16).cuda()
    a = pk.mem_search(q, K, k)
    b = pk.mem_search_extra(q, K, k, torch.zeros((T, H, 0), dtype=torch.int64, device="cuda"))
    torch.cuda.synchronize()
    for x, y in zip(a[:3], b[:3]):
        assert torch.equal(x, y)


def test_search_extra_float_inputs(gpu_lib):
    S, H, n, k, r, T = 1024, 4, 512, 32, 16, 256
    g = torch.Generator().manual_seed(61)
    q = torch.randn((T, H, n), generator=g).to(torch.bfloat16)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 16).to(torch.bfloat16)
    ex = extra_indices(T, H, r, S, 62)
    idx, w, score, _ = pk.mem_search_extra(q.cuda(), K.cuda(), k, ex.cuda())
    torch.cuda.synchronize()
    qh, Kh = h64(q), h64(K)
    ref = oracle.search_extra(qh, Kh, k, ex.numpy())
    gi = idx.cpu().numpy()
    np.testing.assert_array_equal(gi[..., k:], ex.numpy())
    plain = {kk: v[..., :k] for kk, v in ref.items() if kk in ("idx", "score")}
    assert _certify_near_ties(qh, Kh, k, gi[..., :k], plain) == 0
    ok = (gi[..., :k] == ref["idx"][..., :k]).all(-1)
    assert ok.mean() > 0.9
    # extra scores: fp32 sums of exact bf16 products
    assert normwise(h64(score)[..., k:], ref["score"][..., k:]) <= TOL_F32
    assert normwise(h64(score)[ok], ref["score"][ok]) <= TOL_F32
    assert normwise(h64(w)[ok], ref["w"][ok]) <= TOL_F32


def test_extra_slots_through_bag_and_search_backward(gpu_lib):
    """The bag forward / backward and the search backward take the k + r
    slots unchanged: each against the oracle on the same selection."""
    S, H, n, k, r, T, N, D = 64, 2, 64, 8, 4, 150, 64 * 64, 256
    dt = torch.bfloat16
    q = int_tensor((T, H, n), 71, dt)
    K = int_tensor((H, 2, S, n // 2), 72, dt)
    ex = extra_indices(T, H, r, S, 73)
    g = torch.Generator().manual_seed(74)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt)
    dy = torch.randn((T, D), generator=g).to(dt)
    idx, w, score, _ = pk.mem_search_extra(q.cuda(), K.cuda(), k, ex.cuda())
    y = pk.mem_bag_forward(V.cuda(), idx.view(T, -1), w.view(T, -1))
    gv = torch.zeros((N, D), dtype=torch.float32, device="cuda")
    gv, gw, gz = pk.mem_bag_backward(dy.cuda(), V.cuda(), idx, w, grad_values=gv, mode="sorted")
    gq, gK = pk.mem_search_backward(q.cuda(), K.cuda(), idx, gz)
    torch.cuda.synchronize()
    ref = oracle.search_extra(h64(q), h64(K), k, ex.numpy())
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    kk = k + r
    yref = oracle.bag_forward(h64(V), ref["idx"].reshape(T, -1), ref["w"].reshape(T, -1))
    assert normwise(h64(y), yref) <= TOL_BF16
    b = oracle.bag_backward(h64(dy), h64(V), ref["idx"], ref["w"], H, kk)
    assert normwise(h64(gv), b["grad_values"]) <= TOL_F32
    assert normwise(h64(gw), b["grad_w"]) <= TOL_F32
    assert normwise(h64(gz), b["grad_z"]) <= TOL_F32
    s = oracle.search_backward(h64(q), h64(K), ref["idx"], b["grad_z"])
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32


def test_search_extra_full_size_sampled(gpu_lib):
    """1M-key workload at full size with 16 extra pairs per (token, head):
    sampled tokens against the oracle."""
    wl = WORKLOADS["pk1m_d1024"]
    dev = torch.device("cuda:0")
    q = gen_queries(wl, dev)
    K = gen_subkeys(wl, dev)
    r = 16
    ex = torch.randint(0, wl.N, (wl.T, wl.H, r), generator=torch.Generator().manual_seed(81),
                       dtype=torch.int64)
    idx, w, score, _ = pk.mem_search_extra(q, K, wl.k, ex.to(dev))
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    samp = np.unique(np.concatenate([np.arange(8), np.arange(wl.T - 8, wl.T),
                                     rng.choice(np.arange(8, wl.T - 8), 16, replace=False)]))
    st = torch.from_numpy(samp).to(dev)
    qh, Kh = h64(q[st]), h64(K)
    ref = oracle.search_extra(qh, Kh, wl.k, ex[torch.from_numpy(samp)].numpy())
    gi = idx[st].cpu().numpy()
    np.testing.assert_array_equal(gi[..., wl.k:], ref["idx"][..., wl.k:])
    plain = {kk: v[..., :wl.k] for kk, v in ref.items() if kk in ("idx", "score")}
    assert _certify_near_ties(qh, Kh, wl.k, gi[..., :wl.k], plain) == 0
    ok = (gi == ref["idx"]).all(-1)
    assert ok.mean() > 0.9
    assert normwise(h64(score[st])[..., wl.k:], ref["score"][..., wl.k:]) <= TOL_F32
    assert normwise(h64(w[st])[ok], ref["w"][ok]) <= TOL_F32


def test_extra_slots_beyond_S_through_search_backward(gpu_lib):
    """k + r may exceed S (S = 6, k = 6, r = 5: 11 slots, every extra a repeat
    of some selected key): the search backward takes all 11 slots."""
    S, H, n, k, r, T = 6, 2, 16, 6, 5, 90
    dt = torch.bfloat16
    q = int_tensor((T, H, n), 75, dt)
    K = int_tensor((H, 2, S, n // 2), 76, dt)
    ex = extra_indices(T, H, r, S, 77)
    gz = torch.randn((T, H, k + r), generator=torch.Generator().manual_seed(78))
    idx, w, score, _ = pk.mem_search_extra(q.cuda(), K.cuda(), k, ex.cuda())
    gq, gK = pk.mem_search_backward(q.cuda(), K.cuda(), idx, gz.cuda())
    torch.cuda.synchronize()
    ref = oracle.search_extra(h64(q), h64(K), k, ex.numpy())
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    s = oracle.search_backward(h64(q), h64(K), ref["idx"], h64(gz))
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32
