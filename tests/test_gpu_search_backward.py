"""GPU parity of mem_search_backward (gradients into queries and sub-keys)
against the fp64 oracle.  Integer-valued queries and sub-keys make the
selection exact, so the oracle's own selection equals the GPU's; fp32
outputs within 1e-5 normwise."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_queries, gen_subkeys
from tests.test_gpu_parity import TOL_F32, _certify_near_ties, h64, int_tensor, normwise

pytestmark = pytest.mark.gpu

CASES = [
    ("tiny_f32_S64_k8", 64, 1, 64, 8, 256, torch.float32),
    ("bf16_S1024_H4_k32", 1024, 4, 512, 32, 200, torch.bfloat16),
    ("bf16_S100_d32", 100, 2, 64, 16, 130, torch.bfloat16),
    ("bf16_k64_d64", 256, 2, 128, 64, 70, torch.bfloat16),
    ("f32_d64_S200", 200, 2, 128, 20, 99, torch.float32),
    ("bf16_d8_ties", 50, 3, 16, 10, 77, torch.bfloat16),
    ("bf16_S8192_d256", 8192, 1, 512, 16, 300, torch.bfloat16),
    ("f32_S3000_d24_k64", 3000, 2, 48, 64, 45, torch.float32),
    ("bf16_S1_k1", 1, 2, 16, 1, 70, torch.bfloat16),
    ("bf16_S2_k2_H8", 2, 8, 16, 2, 300, torch.bfloat16),
    ("bf16_H16_S64", 64, 16, 32, 8, 40, torch.bfloat16),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_search_backward_integer_inputs(gpu_lib, case):
    name, S, H, n, k, T, dt = case
    print(f"[search-bwd] {name}", flush=True)
    q = int_tensor((T, H, n), 21, dt)
    K = int_tensor((H, 2, S, n // 2), 22, dt)
    gz = torch.randn((T, H, k), generator=torch.Generator().manual_seed(23))
    base = torch.randn((H, 2, S, n // 2), generator=torch.Generator().manual_seed(24))
    idx, w, _, _ = pk.mem_search(q.cuda(), K.cuda(), k)
    gq, gK = pk.mem_search_backward(q.cuda(), K.cuda(), idx, gz.cuda(), grad_subkeys=base.clone().cuda())
    torch.cuda.synchronize()
    s = oracle.search(h64(q), h64(K), k)
    np.testing.assert_array_equal(idx.cpu().numpy(), s["idx"])
    ref = oracle.search_backward(h64(q), h64(K), s["idx"], gz.double().numpy())
    assert normwise(h64(gq), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(gK) - base.double().numpy(), ref["grad_K"]) <= TOL_F32


def test_search_backward_optional_outputs(gpu_lib):
    S, H, n, k, T = 64, 2, 64, 8, 40
    q = int_tensor((T, H, n), 31, torch.bfloat16).cuda()
    K = int_tensor((H, 2, S, n // 2), 32, torch.bfloat16).cuda()
    gz = torch.randn((T, H, k), generator=torch.Generator().manual_seed(33)).cuda()
    idx, _, _, _ = pk.mem_search(q, K, k)
    gq_only, none_k = pk.mem_search_backward(q, K, idx, gz, want_grad_subkeys=False)
    none_q, gk_only = pk.mem_search_backward(q, K, idx, gz, want_grad_q=False)
    gq, gk = pk.mem_search_backward(q, K, idx, gz)
    torch.cuda.synchronize()
    assert none_k is None and none_q is None
    assert torch.equal(gq_only, gq)
    assert normwise(h64(gk_only), h64(gk)) <= TOL_F32


def test_search_backward_full_size_sampled(gpu_lib):
    """4M-key workload at full size; grad_scores zero outside 48 sampled tokens,
    so the accumulated sub-key gradient holds exactly their contributions."""
    wl = WORKLOADS["pk4m_d2048"]
    dev = torch.device("cuda:0")
    T, H, k = wl.T, wl.H, wl.k
    q = gen_queries(wl, dev)
    K = gen_subkeys(wl, dev)
    idx, w, _, _ = pk.mem_search(q, K, k)
    rng = np.random.default_rng(5)
    samp = np.unique(np.concatenate([np.arange(16), np.arange(T - 16, T),
                                     rng.choice(np.arange(16, T - 16), 16, replace=False)]))
    st = torch.from_numpy(samp).to(dev)
    qh, Kh = h64(q[st]), h64(K)
    s = oracle.search(qh, Kh, k)
    gi = idx[st].cpu().numpy()
    assert _certify_near_ties(qh, Kh, k, gi, s) == 0
    ok = (gi == s["idx"]).all(-1).all(-1)
    keep = samp[ok]
    assert len(keep) >= 40
    gz = torch.zeros((T, H, k), device=dev)
    gz_keep = torch.randn((len(keep), H, k), generator=torch.Generator().manual_seed(7)).to(dev)
    gz[torch.from_numpy(keep).to(dev)] = gz_keep
    gq, gK = pk.mem_search_backward(q, K, idx, gz)
    torch.cuda.synchronize()
    ref = oracle.search_backward(qh[ok], Kh, s["idx"][ok], gz_keep.double().cpu().numpy())
    assert normwise(h64(gq[torch.from_numpy(keep).to(dev)]), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), ref["grad_K"]) <= TOL_F32
    others = torch.ones(T, dtype=torch.bool, device=dev)
    others[torch.from_numpy(keep).to(dev)] = False
    assert float(gq[others].abs().max()) == 0.0


def test_search_backward_deterministic_and_skips_invalid_indices(gpu_lib):
    """Two calls give bitwise-equal gradients (sorted, atomic-free sums), and a
    lookup whose index lies outside [0, S*S) contributes nothing: the result
    equals the oracle's with that lookup's gradient set to zero."""
    S, H, n, k, T = 128, 2, 64, 16, 300
    g = torch.Generator().manual_seed(41)
    q = torch.randn((T, H, n), generator=g).to(torch.bfloat16)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 8).to(torch.bfloat16)
    gz = torch.randn((T, H, k), generator=g)
    idx, _, _, _ = pk.mem_search(q.cuda(), K.cuda(), k)
    bad = [(0, 0, 3), (5, 1, 0), (299, 1, 15)]
    for (t, h, j), v in zip(bad, (-1, S * S, 1 << 40)):
        idx[t, h, j] = v
    runs = [pk.mem_search_backward(q.cuda(), K.cuda(), idx, gz.cuda()) for _ in range(2)]
    torch.cuda.synchronize()
    assert torch.equal(runs[0][0], runs[1][0]) and torch.equal(runs[0][1], runs[1][1])
    idx_ref = idx.cpu().numpy().copy()
    gz_ref = gz.double().numpy().copy()
    for t, h, j in bad:
        idx_ref[t, h, j] = 0
        gz_ref[t, h, j] = 0.0
    ref = oracle.search_backward(h64(q), h64(K), idx_ref, gz_ref)
    assert normwise(h64(runs[0][0]), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(runs[0][1]), ref["grad_K"]) <= TOL_F32


@pytest.mark.parametrize("qnorm", [False, True], ids=["plain", "qnorm"])
def test_search_backward_long_segments(gpu_lib, qnorm):
    """Sub-keys chosen by thousands of tokens: 3000 of the 3500 tokens select
    the same 8 composed indices (2 x 4 sub-keys per head), so their sub-key
    segments hold more than 2048 pairs and are summed by a workgroup each; the
    other tokens' indices are uniform (short segments).  Against the oracle,
    and bitwise repeatable."""
    S, H, n, k, T, hot = 64, 2, 64, 8, 3500, 3000
    q = int_tensor((T, H, n), 131, torch.bfloat16)
    K = int_tensor((H, 2, S, n // 2), 132, torch.bfloat16)
    g = torch.Generator().manual_seed(133)
    j = torch.arange(k)
    idx = torch.randint(0, S * S, (T, H, k), generator=g)
    idx[:hot] = ((j // 4) * S + (j % 4)).view(1, 1, k)
    idx = idx[torch.randperm(T, generator=g)].contiguous()  # hot tokens spread over the batch
    gz = torch.randn((T, H, k), generator=g)
    args = (q.cuda(), K.cuda(), idx.cuda(), gz.cuda())
    if qnorm:
        a = pk.mem_search_backward_qnorm(*args, 1e-5)
        b = pk.mem_search_backward_qnorm(*args, 1e-5)
        ref = oracle.search_backward_qnorm(h64(q), h64(K), idx.numpy(), h64(gz), 1e-5, "bf16")
    else:
        a = pk.mem_search_backward(*args)
        b = pk.mem_search_backward(*args)
        ref = oracle.search_backward(h64(q), h64(K), idx.numpy(), h64(gz))
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    assert normwise(h64(a[0]), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(a[1]), ref["grad_K"]) <= TOL_F32
    # the hot sub-key rows themselves (the long segments)
    for p, rows in ((0, [0, 1]), (1, [0, 1, 2, 3])):
        assert normwise(h64(a[1])[:, p, rows], ref["grad_K"][:, p, rows]) <= TOL_F32
