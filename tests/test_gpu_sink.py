"""GPU parity of mem_search_sink / mem_search_backward_sink (a fixed key-value
pair per head beside the selection, Sec. 5.4) against the fp64 oracle.
Integer inputs make every score exact, so indices and scores must match bit
for bit; weights and gradients within 1e-5 (normwise).  The sink's value is a
row of the value table after the S*S key rows, so the unchanged bag forward
and backward carry it."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_queries, gen_subkeys
from tests.test_gpu_parity import TOL_BF16, TOL_F32, h64, int_tensor, normwise

pytestmark = pytest.mark.gpu

CASES = [
    # (name, S, H, n, k, r, T, dtype)
    ("bf16_S1024_H4_k32_r0_ragged", 1024, 4, 512, 32, 0, 200, torch.bfloat16),
    ("bf16_S1024_H4_k32_r16", 1024, 4, 512, 32, 16, 130, torch.bfloat16),
    ("bf16_k1_r0", 512, 1, 16, 1, 0, 300, torch.bfloat16),
    ("bf16_k55_r8_64_slots", 256, 2, 128, 55, 8, 70, torch.bfloat16),
    ("bf16_k63_r0_64_slots", 256, 2, 64, 63, 0, 33, torch.bfloat16),
    ("f32_S200_d64_r5", 200, 2, 128, 20, 5, 99, torch.float32),
]


def _extras(T, H, r, S, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.randint(0, S * S, (T, H, r), generator=g, dtype=torch.int64)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_search_sink_integer_inputs(gpu_lib, case):
    name, S, H, n, k, r, T, dt = case
    print(f"[sink] {name}", flush=True)
    q = int_tensor((T, H, n), 91, dt)
    K = int_tensor((H, 2, S, n // 2), 92, dt)
    ks = int_tensor((H, n), 93, dt, -1, 1)
    ex = _extras(T, H, r, S, 94)
    row0 = S * S + 5
    idx, w, score, hidx = pk.mem_search_sink(q.cuda(), K.cuda(), k, ks.cuda(), row0, ex.cuda(),
                                             want_half=True)
    torch.cuda.synchronize()
    ref = oracle.search_sink(h64(q), h64(K), k, ex.numpy(), h64(ks), row0)
    assert idx.shape == (T, H, k + r + 1)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    np.testing.assert_array_equal(hidx.cpu().numpy(), ref["half_idx"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32
    np.testing.assert_allclose(h64(w).sum(-1), 1.0, rtol=1e-5)


def test_zero_sink_key_adds_one_to_the_denominator(gpu_lib):
    """Zero key: logit 0 in the sink slot, so every weight is exp(z_j) / (1 +
    sum exp(z)): w_j / w_sink = exp(z_j) on the call's own scores, which equal
    mem_search's (scores scaled small so that the sink's weight is not
    negligible)."""
    S, H, n, k, T = 512, 2, 128, 16, 257
    g = torch.Generator().manual_seed(95)
    q = (torch.randn((T, H, n), generator=g) * 0.05).to(torch.bfloat16).cuda()
    K = (torch.randn((H, 2, S, n // 2), generator=g) * 0.05).to(torch.bfloat16).cuda()
    ks = torch.zeros((H, n), dtype=torch.bfloat16, device="cuda")
    plain_idx, _, plain_score, _ = pk.mem_search(q, K, k)
    idx, w, score, _ = pk.mem_search_sink(q, K, k, ks, S * S)
    torch.cuda.synchronize()
    assert torch.equal(idx[..., :k], plain_idx) and torch.equal(score[..., :k], plain_score)
    assert float(score[..., k].abs().max()) == 0.0
    wh = h64(w)
    assert normwise(wh[..., :k] / wh[..., k:], np.exp(h64(score)[..., :k])) <= TOL_F32
    np.testing.assert_allclose(wh.sum(-1), 1.0, rtol=1e-5)
    assert wh[..., k].min() > 0.01
    np.testing.assert_array_equal(idx[..., k].cpu().numpy(), S * S + np.arange(H)[None, :].repeat(T, 0))


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_sink_through_bag_and_search_backward(gpu_lib, dt):
    """search_sink -> bag forward -> sorted bag backward -> search_backward_sink,
    each against the oracle on the same selection; grad_subkeys and grad_sink
    accumulate into non-zero tables."""
    S, H, n, k, r, T, D = 64, 2, 64, 8, 3, 700, 256  # T spans 3 chunks of 256 and a ragged tail
    N = S * S + H
    q = int_tensor((T, H, n), 101, dt)
    K = int_tensor((H, 2, S, n // 2), 102, dt)
    ks = int_tensor((H, n), 103, dt, -1, 1)
    ex = _extras(T, H, r, S, 104)
    g = torch.Generator().manual_seed(105)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt)
    dy = torch.randn((T, D), generator=g).to(dt)
    gK0 = torch.randn((H, 2, S, n // 2), generator=g)
    gs0 = torch.randn((H, n), generator=g)
    idx, w, score, _ = pk.mem_search_sink(q.cuda(), K.cuda(), k, ks.cuda(), S * S, ex.cuda())
    kk = k + r + 1
    y = pk.mem_bag_forward(V.cuda(), idx.view(T, -1), w.view(T, -1))
    gv = torch.zeros((N, D), dtype=torch.float32, device="cuda")
    gv, gw, gz = pk.mem_bag_backward(dy.cuda(), V.cuda(), idx, w, grad_values=gv, mode="sorted")
    gq, gK, gs = pk.mem_search_backward_sink(q.cuda(), K.cuda(), idx, gz, ks.cuda(),
                                             grad_subkeys=gK0.cuda(), grad_sink=gs0.cuda())
    torch.cuda.synchronize()
    ref = oracle.search_sink(h64(q), h64(K), k, ex.numpy(), h64(ks), S * S)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    yref = oracle.bag_forward(h64(V), ref["idx"].reshape(T, -1), ref["w"].reshape(T, -1))
    assert normwise(h64(y), yref) <= (TOL_BF16 if dt == torch.bfloat16 else TOL_F32)
    b = oracle.bag_backward(h64(dy), h64(V), ref["idx"], ref["w"], H, kk)
    assert normwise(h64(gv), b["grad_values"]) <= TOL_F32
    assert normwise(h64(gv)[S * S:], b["grad_values"][S * S:]) <= TOL_F32  # the sink values' rows
    assert normwise(h64(gz), b["grad_z"]) <= TOL_F32
    s = oracle.search_backward_sink(h64(q), h64(K), ref["idx"], b["grad_z"], h64(ks),
                                    h64(gK0), h64(gs0))
    assert normwise(h64(gq), s["grad_q"]) <= TOL_F32
    assert normwise(h64(gK), s["grad_K"]) <= TOL_F32
    assert normwise(h64(gs), s["grad_sink"]) <= TOL_F32
    assert normwise(h64(gs) - h64(gs0), s["grad_sink"] - h64(gs0)) <= TOL_F32


def test_search_backward_sink_deterministic_and_parts(gpu_lib):
    """Bitwise repeatable; each output alone equals the same output of the
    full call; a second call adds exactly the same sums (x + x = 2x); the sink
    slot never reaches the sub-key gradients.  Integer inputs: the selection is
    the oracle's exactly."""
    S, H, n, k, T = 128, 4, 256, 16, 1300
    dev = torch.device("cuda:0")
    q = int_tensor((T, H, n), 111, torch.bfloat16)
    K = int_tensor((H, 2, S, n // 2), 112, torch.bfloat16)
    ks = int_tensor((H, n), 113, torch.bfloat16, -1, 1)
    gz = torch.randn((T, H, k + 1), generator=torch.Generator().manual_seed(114))
    qd, Kd, ksd, gzd = q.to(dev), K.to(dev), ks.to(dev), gz.to(dev)
    idx, w, _, _ = pk.mem_search_sink(qd, Kd, k, ksd, S * S)
    a = pk.mem_search_backward_sink(qd, Kd, idx, gzd, ksd)
    b = pk.mem_search_backward_sink(qd, Kd, idx, gzd, ksd)
    only_q = pk.mem_search_backward_sink(qd, Kd, idx, gzd, ksd, want_grad_subkeys=False,
                                         want_grad_sink=False)[0]
    only_s = pk.mem_search_backward_sink(qd, Kd, idx, gzd, ksd, want_grad_q=False,
                                         want_grad_subkeys=False)[2]
    twice = pk.mem_search_backward_sink(qd, Kd, idx, gzd, ksd, grad_subkeys=a[1].clone(),
                                        grad_sink=a[2].clone())
    _, gK_plain = pk.mem_search_backward(qd, Kd, idx[..., :k].contiguous(), gzd[..., :k].contiguous())
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    assert torch.equal(only_q, a[0]) and torch.equal(only_s, a[2])
    assert torch.equal(twice[2], 2 * a[2]) and torch.equal(twice[1], 2 * a[1])
    assert torch.equal(gK_plain, a[1])
    sel = oracle.search_sink(h64(q), h64(K), k, np.zeros((T, H, 0), dtype=np.int64), h64(ks), S * S)
    np.testing.assert_array_equal(idx.cpu().numpy(), sel["idx"])
    ref = oracle.search_backward_sink(h64(q), h64(K), sel["idx"], h64(gz), h64(ks))
    assert normwise(h64(a[0]), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(a[1]), ref["grad_K"]) <= TOL_F32
    assert normwise(h64(a[2]), ref["grad_sink"]) <= TOL_F32


def test_search_sink_full_size_sampled(gpu_lib):
    """4M-key workload at full size (32768 tokens, 4 heads, n = 512) with a
    sink, in the launch configuration of the benchmark: sampled tokens of the
    forward against the oracle; grad_sink (a sum over every token) against the
    oracle in full; grad_q on the sampled tokens whose selection is the
    oracle's (grad_scores zero elsewhere)."""
    wl = WORKLOADS["pk4m_d2048"]
    dev = torch.device("cuda:0")
    T, H, k = wl.T, wl.H, wl.k
    q = gen_queries(wl, dev)
    K = gen_subkeys(wl, dev)
    g = torch.Generator().manual_seed(121)
    ks = (torch.randn((H, wl.n), generator=g) / 16).to(q.dtype)
    idx, w, score, _ = pk.mem_search_sink(q, K, k, ks.to(dev), wl.N)
    rng = np.random.default_rng(4)
    samp = np.unique(np.concatenate([np.arange(4), np.arange(T - 4, T),
                                     rng.choice(np.arange(4, T - 4), 16, replace=False)]))
    st = torch.from_numpy(samp).to(dev)
    qs, Kh = h64(q[st]), h64(K)
    sel = oracle.search_sink(qs, Kh, k, np.zeros((len(samp), H, 0), dtype=np.int64), h64(ks), wl.N)
    gi = idx[st].cpu().numpy()
    np.testing.assert_array_equal(gi[..., -1], sel["idx"][..., -1])
    assert normwise(h64(score[st])[..., -1], sel["score"][..., -1]) <= TOL_F32
    ok = (gi == sel["idx"]).all(-1).all(-1)
    assert ok.mean() > 0.8
    keep = samp[ok]
    # grad_scores: the sink slot everywhere, the product-key slots on the kept samples
    gz = torch.zeros((T, H, k + 1))
    gz[..., k] = torch.randn((T, H), generator=g) * 0.01
    gz[torch.from_numpy(keep), :, :k] = torch.randn((len(keep), H, k), generator=g) * 0.01
    gq, _, gs = pk.mem_search_backward_sink(q, K, idx, gz.to(dev), ks.to(dev), want_grad_subkeys=False)
    torch.cuda.synchronize()
    ref = oracle.search_backward_sink(qs[ok], Kh, sel["idx"][ok], h64(gz[torch.from_numpy(keep)]), h64(ks))
    assert normwise(h64(gq[torch.from_numpy(keep).to(dev)]), ref["grad_q"]) <= TOL_F32
    # grad_sink over all tokens: the oracle on the sink slot alone
    sink_idx = np.broadcast_to(wl.N + np.arange(H)[None, :, None], (T, H, 1))
    full = oracle.search_backward_sink(h64(q), Kh[:, :, :1], sink_idx, h64(gz[..., k:]), h64(ks))
    assert normwise(h64(gs), full["grad_sink"]) <= TOL_F32
