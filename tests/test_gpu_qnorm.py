"""GPU parity of the search with query normalisation fused in front of the
scoring (mem_search_qnorm, mem_search_backward_qnorm) against the fp64 oracle.

Exact cases: eps = 0 on rows built as c + 2^m x (mean c, variance 4 * 4^m)
normalise to x / 2 exactly in binary arithmetic, and integer sub-keys make
every score exact, so indices must match bit for bit.  Float cases (eps =
1e-5): the normalised queries are compared with the oracle's (fp32 statistics
against fp64 may move a bf16 rounding by one unit), and the selection is
accepted where it differs from the oracle's only within the score change
that those rounding differences can cause."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_queries, gen_subkeys
from tests.oracle_pins import exact_norm_rows
from tests.test_gpu_parity import TOL_F32, h64, int_tensor, normwise

pytestmark = pytest.mark.gpu

DT = {torch.bfloat16: "bf16", torch.float32: "fp32"}

EXACT_CASES = [
    # (name, S, H, n, k, T, dtype)
    ("bf16_S1024_H4_k32_ragged", 1024, 4, 512, 32, 200, torch.bfloat16),
    ("bf16_S100_d32", 100, 2, 64, 16, 130, torch.bfloat16),
    ("bf16_k_eq_S", 37, 3, 32, 37, 65, torch.bfloat16),
    ("bf16_k1", 512, 1, 16, 1, 300, torch.bfloat16),
    ("bf16_k64_S8192", 8192, 1, 512, 64, 40, torch.bfloat16),
    ("f32_S200_d64", 200, 2, 128, 20, 99, torch.float32),
    ("f32_S64_k8", 64, 1, 64, 8, 256, torch.float32),
    ("bf16_T1", 2048, 4, 512, 32, 1, torch.bfloat16),
]


def exact_inputs(T, H, n, S, seed, dt):
    rng = np.random.default_rng(seed)
    q, half = exact_norm_rows(rng, T, H, n)
    K = int_tensor((H, 2, S, n // 2), seed + 1, dt)
    return torch.from_numpy(q).to(dt), half, K


@pytest.mark.parametrize("case", EXACT_CASES, ids=[c[0] for c in EXACT_CASES])
def test_search_qnorm_exact(gpu_lib, case):
    name, S, H, n, k, T, dt = case
    print(f"[qnorm-exact] {name}", flush=True)
    q, half, K = exact_inputs(T, H, n, S, 11, dt)
    idx, w, score, hidx, qhat, stats = pk.mem_search_qnorm(
        q.cuda(), K.cuda(), k, 0.0, want_half=True, want_qhat=True, want_stats=True)
    torch.cuda.synchronize()
    ref = oracle.search_qnorm(h64(q), h64(K), k, 0.0, DT[dt])
    np.testing.assert_array_equal(ref["qhat"], half)  # the rows normalise exactly
    np.testing.assert_array_equal(h64(qhat), half)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref["idx"])
    np.testing.assert_array_equal(hidx.cpu().numpy(), ref["half_idx"])
    np.testing.assert_array_equal(h64(score), ref["score"])
    assert normwise(h64(w), ref["w"]) <= TOL_F32
    np.testing.assert_array_equal(h64(stats)[..., 0], ref["mean"])
    np.testing.assert_array_equal(h64(stats)[..., 1], ref["rstd"])


def test_search_qnorm_matches_normalise_then_search(gpu_lib):
    """The fused normalisation equals searching the normalised queries it
    reports (mem_search on qhat_out): bitwise, at the 1M-key workload's
    shape with raw N(0, 1) queries shifted and scaled per token."""
    wl = WORKLOADS["pk1m_d1024"]
    T = 4096
    g = torch.Generator().manual_seed(61)
    raw = torch.randn((T, wl.H, wl.n), generator=g) * (1 + 3 * torch.rand((T, wl.H, 1), generator=g))
    raw = (raw + torch.randn((T, wl.H, 1), generator=g)).to(torch.bfloat16).cuda()
    K = gen_subkeys(wl, "cuda")
    idx, w, score, _, qhat, _ = pk.mem_search_qnorm(raw, K, wl.k, 1e-5, want_qhat=True)
    idx2, w2, score2, _ = pk.mem_search(qhat, K, wl.k)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2) and torch.equal(w, w2) and torch.equal(score, score2)


def _qhat_row_bound(qh_gpu, qh_ref, K):
    """Per (t, h): an upper bound on |score(qhat_gpu) - score(qhat_ref)| over
    every full key, from the elementwise qhat differences."""
    T, H, n = qh_ref.shape
    d = n // 2
    kmax = np.abs(K).max(axis=2)  # [H, 2, d]
    dq = np.abs(qh_gpu - qh_ref)
    return (dq[..., :d] * kmax[None, :, 0]).sum(-1) + (dq[..., d:] * kmax[None, :, 1]).sum(-1)


def _certify(qh_ref, K, k, gpu_idx, ref, bound, rel_gap=1e-4):
    T, H, n = qh_ref.shape
    d = n // 2
    S = K.shape[2]
    bad = 0
    for t, h in zip(*np.nonzero((gpu_idx != ref["idx"]).any(-1))):
        i = gpu_idx[t, h]
        full = qh_ref[t, h, :d] @ K[h, 0, i // S].T + qh_ref[t, h, d:] @ K[h, 1, i % S].T
        scale = np.abs(ref["score"][t, h]).max()
        gap = np.abs(np.sort(full)[::-1] - ref["score"][t, h])
        if not np.all(gap <= rel_gap * scale + 2.0 * bound[t, h]):
            bad += 1
    return bad


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_search_qnorm_float_inputs(gpu_lib, dt):
    S, H, n, k, T = (1024, 4, 512, 32, 300) if dt == torch.bfloat16 else (256, 2, 128, 16, 300)
    print(f"[qnorm-float] {DT[dt]}", flush=True)
    g = torch.Generator().manual_seed(71)
    q = (2.5 * torch.randn((T, H, n), generator=g) + 0.75).to(dt)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 16).to(dt)
    idx, w, score, _, qhat, stats = pk.mem_search_qnorm(q.cuda(), K.cuda(), k, 1e-5,
                                                        want_qhat=True, want_stats=True)
    torch.cuda.synchronize()
    ref = oracle.search_qnorm(h64(q), h64(K), k, 1e-5, DT[dt])
    qg = h64(qhat)
    # statistics in fp32 against fp64
    assert normwise(h64(stats)[..., 1], ref["rstd"]) <= TOL_F32
    assert np.all(np.abs(h64(stats)[..., 0] - ref["mean"]) <= 1e-5 / ref["rstd"])
    if dt == torch.bfloat16:
        # one bf16 unit at most, on a small share of the elements
        diff = np.abs(qg - ref["qhat"])
        assert np.all(diff <= np.abs(ref["qhat"]) * 2.0 ** -7 + 1e-30)
        assert np.count_nonzero(diff) <= 0.01 * diff.size
    else:
        assert normwise(qg, ref["qhat"]) <= TOL_F32
    bound = _qhat_row_bound(qg, ref["qhat"], h64(K))
    gi = idx.cpu().numpy()
    assert _certify(ref["qhat"], h64(K), k, gi, ref, bound) == 0
    ok = (gi == ref["idx"]).all(-1)
    assert ok.mean() > 0.9
    # bf16: rows whose normalised query is bitwise the oracle's; fp32: every
    # matching row (its qhat differs from the oracle's by fp32 rounding only)
    same = ok & (bound == 0) if dt == torch.bfloat16 else ok
    assert same.sum() >= 0.5 * same.size
    assert normwise(h64(score)[same], ref["score"][same]) <= TOL_F32
    assert normwise(h64(w)[same], ref["w"][same]) <= TOL_F32


BWD_CASES = [
    ("bf16_S1024_H4_k32", 1024, 4, 512, 32, 200, torch.bfloat16),
    ("bf16_S100_d32", 100, 2, 64, 16, 130, torch.bfloat16),
    ("f32_S200_d64", 200, 2, 128, 20, 99, torch.float32),
    ("bf16_S8192_d256", 8192, 1, 512, 16, 300, torch.bfloat16),
]


@pytest.mark.parametrize("case", BWD_CASES, ids=[c[0] for c in BWD_CASES])
def test_search_backward_qnorm_exact(gpu_lib, case):
    name, S, H, n, k, T, dt = case
    print(f"[qnorm-bwd] {name}", flush=True)
    q, half, K = exact_inputs(T, H, n, S, 31, dt)
    gz = torch.randn((T, H, k), generator=torch.Generator().manual_seed(33))
    base = torch.randn((H, 2, S, n // 2), generator=torch.Generator().manual_seed(34))
    idx, _, _, _, _, _ = pk.mem_search_qnorm(q.cuda(), K.cuda(), k, 0.0)
    gq, gK = pk.mem_search_backward_qnorm(q.cuda(), K.cuda(), idx, gz.cuda(), 0.0,
                                          grad_subkeys=base.clone().cuda())
    torch.cuda.synchronize()
    s = oracle.search_qnorm(h64(q), h64(K), k, 0.0, DT[dt])
    np.testing.assert_array_equal(idx.cpu().numpy(), s["idx"])
    ref = oracle.search_backward_qnorm(h64(q), h64(K), s["idx"], gz.double().numpy(), 0.0, DT[dt])
    assert normwise(h64(gq), ref["grad_q"]) <= TOL_F32
    assert normwise(h64(gK) - base.double().numpy(), ref["grad_K"]) <= TOL_F32


@pytest.mark.parametrize("dt", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
def test_search_backward_qnorm_float_inputs(gpu_lib, dt):
    """eps = 1e-5, float queries: rows whose selection and normalised query
    match the oracle's exactly carry the gradient (gz = 0 elsewhere).  grad_q
    within 1e-5; grad_K too (it uses qhat, equal on the kept rows)."""
    S, H, n, k, T = (512, 2, 256, 16, 256) if dt == torch.bfloat16 else (128, 2, 64, 8, 256)
    g = torch.Generator().manual_seed(81)
    q = (1.5 * torch.randn((T, H, n), generator=g) - 0.3).to(dt)
    K = (torch.randn((H, 2, S, n // 2), generator=g) / 8).to(dt)
    idx, _, _, _, qhat, _ = pk.mem_search_qnorm(q.cuda(), K.cuda(), k, 1e-5, want_qhat=True)
    torch.cuda.synchronize()
    s = oracle.search_qnorm(h64(q), h64(K), k, 1e-5, DT[dt])
    same_q = (h64(qhat) == s["qhat"]).all(-1) if dt == torch.bfloat16 else np.ones((T, H), bool)
    keep = ((idx.cpu().numpy() == s["idx"]).all(-1) & same_q).all(-1)
    assert keep.mean() > 0.8
    gz = torch.randn((T, H, k), generator=torch.Generator().manual_seed(83))
    gz[torch.from_numpy(~keep)] = 0.0
    gq, gK = pk.mem_search_backward_qnorm(q.cuda(), K.cuda(), idx, gz.cuda(), 1e-5)
    runs = pk.mem_search_backward_qnorm(q.cuda(), K.cuda(), idx, gz.cuda(), 1e-5)
    torch.cuda.synchronize()
    assert torch.equal(gq, runs[0]) and torch.equal(gK, runs[1])  # deterministic
    ref = oracle.search_backward_qnorm(h64(q)[keep], h64(K), s["idx"][keep],
                                       gz.double().numpy()[keep], 1e-5, DT[dt])
    assert normwise(h64(gq)[keep], ref["grad_q"]) <= TOL_F32
    assert not h64(gq)[~keep].any()
    assert normwise(h64(gK), ref["grad_K"]) <= TOL_F32


def test_search_qnorm_full_size_sampled(gpu_lib):
    """4M-key workload shape with raw N(0, 1) queries, shifted: sampled tokens
    against the oracle (normalised query and selection)."""
    wl = WORKLOADS["pk4m_d2048"]
    dev = torch.device("cuda:0")
    q = (gen_queries(wl, dev).float() * 2.0 + 0.5).to(torch.bfloat16)
    K = gen_subkeys(wl, dev)
    idx, w, score, _, qhat, _ = pk.mem_search_qnorm(q, K, wl.k, 1e-5, want_qhat=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(9)
    samp = np.unique(np.concatenate([np.arange(8), np.arange(wl.T - 8, wl.T),
                                     rng.choice(np.arange(8, wl.T - 8), 16, replace=False)]))
    st = torch.from_numpy(samp).to(dev)
    Kh = h64(K)
    ref = oracle.search_qnorm(h64(q[st]), Kh, wl.k, 1e-5, "bf16")
    qg = h64(qhat[st])
    assert np.all(np.abs(qg - ref["qhat"]) <= np.abs(ref["qhat"]) * 2.0 ** -7 + 1e-30)
    bound = _qhat_row_bound(qg, ref["qhat"], Kh)
    gi = idx[st].cpu().numpy()
    assert _certify(ref["qhat"], Kh, wl.k, gi, ref, bound) == 0
    ok = (gi == ref["idx"]).all(-1) & (bound == 0)
    assert ok.sum() >= 0.5 * ok.size
    assert normwise(h64(w[st])[ok], ref["w"][ok]) <= TOL_F32


def test_search_qnorm_constant_rows_and_empty(gpu_lib):
    """A constant query with eps = 0 normalises to zeros (every score 0: the
    k lowest composed indices, uniform weights); T = 0 is a no-op."""
    T, H, n, S, k = 20, 2, 32, 50, 6
    q = torch.full((T, H, n), 3.0, dtype=torch.bfloat16).cuda()
    K = int_tensor((H, 2, S, n // 2), 5, torch.bfloat16).cuda()
    idx, w, score, _, qhat, stats = pk.mem_search_qnorm(q, K, k, 0.0, want_qhat=True, want_stats=True)
    torch.cuda.synchronize()
    assert float(qhat.float().abs().max()) == 0.0
    np.testing.assert_array_equal(idx.cpu().numpy(), np.broadcast_to(np.arange(k), (T, H, k)))
    np.testing.assert_allclose(w.cpu().numpy(), 1.0 / k, rtol=1e-6)
    assert float(stats[..., 1].abs().max()) == 0.0
    e = torch.zeros((0, H, n), dtype=torch.bfloat16).cuda()
    idx0, _, _, _, _, _ = pk.mem_search_qnorm(e, K, k)
    gq0, _ = pk.mem_search_backward_qnorm(e, K, idx0, torch.zeros((0, H, k)).cuda())
    torch.cuda.synchronize()
    assert idx0.shape == (0, H, k) and gq0.shape == (0, H, n)
