"""Full-size parity: every large workload at its real shape, through the same
C-ABI calls and launch configuration the benchmark times, checked on sampled
tokens against the fp64 oracle and on properties that hold at any size.

Per workload:
  * search on all T tokens; the oracle recomputes a sample of 48 tokens (first
    16, last 16, 16 seeded random) from host copies of their queries and the
    full sub-key tables; index mismatches must be certified near-ties (float
    inputs), scores and weights match to 1e-5 elsewhere;
  * bag forward on all tokens; sampled tokens compared with the oracle's bag of
    its own selection (bf16 output: 2e-2, one rounding);
  * bag backward with dy zero outside the sample (the backward is linear in dy,
    so the value gradient then holds exactly the sample's contributions):
    sampled grad_w / grad_scores and the touched gradient rows against the
    oracle; grad_w of unsampled tokens exactly zero; no gradient outside the
    touched rows.
The headline workload also runs with integer-valued queries and sub-keys, where
every index must match exactly.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_dy, gen_queries, gen_subkeys, gen_values
from tests.test_gpu_parity import TOL_BF16, TOL_F32, _certify_near_ties, h64, normwise

pytestmark = pytest.mark.gpu


def abs_sum(t, rows_per_chunk=1 << 18):
    """sum |t| in float64, in row chunks (no full-size temporaries)."""
    tot = 0.0
    for r0 in range(0, t.shape[0], rows_per_chunk):
        tot += float(t[r0:r0 + rows_per_chunk].abs().sum(dtype=torch.float64))
    return tot


def sample_tokens(T, seed=0):
    rng = np.random.default_rng(seed)
    mid = rng.choice(np.arange(16, T - 16), size=16, replace=False)
    return np.unique(np.concatenate([np.arange(16), np.arange(T - 16, T), mid]))


@pytest.fixture(autouse=True)
def _free_device_memory():
    yield
    torch.cuda.empty_cache()


CASES = [("pk1m_d1024", False), ("pk4m_d2048", False), ("pk4m_d2048", True),
         ("pk16m_d2048", False), ("pk64m_d256", False)]


@pytest.mark.parametrize("name,integer", CASES, ids=[f"{n}{'-int' if i else ''}" for n, i in CASES])
def test_full_size_sampled(gpu_lib, name, integer):
    wl = WORKLOADS[name]
    dev = torch.device("cuda:0")
    T, H, k, N, D = wl.T, wl.H, wl.k, wl.N, wl.D
    print(f"[fullsize] {name} integer={integer}: generating", flush=True)
    q = gen_queries(wl, dev, integer=integer)
    K = gen_subkeys(wl, dev, integer=integer)
    V = gen_values(wl, dev)
    dy_full = gen_dy(wl, dev)
    samp = sample_tokens(T)
    st = torch.from_numpy(samp).to(dev)

    # --- search (all tokens) ---------------------------------------------
    idx, w, score, _ = pk.mem_search(q, K, k)
    torch.cuda.synchronize()
    qh, Kh = h64(q[st]), h64(K)
    ref = oracle.search(qh, Kh, k)
    gi = idx[st].cpu().numpy()
    if integer:
        np.testing.assert_array_equal(gi, ref["idx"])
    else:
        assert _certify_near_ties(qh, Kh, k, gi, ref) == 0
    same = (gi == ref["idx"]).all(-1)          # [n_samp, H]
    assert same.mean() >= 0.98, f"too many certified near-ties: {1 - same.mean():.3f}"
    assert normwise(h64(score[st])[same], ref["score"][same]) <= TOL_F32
    assert normwise(h64(w[st])[same], ref["w"][same]) <= TOL_F32
    tok_ok = same.all(-1)                        # tokens whose whole selection matches
    print(f"[fullsize] {name}: search ok ({tok_ok.sum()}/{len(samp)} tokens exact)", flush=True)

    # --- bag forward (all tokens) ------------------------------------------
    y = pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1))
    torch.cuda.synchronize()
    rows, inv = np.unique(ref["idx"], return_inverse=True)
    Vs = h64(V[torch.from_numpy(rows).to(dev)])
    loc = inv.reshape(ref["idx"].shape)
    yref = oracle.bag_forward(Vs, loc.reshape(len(samp), -1), ref["w"].reshape(len(samp), -1))
    ys = h64(y[st])
    tol = TOL_F32 if wl.value_dtype == "f32" else TOL_BF16
    assert normwise(ys[tok_ok], yref[tok_ok]) <= tol
    print(f"[fullsize] {name}: bag forward ok", flush=True)

    # --- bag backward (dy zero outside the sample) -------------------------
    # Only sampled tokens whose selection matches the oracle's keep their dy.
    keep = samp[tok_ok]
    sk = torch.from_numpy(keep).to(dev)
    dy = torch.zeros_like(dy_full)
    dy[sk] = dy_full[sk]
    del dy_full
    b = oracle.bag_backward_rows(h64(dy[sk]), Vs, loc[tok_ok], ref["w"][tok_ok], H, k)
    touched = rows[b["rows"]]                    # global row ids touched by the kept tokens
    if wl.sparse_grad:
        rows_out, grows, gw, gz = pk.mem_bag_backward_sparse(dy, V, idx, w)
        torch.cuda.synchronize()
        # every row any lookup touched appears once, ascending
        assert torch.equal(rows_out, torch.unique(idx.view(-1)))
        pos = torch.searchsorted(rows_out, torch.from_numpy(touched).to(dev))
        assert normwise(h64(grows[pos]), b["grad_rows"]) <= TOL_F32
        # rows touched only by tokens with zero dy carry a zero gradient
        assert abs_sum(grows) == pytest.approx(abs_sum(grows[pos]), rel=1e-12, abs=0.0)
    else:
        gv = torch.zeros((N, D), dtype=torch.float32, device=dev)
        gv, gw, gz = pk.mem_bag_backward(dy, V, idx, w, grad_values=gv, mode="auto")
        torch.cuda.synchronize()
        tt = torch.from_numpy(touched).to(dev)
        assert normwise(h64(gv[tt]), b["grad_rows"]) <= TOL_F32
        # no gradient outside the rows the kept tokens touched
        assert abs_sum(gv) == pytest.approx(abs_sum(gv[tt]), rel=1e-12, abs=0.0)
        del gv
    assert normwise(h64(gw[sk]), b["grad_w"]) <= TOL_F32
    assert normwise(h64(gz[sk]), b["grad_z"]) <= TOL_F32
    others = torch.ones(T, dtype=torch.bool, device=dev)
    others[sk] = False
    assert float(gw[others].abs().max()) == 0.0
    print(f"[fullsize] {name}: bag backward ok", flush=True)
