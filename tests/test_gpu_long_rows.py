"""Rows chosen by more than 1024 lookups: the sorted backward lists them and
cuts each into chunks of 1024 lookups, each chunk summed by a workgroup of its
own (contiguous runs of lookups per lane group, partial rows added in group
order), the chunks' partial rows added in chunk order.  Against the fp64 oracle, dense and
sparse, across row widths; bitwise deterministic run to run; lengths at and
just past the split threshold."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from tests.test_gpu_parity import TOL_F32, h64, normwise

pytestmark = pytest.mark.gpu

LONG = 1024


def skewed_inputs(N, D, T, H, k, dt, seed, hot_rows, hot_frac):
    """Lookups: a share hot_frac goes to the first hot_rows rows, the rest is
    uniform over N."""
    g = torch.Generator().manual_seed(seed)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt)
    idx = torch.randint(0, N, (T, H, k), generator=g)
    hot = torch.rand((T, H, k), generator=g) < hot_frac
    idx[hot] = torch.randint(0, hot_rows, (int(hot.sum()),), generator=g)
    z = torch.randn((T, H, k), generator=g, dtype=torch.float64)
    w = torch.softmax(z, -1).float()
    dy = torch.randn((T, D), generator=g).to(dt)
    return V, idx, w, dy


CASES = [
    # (name, N, D, T, H, k, dtype, hot_rows, hot_frac)
    ("bf16_D2048_three_hot", 3000, 2048, 400, 4, 8, torch.bfloat16, 3, 0.9),
    ("bf16_D4096_two_hot", 700, 4096, 200, 2, 16, torch.bfloat16, 2, 0.8),
    ("bf16_D256_many_hot", 5000, 256, 1500, 4, 16, torch.bfloat16, 20, 0.7),
    ("bf16_D8_hot", 300, 8, 2000, 2, 4, torch.bfloat16, 4, 0.9),
    ("f32_D64_hot", 1000, 64, 1200, 2, 8, torch.float32, 5, 0.8),
    ("bf16_D1024_one_row", 10, 1024, 800, 4, 8, torch.bfloat16, 1, 1.0),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_long_rows_dense_and_sparse(gpu_lib, case):
    name, N, D, T, H, k, dt, hot_rows, hot_frac = case
    print(f"[long-rows] {name}", flush=True)
    V, idx, w, dy = skewed_inputs(N, D, T, H, k, dt, 17, hot_rows, hot_frac)
    counts = np.bincount(idx.numpy().ravel(), minlength=N)
    assert counts.max() > LONG  # the split path runs
    ref = oracle.bag_backward(h64(dy), h64(V), idx.numpy(), h64(w), H, k)
    base = torch.randn((N, D), generator=torch.Generator().manual_seed(18))
    gv, gw, gz = gpu_lib.mem_bag_backward(dy.cuda(), V.cuda(), idx.cuda(), w.cuda(),
                                          grad_values=base.clone().cuda(), mode="sorted")
    gv2, gw2, gz2 = gpu_lib.mem_bag_backward(dy.cuda(), V.cuda(), idx.cuda(), w.cuda(),
                                             grad_values=base.clone().cuda(), mode="sorted")
    rows, grows, gws, gzs = gpu_lib.mem_bag_backward_sparse(dy.cuda(), V.cuda(), idx.cuda(), w.cuda())
    torch.cuda.synchronize()
    assert torch.equal(gv, gv2) and torch.equal(gw, gw2) and torch.equal(gz, gz2)  # deterministic
    assert normwise(h64(gv) - base.double().numpy(), ref["grad_values"]) <= TOL_F32
    assert normwise(h64(gw), ref["grad_w"]) <= TOL_F32
    # grad_z = w * (grad_w - <w, grad_w>) cancels to zero when every lookup of
    # a (token, head) hits one row: measure it against the terms that cancel
    scale = np.abs(h64(w) * ref["grad_w"]).max()
    assert np.abs(h64(gz) - ref["grad_z"]).max() <= TOL_F32 * scale
    np.testing.assert_array_equal(rows.cpu().numpy(), ref["rows"])
    assert normwise(h64(grows), ref["grad_rows"]) <= TOL_F32
    assert torch.equal(gws, gw)


def test_segments_at_the_split_threshold(gpu_lib):
    """Rows with exactly 1024 lookups (kept whole) and 1025 (split) next to
    short ones: both paths in one call."""
    N, D, T, H, k = 64, 512, 1025, 1, 4
    idx = torch.zeros((T, H, k), dtype=torch.int64)
    idx[:, 0, 0] = 5                       # row 5: 1025 lookups (split)
    idx[:1024, 0, 1] = 9                   # row 9: 1024 lookups (whole)
    idx[1024, 0, 1] = 10
    g = torch.Generator().manual_seed(21)
    idx[:, 0, 2:] = torch.randint(11, N, (T, k - 2), generator=g)
    V = (torch.randn((N, D), generator=g) * 0.02).to(torch.bfloat16)
    w = torch.softmax(torch.randn((T, H, k), generator=g, dtype=torch.float64), -1).float()
    dy = torch.randn((T, D), generator=g).to(torch.bfloat16)
    ref = oracle.bag_backward(h64(dy), h64(V), idx.numpy(), h64(w), H, k)
    gv, gw, gz = gpu_lib.mem_bag_backward(dy.cuda(), V.cuda(), idx.cuda(), w.cuda(), mode="sorted")
    torch.cuda.synchronize()
    assert normwise(h64(gv), ref["grad_values"]) <= TOL_F32
    assert normwise(h64(gw), ref["grad_w"]) <= TOL_F32
    assert np.abs(h64(gz) - ref["grad_z"]).max() <= TOL_F32 * np.abs(h64(w) * ref["grad_w"]).max()


@pytest.mark.parametrize("mode", ["sorted", "atomic"])
def test_backward_without_value_gradient(gpu_lib, mode):
    """grad_values not requested (NULL): grad_w and grad_scores are bitwise
    those of the full call (including rows long enough for the split path),
    and match the oracle."""
    N, D, T, H, k = 3000, 512, 900, 4, 8
    V, idx, w, dy = skewed_inputs(N, D, T, H, k, torch.bfloat16, 141, 3, 0.6)
    args = (dy.cuda(), V.cuda(), idx.cuda(), w.cuda())
    _, gw_full, gz_full = pk.mem_bag_backward(*args, mode=mode)
    gv_none, gw, gz = pk.mem_bag_backward(*args, want_grad_values=False, mode=mode)
    torch.cuda.synchronize()
    assert gv_none is None
    assert torch.equal(gw, gw_full) and torch.equal(gz, gz_full)
    ref = oracle.bag_backward(h64(dy), h64(V), idx.numpy(), h64(w), H, k)
    assert normwise(h64(gw), ref["grad_w"]) <= TOL_F32
    assert normwise(h64(gz), ref["grad_z"]) <= TOL_F32


def test_row_chosen_by_most_tokens(gpu_lib):
    """One row chosen by about 60% of 65,536 tokens (about 39,000 lookups):
    its lookups are cut into chunks summed by many workgroups and added in
    chunk order.  Against the oracle, dense and sparse, bitwise deterministic."""
    N, D, T, H, k = 1 << 16, 256, 65536, 1, 4
    g = torch.Generator().manual_seed(31)
    idx = torch.randint(0, N, (T, H, k), generator=g)
    hot = torch.rand((T,), generator=g) < 0.6
    idx[hot, 0, 0] = 7
    V = (torch.randn((N, D), generator=g) * 0.02).to(torch.bfloat16)
    w = torch.softmax(torch.randn((T, H, k), generator=g, dtype=torch.float64), -1).float()
    dy = torch.randn((T, D), generator=g).to(torch.bfloat16)
    counts = np.bincount(idx.numpy().ravel(), minlength=N)
    assert counts[7] >= T // 2
    print(f"[long-rows] hot row lookups {counts[7]}", flush=True)
    args = (dy.cuda(), V.cuda(), idx.cuda(), w.cuda())
    gv, gw, gz = gpu_lib.mem_bag_backward(*args, mode="sorted")
    gv2, gw2, gz2 = gpu_lib.mem_bag_backward(*args, mode="sorted")
    rows, grows, _, _ = gpu_lib.mem_bag_backward_sparse(*args)
    torch.cuda.synchronize()
    assert torch.equal(gv, gv2) and torch.equal(gw, gw2) and torch.equal(gz, gz2)
    ref = oracle.bag_backward_rows(h64(dy), h64(V), idx.numpy(), h64(w), H, k)
    np.testing.assert_array_equal(rows.cpu().numpy(), ref["rows"])
    assert normwise(h64(grows), ref["grad_rows"]) <= TOL_F32
    hot_u = int(np.searchsorted(ref["rows"], 7))
    assert normwise(h64(grows[hot_u]), ref["grad_rows"][hot_u]) <= TOL_F32
    assert normwise(h64(gv[torch.from_numpy(ref["rows"]).cuda()]), ref["grad_rows"]) <= TOL_F32
    assert normwise(h64(gw), ref["grad_w"]) <= TOL_F32
