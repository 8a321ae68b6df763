"""The value table sharded by embedding dimension (the parallel memory of
Sec. 3.1.2), on one GPU: each of G column shards [N, D/G] is an ordinary
table for the library.  Per-shard forwards concatenate to the unsharded
output: bitwise when shard and table rows both take one 64-lane group (then
every output element sums the same lookups in the same order), otherwise
within one rounding (narrow rows split a wave into lane groups whose partial
sums combine in a different order); per-shard value gradients are column
slices of the unsharded one, bitwise (each element sums its lookups in
lookup order in every layout); per-shard grad_w are partial dot products
whose sum (the reduce-scatter of a G-GPU run) matches the unsharded grad_w
to fp32 rounding.  The collectives themselves need several GPUs and are not
here."""
import pytest
import torch

import paper_2412_09764_amd as pk
from tests.test_gpu_parity import TOL_BF16, TOL_F32, h64, normwise

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("G,D,dt,exact", [(4, 2048, torch.bfloat16, True), (8, 256, torch.bfloat16, False),
                                           (2, 64, torch.float32, False)])
def test_dimension_sharded_bag_equals_unsharded(gpu_lib, G, D, dt, exact):
    N, T, H, k = 3000, 97, 4, 16
    g = torch.Generator().manual_seed(101 + G)
    V = (torch.randn((N, D), generator=g) * 0.02).to(dt).cuda()
    idx = torch.randint(0, N, (T, H, k), generator=g).cuda()
    w = torch.softmax(torch.randn((T, H, k), generator=g), -1).cuda()
    dy = torch.randn((T, D), generator=g).to(dt).cuda()
    y = pk.mem_bag_forward(V, idx.view(T, -1), w.view(T, -1))
    gv, gw, _ = pk.mem_bag_backward(dy, V, idx, w, mode="sorted")
    Ds = D // G
    ys, gvs, gws = [], [], []
    for s in range(G):
        Vs = V[:, s * Ds:(s + 1) * Ds].contiguous()
        ys.append(pk.mem_bag_forward(Vs, idx.view(T, -1), w.view(T, -1)))
        gv_s, gw_s, _ = pk.mem_bag_backward(dy[:, s * Ds:(s + 1) * Ds].contiguous(), Vs, idx, w,
                                            mode="sorted")
        gvs.append(gv_s)
        gws.append(gw_s)
    torch.cuda.synchronize()
    if exact:
        assert torch.equal(torch.cat(ys, dim=1), y)
    else:
        tol = TOL_F32 if dt == torch.float32 else TOL_BF16
        assert normwise(h64(torch.cat(ys, dim=1)), h64(y)) <= tol
    assert torch.equal(torch.cat(gvs, dim=1), gv)
    assert normwise(h64(sum(gws)), h64(gw)) <= TOL_F32
