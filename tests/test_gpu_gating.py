"""GPU parity of the Memory+ gating (Sec. 3.1.4) through the C ABI:
mem_bag_forward_gated (out = bag * silu(gate), fused into the gather) and
mem_gate_backward, against the fp64 oracle.  The un-gated bag the gated call
writes must equal mem_bag_forward's output bitwise (same accumulation)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_09764_amd as pk
from paper_2412_09764_amd.inputs import WORKLOADS, gen_dy, gen_values
from tests.test_gpu_parity import TOL_BF16, TOL_F32, h64, normwise

pytestmark = pytest.mark.gpu

# name, N, D, T, bag, dtype
CASES = [
    ("bf16_D2048", 5000, 2048, 77, 128, torch.bfloat16),
    ("bf16_D1024_tail", 3000, 1024, 130, 96, torch.bfloat16),
    ("bf16_D200_ragged", 700, 200, 65, 20, torch.bfloat16),
    ("bf16_D8", 50, 8, 33, 7, torch.bfloat16),
    ("f32_D64", 4096, 64, 256, 8, torch.float32),
    ("f32_D1000", 900, 1000, 40, 64, torch.float32),
]


def _inputs(N, D, T, bag, dt, seed):
    g = torch.Generator().manual_seed(seed)
    V = (torch.randn((N, D), generator=g) * 0.05).to(dt)
    idx = torch.randint(0, N, (T, bag), generator=g)
    w = torch.rand((T, bag), generator=g)
    gate = (torch.randn((T, D), generator=g) * 2.0)
    gate[0, :4] = torch.tensor([30.0, -30.0, 0.0, -88.0])[: min(4, D)]
    return V, idx, w, gate.to(dt)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_gated_forward_and_backward(gpu_lib, case):
    name, N, D, T, bag, dt = case
    print(f"[gating] {name}", flush=True)
    V, idx, w, gate = _inputs(N, D, T, bag, dt, 91)
    Vd, idd, wd, gd = V.cuda(), idx.cuda(), w.cuda(), gate.cuda()
    out, y = pk.mem_bag_forward_gated(Vd, idd, wd, gd)
    plain = pk.mem_bag_forward(Vd, idd, wd)
    torch.cuda.synchronize()
    assert torch.equal(y, plain)
    tol = TOL_F32 if dt == torch.float32 else TOL_BF16
    yref = oracle.bag_forward(h64(V), idx.numpy(), w.double().numpy())
    assert normwise(h64(y), yref) <= tol
    assert normwise(h64(out), oracle.gated_output(yref, h64(gate))) <= tol
    # backward: both sides take the same y, the oracle's bag rounded to the
    # value dtype (an input of the gate backward, like d_out and the gate)
    d_out = (torch.randn((T, D), generator=torch.Generator().manual_seed(92))).to(dt)
    y_in = torch.from_numpy(yref).to(dt)
    dy, dg = pk.mem_gate_backward(d_out.cuda(), gd, y_in.cuda())
    torch.cuda.synchronize()
    ref = oracle.gated_backward(h64(d_out), h64(y_in), h64(gate))
    assert normwise(h64(dy), ref["dy"]) <= tol
    assert normwise(h64(dg), ref["dg"]) <= TOL_F32


def test_gated_forward_without_y(gpu_lib):
    V, idx, w, gate = _inputs(300, 256, 50, 16, torch.bfloat16, 93)
    out_a, none = pk.mem_bag_forward_gated(V.cuda(), idx.cuda(), w.cuda(), gate.cuda(), want_y=False)
    out_b, _ = pk.mem_bag_forward_gated(V.cuda(), idx.cuda(), w.cuda(), gate.cuda())
    torch.cuda.synchronize()
    assert none is None and torch.equal(out_a, out_b)


def test_gated_chain_into_value_backward(gpu_lib):
    """gated forward -> gate backward -> bag backward, against the oracle's own
    chain.  The GPU stores dy in the value dtype between the two backwards; the
    oracle rounds its fp64 dy to bfloat16 the same way (round_bf16), so dy must
    match bit for bit and the value-side results are held to 1e-5.  A dy element
    whose exact value lies within fp32 evaluation error of a bfloat16 rounding
    midpoint may round either way: each such element is certified as a near-tie
    that took the other neighbour, and the tokens holding one (with every value
    row they touch) are left out of the value-side comparison, which then
    compares only what is unique."""
    N, D, T, H, k = 600, 512, 90, 4, 8
    V, idx, w, gate = _inputs(N, D, T, H * k, torch.bfloat16, 94)
    idx3, w3 = idx.view(T, H, k), w.view(T, H, k)
    d_out = torch.randn((T, D), generator=torch.Generator().manual_seed(95)).to(torch.bfloat16)
    out, y = pk.mem_bag_forward_gated(V.cuda(), idx.cuda(), w.cuda(), gate.cuda())
    dy, dg = pk.mem_gate_backward(d_out.cuda(), gate.cuda(), y)
    gv, gw, gz = pk.mem_bag_backward(dy, V.cuda(), idx3.cuda().contiguous(), w3.cuda().contiguous(),
                                     mode="sorted")
    torch.cuda.synchronize()
    yref = oracle.bag_forward(h64(V), idx.numpy(), w.double().numpy())
    dy_exact = oracle.gated_backward(h64(d_out), yref, h64(gate))["dy"]
    dy_ref = oracle.round_bf16(dy_exact)
    gdy = h64(dy)
    flip = gdy != dy_ref
    if flip.any():
        m, e = np.frexp(dy_exact[flip])
        frac = np.abs(m) * 256.0 - np.floor(np.abs(m) * 256.0)
        assert np.all(np.abs(frac - 0.5) <= 2.0 ** -10), "dy differs away from a rounding midpoint"
        assert np.all(np.abs(gdy[flip] - dy_ref[flip]) == np.ldexp(1.0, e - 8)), "not a neighbour"
    assert flip.sum() <= 8
    ok_t = ~flip.any(1)
    bad_rows = np.unique(idx3.numpy()[~ok_t])
    ok_r = np.ones(N, bool)
    ok_r[bad_rows] = False
    b = oracle.bag_backward(dy_ref, h64(V), idx3.numpy(), w3.double().numpy(), H, k)
    assert normwise(gdy, dy_exact) <= TOL_BF16
    assert normwise(h64(gv)[ok_r], b["grad_values"][ok_r]) <= 1e-5
    assert normwise(h64(gw)[ok_t], b["grad_w"][ok_t]) <= 1e-5
    assert ok_r.sum() >= N // 2


def test_gated_full_size_sampled(gpu_lib):
    """4M x 2048 bf16 values, 32768 tokens of 128 lookups: the gated gather on
    every token in the benchmark's launch configuration, 48 tokens against the
    oracle; the un-gated output equals mem_bag_forward's bitwise."""
    wl = WORKLOADS["pk4m_d2048"]
    dev = torch.device("cuda:0")
    T, D, N, bag = wl.T, wl.D, wl.N, wl.bag
    V = gen_values(wl, dev)
    g = torch.Generator(device=dev).manual_seed(96)
    idx = torch.randint(0, N, (T, bag), generator=g, device=dev)
    w = torch.rand((T, bag), generator=g, device=dev)
    gate = gen_dy(wl, dev)   # N(0,1) in the value dtype: the gate pre-activation
    out, y = pk.mem_bag_forward_gated(V, idx, w, gate)
    plain = pk.mem_bag_forward(V, idx, w)
    torch.cuda.synchronize()
    assert torch.equal(y, plain)
    del plain
    rng = np.random.default_rng(97)
    samp = np.unique(np.concatenate([np.arange(16), np.arange(T - 16, T),
                                     rng.choice(np.arange(16, T - 16), 16, replace=False)]))
    st = torch.from_numpy(samp).to(dev)
    rows, inv = np.unique(idx[st].cpu().numpy(), return_inverse=True)
    Vs = h64(V[torch.from_numpy(rows).to(dev)])
    yref = oracle.bag_forward(Vs, inv.reshape(len(samp), -1), w[st].double().cpu().numpy())
    assert normwise(h64(out[st]), oracle.gated_output(yref, h64(gate[st]))) <= TOL_BF16
    # gate backward on every token with a seeded y input (both sides)
    y_in = torch.randn((T, D), generator=torch.Generator(device=dev).manual_seed(98),
                       device=dev).to(y.dtype)
    dy, dg = pk.mem_gate_backward(gen_dy(wl, dev), gate, y_in)
    torch.cuda.synchronize()
    ref = oracle.gated_backward(h64(gen_dy(wl, dev)[st]), h64(y_in[st]), h64(gate[st]))
    assert normwise(h64(dy[st]), ref["dy"]) <= TOL_BF16
    assert normwise(h64(dg[st]), ref["dg"]) <= TOL_F32
