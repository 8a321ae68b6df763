"""Random argument tuples through every compute entry point of the C ABI, on
a host without a GPU: every call must return one of the documented status
codes (argument errors are found on the host; anything that passes them
fails at its first HIP call with PKMEM_ERR_HIP here) and never crash.
Pointers are fake, aligned or not, and never dereferenced on the host; the
test refuses to run where a GPU is present, since a call that passed the
checks would launch kernels on them."""
import numpy as np
import pytest
import torch

import paper_2412_09764_amd as pk

CODES = {0, -1, -2, -3, -4}
BIG = 1 << 40


@pytest.fixture(scope="module")
def lib():
    if torch.cuda.is_available():
        pytest.skip("fake device pointers: host-only test")
    return pk.load()


def _ptr(rng):
    return int(rng.choice([0, 0x10000, 0x10008, 0x10004, 0x20000]))


def _dt(rng):
    return int(rng.choice([0, 1, 1, 1, 7]))


def _sz(rng, lo, hi):
    return int(rng.integers(lo, hi))


@pytest.mark.parametrize("seed", range(4))
def test_search_family(lib, seed):
    rng = np.random.default_rng(seed)
    for _ in range(400):
        dt = _dt(rng)
        a = dict(T=_sz(rng, -2, 300), H=_sz(rng, -1, 6), n=_sz(rng, -2, 700), S=_sz(rng, -1, 9000),
                 k=_sz(rng, -1, 70))
        ws = int(rng.choice([0, 16, BIG]))
        args = (_ptr(rng), dt, _ptr(rng), dt if rng.random() < 0.9 else _dt(rng), a["T"], a["H"],
                a["n"], a["S"], a["k"])
        outs = (_ptr(rng), _ptr(rng), None, None)
        assert lib.mem_search(*args, *outs, _ptr(rng), ws, None) in CODES
        assert lib.mem_search_qnorm(*args, float(rng.choice([1e-5, 0.0, -1.0, np.nan])), *outs,
                                    None, None, _ptr(rng), ws, None) in CODES
        assert lib.mem_search_extra(*args, _sz(rng, -1, 40), _ptr(rng), *outs, _ptr(rng), ws,
                                    None) in CODES
        assert lib.mem_search_backward(*args, _ptr(rng), _ptr(rng), _ptr(rng), _ptr(rng),
                                       _ptr(rng), ws, None) in CODES
        assert lib.mem_search_backward_qnorm(*args, 1e-5, _ptr(rng), _ptr(rng), _ptr(rng),
                                             _ptr(rng), _ptr(rng), ws, None) in CODES
        row0 = int(rng.choice([-1, 0, max(a["S"], 0) ** 2, 1 << 40, (1 << 63) - 1]))
        assert lib.mem_search_sink(*args, _sz(rng, -1, 40), _ptr(rng), _ptr(rng), row0, *outs,
                                   _ptr(rng), ws, None) in CODES
        assert lib.mem_search_backward_sink(*args, _ptr(rng), _ptr(rng), _ptr(rng), _ptr(rng),
                                            _ptr(rng), _ptr(rng), _ptr(rng), ws, None) in CODES


@pytest.mark.parametrize("seed", range(4))
def test_bag_family(lib, seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(400):
        vdt = _dt(rng)
        N, D, T = _sz(rng, -1, 5000), _sz(rng, -8, 5000), _sz(rng, -2, 300)
        H, k = _sz(rng, -1, 6), _sz(rng, -1, 70)
        ws = int(rng.choice([0, 16, BIG]))
        mode = int(rng.choice([0, 1, 2, 5]))
        assert lib.mem_bag_forward(_ptr(rng), vdt, N, D, _ptr(rng), _ptr(rng), T, H * k,
                                   _ptr(rng), None) in CODES
        assert lib.mem_bag_forward_gated(_ptr(rng), vdt, N, D, _ptr(rng), _ptr(rng), T, H * k,
                                         _ptr(rng), None, _ptr(rng), None) in CODES
        assert lib.mem_gate_backward(_ptr(rng), _ptr(rng), _ptr(rng), vdt, T, D, _ptr(rng),
                                     _ptr(rng), None) in CODES
        assert lib.mem_bag_backward(_ptr(rng), _ptr(rng), vdt, N, D, _ptr(rng), _ptr(rng), T, H, k,
                                    _ptr(rng), _ptr(rng), _ptr(rng), mode, _ptr(rng), ws,
                                    None) in CODES
        import ctypes
        nrows = ctypes.c_int64(0)
        assert lib.mem_bag_backward_sparse(_ptr(rng), _ptr(rng), vdt, N, D, _ptr(rng), _ptr(rng),
                                           T, H, k, _ptr(rng), _ptr(rng), _sz(rng, -1, 10 ** 6),
                                           ctypes.addressof(nrows), None, None, _ptr(rng), ws,
                                           None) in CODES


def test_workspace_queries_never_fail(lib):
    rng = np.random.default_rng(7)
    for _ in range(500):
        T, H, S, k = _sz(rng, -5, 10 ** 6), _sz(rng, -2, 64), _sz(rng, -2, 9000), _sz(rng, -2, 70)
        assert lib.mem_search_workspace_size(T, H, S, k) >= 0
        assert lib.mem_search_backward_workspace_size(T, H, S, k) >= 0
        assert lib.mem_search_backward_sink_workspace_size(T, H, _sz(rng, -2, 600), S, k) >= 0
        assert lib.mem_bag_backward_workspace_size(T, H, k, _sz(rng, -1, 10 ** 7),
                                                   _sz(rng, -8, 5000), int(rng.choice([0, 1, 2, 9]))) >= 0
