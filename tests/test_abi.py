"""C ABI checks that need no GPU: the library loads, exports every function
include/pkmem.h declares, and rejects bad arguments on the host with the
documented status codes before any HIP call (pointer arguments here are fake,
aligned addresses that are never dereferenced)."""
import ctypes
import os
import re

import pytest

import paper_2412_09764_amd as pk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pkmem.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, -1, -2, -3
F32, BF16 = 0, 1
FAKE = 0x10000  # 256-byte aligned, never dereferenced
BIG_WS = 1 << 40


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*(mem_[a-z_]+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(pk.lib_path()):
        pytest.fail("libpkmem.so is not built (run __graft_entry__.build())")
    return pk.load()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("mem_search", "mem_bag_forward", "mem_bag_backward", "mem_bag_backward_sparse",
              "mem_search_workspace_size", "mem_bag_backward_workspace_size", "mem_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert lib.mem_version() == 1


def search(lib, q=FAKE, qdt=BF16, K=FAKE, kdt=BF16, T=8, H=2, n=64, S=16, k=4, idx=FAKE, w=FAKE,
           ws=FAKE, ws_bytes=BIG_WS):
    return lib.mem_search(q, qdt, K, kdt, T, H, n, S, k, idx, w, None, None, ws, ws_bytes, None)


def msg(lib):
    return lib.mem_last_error().decode()


@pytest.mark.parametrize("kw,code,text", [
    (dict(n=63), INVALID, "even"),
    (dict(n=0), INVALID, "even"),
    (dict(k=0), INVALID, "k <= S"),
    (dict(k=17), INVALID, "k <= S"),
    (dict(S=100, k=65), UNSUPPORTED, "k >"),
    (dict(S=8193), UNSUPPORTED, "S >"),
    (dict(S=0), INVALID, "S must"),
    (dict(H=0), INVALID, "H must"),
    (dict(T=-1), INVALID, "T must"),
    (dict(n=20), UNSUPPORTED, "multiple of 8"),
    (dict(n=1024), UNSUPPORTED, "<= 256"),
    (dict(qdt=F32, kdt=F32, n=256), UNSUPPORTED, "fp32"),
    (dict(qdt=F32), UNSUPPORTED, "share a dtype"),
    (dict(qdt=7, kdt=7), INVALID, "dtype"),
    (dict(q=0), INVALID, "null"),
    (dict(idx=0), INVALID, "null"),
    (dict(q=FAKE + 8), INVALID, "aligned"),
    (dict(ws=0), WORKSPACE, "workspace"),
    (dict(ws_bytes=16), WORKSPACE, "workspace"),
    (dict(ws=FAKE + 64), INVALID, "256-byte"),
])
def test_search_rejects(lib, kw, code, text):
    assert search(lib, **kw) == code
    assert text in msg(lib)


def test_search_empty_batch_is_a_noop(lib):
    assert search(lib, T=0) == OK


def test_workspace_sizes(lib):
    a = lib.mem_search_workspace_size(1000, 4, 2048, 32)
    b = lib.mem_search_workspace_size(2000, 4, 2048, 32)
    assert 0 < a < b
    assert lib.mem_search_workspace_size(-1, 4, 2048, 32) == 0
    s = lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 2)
    at = lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 1)
    assert s > at >= 1000 * 4 * 32 * 4
    # auto picks the sorted strategy for wide rows and atomics for narrow ones
    assert lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 0) == s
    assert lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 64, 0) == at


def fwd(lib, V=FAKE, vdt=BF16, N=4096, D=64, idx=FAKE, w=FAKE, T=4, bag=8, y=FAKE):
    return lib.mem_bag_forward(V, vdt, N, D, idx, w, T, bag, y, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(D=12), UNSUPPORTED, "multiple of 8"),
    (dict(D=0), UNSUPPORTED, "multiple of 8"),
    (dict(D=4104), UNSUPPORTED, "8 KiB"),
    (dict(vdt=F32, D=2056), UNSUPPORTED, "8 KiB"),
    (dict(N=0), INVALID, "N must"),
    (dict(bag=0), INVALID, "bag"),
    (dict(T=-2), INVALID, "T must"),
    (dict(vdt=5), INVALID, "dtype"),
    (dict(V=0), INVALID, "null"),
    (dict(y=0), INVALID, "null"),
    (dict(y=FAKE + 4), INVALID, "aligned"),
])
def test_bag_forward_rejects(lib, kw, code, text):
    assert fwd(lib, **kw) == code
    assert text in msg(lib)


def test_bag_forward_empty_batch_is_a_noop(lib):
    assert fwd(lib, T=0) == OK


def bwd(lib, dy=FAKE, V=FAKE, vdt=BF16, N=4096, D=64, idx=FAKE, w=FAKE, T=4, H=2, k=4, gv=FAKE,
        gw=FAKE, gz=FAKE, mode=0, ws=FAKE, ws_bytes=BIG_WS):
    return lib.mem_bag_backward(dy, V, vdt, N, D, idx, w, T, H, k, gv, gw, gz, mode, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(mode=3), INVALID, "mode"),
    (dict(H=0), INVALID, "H and k"),
    (dict(k=0), INVALID, "H and k"),
    (dict(D=9), UNSUPPORTED, "multiple of 8"),
    (dict(dy=0), INVALID, "null"),
    (dict(ws=0), WORKSPACE, "workspace"),
    (dict(ws_bytes=100), WORKSPACE, "workspace"),
    (dict(ws=FAKE + 128), INVALID, "256-byte"),
    (dict(gv=FAKE + 4), INVALID, "aligned"),
])
def test_bag_backward_rejects(lib, kw, code, text):
    assert bwd(lib, **kw) == code
    assert text in msg(lib)


def test_bag_backward_empty_batch_is_a_noop(lib):
    assert bwd(lib, T=0) == OK


def test_sparse_backward_rejects(lib):
    nrows = ctypes.c_int64(-1)
    f = lib.mem_bag_backward_sparse
    # cap below min(T*H*k, N)
    rc = f(FAKE, FAKE, BF16, 4096, 64, FAKE, FAKE, 4, 2, 4, FAKE, FAKE, 31, ctypes.addressof(nrows),
           None, None, FAKE, BIG_WS, None)
    assert rc == INVALID and "cap" in msg(lib)
    rc = f(FAKE, FAKE, BF16, 4096, 64, FAKE, FAKE, 4, 2, 4, None, FAKE, 32, ctypes.addressof(nrows),
           None, None, FAKE, BIG_WS, None)
    assert rc == INVALID and "required" in msg(lib)
    rc = f(FAKE, FAKE, BF16, 4096, 64, FAKE, FAKE, 0, 2, 4, FAKE, FAKE, 32, ctypes.addressof(nrows),
           None, None, FAKE, BIG_WS, None)
    assert rc == OK and nrows.value == 0


def sbwd(lib, q=FAKE, qdt=BF16, K=FAKE, kdt=BF16, T=8, H=2, n=64, S=16, k=4, idx=FAKE, gz=FAKE,
         gq=FAKE, gk=FAKE, ws=FAKE, ws_bytes=BIG_WS):
    return lib.mem_search_backward(q, qdt, K, kdt, T, H, n, S, k, idx, gz, gq, gk, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(n=63), INVALID, "even"),
    (dict(k=0), INVALID, "k <= S"),
    (dict(k=65), UNSUPPORTED, "k > 64"),
    (dict(S=9000), UNSUPPORTED, "S >"),
    (dict(qdt=F32), UNSUPPORTED, "share a dtype"),
    (dict(idx=0), INVALID, "null"),
    (dict(gz=0), INVALID, "null"),
    (dict(q=FAKE + 2), INVALID, "aligned"),
    (dict(ws=0), WORKSPACE, "workspace"),
    (dict(ws_bytes=8), WORKSPACE, "workspace"),
    (dict(ws=FAKE + 8), INVALID, "256-byte"),
    (dict(T=1 << 26, H=4, k=16), UNSUPPORTED, "2^32"),
    (dict(T=1, H=1 << 18, S=8192, k=1), UNSUPPORTED, "2^31"),
    (dict(gk=FAKE + 4), INVALID, "16-byte"),
])
def test_search_backward_rejects(lib, kw, code, text):
    assert sbwd(lib, **kw) == code
    assert text in msg(lib)


def test_search_backward_noops(lib):
    assert sbwd(lib, T=0) == OK
    assert sbwd(lib, gq=None, gk=None) == OK          # nothing requested
    # k counts slots (k + r after extra pairs) and may exceed S
    assert sbwd(lib, T=0, k=17) == OK
    assert lib.mem_search_backward_workspace_size(100, 4, 2048, 32) >= 100 * 4 * 2 * 32 * 8


def fwdg(lib, V=FAKE, vdt=BF16, N=4096, D=64, idx=FAKE, w=FAKE, T=4, bag=8, gate=FAKE, y=FAKE, out=FAKE):
    return lib.mem_bag_forward_gated(V, vdt, N, D, idx, w, T, bag, gate, y, out, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(D=12), UNSUPPORTED, "multiple of 8"),
    (dict(vdt=5), INVALID, "dtype"),
    (dict(gate=0), INVALID, "null"),
    (dict(out=0), INVALID, "null"),
    (dict(gate=FAKE + 8), INVALID, "aligned"),
    (dict(y=FAKE + 4), INVALID, "aligned"),
    (dict(bag=0), INVALID, "bag"),
])
def test_bag_forward_gated_rejects(lib, kw, code, text):
    assert fwdg(lib, **kw) == code
    assert text in msg(lib)


def gbwd(lib, d=FAKE, g=FAKE, y=FAKE, vdt=BF16, T=4, D=64, dy=FAKE, gg=FAKE):
    return lib.mem_gate_backward(d, g, y, vdt, T, D, dy, gg, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(D=12), UNSUPPORTED, "multiple of 8"),
    (dict(vdt=9), INVALID, "dtype"),
    (dict(T=-1), INVALID, "T must"),
    (dict(y=0), INVALID, "null"),
    (dict(gg=0), INVALID, "null"),
    (dict(gg=FAKE + 4), INVALID, "aligned"),
])
def test_gate_backward_rejects(lib, kw, code, text):
    assert gbwd(lib, **kw) == code
    assert text in msg(lib)


def test_gating_empty_batch_is_a_noop(lib):
    assert fwdg(lib, T=0) == OK
    assert gbwd(lib, T=0) == OK


def test_bwd_auto_rule(lib, monkeypatch):
    """PKMEM_BWD_AUTO: atomic when T*H*k*D <= 2^26 and D <= 1024 (the measured
    crossover), sorted otherwise; seen through the workspace sizes."""
    monkeypatch.delenv("PKMEM_BWD_MODE", raising=False)
    ws = lambda T, D, m: lib.mem_bag_backward_workspace_size(T, 4, 32, 1 << 22, D, m)  # noqa: E731
    for T, D, want in [(256, 64, 1), (8192, 64, 1), (16384, 64, 2), (4096, 128, 1),
                       (8192, 128, 2), (256, 1024, 1), (1024, 1024, 2), (256, 2048, 2),
                       (32768, 2048, 2)]:
        assert ws(T, D, 0) == ws(T, D, want), (T, D, want)
        assert ws(T, D, 1) != ws(T, D, 2)


def test_bwd_mode_environment_override(lib, monkeypatch):
    args = (1000, 4, 32, 1 << 22, 2048, 0)
    atomic = lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 1)
    sorted_ = lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 2)
    assert lib.mem_bag_backward_workspace_size(*args) == sorted_
    monkeypatch.setenv("PKMEM_BWD_MODE", "atomic")
    assert lib.mem_bag_backward_workspace_size(*args) == atomic
    monkeypatch.setenv("PKMEM_BWD_MODE", "sorted")
    assert (lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 64, 0) ==
            lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 64, 2))
    # an explicit mode is never overridden
    assert lib.mem_bag_backward_workspace_size(1000, 4, 32, 1 << 22, 2048, 1) == atomic


def searchqn(lib, q=FAKE, qdt=BF16, K=FAKE, kdt=BF16, T=8, H=2, n=64, S=16, k=4, eps=1e-5,
             idx=FAKE, w=FAKE, qhat=None, stats=None, ws=FAKE, ws_bytes=BIG_WS):
    return lib.mem_search_qnorm(q, qdt, K, kdt, T, H, n, S, k, eps, idx, w, None, None, qhat, stats,
                                ws, ws_bytes, None)


def sbwdqn(lib, T=8, eps=1e-5, gq=FAKE, gk=FAKE, ws=FAKE, ws_bytes=BIG_WS, n=64):
    return lib.mem_search_backward_qnorm(FAKE, BF16, FAKE, BF16, T, 2, n, 16, 4, eps, FAKE, FAKE, gq, gk,
                                         ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(eps=-1e-3), INVALID, "eps"),
    (dict(eps=float("nan")), INVALID, "eps"),
    (dict(eps=float("inf")), INVALID, "eps"),
    (dict(qhat=FAKE + 8), INVALID, "qhat_out"),
    (dict(stats=FAKE + 4), INVALID, "stats_out"),
    (dict(n=63), INVALID, "even"),
    (dict(k=17), INVALID, "k <= S"),
    (dict(idx=0), INVALID, "null"),
    (dict(ws_bytes=16), WORKSPACE, "workspace"),
])
def test_search_qnorm_rejects(lib, kw, code, text):
    assert searchqn(lib, **kw) == code
    assert text in msg(lib)


def test_search_qnorm_noops_and_workspace(lib):
    assert searchqn(lib, T=0) == OK
    assert searchqn(lib, T=0, eps=0.0) == OK
    assert sbwdqn(lib, T=0) == OK
    assert sbwdqn(lib, gq=None, gk=None) == OK
    assert sbwdqn(lib, eps=-1.0) == INVALID and "eps" in msg(lib)
    assert sbwdqn(lib, n=63) == INVALID
    # room for the per-query statistics on top of the plain search backward's needs
    need = lib.mem_search_backward_workspace_size(8, 2, 16, 4)
    assert sbwdqn(lib, ws_bytes=need - 1) == WORKSPACE


def searchx(lib, T=8, k=4, r=3, ex=FAKE, S=16, ws_bytes=BIG_WS):
    return lib.mem_search_extra(FAKE, BF16, FAKE, BF16, T, 2, 64, S, k, r, ex, FAKE, FAKE, None, None,
                                FAKE, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(r=-1), INVALID, "r must"),
    (dict(k=40, r=25, S=100), UNSUPPORTED, "k + r"),
    (dict(ex=0), INVALID, "null"),
    (dict(k=17), INVALID, "k <= S"),
    (dict(ws_bytes=16), WORKSPACE, "workspace"),
])
def test_search_extra_rejects(lib, kw, code, text):
    assert searchx(lib, **kw) == code
    assert text in msg(lib)


def test_search_extra_noops(lib):
    assert searchx(lib, T=0) == OK
    assert searchx(lib, T=0, ex=0) == OK
    assert searchx(lib, T=0, r=0, ex=0) == OK


def searchs(lib, T=8, k=4, r=3, ex=FAKE, S=16, sink=FAKE, row0=256, ws_bytes=BIG_WS, idx=FAKE):
    return lib.mem_search_sink(FAKE, BF16, FAKE, BF16, T, 2, 64, S, k, r, ex, sink, row0, idx, FAKE,
                               None, None, FAKE, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(r=-1), INVALID, "r must"),
    (dict(k=40, r=24, S=100), UNSUPPORTED, "k + r + 1"),
    (dict(ex=0), INVALID, "null"),
    (dict(sink=0), INVALID, "null"),
    (dict(sink=FAKE + 8), INVALID, "sink_keys"),
    (dict(row0=255), INVALID, "sink_row0"),
    (dict(row0=-1), INVALID, "sink_row0"),
    (dict(row0=(1 << 63) - 1), INVALID, "sink_row0"),
    (dict(idx=0), INVALID, "null"),
    (dict(k=17), INVALID, "k <= S"),
    (dict(ws_bytes=16), WORKSPACE, "workspace"),
])
def test_search_sink_rejects(lib, kw, code, text):
    assert searchs(lib, **kw) == code
    assert text in msg(lib)


def test_search_sink_noops(lib):
    assert searchs(lib, T=0) == OK
    assert searchs(lib, T=0, sink=0, ex=0) == OK
    assert searchs(lib, T=0, r=0, ex=0) == OK
    assert searchs(lib, T=0, k=40, r=23, S=100, row0=10000) == OK   # 64 slots
    assert searchs(lib, T=0, k=40, r=24, S=100, row0=10000) == UNSUPPORTED


def sbwds(lib, T=8, H=2, n=64, S=16, k=4, sink=FAKE, gq=FAKE, gk=FAKE, gs=FAKE, ws=FAKE,
          ws_bytes=BIG_WS):
    return lib.mem_search_backward_sink(FAKE, BF16, FAKE, BF16, T, H, n, S, k, FAKE, FAKE, sink, gq,
                                        gk, gs, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code,text", [
    (dict(k=64), UNSUPPORTED, "slots"),
    (dict(k=0), INVALID, "k <= S"),
    (dict(sink=0), INVALID, "null"),
    (dict(sink=FAKE + 8), INVALID, "sink_keys"),
    (dict(gs=FAKE + 2), INVALID, "grad_sink"),
    (dict(ws_bytes=16), WORKSPACE, "workspace"),
    (dict(n=63), INVALID, "even"),
])
def test_search_backward_sink_rejects(lib, kw, code, text):
    assert sbwds(lib, **kw) == code
    assert text in msg(lib)


def test_search_backward_sink_noops_and_workspace(lib):
    assert sbwds(lib, T=0) == OK
    assert sbwds(lib, gq=None, gk=None, gs=None) == OK
    assert sbwds(lib, T=0, gq=None, gs=None, sink=0) == OK   # only grad_subkeys: the sink is not read
    assert sbwds(lib, k=63, T=0) == OK
    # the plain search backward's needs plus the partial sums of grad_sink (one
    # row of n floats per head and chunk of 256 tokens)
    T, H, n, S, k = 1000, 4, 512, 2048, 33
    need = lib.mem_search_backward_sink_workspace_size(T, H, n, S, k)
    plain = lib.mem_search_backward_workspace_size(T, H, S, k) - ((T * H * 8 + 255) // 256) * 256
    assert need >= plain + 4 * H * n * 4
    assert sbwds(lib, T=T, H=H, n=n, S=S, k=k, ws_bytes=need - 1) == WORKSPACE
    assert lib.mem_search_backward_sink_workspace_size(-1, 4, 64, 16, 4) == 0
