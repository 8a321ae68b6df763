"""Product-key memory hot path on MI355X: thin binding of libpkmem.so.

The library (include/pkmem.h) implements the product-key search of Sec. 3.1.1
of "Memory Layers at Scale" (arXiv 2412.09764) followed by the softmax of
Sec. 3, Eq. (1), and the weighted EmbeddingBag forward and backward of
Sec. 3.1.4, as hand-written HIP kernels for gfx950.

This module only marshals arguments: it checks tensor placement and dtype,
allocates outputs and workspaces with torch on the current device (on the
`stream` argument when one is given, else on the current stream), passes raw
pointers and that HIP stream through the C ABI, and turns a non-zero status
into PkmemError.  Every step of the computation runs in the library;
there is no fallback: without the built library every call raises.
"""
from __future__ import annotations

import contextlib
import ctypes
import functools
import os

import torch  # noqa: F401  (first: the library binds to the HIP runtime torch loads)

__all__ = [
    "PkmemError", "load", "lib_path", "mem_search", "mem_search_noalloc", "mem_search_backward",
    "mem_search_qnorm", "NOALLOC_SCRATCH_BYTES",
    "mem_search_backward_qnorm", "mem_search_extra", "mem_search_sink",
    "mem_search_backward_sink", "mem_bag_forward",
    "mem_bag_forward_gated", "mem_gate_backward",
    "mem_bag_backward",
    "mem_bag_backward_sparse", "mem_search_workspace_size", "mem_bag_backward_workspace_size",
    "BWD_MODES", "F32", "BF16", "mem_timer_start", "mem_timer_stop", "mem_timer_read",
]

F32, BF16 = 0, 1
NOALLOC_SCRATCH_BYTES = 128 << 20  # PKMEM_NOALLOC_SCRATCH_BYTES
BWD_MODES = {"auto": 0, "atomic": 1, "sorted": 2}
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


class PkmemError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"pkmem status {code}: {msg}")
        self.code = code


def lib_path() -> str:
    return os.environ.get("PKMEM_LIB", os.path.join(_HERE, "libpkmem.so"))


def load() -> ctypes.CDLL:
    """Load libpkmem.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2412_09764_amd.build`")
    L = ctypes.CDLL(path)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t
    L.mem_search_workspace_size.argtypes = [I64, I32, I32, I32]
    L.mem_search_workspace_size.restype = SZ
    L.mem_search.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, SZ, P]
    L.mem_search.restype = I32
    L.mem_search_noalloc.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P]
    L.mem_search_noalloc.restype = I32
    L.mem_search_backward_workspace_size.argtypes = [I64, I32, I32, I32]
    L.mem_search_backward_workspace_size.restype = SZ
    L.mem_search_backward.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, SZ, P]
    L.mem_search_backward.restype = I32
    F32 = ctypes.c_float
    L.mem_search_qnorm.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, F32, P, P, P, P, P, P,
                                   P, SZ, P]
    L.mem_search_qnorm.restype = I32
    L.mem_search_backward_qnorm.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, F32, P, P, P,
                                            P, P, SZ, P]
    L.mem_search_backward_qnorm.restype = I32
    L.mem_search_extra.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, I32, P, P, P, P, P, P, SZ,
                                   P]
    L.mem_search_extra.restype = I32
    L.mem_search_sink.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, I32, P, P, I64, P, P, P,
                                  P, P, SZ, P]
    L.mem_search_sink.restype = I32
    L.mem_search_backward_sink_workspace_size.argtypes = [I64, I32, I32, I32, I32]
    L.mem_search_backward_sink_workspace_size.restype = SZ
    L.mem_search_backward_sink.argtypes = [P, I32, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, P,
                                           P, SZ, P]
    L.mem_search_backward_sink.restype = I32
    L.mem_bag_forward.argtypes = [P, I32, I64, I32, P, P, I64, I32, P, P]
    L.mem_bag_forward.restype = I32
    L.mem_bag_forward_gated.argtypes = [P, I32, I64, I32, P, P, I64, I32, P, P, P, P]
    L.mem_bag_forward_gated.restype = I32
    L.mem_gate_backward.argtypes = [P, P, P, I32, I64, I32, P, P, P]
    L.mem_gate_backward.restype = I32
    L.mem_bag_backward_workspace_size.argtypes = [I64, I32, I32, I64, I32, I32]
    L.mem_bag_backward_workspace_size.restype = SZ
    L.mem_bag_backward.argtypes = [P, P, I32, I64, I32, P, P, I64, I32, I32, P, P, P, I32, P, SZ, P]
    L.mem_bag_backward.restype = I32
    L.mem_bag_backward_sparse.argtypes = [P, P, I32, I64, I32, P, P, I64, I32, I32, P, P, I64, P,
                                          P, P, P, SZ, P]
    L.mem_bag_backward_sparse.restype = I32
    L.mem_last_error.argtypes = []
    L.mem_last_error.restype = ctypes.c_char_p
    L.mem_version.argtypes = []
    L.mem_version.restype = I32
    L.mem_timer_start.argtypes = [ctypes.c_char_p]
    L.mem_timer_start.restype = I32
    L.mem_timer_stop.argtypes = []
    L.mem_timer_stop.restype = I32
    L.mem_timer_read.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.POINTER(ctypes.c_int), I32]
    L.mem_timer_read.restype = I32
    _LIB = L
    return L


def _check(rc: int) -> None:
    if rc != 0:
        raise PkmemError(rc, load().mem_last_error().decode(errors="replace"))


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _dev(*ts: torch.Tensor) -> None:
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _on(stream):
    """Context making `stream` (if given) torch's current stream, so that the
    outputs and workspaces allocated inside belong to the stream the library
    launches on and any zero-fill is ordered before the launch."""
    return contextlib.nullcontext() if stream is None else torch.cuda.stream(stream)


def _launches_on_stream(fn):
    """Runs fn with its `stream` argument (if given) as torch's current stream:
    outputs, workspaces and zero-filled accumulators allocated by the wrapper
    then belong to the stream the library launches on, and the fills are
    ordered before the launch on that stream."""
    @functools.wraps(fn)
    def wrapper(*args, stream=None, **kw):
        with _on(stream):
            return fn(*args, stream=stream, **kw)
    return wrapper


def _workspace(nbytes: int, device, ws):
    if ws is not None:
        if ws.numel() * ws.element_size() < nbytes:
            raise ValueError(f"workspace too small: {nbytes} bytes needed")
        return ws
    return torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)


def mem_timer_start(*kernels: str) -> None:
    """Record HIP events around every launch of the named kernels (pkmem.h)."""
    _check(load().mem_timer_start(",".join(kernels).encode()))


def mem_timer_stop() -> None:
    _check(load().mem_timer_stop())


def mem_timer_read(cap: int = 1 << 16) -> list:
    """[(kernel_position, ms)] of the launches recorded since the last read."""
    ms = (ctypes.c_float * cap)()
    which = (ctypes.c_int * cap)()
    n = load().mem_timer_read(ms, which, cap)
    if n < 0:
        _check(n)
    return [(int(which[i]), float(ms[i])) for i in range(min(n, cap))]


def mem_search_workspace_size(T: int, H: int, S: int, k: int) -> int:
    return int(load().mem_search_workspace_size(T, H, S, k))


def mem_bag_backward_workspace_size(T: int, H: int, k: int, N: int, D: int, mode="auto") -> int:
    m = BWD_MODES[mode] if isinstance(mode, str) else int(mode)
    return int(load().mem_bag_backward_workspace_size(T, H, k, N, D, m))


@_launches_on_stream
def mem_search(q: torch.Tensor, subkeys: torch.Tensor, k: int, *, idx_out=None, w_out=None,
               score_out=None, half_idx_out=None, want_score: bool = True,
               want_half: bool = False, workspace=None, stream=None):
    """Product-key search + softmax.  q [T, H, n], subkeys [H, 2, S, n/2].

    Returns (idx int64 [T,H,k], w fp32 [T,H,k], score fp32 [T,H,k] or None,
    half_idx int32 [T,H,2,k] or None).
    """
    return _search(q, subkeys, k, None, idx_out, w_out, score_out, half_idx_out, want_score,
                   want_half, None, None, workspace, stream)[:4]


@_launches_on_stream
def mem_search_noalloc(q: torch.Tensor, subkeys: torch.Tensor, k: int, *, idx_out=None,
                       w_out=None, score_out=None, half_idx_out=None, want_score: bool = True,
                       want_half: bool = False, stream=None):
    """mem_search with its workspace in the library's static device scratch
    array (no workspace argument; the C call allocates nothing).  Outputs not
    given are allocated here with torch; pass them all to allocate nothing.
    Requires mem_search_workspace_size(T, H, S, k) <= NOALLOC_SCRATCH_BYTES."""
    L = load()
    _dev(q, subkeys)
    T, H, n = q.shape
    S = subkeys.shape[2]
    dev = q.device
    if idx_out is None:
        idx_out = torch.empty((T, H, k), dtype=torch.int64, device=dev)
    if w_out is None:
        w_out = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    if score_out is None and want_score:
        score_out = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    if half_idx_out is None and want_half:
        half_idx_out = torch.empty((T, H, 2, k), dtype=torch.int32, device=dev)
    _dev(idx_out, w_out, score_out, half_idx_out)
    _check(L.mem_search_noalloc(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k,
                                _ptr(idx_out), _ptr(w_out), _ptr(score_out), _ptr(half_idx_out),
                                _stream(stream)))
    return idx_out, w_out, score_out, half_idx_out


@_launches_on_stream
def mem_search_qnorm(q: torch.Tensor, subkeys: torch.Tensor, k: int, eps: float = 1e-5, *,
                     idx_out=None, w_out=None, score_out=None, half_idx_out=None,
                     want_score: bool = True, want_half: bool = False, qhat_out=None,
                     stats_out=None, want_qhat: bool = False, want_stats: bool = False,
                     workspace=None, stream=None):
    """mem_search of the LayerNorm-normalised queries (no affine, eps), the
    normalisation fused into the scoring.  Returns (idx, w, score, half_idx,
    qhat [T,H,n] in q's dtype or None, stats fp32 [T,H,2] (mean, rstd) or None)."""
    T, H, n = q.shape
    if qhat_out is None and want_qhat:
        qhat_out = torch.empty((T, H, n), dtype=q.dtype, device=q.device)
    if stats_out is None and want_stats:
        stats_out = torch.empty((T, H, 2), dtype=torch.float32, device=q.device)
    return _search(q, subkeys, k, float(eps), idx_out, w_out, score_out, half_idx_out, want_score,
                   want_half, qhat_out, stats_out, workspace, stream)


@_launches_on_stream
def mem_search_extra(q: torch.Tensor, subkeys: torch.Tensor, k: int, extra_idx: torch.Tensor, *,
                     idx_out=None, w_out=None, score_out=None, half_idx_out=None,
                     want_score: bool = True, want_half: bool = False, workspace=None,
                     stream=None):
    """mem_search plus r extra key-value pairs per (token, head): extra_idx
    [T, H, r] int64 composed indices, scored as full keys, in slots k..k+r-1;
    softmax over all k + r.  Returns (idx, w, score, half_idx) with k + r slots."""
    return _search_extra(q, subkeys, k, extra_idx, None, 0, idx_out, w_out, score_out,
                         half_idx_out, want_score, want_half, workspace, stream)


@_launches_on_stream
def mem_search_sink(q: torch.Tensor, subkeys: torch.Tensor, k: int, sink_keys: torch.Tensor,
                    sink_row0: int, extra_idx=None, *, idx_out=None, w_out=None, score_out=None,
                    half_idx_out=None, want_score: bool = True, want_half: bool = False,
                    workspace=None, stream=None):
    """mem_search_extra (extra_idx [T, H, r] or None) plus one fixed key-value
    pair per head in the last slot: key sink_keys [H, n] (subkeys' dtype),
    scored q . sink_keys[h]; index sink_row0 + h (>= S*S, the value-table row of
    head h's sink value).  Returns (idx, w, score, half_idx) with k + r + 1 slots."""
    if extra_idx is None:
        T, H, _ = q.shape
        extra_idx = torch.empty((T, H, 0), dtype=torch.int64, device=q.device)
    return _search_extra(q, subkeys, k, extra_idx, sink_keys, int(sink_row0), idx_out, w_out,
                         score_out, half_idx_out, want_score, want_half, workspace, stream)


def _search_extra(q, subkeys, k, extra_idx, sink_keys, sink_row0, idx_out, w_out, score_out,
                  half_idx_out, want_score, want_half, workspace, stream):
    L = load()
    _dev(q, subkeys, extra_idx, sink_keys)
    T, H, n = q.shape
    S = subkeys.shape[2]
    r = extra_idx.shape[2] if extra_idx.dim() == 3 else 0
    if extra_idx.dtype != torch.int64:
        raise ValueError("extra_idx must be int64")
    if sink_keys is not None and (sink_keys.shape != (H, n) or sink_keys.dtype != subkeys.dtype):
        raise ValueError("sink_keys must be [H, n] in the sub-keys' dtype")
    dev = q.device
    kk = k + r + (1 if sink_keys is not None else 0)
    if idx_out is None:
        idx_out = torch.empty((T, H, kk), dtype=torch.int64, device=dev)
    if w_out is None:
        w_out = torch.empty((T, H, kk), dtype=torch.float32, device=dev)
    if score_out is None and want_score:
        score_out = torch.empty((T, H, kk), dtype=torch.float32, device=dev)
    if half_idx_out is None and want_half:
        half_idx_out = torch.empty((T, H, 2, k), dtype=torch.int32, device=dev)
    _dev(idx_out, w_out, score_out, half_idx_out)
    ws = _workspace(mem_search_workspace_size(T, H, S, k), dev, workspace)
    outs = (_ptr(idx_out), _ptr(w_out), _ptr(score_out), _ptr(half_idx_out), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream))
    if sink_keys is None:
        _check(L.mem_search_extra(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k, r,
                                  _ptr(extra_idx), *outs))
    else:
        _check(L.mem_search_sink(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k, r,
                                 _ptr(extra_idx), _ptr(sink_keys), sink_row0, *outs))
    return idx_out, w_out, score_out, half_idx_out


def _search(q, subkeys, k, eps, idx_out, w_out, score_out, half_idx_out, want_score, want_half,
            qhat_out, stats_out, workspace, stream):
    L = load()
    _dev(q, subkeys)
    T, H, n = q.shape
    S = subkeys.shape[2]
    dev = q.device
    if idx_out is None:
        idx_out = torch.empty((T, H, k), dtype=torch.int64, device=dev)
    if w_out is None:
        w_out = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    if score_out is None and want_score:
        score_out = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    if half_idx_out is None and want_half:
        half_idx_out = torch.empty((T, H, 2, k), dtype=torch.int32, device=dev)
    _dev(idx_out, w_out, score_out, half_idx_out)
    nbytes = mem_search_workspace_size(T, H, S, k)
    ws = _workspace(nbytes, dev, workspace)
    if eps is None:
        _check(L.mem_search(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k,
                            _ptr(idx_out), _ptr(w_out), _ptr(score_out), _ptr(half_idx_out),
                            _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    else:
        _dev(qhat_out, stats_out)
        _check(L.mem_search_qnorm(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k, eps,
                                  _ptr(idx_out), _ptr(w_out), _ptr(score_out), _ptr(half_idx_out),
                                  _ptr(qhat_out), _ptr(stats_out), _ptr(ws),
                                  ws.numel() * ws.element_size(), _stream(stream)))
    return idx_out, w_out, score_out, half_idx_out, qhat_out, stats_out


@_launches_on_stream
def mem_search_backward(q: torch.Tensor, subkeys: torch.Tensor, idx: torch.Tensor,
                        grad_scores: torch.Tensor, *, grad_q=None, grad_subkeys=None,
                        want_grad_q: bool = True, want_grad_subkeys: bool = True, workspace=None,
                        stream=None):
    """Gradients of the selected scores into q ([T,H,n], written) and the
    sub-keys ([H,2,S,n/2], ACCUMULATED; a zero table is allocated if none is
    given).  Returns (grad_q, grad_subkeys)."""
    return _search_backward(q, subkeys, idx, grad_scores, None, grad_q, grad_subkeys, want_grad_q,
                            want_grad_subkeys, workspace, stream)


@_launches_on_stream
def mem_search_backward_qnorm(q: torch.Tensor, subkeys: torch.Tensor, idx: torch.Tensor,
                              grad_scores: torch.Tensor, eps: float = 1e-5, *, grad_q=None,
                              grad_subkeys=None, want_grad_q: bool = True,
                              want_grad_subkeys: bool = True, workspace=None, stream=None):
    """mem_search_backward through the query normalisation of
    mem_search_qnorm (same q and eps): grad_q with respect to the raw
    queries, grad_subkeys accumulated from the normalised ones."""
    return _search_backward(q, subkeys, idx, grad_scores, float(eps), grad_q, grad_subkeys,
                            want_grad_q, want_grad_subkeys, workspace, stream)


@_launches_on_stream
def mem_search_backward_sink(q: torch.Tensor, subkeys: torch.Tensor, idx: torch.Tensor,
                             grad_scores: torch.Tensor, sink_keys: torch.Tensor, *, grad_q=None,
                             grad_subkeys=None, grad_sink=None, want_grad_q: bool = True,
                             want_grad_subkeys: bool = True, want_grad_sink: bool = True,
                             workspace=None, stream=None):
    """Search backward of mem_search_sink: idx and grad_scores [T, H, k + 1]
    (last slot the sink's).  grad_q written; grad_subkeys and grad_sink
    ([H, n] fp32) ACCUMULATED (zero tables allocated if none are given).
    Returns (grad_q, grad_subkeys, grad_sink)."""
    L = load()
    _dev(q, subkeys, idx, grad_scores, sink_keys)
    T, H, n = q.shape
    S = subkeys.shape[2]
    k = idx.shape[2] - 1
    if grad_q is None and want_grad_q:
        grad_q = torch.empty((T, H, n), dtype=torch.float32, device=q.device)
    if grad_subkeys is None and want_grad_subkeys:
        grad_subkeys = torch.zeros(subkeys.shape, dtype=torch.float32, device=q.device)
    if grad_sink is None and want_grad_sink:
        grad_sink = torch.zeros((H, n), dtype=torch.float32, device=q.device)
    _dev(grad_q, grad_subkeys, grad_sink)
    nbytes = int(L.mem_search_backward_sink_workspace_size(T, H, n, S, k))
    ws = _workspace(nbytes, q.device, workspace)
    _check(L.mem_search_backward_sink(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k,
                                      _ptr(idx), _ptr(grad_scores), _ptr(sink_keys), _ptr(grad_q),
                                      _ptr(grad_subkeys), _ptr(grad_sink), _ptr(ws),
                                      ws.numel() * ws.element_size(), _stream(stream)))
    return grad_q, grad_subkeys, grad_sink


def _search_backward(q, subkeys, idx, grad_scores, eps, grad_q, grad_subkeys, want_grad_q,
                     want_grad_subkeys, workspace, stream):
    L = load()
    _dev(q, subkeys, idx, grad_scores)
    T, H, n = q.shape
    S = subkeys.shape[2]
    k = idx.shape[2]
    if grad_q is None and want_grad_q:
        grad_q = torch.empty((T, H, n), dtype=torch.float32, device=q.device)
    if grad_subkeys is None and want_grad_subkeys:
        grad_subkeys = torch.zeros(subkeys.shape, dtype=torch.float32, device=q.device)
    _dev(grad_q, grad_subkeys)
    nbytes = int(L.mem_search_backward_workspace_size(T, H, S, k))
    ws = _workspace(nbytes, q.device, workspace)
    args = (_ptr(idx), _ptr(grad_scores), _ptr(grad_q), _ptr(grad_subkeys), _ptr(ws),
            ws.numel() * ws.element_size(), _stream(stream))
    if eps is None:
        _check(L.mem_search_backward(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n, S, k,
                                     *args))
    else:
        _check(L.mem_search_backward_qnorm(_ptr(q), _dt(q), _ptr(subkeys), _dt(subkeys), T, H, n,
                                           S, k, eps, *args))
    return grad_q, grad_subkeys


@_launches_on_stream
def mem_bag_forward(values: torch.Tensor, idx: torch.Tensor, w: torch.Tensor, *, y_out=None,
                    stream=None):
    """y[t] = sum_j w[t, j] values[idx[t, j]]; idx, w of shape [T, ...] (bag = rest)."""
    L = load()
    _dev(values, idx, w)
    N, D = values.shape
    T = idx.shape[0]
    bag = idx.numel() // T if T else (idx[0].numel() if idx.dim() > 1 else 1)
    if idx.dtype != torch.int64 or w.dtype != torch.float32:
        raise TypeError("idx must be int64 and w float32")
    if y_out is None:
        y_out = torch.empty((T, D), dtype=values.dtype, device=values.device)
    _dev(y_out)
    _check(L.mem_bag_forward(_ptr(values), _dt(values), N, D, _ptr(idx), _ptr(w), T, bag,
                             _ptr(y_out), _stream(stream)))
    return y_out


@_launches_on_stream
def mem_bag_forward_gated(values: torch.Tensor, idx: torch.Tensor, w: torch.Tensor,
                          gate: torch.Tensor, *, want_y=True, out=None, y_out=None, stream=None):
    """Memory+ epilogue: out = bag * silu(gate), gate [T, D] in the value dtype.
    Returns (out, y) with y the un-gated bag (None unless want_y)."""
    L = load()
    _dev(values, idx, w, gate)
    N, D = values.shape
    T = idx.shape[0]
    bag = idx.numel() // T if T else (idx[0].numel() if idx.dim() > 1 else 1)
    if idx.dtype != torch.int64 or w.dtype != torch.float32:
        raise TypeError("idx must be int64 and w float32")
    if gate.dtype != values.dtype or tuple(gate.shape) != (T, D) or not gate.is_contiguous():
        raise ValueError("gate must be a contiguous [T, D] tensor of the value dtype")
    if out is None:
        out = torch.empty((T, D), dtype=values.dtype, device=values.device)
    if y_out is None and want_y:
        y_out = torch.empty((T, D), dtype=values.dtype, device=values.device)
    _dev(out, y_out)
    _check(L.mem_bag_forward_gated(_ptr(values), _dt(values), N, D, _ptr(idx), _ptr(w), T, bag,
                                   _ptr(gate), _ptr(y_out), _ptr(out), _stream(stream)))
    return out, y_out


@_launches_on_stream
def mem_gate_backward(d_out: torch.Tensor, gate: torch.Tensor, y: torch.Tensor, *, dy_out=None,
                      grad_gate=None, stream=None):
    """Backward of out = y * silu(gate): returns (dy [value dtype], grad_gate fp32)."""
    L = load()
    _dev(d_out, gate, y)
    T, D = d_out.shape
    for t_ in (gate, y):
        if t_.dtype != d_out.dtype or tuple(t_.shape) != (T, D) or not t_.is_contiguous():
            raise ValueError("gate and y must be contiguous [T, D] tensors of d_out's dtype")
    if dy_out is None:
        dy_out = torch.empty((T, D), dtype=d_out.dtype, device=d_out.device)
    if grad_gate is None:
        grad_gate = torch.empty((T, D), dtype=torch.float32, device=d_out.device)
    _dev(dy_out, grad_gate)
    _check(L.mem_gate_backward(_ptr(d_out), _ptr(gate), _ptr(y), _dt(d_out), T, D, _ptr(dy_out),
                               _ptr(grad_gate), _stream(stream)))
    return dy_out, grad_gate


@_launches_on_stream
def mem_bag_backward(dy: torch.Tensor, values: torch.Tensor, idx: torch.Tensor, w: torch.Tensor,
                     *, grad_values=None, grad_w=None, grad_scores=None, want_grad_values=True,
                     want_grad_w=True, want_grad_scores=True, mode="auto", workspace=None,
                     stream=None):
    """EmbeddingBag + softmax backward.  idx, w [T, H, k].  grad_values is
    ACCUMULATED into (a zero table is allocated if none is given)."""
    Lb = load()
    _dev(dy, values, idx, w)
    N, D = values.shape
    T, H, k = idx.shape
    dev = values.device
    if grad_values is None and want_grad_values:
        grad_values = torch.zeros((N, D), dtype=torch.float32, device=dev)
    if grad_w is None and want_grad_w:
        grad_w = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    if grad_scores is None and want_grad_scores:
        grad_scores = torch.empty((T, H, k), dtype=torch.float32, device=dev)
    _dev(grad_values, grad_w, grad_scores)
    m = BWD_MODES[mode] if isinstance(mode, str) else int(mode)
    nbytes = int(Lb.mem_bag_backward_workspace_size(T, H, k, N, D, m))
    ws = _workspace(nbytes, dev, workspace)
    _check(Lb.mem_bag_backward(_ptr(dy), _ptr(values), _dt(values), N, D, _ptr(idx), _ptr(w), T,
                               H, k, _ptr(grad_values), _ptr(grad_w), _ptr(grad_scores), m,
                               _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    return grad_values, grad_w, grad_scores


@_launches_on_stream
def mem_bag_backward_sparse(dy: torch.Tensor, values: torch.Tensor, idx: torch.Tensor,
                            w: torch.Tensor, *, want_grad_w=True, want_grad_scores=True,
                            workspace=None, stream=None):
    """Backward with the value gradient as touched rows only.

    Returns (rows int64 [U], grad_rows fp32 [U, D], grad_w, grad_scores); waits
    for the stream to learn U.
    """
    Lb = load()
    _dev(dy, values, idx, w)
    N, D = values.shape
    T, H, k = idx.shape
    dev = values.device
    cap = max(1, min(T * H * k, N))
    rows = torch.empty((cap,), dtype=torch.int64, device=dev)
    grad_rows = torch.empty((cap, D), dtype=torch.float32, device=dev)
    grad_w = torch.empty((T, H, k), dtype=torch.float32, device=dev) if want_grad_w else None
    grad_scores = torch.empty((T, H, k), dtype=torch.float32, device=dev) if want_grad_scores else None
    nbytes = int(Lb.mem_bag_backward_workspace_size(T, H, k, N, D, BWD_MODES["sorted"]))
    ws = _workspace(nbytes, dev, workspace)
    U = ctypes.c_int64(0)
    _check(Lb.mem_bag_backward_sparse(_ptr(dy), _ptr(values), _dt(values), N, D, _ptr(idx),
                                      _ptr(w), T, H, k, _ptr(rows), _ptr(grad_rows), cap,
                                      ctypes.addressof(U), _ptr(grad_w), _ptr(grad_scores),
                                      _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))
    u = int(U.value)
    return rows[:u], grad_rows[:u], grad_w, grad_scores
