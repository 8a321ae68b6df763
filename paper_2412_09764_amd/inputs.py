"""Seeded synthetic inputs for the product-key memory workloads.

This module only draws random numbers and reshapes them; it holds none of
the method's arithmetic.  The tests, the benchmark and the smoke check use it
to feed the same tensors to the HIP library and to the CPU oracle.

The paper trains on text corpora that are not available here; Gaussian draws
at the paper's memory shapes stand in for the activations (value dim 2048 and
N in {1024^2 .. 8192^2} as in its memory-size scaling study; 1M x 1024 values
and key dim 512 as in its key/value-dimension ablation).

Per workload, every tensor has its own generator seeded with
`seed_base + slot` (slot 0 queries, 1 sub-keys, 2 values, 3 upstream
gradient, 4 cluster centres, 5 cluster ids), so a tensor never depends on
the order in which the others were drawn.  `N(0, x)` below means standard
deviation x.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

__all__ = ["Workload", "WORKLOADS", "gen_queries", "gen_subkeys", "gen_values",
           "gen_dy", "torch_dtype"]


@dataclass(frozen=True)
class Workload:
    name: str
    S: int            # sub-keys per half; N = S * S values
    H: int            # heads (independent query / sub-key pairs per token)
    n: int            # query dim per head; d = n / 2 per half
    D: int            # value dim
    k: int            # top-k per half and overall
    T: int            # tokens per step
    key_dtype: str    # dtype of queries and sub-keys: "f32" | "bf16"
    value_dtype: str  # dtype of values, output and upstream gradient
    subkey_std: float
    value_std: float
    query: str        # "normal" | "layernorm" | "clusters"
    sparse_grad: bool  # value gradient as touched rows only
    seed_base: int

    @property
    def N(self) -> int:
        return self.S * self.S

    @property
    def d(self) -> int:
        return self.n // 2

    @property
    def bag(self) -> int:
        return self.H * self.k


WORKLOADS = {
    # 64^2 = 4096 keys, 1 head, n = 64, 4096 x 64 fp32 values, k = 8, 256 tokens.
    "pk4k_d64_f32": Workload("pk4k_d64_f32", S=64, H=1, n=64, D=64, k=8, T=256,
                             key_dtype="f32", value_dtype="f32", subkey_std=1.0,
                             value_std=0.02, query="normal", sparse_grad=False,
                             seed_base=1000),
    # 1024^2 keys, 4 heads, n = 512, 1M x 1024 bf16 values, k = 32, 16384 tokens,
    # queries layer-normalised per (token, head).
    "pk1m_d1024": Workload("pk1m_d1024", S=1024, H=4, n=512, D=1024, k=32, T=16384,
                           key_dtype="bf16", value_dtype="bf16", subkey_std=1.0 / 256,
                           value_std=0.02, query="layernorm", sparse_grad=False,
                           seed_base=2000),
    # 2048^2 = 4M keys, 4 heads, n = 512, 4M x 2048 bf16 values (16 GiB),
    # k = 32, 32768 tokens (8 sequences x 4096).
    "pk4m_d2048": Workload("pk4m_d2048", S=2048, H=4, n=512, D=2048, k=32, T=32768,
                           key_dtype="bf16", value_dtype="bf16", subkey_std=1.0 / 256,
                           value_std=0.02, query="normal", sparse_grad=False,
                           seed_base=3000),
    # 4096^2 = 16M keys, 16M x 2048 bf16 values (64 GiB), sparse value gradient.
    "pk16m_d2048": Workload("pk16m_d2048", S=4096, H=4, n=512, D=2048, k=32, T=32768,
                            key_dtype="bf16", value_dtype="bf16", subkey_std=1.0 / 256,
                            value_std=0.02, query="normal", sparse_grad=True,
                            seed_base=4000),
    # 8192^2 = 64M keys, 64M x 256 bf16 values (an embedding-dim slice, 32 GiB),
    # 65536 tokens whose queries come from a 64-cluster Gaussian mixture.
    "pk64m_d256": Workload("pk64m_d256", S=8192, H=4, n=512, D=256, k=32, T=65536,
                           key_dtype="bf16", value_dtype="bf16", subkey_std=1.0 / 256,
                           value_std=0.02, query="clusters", sparse_grad=False,
                           seed_base=5000),
}

_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def torch_dtype(name: str) -> torch.dtype:
    return _DT[name]


def _gen(wl: Workload, slot: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed_base + slot)
    return g


def _int_uniform(shape, g, device) -> torch.Tensor:
    """Integers uniform over {-4..4}: exact in bf16 and fp32, and every
    dot product of length <= 2^16 of them is an exact integer in fp32."""
    return torch.randint(-4, 5, shape, generator=g, device=device).to(torch.float32)


def gen_queries(wl: Workload, device="cpu", integer: bool = False, T: int | None = None) -> torch.Tensor:
    """Queries [T, H, n] in the workload's key dtype.

    A smaller T is its own draw, not necessarily a prefix of the full one
    (device generators place values by launch geometry): to compare a token
    slice, draw the full tensor and slice it."""
    T = wl.T if T is None else T
    shape = (T, wl.H, wl.n)
    g = _gen(wl, 0, device)
    if integer:
        q = _int_uniform(shape, g, device)
    elif wl.query == "normal":
        q = torch.randn(shape, generator=g, device=device)
    elif wl.query == "layernorm":
        x = torch.randn(shape, generator=g, device=device)
        # LayerNorm without affine parameters, eps 1e-5, per (token, head).
        q = torch.nn.functional.layer_norm(x, (wl.n,), eps=1e-5)
    elif wl.query == "clusters":
        # 64 centres per head with unit-variance entries; one cluster id per
        # token shared by its heads; q = centre + 0.1 * noise.
        gc = _gen(wl, 4, device)
        gi = _gen(wl, 5, device)
        centres = torch.randn((64, wl.H, wl.n), generator=gc, device=device)
        ids = torch.randint(0, 64, (T,), generator=gi, device=device)
        q = centres[ids] + 0.1 * torch.randn(shape, generator=g, device=device)
    else:
        raise ValueError(wl.query)
    return q.to(_DT[wl.key_dtype]).contiguous()


def gen_subkeys(wl: Workload, device="cpu", integer: bool = False) -> torch.Tensor:
    """Sub-keys [H, 2, S, d]: [h, 0] pairs with q[..., :d], [h, 1] with q[..., d:]."""
    shape = (wl.H, 2, wl.S, wl.d)
    g = _gen(wl, 1, device)
    if integer:
        K = _int_uniform(shape, g, device)
    else:
        K = torch.randn(shape, generator=g, device=device) * wl.subkey_std
    return K.to(_DT[wl.key_dtype]).contiguous()


def gen_values(wl: Workload, device="cpu", rows: int | None = None,
               chunk_elems: int = 1 << 28) -> torch.Tensor:
    """Value table [N, D] ~ N(0, value_std) in the value dtype.

    Drawn in fp32 chunks of at most `chunk_elems` elements and cast per
    chunk, so a 16-64 GiB bf16 table never needs an fp32 copy.  `rows`
    draws a smaller table of that many rows (its own draw, not a prefix).
    """
    N = wl.N if rows is None else rows
    out = torch.empty((N, wl.D), dtype=_DT[wl.value_dtype], device=device)
    g = _gen(wl, 2, device)
    step = max(1, chunk_elems // wl.D)
    for r0 in range(0, N, step):
        r1 = min(N, r0 + step)
        out[r0:r1] = (torch.randn((r1 - r0, wl.D), generator=g, device=device)
                      * wl.value_std).to(out.dtype)
    return out


def gen_dy(wl: Workload, device="cpu", T: int | None = None) -> torch.Tensor:
    """Upstream gradient [T, D] ~ N(0, 1) in the value dtype."""
    T = wl.T if T is None else T
    g = _gen(wl, 3, device)
    return torch.randn((T, wl.D), generator=g, device=device).to(_DT[wl.value_dtype]).contiguous()
