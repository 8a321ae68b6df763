"""Plain fp64 CPU oracle for the product-key memory hot path.

TEST INFRASTRUCTURE ONLY.  This module is the checker, not the product:
only the test suite, the smoke check and the benchmark's CPU-baseline leg
may import it.  It shares no code with the HIP library and never imports
it.  It is deliberately slow and literal: per-token Python loops over
NumPy float64 arrays, one library primitive per step (a dot product, a
lexicographic sort, an exponential), no blocking, no fusion, no pruning.

Paper: "Memory Layers at Scale" (arXiv 2412.09764).

  Sec. 3, Eq. (1)              I = SelectTopkIndices(K q),
                               s = Softmax(K_I q),  y = s V_I,
                               each token independently.
  Sec. 3.1.1 (Product-key lookup)
                               K1, K2 in R^{sqrt(N) x n/2}; the full key set
                               (never instantiated) is their product; split
                               q into q1, q2; top-k per half; the result is
                               the best k of the k x k sums s1[i1] + s2[i2].
  Sec. 3.1.4 (Performance and stability improvements)
                               the weighted sum is an EmbeddingBag; its
                               backward propagates several output gradients
                               into the same value-gradient row.

Readings where the paper is silent:
  * heads: H independent (query, sub-key pair) per token, one shared value
    table, per-head top-k and softmax, one bag of H*k rows summed;
  * composed index i = i1 * S + i2, with q1 = q[:n/2] scored against
    sub-key half 0, so full key row i is [K1[i // S]; K2[i % S]];
  * "argmax over I1 x I2" means the top k of the k*k sums;
  * order: score descending, index ascending (lower index wins a tie), at
    both levels; outputs are in that rank order;
  * raw dot-product scores: no scale, no temperature, no bias;
  * softmax over the k selected scores of one (token, head);
  * value gradients accumulate (+=) into the caller's table, because one
    value pool is shared by several memory layers (Sec. 3.1.3).

Function pins (tests under tests/test_oracle_*.py):
  search           brute force over the instantiated full key set; all-equal
                   sub-keys; k = 1 argmax; hand-worked golden fixture
  softmax          closed form for two entries; sum/positivity/order/shift
  bag_forward      torch embedding_bag (fp64, CPU); dense A @ V; one-hot rows
  bag_backward     torch autograd (fp64, CPU); central finite differences;
                   dense A.T @ dy; sum of score gradients is zero
  invert_index     multiset and ordering invariants
  search_backward  central finite differences of the selected scores at a fixed
                   selection; torch autograd (fp64); the bilinear identities
                   sum(grad_q * q) = sum(grad_z * z) = sum(grad_K * K)
  silu, gated_output, gated_backward
                   torch.nn.functional.silu and torch autograd (fp64, CPU);
                   closed forms silu(0) = 0, silu(ln 3) = (3/4) ln 3,
                   silu'(0) = 1/2; central finite differences; limits
  query_layernorm  torch.nn.functional.layer_norm (fp64, CPU); closed form for
                   [1, 2, 3, 4]; zero mean, mean square var / (var + eps);
                   invariance to shift and (eps = 0) positive scale
  round_bf16       torch's bf16 conversion of fp32 values; hand-worked ties
  search_qnorm     eps = 0 on rows built with mean 0 and variance 4: equals
                   the plain search (and brute force) on q / 2
  search_backward_qnorm
                   central finite differences in the raw queries at a fixed
                   selection; torch autograd through layer_norm (fp64)
  search_sink, search_backward_sink
                   zero sink key: logit 0, weights exp(z) / (1 + sum exp(z));
                   a sink whose score dominates takes the whole weight; the
                   other slots as `search_extra`; gradients by central
                   differences and torch autograd (fp64)
  search_extra     r = 0 gives `search`; every extra slot's score equals the
                   brute-force full-key score of its index; an extra that
                   repeats a selected index repeats its score; the weights
                   are the closed-form softmax of the k + r scores

Fixed ("sink") key-value pair (Sec. 5.4, model ablations, names one fixed
key-value pair added to the selected ones as an anchor, without a formula).
Reading: per head a key k_s[h] in R^n and a value row given by the caller (a
row of the value table the caller adds, so the bag treats it as any other
lookup); its score is the query's dot product with k_s[h], like any key's;
it takes one more slot after the selected (and extra) ones and joins their
softmax.  k_s = 0 gives the constant logit 0, the softmax with one added to
its denominator.

Extra key-value pairs (Sec. 5.4, model ablations, names adding random
key-value pairs beside the top-k during pre-training, without a formula).
Reading: per (token, head) the caller draws r indices in [0, S*S) (the
random numbers are inputs); each is scored like any full key, s1[i1] + s2[i2],
and occupies its own slot after the k selected ones (a repeat of a selected
index is a separate slot); the softmax runs over all k + r scores.

Query normalisation (qk-normalisation, named in Sec. 3.1.4 as the remedy for
unstable training of large memories, citing a LayerNorm of queries and keys).
The paper gives no formula; reading: LayerNorm without affine parameters over
each (token, head) query of n elements, biased variance, eps inside the
square root; a query with zero variance and eps = 0 normalises to zeros.  The
normalised query is stored in the query dtype (bf16 or fp32) before scoring,
and that rounding passes gradients unchanged.  Sub-keys are parameters and are
not normalised here.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "rank_order",
    "order_desc",
    "topk_desc",
    "half_scores",
    "search",
    "brute_force_search",
    "softmax",
    "bag_forward",
    "bag_backward",
    "bag_backward_rows",
    "invert_index",
    "search_backward",
    "silu",
    "gated_output",
    "gated_backward",
    "round_bf16",
    "round_to",
    "query_layernorm",
    "search_qnorm",
    "search_backward_qnorm",
    "search_extra",
    "search_sink",
    "search_backward_sink",
]


def _f64(a) -> np.ndarray:
    """Exact widening of stored fp32 / bf16-in-fp32 values to fp64."""
    return np.asarray(a, dtype=np.float64)


def rank_order(scores: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Positions sorted by (score descending, id ascending).

    The tie rule (lower index first) is the reading taken for a point the
    paper leaves open; it makes every selection unique.
    """
    scores = np.asarray(scores, dtype=np.float64)
    # lexsort sorts by the last key first: primary -score, secondary id.
    return np.lexsort((np.asarray(ids), -scores))


def order_desc(scores: np.ndarray) -> np.ndarray:
    """Positions of `scores` sorted by (score descending, position ascending)."""
    return rank_order(scores, np.arange(np.asarray(scores).shape[0]))


def topk_desc(scores: np.ndarray, k: int) -> np.ndarray:
    """First k positions of order_desc(scores) (Sec. 3, Eq. (1): top-k)."""
    return order_desc(scores)[:k]


def half_scores(q_half: np.ndarray, subkeys_half: np.ndarray) -> np.ndarray:
    """Scores of one query half against one sub-key table (Sec. 3.1.1).

    q_half: [d]; subkeys_half: [S, d].  Returns [S] = subkeys_half @ q_half.
    """
    return _f64(subkeys_half) @ _f64(q_half)


def softmax(z: np.ndarray) -> np.ndarray:
    """Softmax over the selected scores (Sec. 3, Eq. (1)), max-subtracted."""
    z = _f64(z)
    e = np.exp(z - z.max())
    return e / e.sum()


def search(q: np.ndarray, subkeys: np.ndarray, k: int) -> dict:
    """Multi-head product-key search (Sec. 3.1.1) followed by softmax (Eq. (1)).

    q:       [T, H, n] query per token and head, n even, d = n / 2.
    subkeys: [H, 2, S, d]; subkeys[h, 0] is K1 (paired with q[..., :d]),
             subkeys[h, 1] is K2 (paired with q[..., d:]).
    k:       1 <= k <= S.

    Returns a dict of
      idx        [T, H, k] int64   composed index i1 * S + i2, rank order
      score      [T, H, k] fp64    s1[i1] + s2[i2] = full-key score K_I q
      w          [T, H, k] fp64    softmax of `score` over k
      half_idx   [T, H, 2, k] int64  per-half top-k, rank order
      half_score [T, H, 2, k] fp64
    """
    q = _f64(q)
    K = _f64(subkeys)
    T, H, n = q.shape
    assert n % 2 == 0, "query dim must be even"
    d = n // 2
    assert K.shape[0] == H and K.shape[1] == 2 and K.shape[3] == d
    S = K.shape[2]
    assert 1 <= k <= S
    assert np.all(np.isfinite(q)) and np.all(np.isfinite(K))

    idx = np.zeros((T, H, k), dtype=np.int64)
    score = np.zeros((T, H, k))
    w = np.zeros((T, H, k))
    half_idx = np.zeros((T, H, 2, k), dtype=np.int64)
    half_score = np.zeros((T, H, 2, k))
    for t in range(T):
        for h in range(H):
            # Split the query into its two halves.
            q1 = q[t, h, :d]
            q2 = q[t, h, d:]
            # Score each half against its own sqrt(N) sub-keys.
            s1 = half_scores(q1, K[h, 0])
            s2 = half_scores(q2, K[h, 1])
            # Top-k of each half.
            I1 = topk_desc(s1, k)
            I2 = topk_desc(s2, k)
            half_idx[t, h, 0] = I1
            half_idx[t, h, 1] = I2
            half_score[t, h, 0] = s1[I1]
            half_score[t, h, 1] = s2[I2]
            # All k*k combinations: summed score and composed index.
            cand_score = (s1[I1][:, None] + s2[I2][None, :]).ravel()
            cand_idx = (I1[:, None] * S + I2[None, :]).ravel()
            # Best k by (score desc, composed index asc).
            order = rank_order(cand_score, cand_idx)[:k]
            idx[t, h] = cand_idx[order]
            score[t, h] = cand_score[order]
            # Softmax over the k selected scores.
            w[t, h] = softmax(score[t, h])
    return dict(idx=idx, score=score, w=w, half_idx=half_idx, half_score=half_score)


def brute_force_search(q: np.ndarray, subkeys: np.ndarray, k: int) -> dict:
    """Eq. (1) taken literally: instantiate all N = S^2 full keys.

    Full key row i = concat(K1[i // S], K2[i % S]).  Only for tiny inputs;
    this is the definition that the product-key search must reproduce.
    Returns idx [T, H, k] and score [T, H, k].
    """
    q = _f64(q)
    K = _f64(subkeys)
    T, H, n = q.shape
    d = n // 2
    S = K.shape[2]
    N = S * S
    idx = np.zeros((T, H, k), dtype=np.int64)
    score = np.zeros((T, H, k))
    for h in range(H):
        full = np.zeros((N, n))
        for i in range(N):
            full[i, :d] = K[h, 0, i // S]
            full[i, d:] = K[h, 1, i % S]
        for t in range(T):
            f = full @ q[t, h]
            sel = topk_desc(f, k)
            idx[t, h] = sel
            score[t, h] = f[sel]
    return dict(idx=idx, score=score)


def bag_forward(values: np.ndarray, idx: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Weighted EmbeddingBag, sum mode (Eq. (1) y = s V_I; Sec. 3.1.4).

    values: [N, D]; idx, w: [T, B] with B = H * k lookups per token (any
    leading shape that flattens to T rows).  y[t] = sum_j w[t, j] V[idx[t, j]].
    A row chosen by two heads contributes twice.
    """
    V = _f64(values)
    idx = np.asarray(idx).reshape(idx.shape[0], -1)
    w = _f64(w).reshape(idx.shape[0], -1)
    T, B = idx.shape
    y = np.zeros((T, V.shape[1]))
    for t in range(T):
        for j in range(B):
            y[t] += w[t, j] * V[idx[t, j]]
    return y


def bag_backward_rows(dy: np.ndarray, values: np.ndarray, idx: np.ndarray,
                      w: np.ndarray, H: int, k: int) -> dict:
    """Backward of bag_forward and of the softmax in front of it.

    Differentiates y[t] = sum_{h,j} w[t,h,j] V[idx[t,h,j]] with
    w[t,h,:] = softmax(z[t,h,:]) (Sec. 3, Eq. (1); Sec. 3.1.4):
      grad_w[t,h,j]  = dy[t] . V[idx[t,h,j]]
      grad_z[t,h,j]  = w[t,h,j] * (grad_w[t,h,j] - sum_j' w[t,h,j'] grad_w[t,h,j'])
      grad_V[r]     += sum over lookups (t,h,j) with idx = r of w[t,h,j] dy[t]

    Returns grad_w [T,H,k], grad_z [T,H,k] and the value gradient as
    touched rows only: rows (ascending int64) and grad_rows [U, D].
    """
    dy = _f64(dy)
    V = _f64(values)
    T = dy.shape[0]
    idx = np.asarray(idx).reshape(T, H, k)
    w = _f64(w).reshape(T, H, k)
    grad_w = np.zeros((T, H, k))
    grad_z = np.zeros((T, H, k))
    acc: dict[int, np.ndarray] = {}
    for t in range(T):
        for h in range(H):
            for j in range(k):
                r = int(idx[t, h, j])
                grad_w[t, h, j] = dy[t] @ V[r]
                if r not in acc:
                    acc[r] = np.zeros(V.shape[1])
                acc[r] += w[t, h, j] * dy[t]
            # Softmax backward: Jacobian diag(w) - w w^T applied to grad_w.
            inner = w[t, h] @ grad_w[t, h]
            grad_z[t, h] = w[t, h] * (grad_w[t, h] - inner)
    rows = np.array(sorted(acc), dtype=np.int64)
    grad_rows = np.stack([acc[int(r)] for r in rows]) if len(rows) else np.zeros((0, V.shape[1]))
    return dict(grad_w=grad_w, grad_z=grad_z, rows=rows, grad_rows=grad_rows)


def bag_backward(dy: np.ndarray, values: np.ndarray, idx: np.ndarray,
                 w: np.ndarray, H: int, k: int, grad_values_in=None) -> dict:
    """bag_backward_rows with a dense [N, D] value gradient.

    The dense gradient is grad_values_in (default zeros) plus the touched
    rows' sums: accumulate semantics, as for a value pool shared by layers.
    """
    out = bag_backward_rows(dy, values, idx, w, H, k)
    N, D = np.asarray(values).shape
    gV = np.zeros((N, D)) if grad_values_in is None else _f64(grad_values_in).copy()
    for r, g in zip(out["rows"], out["grad_rows"]):
        gV[int(r)] += g
    out["grad_values"] = gV
    return out


def invert_index(idx: np.ndarray) -> dict:
    """Invert the lookup -> row mapping (Sec. 3.1.4, "reverse indices").

    idx: [L] rows of the flattened lookups l = 0..L-1.  Returns
      rows     [U]   distinct rows, ascending
      row_ptr  [U+1] CSR offsets into `lookups`
      lookups  [L]   lookup ids grouped by row, ascending within a row
    """
    idx = np.asarray(idx).ravel().astype(np.int64)
    groups: dict[int, list[int]] = {}
    for l, r in enumerate(idx.tolist()):
        groups.setdefault(r, []).append(l)
    rows = np.array(sorted(groups), dtype=np.int64)
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    lookups = []
    for u, r in enumerate(rows.tolist()):
        lookups.extend(groups[r])
        row_ptr[u + 1] = len(lookups)
    return dict(rows=rows, row_ptr=row_ptr, lookups=np.array(lookups, dtype=np.int64))


def search_backward(q: np.ndarray, subkeys: np.ndarray, idx: np.ndarray,
                    grad_z: np.ndarray, grad_subkeys_in=None) -> dict:
    """Gradient of the selected scores with respect to queries and sub-keys.

    The keys are trainable parameters (Sec. 3); the selection itself is
    piecewise constant and passes no gradient.  With the composed index
    i = i1 * S + i2 of Sec. 3.1.1, the selected score of rank j is
      z[t,h,j] = q[t,h,:d] . K[h,0,i1] + q[t,h,d:] . K[h,1,i2]
    so, given grad_z = dL/dz:
      grad_q[t,h,:d]  = sum_j grad_z[t,h,j] K[h,0,i1_j]
      grad_q[t,h,d:]  = sum_j grad_z[t,h,j] K[h,1,i2_j]
      grad_K[h,0,i]  += sum over (t,j) with i1_j = i of grad_z[t,h,j] q[t,h,:d]
      grad_K[h,1,i]  += sum over (t,j) with i2_j = i of grad_z[t,h,j] q[t,h,d:]
    grad_K accumulates onto grad_subkeys_in (default zeros).
    Returns grad_q [T,H,n] and grad_K [H,2,S,d].
    """
    q = _f64(q)
    K = _f64(subkeys)
    T, H, n = q.shape
    d = n // 2
    S = K.shape[2]
    idx = np.asarray(idx)
    gz = _f64(grad_z)
    k = idx.shape[2]
    grad_q = np.zeros((T, H, n))
    grad_K = np.zeros(K.shape) if grad_subkeys_in is None else _f64(grad_subkeys_in).copy()
    for t in range(T):
        for h in range(H):
            for j in range(k):
                i1, i2 = divmod(int(idx[t, h, j]), S)
                g = gz[t, h, j]
                grad_q[t, h, :d] += g * K[h, 0, i1]
                grad_q[t, h, d:] += g * K[h, 1, i2]
                grad_K[h, 0, i1] += g * q[t, h, :d]
                grad_K[h, 1, i2] += g * q[t, h, d:]
    return dict(grad_q=grad_q, grad_K=grad_K)


def silu(x: np.ndarray) -> np.ndarray:
    """silu(x) = x * sigmoid(x) (Sec. 3.1.4, Memory+), in fp64.  The sigmoid
    is taken as 1 / (1 + exp(-x)) for x >= 0 and exp(x) / (1 + exp(x)) for
    x < 0, so neither branch overflows."""
    x = _f64(x)
    e = np.exp(-np.abs(x))
    sig = np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return x * sig


def gated_output(y: np.ndarray, gate: np.ndarray) -> np.ndarray:
    """Memory+ gating (Sec. 3.1.4): the memory output becomes
    (y * silu(x^T W1))^T W2.  The two projections are plain matrix products
    done by the caller; the part on the memory path is the element-wise
    out = y * silu(gate) with gate = x^T W1, both [T, D]."""
    return _f64(y) * silu(gate)


def gated_backward(d_out: np.ndarray, y: np.ndarray, gate: np.ndarray) -> dict:
    """Backward of out = y * silu(g), element-wise, given d_out = dL/dout:
      dy = d_out * silu(g)
      dg = d_out * y * silu'(g),  silu'(g) = sig(g) * (1 + g * (1 - sig(g)))
    (the derivative of g * sig(g), using sig' = sig * (1 - sig)).  dy then
    feeds the bag backward in place of the plain memory output's gradient."""
    d = _f64(d_out)
    yy = _f64(y)
    g = _f64(gate)
    e = np.exp(-np.abs(g))
    sig = np.where(g >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return dict(dy=d * (g * sig), dg=d * yy * (sig * (1.0 + g * (1.0 - sig))))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest value with an 8-bit significand (bfloat16's), ties to even,
    from the exact fp64 value (no intermediate fp32 rounding).  Finite inputs
    within bfloat16's normal range, or zero."""
    x = _f64(x)
    m, e = np.frexp(x)             # x = m * 2**e, 0.5 <= |m| < 1
    m = np.rint(m * 256.0) / 256.0  # 8 significant bits; rint rounds half to even
    return np.ldexp(m, e)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """The value a kernel stores in `dtype`: "bf16", "fp32", or "fp64" (no rounding)."""
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "fp32":
        return _f64(np.asarray(x, dtype=np.float64).astype(np.float32))
    if dtype == "fp64":
        return _f64(x)
    raise ValueError(dtype)


def query_layernorm(q: np.ndarray, eps: float) -> dict:
    """LayerNorm without affine parameters over the last axis (each (t, h)
    query of n elements): mean, biased variance, rstd = 1 / sqrt(var + eps),
    qhat = (q - mean) * rstd.  rstd is 0 where var + eps == 0."""
    x = _f64(q)
    mean = x.mean(axis=-1)
    xc = x - mean[..., None]
    var = (xc * xc).mean(axis=-1)
    ve = var + float(eps)
    rstd = np.where(ve > 0, 1.0 / np.sqrt(np.where(ve > 0, ve, 1.0)), 0.0)
    return dict(qhat=xc * rstd[..., None], mean=mean, rstd=rstd, var=var)


def search_qnorm(q: np.ndarray, subkeys: np.ndarray, k: int, eps: float,
                 dtype: str = "fp64") -> dict:
    """Product-key search of the normalised queries: qhat from
    query_layernorm, rounded to the storage dtype, then `search`.  The result
    also carries qhat (as scored), mean and rstd."""
    ln = query_layernorm(q, eps)
    qs = round_to(ln["qhat"], dtype)
    out = search(qs, subkeys, k)
    out.update(qhat=qs, mean=ln["mean"], rstd=ln["rstd"])
    return out


def search_backward_qnorm(q: np.ndarray, subkeys: np.ndarray, idx: np.ndarray,
                          grad_z: np.ndarray, eps: float, dtype: str = "fp64",
                          grad_subkeys_in=None) -> dict:
    """Search backward through the query normalisation.  With g = dL/dqhat
    from `search_backward` at the stored qhat (which also gives grad_K, built
    from qhat as scored), the LayerNorm backward over each query is
      grad_q = rstd * (g - mean(g) - xhat * mean(g * xhat)),
    xhat = (q - mean) * rstd unrounded (the storage rounding passes the
    gradient unchanged)."""
    ln = query_layernorm(q, eps)
    qs = round_to(ln["qhat"], dtype)
    r = search_backward(qs, subkeys, idx, grad_z, grad_subkeys_in)
    g = r["grad_q"]
    xh = ln["qhat"]
    gm = g.mean(axis=-1, keepdims=True)
    gxm = (g * xh).mean(axis=-1, keepdims=True)
    grad_q = ln["rstd"][..., None] * (g - gm - xh * gxm)
    return dict(grad_q=grad_q, grad_K=r["grad_K"])


def search_extra(q: np.ndarray, subkeys: np.ndarray, k: int, extra_idx: np.ndarray) -> dict:
    """The search of `search` plus r extra key-value pairs per (token, head).

    extra_idx: [T, H, r] int, each in [0, S*S): composed indices chosen by the
    caller.  Slot j < k is the j-th selected key (rank order), slot k + e the
    e-th extra index, scored s1[i1] + s2[i2] with i1 = i // S, i2 = i % S.
    Returns idx, score, w of shape [T, H, k + r] (softmax over all k + r
    scores of a (token, head)); half_idx / half_score as in `search`.
    """
    q = _f64(q)
    K = _f64(subkeys)
    T, H, n = q.shape
    d = n // 2
    S = K.shape[2]
    ex = np.asarray(extra_idx, dtype=np.int64)
    r = ex.shape[2]
    assert ex.shape[:2] == (T, H)
    assert np.all((ex >= 0) & (ex < S * S))
    base = search(q, K, k)
    idx = np.zeros((T, H, k + r), dtype=np.int64)
    score = np.zeros((T, H, k + r))
    w = np.zeros((T, H, k + r))
    for t in range(T):
        for h in range(H):
            idx[t, h, :k] = base["idx"][t, h]
            score[t, h, :k] = base["score"][t, h]
            for e in range(r):
                i1, i2 = divmod(int(ex[t, h, e]), S)
                idx[t, h, k + e] = ex[t, h, e]
                score[t, h, k + e] = q[t, h, :d] @ K[h, 0, i1] + q[t, h, d:] @ K[h, 1, i2]
            w[t, h] = softmax(score[t, h])
    return dict(idx=idx, score=score, w=w, half_idx=base["half_idx"], half_score=base["half_score"])


def search_sink(q: np.ndarray, subkeys: np.ndarray, k: int, extra_idx: np.ndarray,
                sink_keys: np.ndarray, sink_row0: int) -> dict:
    """`search_extra` plus one fixed key-value pair per head in the last slot:
    score q[t,h] . sink_keys[h] (over all n elements), index sink_row0 + h
    (the value-table row holding head h's sink value).  Softmax over all
    k + r + 1 slots.  Returns idx, score, w of shape [T, H, k + r + 1]."""
    q = _f64(q)
    ks = _f64(sink_keys)
    T, H, n = q.shape
    assert ks.shape == (H, n)
    base = search_extra(q, subkeys, k, extra_idx)
    kk = base["idx"].shape[2] + 1
    idx = np.zeros((T, H, kk), dtype=np.int64)
    score = np.zeros((T, H, kk))
    w = np.zeros((T, H, kk))
    for t in range(T):
        for h in range(H):
            idx[t, h, :-1] = base["idx"][t, h]
            score[t, h, :-1] = base["score"][t, h]
            idx[t, h, -1] = sink_row0 + h
            score[t, h, -1] = q[t, h] @ ks[h]
            w[t, h] = softmax(score[t, h])
    return dict(idx=idx, score=score, w=w, half_idx=base["half_idx"], half_score=base["half_score"])


def search_backward_sink(q: np.ndarray, subkeys: np.ndarray, idx: np.ndarray, grad_z: np.ndarray,
                         sink_keys: np.ndarray, grad_subkeys_in=None, grad_sink_in=None) -> dict:
    """Gradients of the scores of `search_sink` (selection fixed): the first
    k + r slots as `search_backward`, the last slot z = q . sink_keys[h]:
      grad_q[t,h]      += grad_z[t,h,-1] * sink_keys[h]
      grad_sink[h]     += sum_t grad_z[t,h,-1] * q[t,h]   (accumulated)."""
    q = _f64(q)
    ks = _f64(sink_keys)
    gz = _f64(grad_z)
    r = search_backward(q, subkeys, np.asarray(idx)[..., :-1], gz[..., :-1], grad_subkeys_in)
    grad_q = r["grad_q"] + gz[..., -1:] * ks[None, :, :]
    grad_sink = np.zeros(ks.shape) if grad_sink_in is None else _f64(grad_sink_in).copy()
    T, H, _ = q.shape
    for h in range(H):
        for t in range(T):
            grad_sink[h] += gz[t, h, -1] * q[t, h]
    return dict(grad_q=grad_q, grad_K=r["grad_K"], grad_sink=grad_sink)
