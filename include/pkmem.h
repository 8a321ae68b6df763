/*
 * pkmem.h - C ABI of the product-key memory hot path on MI355X (gfx950).
 *
 * Paper: "Memory Layers at Scale" (arXiv 2412.09764).
 *   Sec. 3, Eq. (1):  I = SelectTopkIndices(K q), s = Softmax(K_I q), y = s V_I,
 *                     every token independently.
 *   Sec. 3.1.1:       product keys: K1, K2 of sqrt(N) rows of n/2; split q into
 *                     q1, q2; top-k per half; best k of the k*k sums.
 *   Sec. 3.1.4:       the weighted sum is an EmbeddingBag; its backward adds many
 *                     output gradients into the same value-gradient row, either
 *                     with atomics or after inverting the lookup -> row mapping.
 *
 * Conventions for every entry point
 *   - Pointers are DEVICE pointers unless marked "host".  All device buffers are
 *     allocated and owned by the caller; the library allocates no device memory
 *     and keeps no device state between calls (two exceptions: the 4-byte flag
 *     of the PKMEM_DEBUG index check, off by default, see Environment below,
 *     and the static scratch array of mem_search_noalloc).
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = null stream) and
 *     return once the work is enqueued.  mem_bag_backward_sparse is the only call
 *     that waits on the stream (it must report a row count to the host).
 *   - Inputs are read-only.  Outputs are written, except grad_values, which is
 *     accumulated (+=): one value pool may be shared by several memory layers.
 *   - Layouts are dense row-major with the last dimension contiguous.
 *   - A non-zero return means nothing was enqueued (argument errors are found on
 *     the host before any launch) or a HIP error (PKMEM_ERR_HIP).  No call aborts
 *     or throws; mem_last_error() gives a message for the calling thread.
 *   - Inputs must be finite.  Indices passed to the bag calls must lie in [0, N)
 *     and are not range-checked (they normally come from mem_search).
 *
 * Readings where the paper is silent:
 *   - H heads: per token, H independent queries and sub-key pairs; each head
 *     selects its own k values from ONE shared value table; the output sums the
 *     H*k weighted rows (one bag).  A row chosen by two heads counts twice.
 *   - q[t,h,0:d] (d = n/2) is scored against subkeys[h,0], q[t,h,d:n] against
 *     subkeys[h,1]; the composed value index is i = i1 * S + i2.
 *   - Order: score descending, index ascending (lower index wins ties), for the
 *     per-half lists and for the final selection.  Outputs are in rank order.
 *   - Scores are raw dot products (no scale or temperature); the softmax runs
 *     over the k selected scores of one (token, head).
 *   - Arithmetic: fp32 accumulation everywhere; bf16 outputs are rounded to
 *     nearest even from the fp32 value.
 */
#ifndef PKMEM_H
#define PKMEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { PKMEM_F32 = 0, PKMEM_BF16 = 1 } pkmem_dtype;

typedef enum {
  PKMEM_OK = 0,
  PKMEM_ERR_INVALID = -1,     /* null pointer, bad size, inconsistent shapes */
  PKMEM_ERR_UNSUPPORTED = -2, /* valid request outside the supported limits  */
  PKMEM_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required  */
  PKMEM_ERR_HIP = -4          /* a HIP call or kernel launch failed          */
} pkmem_status;

/* Value-gradient strategies of the EmbeddingBag backward (Sec. 3.1.4). */
typedef enum {
  PKMEM_BWD_AUTO = 0,   /* library's choice: atomic when T*H*k*D <= 2^26 and
                           D <= 1024 (small batches), sorted otherwise
                           (measured crossover on MI355X)                      */
  PKMEM_BWD_ATOMIC = 1, /* fp32 atomic adds straight into grad_values          */
  PKMEM_BWD_SORTED = 2  /* lookups sorted by row, one read-modify-write per
                           touched row, contributors summed in lookup order:
                           bitwise deterministic run to run                    */
} pkmem_bwd_mode;

typedef void* pkmem_stream_t; /* a hipStream_t */

/* Limits (checked on the host; exceeding them gives PKMEM_ERR_UNSUPPORTED). */
#define PKMEM_KMAX 64       /* k per half and overall                       */
#define PKMEM_SMAX 8192     /* sub-keys per half, so N = S*S <= 2^26        */
#define PKMEM_DHALF_MAX 256 /* d = n/2 for bf16 queries; 64 for fp32        */

/* ------------------------------------------------------------------------ *
 * Product-key search (Sec. 3.1.1) and softmax (Sec. 3, Eq. (1)).
 *
 *   q        [T, H, n]      queries, dtype q_dt (PKMEM_F32 or PKMEM_BF16); n even.
 *   subkeys  [H, 2, S, n/2] sub-key tables, same dtype as q.
 *   k        1 <= k <= min(S, PKMEM_KMAX).
 * Outputs (written):
 *   idx_out      [T, H, k] int64  composed index i1*S + i2 of the selected values.
 *   w_out        [T, H, k] fp32   softmax of the selected scores (the bag weights).
 *   score_out    [T, H, k] fp32   selected scores s1[i1] + s2[i2]; may be NULL.
 *   half_idx_out [T, H, 2, k] int32 per-half top-k (half 0 then half 1); may be NULL.
 * Workspace: ws of at least mem_search_workspace_size(T, H, S, k) bytes, 256-byte
 *   aligned, used only during the call (contents on entry are ignored).
 * T = 0 is a valid no-op.
 * ------------------------------------------------------------------------ */
size_t mem_search_workspace_size(int64_t T, int H, int S, int k);

int mem_search(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
               int64_t T, int H, int n, int S, int k,
               int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
               void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * mem_search without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops (search
 * then mem_bag_forward, which needs no workspace), harnesses that forbid
 * allocation.  It runs mem_search's kernels with its workspace carved from a
 * static device array of PKMEM_NOALLOC_SCRATCH_BYTES that the library holds
 * on each GPU it runs on until the process ends; the call itself allocates
 * nothing (no hipMalloc, no allocating library routine).
 *   Arguments and outputs as for mem_search.
 *   Size limit: mem_search_workspace_size(T, H, S, k) <= PKMEM_NOALLOC_SCRATCH_BYTES
 *   (128 MiB: about 28,000 (token, head) rows at k = 32, e.g. T = 7,000 at
 *   H = 4); larger requests return PKMEM_ERR_UNSUPPORTED before touching the
 *   device (use mem_search with a workspace).
 *   Sharing: every call on one GPU uses that GPU's one array, which keeps the
 *   last call's contents (nothing read is assumed to start at zero; the call
 *   clears what it needs with a fill kernel).  Calls that overlap on one GPU
 *   (different streams, or different host threads, without ordering between
 *   them) race on the array and give undefined results: serialise them.
 *   Set-up: the first call on a device looks up that device's address of the
 *   array once (hipGetSymbolAddress) with the device current; a failure there
 *   returns PKMEM_ERR_HIP.
 * ------------------------------------------------------------------------ */
#define PKMEM_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

int mem_search_noalloc(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                       int64_t T, int H, int n, int S, int k,
                       int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
                       pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search with extra key-value pairs beside the top-k (Sec. 5.4, model
 * ablations: random key-value pairs added during pre-training).  For every
 * (t, h) the caller supplies r composed indices (drawn as it likes, e.g.
 * uniformly from [0, S*S)); each is scored like any full key,
 *   z = q[t,h,0:d] . subkeys[h,0,i/S] + q[t,h,d:n] . subkeys[h,1,i%S],
 * and occupies its own slot after the k selected ones (an index that is also
 * selected appears twice); the softmax runs over all k + r scores.
 *   r            0 <= r and k + r <= PKMEM_KMAX.
 *   extra_idx    [T, H, r] int64 in [0, S*S) (not range-checked unless
 *                PKMEM_DEBUG is set; an index outside is scored as index 0
 *                and written out unchanged).
 *   idx_out, w_out, score_out   [T, H, k + r]: slots 0..k-1 as mem_search's,
 *                slots k..k+r-1 the extra pairs in the given order; w sums to
 *                one over all k + r.  half_idx_out [T, H, 2, k] as mem_search's.
 * The value bag and both backwards take these outputs as they are, with
 * k + r in place of k.  Workspace: mem_search_workspace_size(T, H, S, k).
 * ------------------------------------------------------------------------ */
int mem_search_extra(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                     int64_t T, int H, int n, int S, int k, int r, const int64_t* extra_idx,
                     int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
                     void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search with a fixed ("sink") key-value pair (Sec. 5.4, model ablations: one
 * fixed key-value pair added beside the selected ones).  mem_search_extra
 * plus one more slot per (t, h): the key sink_keys[h, 0:n] is scored like any
 * full key, z = q[t,h,:] . sink_keys[h,:] (a zero key gives the constant
 * logit 0, one added to the softmax's denominator), and the slot's index is
 * sink_row0 + h, a row of the value table that holds head h's sink value
 * (the caller appends H such rows after the S*S key rows).
 *   sink_keys    [H, n] dtype k_dt, 16-byte aligned (trainable or fixed).
 *   sink_row0    >= S*S: the value-table row of head 0's sink value.
 *   r, extra_idx as for mem_search_extra (r = 0: none); k + r + 1 <= PKMEM_KMAX.
 *   idx_out, w_out, score_out   [T, H, k + r + 1]: slots 0..k+r-1 as
 *                mem_search_extra's, slot k + r the sink's; the softmax runs
 *                over all k + r + 1.  half_idx_out [T, H, 2, k] as mem_search's.
 * The value bag and its backward take these outputs as they are, with
 * k + r + 1 in place of k (the sink value's gradient lands in its row);
 * the search backward is mem_search_backward_sink.
 * Workspace: mem_search_workspace_size(T, H, S, k).
 * ------------------------------------------------------------------------ */
int mem_search_sink(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                    int64_t T, int H, int n, int S, int k, int r, const int64_t* extra_idx,
                    const void* sink_keys, int64_t sink_row0,
                    int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
                    void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search backward: gradient of the selected scores with respect to the
 * queries and the sub-keys (the keys are trainable parameters, Sec. 3; the
 * selection is piecewise constant and passes no gradient).  With
 * i1 = idx / S, i2 = idx % S the score of rank j is
 *   z[t,h,j] = q[t,h,0:d] . subkeys[h,0,i1] + q[t,h,d:n] . subkeys[h,1,i2].
 *
 *   q, subkeys, T, H, n, S  as for mem_search (same dtype rules and limits).
 *   k            slots per row, 1 <= k <= PKMEM_KMAX (k + r after mem_search_extra,
 *                which may exceed S).
 *   idx          [T, H, k] int64  mem_search's selection; lookups whose index lies
 *                outside [0, S*S) contribute nothing (mem_search never writes one).
 *   grad_scores  [T, H, k] fp32   dL/dz (mem_bag_backward's grad_scores).
 * Outputs (each may be NULL to skip it):
 *   grad_q        [T, H, n] fp32, written:
 *                 grad_q[t,h,0:d] = sum_j gz[t,h,j] subkeys[h,0,i1_j], likewise half 1.
 *   grad_subkeys  [H, 2, S, n/2] fp32, ACCUMULATED (+=):
 *                 += sum over (t,j) with i1_j = i of gz[t,h,j] q[t,h,0:d], likewise half 1.
 *                 Bitwise deterministic: the (lookup, half) pairs are sorted by sub-key
 *                 and each sub-key row is summed by one wave in token order, no atomics.
 *                 Requires 2*T*H*k < 2^32.
 * Workspace: mem_search_backward_workspace_size(T, H, S, k) bytes, 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t mem_search_backward_workspace_size(int64_t T, int H, int S, int k);

int mem_search_backward(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                        int64_t T, int H, int n, int S, int k, const int64_t* idx,
                        const float* grad_scores, float* grad_q, float* grad_subkeys,
                        void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search backward of mem_search_sink (same q, sub-keys, sink keys and
 * selection).  k is the number of product-key slots per row (k + r of the
 * forward); idx and grad_scores are [T, H, k + 1], slot k the sink's (its
 * index is not read).  Slots 0..k-1 as mem_search_backward; the sink's score
 * z = q . sink_keys[h] adds
 *   grad_q[t,h,:]    += grad_scores[t,h,k] * sink_keys[h,:]   (grad_q written),
 *   grad_sink[h,:]   += sum_t grad_scores[t,h,k] * q[t,h,:]   (ACCUMULATED),
 * grad_sink [H, n] fp32, bitwise deterministic (per-chunk partial sums added
 * in chunk order, no atomics); any of the three outputs may be NULL.
 * Limits and errors as for mem_search_backward, with k + 1 <= PKMEM_KMAX.
 * Workspace: mem_search_backward_sink_workspace_size(T, H, n, S, k) bytes,
 * 256-byte aligned.
 * ------------------------------------------------------------------------ */
size_t mem_search_backward_sink_workspace_size(int64_t T, int H, int n, int S, int k);

int mem_search_backward_sink(const void* q, pkmem_dtype q_dt, const void* subkeys,
                             pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k,
                             const int64_t* idx, const float* grad_scores, const void* sink_keys,
                             float* grad_q, float* grad_subkeys, float* grad_sink,
                             void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search with query normalisation (qk-normalisation, Sec. 3.1.4: used for
 * large memories whose training is unstable), fused in front of the scoring.
 * Each query row q[t,h,:] is replaced by LayerNorm without affine parameters,
 *   qhat = (q - mean) * rstd,  rstd = 1 / sqrt(var + eps),
 * mean and biased variance over the n elements in fp32 (rstd = 0 where
 * var + eps == 0), qhat rounded to q_dt (nearest, ties to even) and then
 * searched exactly as mem_search does.  The normalised queries are formed in
 * registers by the scoring kernel; nothing of size [T, H, n] is written unless
 * asked for.
 *   eps          >= 0 and finite (LayerNorm's customary value is 1e-5).
 *   qhat_out     [T, H, n] dtype q_dt, 16-byte aligned: the normalised queries
 *                as scored; may be NULL.
 *   stats_out    [T, H, 2] fp32: (mean, rstd) per query; may be NULL.
 *   Everything else as for mem_search (same workspace size function).
 * ------------------------------------------------------------------------ */
int mem_search_qnorm(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                     int64_t T, int H, int n, int S, int k, float eps,
                     int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
                     void* qhat_out, float* stats_out,
                     void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Search backward through the query normalisation of mem_search_qnorm (same
 * q, eps and selection).  The statistics are recomputed from q, bitwise as
 * the forward computed them.  With g = dL/dqhat (mem_search_backward's
 * grad_q formula at qhat):
 *   grad_q        [T, H, n] fp32, written: rstd * (g - mean(g) - xhat * mean(g * xhat)),
 *                 xhat = (q - mean) * rstd in fp32 (the rounding of qhat to q_dt
 *                 passes the gradient unchanged);
 *   grad_subkeys  [H, 2, S, n/2] fp32, ACCUMULATED: mem_search_backward's sum with
 *                 qhat (as scored) in place of q; bitwise deterministic.
 * Limits, workspace (mem_search_backward_workspace_size) and errors as for
 * mem_search_backward; eps as for mem_search_qnorm.
 * ------------------------------------------------------------------------ */
int mem_search_backward_qnorm(const void* q, pkmem_dtype q_dt, const void* subkeys,
                              pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k, float eps,
                              const int64_t* idx, const float* grad_scores, float* grad_q,
                              float* grad_subkeys, void* ws, size_t ws_bytes,
                              pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Weighted EmbeddingBag forward, sum mode (Sec. 3, Eq. (1) y = s V_I; Sec. 3.1.4).
 *
 *   values [N, D]   value table, dtype v_dt; D % 8 == 0.
 *   idx    [T, bag] int64 rows in [0, N); w [T, bag] fp32 weights.
 *   y_out  [T, D]   dtype v_dt, written: y[t] = sum_j w[t,j] * values[idx[t,j]],
 *                   accumulated in fp32 and rounded once to v_dt.
 * For the memory layer bag = H*k and idx / w are mem_search's outputs.
 * ------------------------------------------------------------------------ */
int mem_bag_forward(const void* values, pkmem_dtype v_dt, int64_t N, int D,
                    const int64_t* idx, const float* w, int64_t T, int bag,
                    void* y_out, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Memory+ gating (Sec. 3.1.4): the layer's output becomes
 * (y * silu(x^T W1))^T W2 with silu(x) = x * sigmoid(x).  The projections
 * x^T W1 and .^T W2 are plain matrix products done by the caller; the
 * element-wise gate is fused into the bag:
 *
 *   values, N, D, idx, w, T, bag   as for mem_bag_forward.
 *   gate   [T, D] dtype v_dt   the gate pre-activation x^T W1.
 *   out    [T, D] dtype v_dt   written: bag(t) * silu(gate[t]) elementwise,
 *                              from the fp32 accumulator, rounded once.
 *   y_out  [T, D] dtype v_dt   written when non-NULL: the un-gated bag (what
 *                              mem_gate_backward needs), rounded once.
 * All buffers 16-byte aligned.
 * ------------------------------------------------------------------------ */
int mem_bag_forward_gated(const void* values, pkmem_dtype v_dt, int64_t N, int D,
                          const int64_t* idx, const float* w, int64_t T, int bag,
                          const void* gate, void* y_out, void* out, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Backward of out = y * silu(g), element-wise over [T, D]:
 *   d_out, gate, y   [T, D] dtype v_dt: dL/dout, the gate, the un-gated bag.
 *   dy_out     [T, D] dtype v_dt, written: d_out * silu(g), rounded once; pass
 *              it to mem_bag_backward as its dy.
 *   grad_gate  [T, D] fp32, written: d_out * y * silu'(g),
 *              silu'(g) = sigmoid(g) * (1 + g * (1 - sigmoid(g))).
 * D % 8 == 0; all buffers 16-byte aligned.  (Not fused into the sorted value
 * backward, which reads dy once per lookup: computing it there would read
 * d_out and the gate once per lookup instead.)
 * ------------------------------------------------------------------------ */
int mem_gate_backward(const void* d_out, const void* gate, const void* y, pkmem_dtype v_dt,
                      int64_t T, int D, void* dy_out, float* grad_gate, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * EmbeddingBag backward and softmax backward (Sec. 3.1.4; Eq. (1)).
 *
 *   dy     [T, D]      upstream gradient of y, dtype v_dt.
 *   values [N, D]      dtype v_dt.   idx, w [T, H, k] as from mem_search.
 * Outputs (all optional; NULL skips the output, not the work it depends on):
 *   grad_values [N, D] fp32, ACCUMULATED: += sum over lookups with idx = r of
 *                      w * dy[t].
 *   grad_w      [T, H, k] fp32, written: dy[t] . values[idx[t,h,j]].
 *   grad_scores [T, H, k] fp32, written: w * (grad_w - sum_j w_j grad_w_j), the
 *                      gradient with respect to the selected scores.
 * mode: pkmem_bwd_mode.  Workspace: mem_bag_backward_workspace_size(...) bytes.
 * ------------------------------------------------------------------------ */
size_t mem_bag_backward_workspace_size(int64_t T, int H, int k, int64_t N, int D, int mode);

int mem_bag_backward(const void* dy, const void* values, pkmem_dtype v_dt, int64_t N, int D,
                     const int64_t* idx, const float* w, int64_t T, int H, int k,
                     float* grad_values, float* grad_w, float* grad_scores,
                     int mode, void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* Sparse form of the value gradient, for tables too large for a dense fp32
 * gradient: the touched rows only.  Same arguments and other outputs as
 * mem_bag_backward (always the sorted strategy), except
 *   rows_out      [cap] int64  touched rows, ascending (cap >= T*H*k is enough).
 *   grad_rows_out [cap, D] fp32, written: row u is the gradient of rows_out[u].
 *   num_rows_out  host int64*: number of touched rows U.  Written after the call
 *                 waits for `stream`.  Entries at and beyond U are not written.
 * Workspace: mem_bag_backward_workspace_size(T, H, k, N, D, PKMEM_BWD_SORTED). */
int mem_bag_backward_sparse(const void* dy, const void* values, pkmem_dtype v_dt, int64_t N,
                            int D, const int64_t* idx, const float* w, int64_t T, int H, int k,
                            int64_t* rows_out, float* grad_rows_out, int64_t cap,
                            int64_t* num_rows_out, float* grad_w, float* grad_scores,
                            void* ws, size_t ws_bytes, pkmem_stream_t stream);

/* ------------------------------------------------------------------------ *
 * Benchmark instrumentation (host-side state; not thread-safe).
 * mem_timer_start(kernels) takes a comma-separated list of kernel names and
 * makes the library record a HIP event pair on the launch stream around every
 * following launch of a listed kernel:
 *   "score_topk", "topk_sort", "cartesian" (mem_search, mem_search_qnorm,
 *                                           mem_search_extra, mem_search_sink)
 *   "qnorm"                                (mem_search_qnorm, mem_search_backward_qnorm)
 *   "search_backward"                      (mem_search_backward[_qnorm|_sink])
 *   "bag_forward"                          (mem_bag_forward, mem_bag_forward_gated)
 *   "gate_backward"                        (mem_gate_backward)
 *   "bag_backward_atomic", "sort_by_row",
 *   "bag_backward_rows", "softmax_backward" (mem_bag_backward[_sparse])
 * ("sort_by_row" spans the whole radix sort and segment pass.)
 * mem_timer_stop() stops recording.  mem_timer_read(ms_out, kernel_out, cap)
 * waits for the recorded events, writes up to cap entries in launch order to
 * the host arrays ms_out (duration in milliseconds) and kernel_out (position
 * of the kernel in the list; either array may be NULL), frees the events, and
 * returns how many launches were recorded (or a negative status).  With no
 * timer running the library creates no events.
 * ------------------------------------------------------------------------ */
int mem_timer_start(const char* kernels);
int mem_timer_stop(void);
int mem_timer_read(float* ms_out, int* kernel_out, int cap);

/* ------------------------------------------------------------------------ *
 * Environment (read at every call):
 *   PKMEM_DEBUG=1       before a kernel indexes with idx (mem_bag_forward[_gated],
 *                       mem_bag_backward[_sparse], mem_search_backward[_qnorm|_sink]
 *                       (product-key slots), mem_search_extra's and
 *                       mem_search_sink's extra_idx) a device
 *                       check that every index lies in [0, N) (or [0, S*S)); the
 *                       call waits for it and returns PKMEM_ERR_INVALID if not.
 *                       Off by default: indices from mem_search are in range by
 *                       construction.  The check's flag is the only device
 *                       memory the library allocates (4 bytes per device).
 *   PKMEM_BWD_MODE=atomic|sorted
 *                       what PKMEM_BWD_AUTO means, for mem_bag_backward and its
 *                       workspace size.
 * ------------------------------------------------------------------------ */

/* Message for the last non-OK status returned to the calling thread. */
const char* mem_last_error(void);

/* Library version, for the binding's sanity check. */
int mem_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PKMEM_H */
