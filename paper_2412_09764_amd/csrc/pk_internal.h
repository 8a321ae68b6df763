// Host-side launchers shared between the kernel files and the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pk {

// Scope guard for benchmark instrumentation: while a timer runs for `name`
// (mem_timer_start), records a HIP event pair around the launches made in its
// scope, on the launch stream.  Costs one string compare otherwise.
class LaunchTimer {
 public:
  LaunchTimer(const char* name, hipStream_t st);
  ~LaunchTimer();
  LaunchTimer(const LaunchTimer&) = delete;
  LaunchTimer& operator=(const LaunchTimer&) = delete;

 private:
  hipStream_t st_;
  hipEvent_t stop_ = nullptr;
};

// Candidate slots kept per (token, head, half) between the filter passes and
// the per-row sort of the search; the 32 rows of a scoring wave share one run
// of 32 * CAND_CAP records.
constexpr int CAND_CAP = 256;
// Waves and tokens per workgroup of the scoring kernel (32 tokens per wave).
#ifndef PK_SEARCH_WAVES
#define PK_SEARCH_WAVES 16
#endif
constexpr int SEARCH_WAVES = PK_SEARCH_WAVES;
constexpr int SEARCH_TOK = 32 * SEARCH_WAVES;

// Number of (i1, i2) rank pairs with (i1 + 1) * (i2 + 1) <= k: only these can
// reach the top k of the k*k sums when both half lists are sorted.
int cartesian_pairs(int k);

// ---- search (search.hip) -------------------------------------------------
// rows = T*H*2 (token, head, half) rows; cand = one run of 32 * CAND_CAP u64
// records per group of 32 tokens, head and half (ceil(T / 32) * H * 2 runs);
// cnts = [rows, 2] u32 (records per run, in its first entries); thr = [rows]
// fp32 (each row's
// final threshold: no score below it can be selected);
// ovf = [1 + rows] u32 (count, then overflowed row ids).
// qstats (nullable) = per (token, head) query (mean, rstd): the scoring then
// normalises the queries as it loads them (see launch_qnorm).
// With sink (a [H, n] key per head, the sub-keys' dtype), sink_part [T*H, 2]
// receives each half's part of q . sink[h].
hipError_t launch_search_half(bool bf16, const void* q, const void* subkeys, int64_t T, int H,
                              int n, int S, int k, const float2* qstats, const void* sink,
                              float* sink_part, uint64_t* cand, uint32_t* cnts, float* thr,
                              int32_t* half_idx, float* half_score, uint32_t* ovf,
                              hipStream_t st);
// LayerNorm statistics of rows = T*H queries of n elements into stats, and
// (qhat non-null) the normalised queries in the query dtype.
hipError_t launch_qnorm(bool bf16, const void* q, int64_t rows, int n, float eps, float2* stats,
                        void* qhat, hipStream_t st);
// nex extra key-value pairs per (token, head) (ex_idx [T,H,nex], scored from q
// and the sub-keys) join the softmax after the k selected; outputs then have
// k + nex slots per row.  nex = 0: q, subkeys and ex_idx are not read.
hipError_t launch_cartesian(const int32_t* half_idx, const float* half_score, int64_t T, int H,
                            int S, int k, bool bf16, const void* q, const void* subkeys, int n,
                            const int64_t* ex_idx, int nex, const float* sink_part,
                            int64_t sink_row0, int64_t* idx_out, float* w_out, float* score_out,
                            hipStream_t st);

// ---- search backward (search_bwd.hip) --------------------------------------
size_t search_backward_ws_bytes(int64_t T, int H, int k);
void sort_u32_inputs(void* ws, int64_t Lmax, uint32_t** keys_in, uint32_t** vals_in);
hipError_t sort_u32_segments(int64_t Lmax, const uint32_t* Ldev, int key_bits, void* ws,
                             const uint32_t** ks, const uint32_t** vs, const uint32_t** seg,
                             const uint32_t** nseg, hipStream_t st);
size_t scan_scratch_u32(int64_t n);
hipError_t scan_exclusive_u32(uint32_t* data, int64_t n, uint32_t* sums, hipStream_t st);
// qstats (nullable): the queries were normalised in the forward (their
// (mean, rstd) from launch_qnorm); grad_q is then taken through the
// normalisation and grad_K uses the normalised queries as scored.
// k product-key slots per row, rows kst apart in idx and gz; with a sink
// (kst = k + 1) slot k is the sink's.  grad_sink needs sink_part of
// sink_chunks(T) * H * n floats.
int64_t sink_chunks(int64_t T);
// Appends to long_list (in no particular order) every segment u < *nseg with
// seg_start[u+1] - seg_start[u] > thresh, counting them in *long_cnt, which
// must be zero on entry.  max_seg bounds *nseg (sizes the grid).
hipError_t launch_list_long(const uint32_t* seg_start, const uint32_t* nseg, int64_t max_seg,
                            uint32_t thresh, uint32_t* long_list, uint32_t* long_cnt,
                            hipStream_t st);
hipError_t launch_search_backward(bool bf16, const void* q, const void* subkeys, int64_t T, int H,
                                  int n, int S, int k, int kst, const int64_t* idx, const float* gz,
                                  const float2* qstats, const void* sink, float* grad_q,
                                  float* grad_K, float* grad_sink, float* sink_part, void* ws,
                                  hipStream_t st);

// ---- bag (bag.hip) ---------------------------------------------------------
hipError_t launch_bag_forward(bool bf16, const void* values, int D, const int64_t* idx,
                              const float* w, int64_t T, int bag, void* y, const void* gate,
                              void* y_plain, hipStream_t st);
hipError_t launch_check_indices(const int64_t* idx, int64_t count, int64_t limit, uint32_t* bad,
                                hipStream_t st);
// The first cols of every row of a [rows, stride] array.
hipError_t launch_check_indices_strided(const int64_t* idx, int64_t rows, int cols, int stride,
                                        int64_t limit, uint32_t* bad, hipStream_t st);
hipError_t launch_gate_backward(bool bf16, const void* d_out, const void* gate, const void* y,
                                int64_t T, int D, void* dy, float* grad_gate, hipStream_t st);
hipError_t launch_bag_backward_atomic(bool bf16, const void* dy, const void* values, int D,
                                      const int64_t* idx, const float* w, int64_t T, int bag,
                                      float* grad_values, float* grad_w, hipStream_t st);
hipError_t launch_softmax_backward(const float* w, const float* grad_w, int64_t rows, int k,
                                   float* grad_scores, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t count, hipStream_t st);

// ---- sorted backward (sorted.hip) ------------------------------------------
size_t sorted_workspace_bytes(int64_t L);
// Partial rows of the chunks of rows with many lookups (see sorted.hip).
size_t long_partial_bytes(int64_t L, int D);
// Sorts the L lookups by row (stable), finds the touched rows, and per row
// computes grad_w of its lookups and the row's gradient sum.  Dense mode adds
// the sum into grad_values[row]; sparse mode writes rows_out / grad_rows_out.
hipError_t launch_bag_backward_sorted(bool bf16, const void* dy, const void* values, int64_t N,
                                      int D, const int64_t* idx, const float* w, int64_t T,
                                      int bag, float* grad_values, int64_t* rows_out,
                                      float* grad_rows_out, float* grad_w, void* ws, float* part,
                                      uint32_t** num_rows_dev, hipStream_t st);

}  // namespace pk
