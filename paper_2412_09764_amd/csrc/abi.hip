// C ABI of the product-key memory hot path: argument checks on the host,
// workspace carving, dispatch to the kernels.  Declared in include/pkmem.h.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "pkmem.h"
#include "pk_internal.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int hip_status(hipError_t e, const char* where) {
  if (e == hipSuccess) return PKMEM_OK;
  return fail(PKMEM_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }
inline size_t esize(pkmem_dtype t) { return t == PKMEM_BF16 ? 2 : 4; }
inline bool dtype_ok(int t) { return t == PKMEM_F32 || t == PKMEM_BF16; }

struct SearchWs {
  uint64_t* cand;
  uint32_t* cnts;
  float* thr;
  int32_t* half_idx;
  float* half_score;
  uint32_t* ovf;
  float2* qstats;  // per (token, head) query (mean, rstd) when normalising
  float* sink_part;  // per (token, head) the two halves' parts of the sink's score
  size_t bytes;
};

// The search workspace carved from base (only its size when base is null).
SearchWs search_ws(void* base, int64_t T, int H, int k) {
  const size_t rows = (size_t)T * H * 2;
  char* p = reinterpret_cast<char*>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* at = p ? p + off : nullptr;
    off += align256(bytes);
    return at;
  };
  // candidate runs come in groups of 32 tokens (one per scoring wave)
  const size_t grows = (size_t)((T + 31) / 32) * 32 * H * 2;
  SearchWs w;
  w.cand = reinterpret_cast<uint64_t*>(take(grows * pk::CAND_CAP * sizeof(uint64_t)));
  w.cnts = reinterpret_cast<uint32_t*>(take(rows * 2 * sizeof(uint32_t)));
  w.thr = reinterpret_cast<float*>(take(rows * sizeof(float)));
  w.half_idx = reinterpret_cast<int32_t*>(take(rows * k * sizeof(int32_t)));
  w.half_score = reinterpret_cast<float*>(take(rows * k * sizeof(float)));
  w.ovf = reinterpret_cast<uint32_t*>(take((rows + 1) * sizeof(uint32_t)));
  w.qstats = reinterpret_cast<float2*>(take((size_t)T * H * sizeof(float2)));
  w.sink_part = reinterpret_cast<float*>(take((size_t)T * H * 2 * sizeof(float)));
  w.bytes = off;
  return w;
}

// k is the selection size (1 <= k <= min(S, KMAX)), or with slots the number
// of product-key slots per row (1 <= k <= KMAX; extras may exceed S).
int check_search_shapes(const char* fn, const void* q, pkmem_dtype q_dt, const void* subkeys,
                        pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k,
                        bool slots = false) {
  if (!dtype_ok(q_dt) || !dtype_ok(k_dt)) return fail(PKMEM_ERR_INVALID, "%s: unknown dtype", fn);
  if (q_dt != k_dt) return fail(PKMEM_ERR_UNSUPPORTED, "%s: queries and sub-keys must share a dtype", fn);
  if (T < 0) return fail(PKMEM_ERR_INVALID, "%s: T must be >= 0", fn);
  if (H < 1) return fail(PKMEM_ERR_INVALID, "%s: H must be >= 1", fn);
  if (n < 2 || n % 2 != 0) return fail(PKMEM_ERR_INVALID, "%s: n must be even and >= 2 (got %d)", fn, n);
  const int d = n / 2;
  if (q_dt == PKMEM_BF16 && (d % 8 != 0 || d > PKMEM_DHALF_MAX))
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: bf16 needs n/2 a multiple of 8 and <= %d (got %d)", fn, PKMEM_DHALF_MAX, d);
  if (q_dt == PKMEM_F32 && (d % 4 != 0 || d > 64))
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: fp32 needs n/2 a multiple of 4 and <= 64 (got %d)", fn, d);
  if (S < 1) return fail(PKMEM_ERR_INVALID, "%s: S must be >= 1", fn);
  if (S > PKMEM_SMAX) return fail(PKMEM_ERR_UNSUPPORTED, "%s: S > %d", fn, PKMEM_SMAX);
  if (k < 1 || (!slots && k > S)) return fail(PKMEM_ERR_INVALID, "%s: need 1 <= k <= S (k=%d, S=%d)", fn, k, S);
  if (k > PKMEM_KMAX) return fail(PKMEM_ERR_UNSUPPORTED, "%s: k > %d", fn, PKMEM_KMAX);
  if ((T * H * 2) > (int64_t)0xFFFFFFFF) return fail(PKMEM_ERR_UNSUPPORTED, "%s: T*H*2 must be < 2^32", fn);
  if (T > 0 && (!q || !subkeys)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(q, 16) || !aligned(subkeys, 16)) return fail(PKMEM_ERR_INVALID, "%s: q and subkeys must be 16-byte aligned", fn);
  return PKMEM_OK;
}

int check_bag_shapes(const char* fn, pkmem_dtype v_dt, int64_t N, int D, int64_t T, int bag) {
  if (!dtype_ok(v_dt)) return fail(PKMEM_ERR_INVALID, "%s: unknown value dtype %d", fn, (int)v_dt);
  if (N < 1) return fail(PKMEM_ERR_INVALID, "%s: N must be >= 1 (got %lld)", fn, (long long)N);
  if (N > (int64_t(1) << 32)) return fail(PKMEM_ERR_UNSUPPORTED, "%s: N > 2^32 rows", fn);
  if (T < 0) return fail(PKMEM_ERR_INVALID, "%s: T must be >= 0", fn);
  if (bag < 1) return fail(PKMEM_ERR_INVALID, "%s: bag (H*k) must be >= 1", fn);
  if (D < 8 || D % 8 != 0) return fail(PKMEM_ERR_UNSUPPORTED, "%s: D must be a positive multiple of 8 (got %d)", fn, D);
  const int chunks = (int)(D * esize(v_dt) / 16);
  if (chunks > 512) return fail(PKMEM_ERR_UNSUPPORTED, "%s: rows wider than 8 KiB are not supported (D=%d)", fn, D);
  if ((T * (int64_t)bag) > (int64_t)0xFFFFFFFF) return fail(PKMEM_ERR_UNSUPPORTED, "%s: T*bag must be < 2^32", fn);
  return PKMEM_OK;
}

// grad_w when the caller passes none; for the sorted strategy the sort, then
// the partial rows of long rows' chunks.
size_t bwd_ws_bytes(int64_t T, int H, int k, int D, int mode) {
  const int64_t L = T * H * k;
  size_t b = align256((size_t)L * sizeof(float));
  if (mode == PKMEM_BWD_SORTED) b += pk::sorted_workspace_bytes(L) + pk::long_partial_bytes(L, D);
  return b;
}

// What PKMEM_BWD_AUTO means for L = T*H*k lookups of rows of D elements:
// atomic adds when L*D <= 2^26 fp32 updates and D <= 1024, the sorted
// strategy otherwise.  Measured on MI355X (uniform indices over 2^20 rows,
// D = 64..2048, L = 32K..2M): the atomic kernel costs about 3.5 ps per
// updated element plus one launch, the sort a fixed ~0.1 ms (eleven
// launches) plus its row streaming, so atomics win only small batches; at
// D = 2048 the sort wins from 256 tokens on.  PKMEM_BWD_MODE=atomic|sorted in
// the environment overrides the choice (read at every call).
int resolve_mode(int mode, int D, int64_t L) {
  if (mode != PKMEM_BWD_AUTO) return mode;
  const char* env = getenv("PKMEM_BWD_MODE");
  if (env && strcmp(env, "atomic") == 0) return PKMEM_BWD_ATOMIC;
  if (env && strcmp(env, "sorted") == 0) return PKMEM_BWD_SORTED;
  return (D <= 1024 && L * (int64_t)D <= (int64_t(1) << 26)) ? PKMEM_BWD_ATOMIC : PKMEM_BWD_SORTED;
}

// PKMEM_DEBUG=1 in the environment (read at every call) checks on the device
// that every index lies in [0, limit) before the kernels that use them run:
// the call waits for the check and fails with PKMEM_ERR_INVALID otherwise.
// The flag it needs is the only device memory the library allocates (4 bytes
// per device, once, and only in debug mode).
bool debug_checks() {
  const char* env = getenv("PKMEM_DEBUG");
  return env && env[0] && strcmp(env, "0") != 0;
}

// The debug check's flag on the current device (allocated at first use).
int debug_flag(const char* fn, uint32_t** flag) {
  static uint32_t* flags[64] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, fn);
  if (dev < 0 || dev >= 64) return fail(PKMEM_ERR_UNSUPPORTED, "%s: device %d", fn, dev);
  if (!flags[dev]) {
    e = hipMalloc(reinterpret_cast<void**>(&flags[dev]), sizeof(uint32_t));
    if (e != hipSuccess) return hip_status(e, fn);
  }
  *flag = flags[dev];
  return PKMEM_OK;
}

// Waits for the check launched (status e) and reads its flag.
int debug_outcome(const char* fn, hipError_t e, uint32_t* flag, int64_t limit, hipStream_t st) {
  uint32_t bad = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&bad, flag, sizeof(bad), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_status(e, fn);
  if (bad) return fail(PKMEM_ERR_INVALID, "%s: an index lies outside [0, %lld) (PKMEM_DEBUG)", fn, (long long)limit);
  return PKMEM_OK;
}

int check_indices(const char* fn, const int64_t* idx, int64_t count, int64_t limit, hipStream_t st) {
  if (!debug_checks() || count <= 0) return PKMEM_OK;
  uint32_t* flag = nullptr;
  int rc = debug_flag(fn, &flag);
  if (rc) return rc;
  hipError_t e = pk::launch_check_indices(idx, count, limit, flag, st);
  return debug_outcome(fn, e, flag, limit, st);
}

// check_indices over the first cols slots of each of rows rows, stride apart.
int check_indices_strided(const char* fn, const int64_t* idx, int64_t rows, int cols, int stride,
                          int64_t limit, hipStream_t st) {
  if (cols == stride) return check_indices(fn, idx, rows * cols, limit, st);
  if (!debug_checks() || rows <= 0) return PKMEM_OK;
  uint32_t* flag = nullptr;
  int rc = debug_flag(fn, &flag);
  if (rc) return rc;
  hipError_t e = pk::launch_check_indices_strided(idx, rows, cols, stride, limit, flag, st);
  return debug_outcome(fn, e, flag, limit, st);
}

int bag_backward_common(const char* fn, const void* dy, const void* values, pkmem_dtype v_dt,
                        int64_t N, int D, const int64_t* idx, const float* w, int64_t T, int H,
                        int k, float* grad_values, int64_t* rows_out, float* grad_rows_out,
                        int64_t cap, int64_t* num_rows_out, float* grad_w, float* grad_scores,
                        int mode, void* ws, size_t ws_bytes, hipStream_t st) {
  if (H < 1 || k < 1) return fail(PKMEM_ERR_INVALID, "%s: H and k must be >= 1", fn);
  int rc = check_bag_shapes(fn, v_dt, N, D, T, H * k);
  if (rc) return rc;
  if (mode != PKMEM_BWD_AUTO && mode != PKMEM_BWD_ATOMIC && mode != PKMEM_BWD_SORTED)
    return fail(PKMEM_ERR_INVALID, "%s: unknown mode %d", fn, mode);
  const bool sparse = rows_out != nullptr || num_rows_out != nullptr;
  const int m = sparse ? PKMEM_BWD_SORTED : resolve_mode(mode, D, T * H * (int64_t)k);
  if (T > 0 && (!dy || !values || !idx || !w))
    return fail(PKMEM_ERR_INVALID, "%s: null input pointer", fn);
  if (!aligned(dy, 16) || !aligned(values, 16))
    return fail(PKMEM_ERR_INVALID, "%s: dy and values must be 16-byte aligned", fn);
  if (grad_values && !aligned(grad_values, 16))
    return fail(PKMEM_ERR_INVALID, "%s: grad_values must be 16-byte aligned", fn);
  const int64_t L = T * H * k;
  if (sparse) {
    if (!rows_out || !grad_rows_out || !num_rows_out)
      return fail(PKMEM_ERR_INVALID, "%s: rows_out, grad_rows_out and num_rows_out are required", fn);
    if (!aligned(grad_rows_out, 16)) return fail(PKMEM_ERR_INVALID, "%s: grad_rows_out must be 16-byte aligned", fn);
    const int64_t need = L < N ? L : N;
    if (cap < need)
      return fail(PKMEM_ERR_INVALID, "%s: cap %lld < min(T*H*k, N) = %lld", fn, (long long)cap, (long long)need);
  }
  const size_t need_ws = bwd_ws_bytes(T, H, k, D, m);
  if (!ws || ws_bytes < need_ws)
    return fail(PKMEM_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need_ws, ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 256)) return fail(PKMEM_ERR_INVALID, "%s: workspace must be 256-byte aligned", fn);
  if (sparse) *num_rows_out = 0;
  if (T == 0) return PKMEM_OK;
  rc = check_indices(fn, idx, L, N, st);
  if (rc) return rc;

  char* p = reinterpret_cast<char*>(ws);
  float* gw = grad_w ? grad_w : reinterpret_cast<float*>(p);
  p += align256((size_t)L * sizeof(float));
  const bool bf16 = v_dt == PKMEM_BF16;
  hipError_t e;
  if (m == PKMEM_BWD_ATOMIC) {
    e = pk::launch_bag_backward_atomic(bf16, dy, values, D, idx, w, T, H * k, grad_values, gw, st);
    if (e != hipSuccess) return hip_status(e, fn);
  } else {
    uint32_t* nrows_dev = nullptr;
    float* part = reinterpret_cast<float*>(p + pk::sorted_workspace_bytes(L));
    e = pk::launch_bag_backward_sorted(bf16, dy, values, N, D, idx, w, T, H * k,
                                       sparse ? nullptr : grad_values, sparse ? rows_out : nullptr,
                                       grad_rows_out, gw, p, part, &nrows_dev, st);
    if (e != hipSuccess) return hip_status(e, fn);
    if (sparse) {
      uint32_t U = 0;
      e = hipMemcpyAsync(&U, nrows_dev, sizeof(U), hipMemcpyDeviceToHost, st);
      if (e == hipSuccess) e = hipStreamSynchronize(st);
      if (e != hipSuccess) return hip_status(e, fn);
      *num_rows_out = U;
    }
  }
  if (grad_scores) {
    e = pk::launch_softmax_backward(w, gw, T * H, k, grad_scores, st);
    if (e != hipSuccess) return hip_status(e, fn);
  }
  return PKMEM_OK;
}

// Benchmark timer state (host side, single-threaded use).
struct TimedLaunch {
  int kernel;  // position of the kernel's name in the timer's list
  hipEvent_t start, stop;
};
struct TimerState {
  std::vector<std::string> names;
  bool on = false;
  std::vector<TimedLaunch> events;
};
TimerState g_timer;

int timer_slot(const char* name) {
  for (size_t i = 0; i < g_timer.names.size(); ++i)
    if (g_timer.names[i] == name) return (int)i;
  return -1;
}

}  // namespace

namespace pk {

LaunchTimer::LaunchTimer(const char* name, hipStream_t st) : st_(st) {
  if (!g_timer.on) return;
  const int slot = timer_slot(name);
  if (slot < 0) return;
  hipEvent_t a, b;
  if (hipEventCreate(&a) != hipSuccess) return;
  if (hipEventCreate(&b) != hipSuccess) { (void)hipEventDestroy(a); return; }
  if (hipEventRecord(a, st_) != hipSuccess) {
    (void)hipEventDestroy(a);
    (void)hipEventDestroy(b);
    return;
  }
  stop_ = b;
  g_timer.events.push_back({slot, a, b});
}

LaunchTimer::~LaunchTimer() {
  if (stop_) (void)hipEventRecord(stop_, st_);
}

}  // namespace pk

extern "C" {

int mem_timer_start(const char* kernels) {
  if (!kernels) return fail(PKMEM_ERR_INVALID, "mem_timer_start: null kernel list");
  g_timer.names.clear();
  std::string cur;
  for (const char* c = kernels;; ++c) {
    if (*c == ',' || *c == '\0') {
      if (!cur.empty()) g_timer.names.push_back(cur);
      cur.clear();
      if (*c == '\0') break;
    } else if (*c != ' ') {
      cur.push_back(*c);
    }
  }
  g_timer.on = !g_timer.names.empty();
  return PKMEM_OK;
}

int mem_timer_stop(void) {
  g_timer.on = false;
  return PKMEM_OK;
}

int mem_timer_read(float* ms_out, int* kernel_out, int cap) {
  int n = 0;
  hipError_t err = hipSuccess;
  for (auto& ev : g_timer.events) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(ev.stop);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, ev.start, ev.stop);
    if (e != hipSuccess && err == hipSuccess) err = e;
    if (n < cap) {
      if (ms_out) ms_out[n] = ms;
      if (kernel_out) kernel_out[n] = ev.kernel;
    }
    ++n;
    (void)hipEventDestroy(ev.start);
    (void)hipEventDestroy(ev.stop);
  }
  g_timer.events.clear();
  if (err != hipSuccess) return hip_status(err, "mem_timer_read");
  return n;
}

const char* mem_last_error(void) { return g_last_error.c_str(); }

int mem_version(void) { return 1; }

size_t mem_search_workspace_size(int64_t T, int H, int S, int k) {
  (void)S;
  if (T < 0 || H < 1 || k < 1) return 0;
  return search_ws(nullptr, T, H, k).bytes;
}

// The search, with the queries normalised (qnorm) or not.
static int search_common(const char* fn, const void* q, pkmem_dtype q_dt, const void* subkeys,
                         pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k, bool qnorm,
                         float eps, int nex, const int64_t* ex_idx, bool has_sink,
                         const void* sink, int64_t sink_row0, int64_t* idx_out, float* w_out, float* score_out,
                         int32_t* half_idx_out, void* qhat_out, float* stats_out, void* ws,
                         size_t ws_bytes, pkmem_stream_t stream) {
  int rc = check_search_shapes(fn, q, q_dt, subkeys, k_dt, T, H, n, S, k);
  if (rc) return rc;
  if (nex < 0) return fail(PKMEM_ERR_INVALID, "%s: r must be >= 0", fn);
  if (k + nex + (has_sink ? 1 : 0) > PKMEM_KMAX)
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: k + r%s must be <= %d (k=%d, r=%d)", fn,
                has_sink ? " + 1" : "", PKMEM_KMAX, k, nex);
  if (has_sink) {
    if (T > 0 && !sink) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
    if (!aligned(sink, 16)) return fail(PKMEM_ERR_INVALID, "%s: sink_keys must be 16-byte aligned", fn);
    if (sink_row0 < (int64_t)S * S || sink_row0 > INT64_MAX - H)
      return fail(PKMEM_ERR_INVALID, "%s: sink_row0 must be >= S*S = %lld (got %lld)", fn,
                  (long long)S * S, (long long)sink_row0);
  }
  if (T > 0 && nex > 0 && !ex_idx) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (T > 0 && (!idx_out || !w_out)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (qnorm && !(eps >= 0.f && eps <= 3.0e38f))
    return fail(PKMEM_ERR_INVALID, "%s: eps must be finite and >= 0", fn);
  if (!aligned(qhat_out, 16) || !aligned(stats_out, 8))
    return fail(PKMEM_ERR_INVALID, "%s: qhat_out must be 16-byte and stats_out 8-byte aligned", fn);
  const SearchWs need = search_ws(nullptr, T, H, k);
  if (!ws || ws_bytes < need.bytes)
    return fail(PKMEM_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need.bytes, ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 256)) return fail(PKMEM_ERR_INVALID, "%s: workspace must be 256-byte aligned", fn);
  if (T == 0) return PKMEM_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  SearchWs w = search_ws(ws, T, H, k);
  const bool bf16 = q_dt == PKMEM_BF16;
  float2* qstats = nullptr;
  hipError_t e = hipSuccess;
  if (qnorm) {
    qstats = stats_out ? reinterpret_cast<float2*>(stats_out) : w.qstats;
    e = pk::launch_qnorm(bf16, q, T * H, n, eps, qstats, qhat_out, st);
    if (e != hipSuccess) return hip_status(e, fn);
  }
  int32_t* hidx = half_idx_out ? half_idx_out : w.half_idx;
  e = pk::launch_search_half(bf16, q, subkeys, T, H, n, S, k, qstats, has_sink ? sink : nullptr,
                             w.sink_part, w.cand, w.cnts, w.thr, hidx, w.half_score, w.ovf, st);
  if (e != hipSuccess) return hip_status(e, fn);
  if (nex > 0) {
    rc = check_indices(fn, ex_idx, T * H * nex, (int64_t)S * S, st);
    if (rc) return rc;
  }
  e = pk::launch_cartesian(hidx, w.half_score, T, H, S, k, bf16, q, subkeys, n, ex_idx, nex,
                           has_sink ? w.sink_part : nullptr, sink_row0, idx_out, w_out, score_out,
                           st);
  if (e != hipSuccess) return hip_status(e, fn);
  return PKMEM_OK;
}

int mem_search(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt, int64_t T,
               int H, int n, int S, int k, int64_t* idx_out, float* w_out, float* score_out,
               int32_t* half_idx_out, void* ws, size_t ws_bytes, pkmem_stream_t stream) {
  return search_common("mem_search", q, q_dt, subkeys, k_dt, T, H, n, S, k, false, 0.f, 0, nullptr,
                       false, nullptr, 0, idx_out, w_out, score_out, half_idx_out, nullptr, nullptr, ws, ws_bytes,
                       stream);
}

}  // extern "C"

// Workspace of mem_search_noalloc: one array per GPU, part of the library's
// code object, held until the process ends.  Host code never uses its name as
// an address: the device address comes from hipGetSymbolAddress, looked up
// once per device with that device current.
static __device__ __align__(256) unsigned char scratch[PKMEM_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[SCRATCH_DEVICES] = {};

// The current device's address of the scratch array (looked up at the first
// call on that device).
int scratch_on_current_device(const char* fn, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, fn);
  if (dev < 0 || dev >= SCRATCH_DEVICES) return fail(PKMEM_ERR_UNSUPPORTED, "%s: device %d", fn, dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, fn);
    if (!p) return fail(PKMEM_ERR_HIP, "%s: no device address for the scratch array", fn);
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PKMEM_OK;
}

}  // namespace

extern "C" {

int mem_search_noalloc(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                       int64_t T, int H, int n, int S, int k, int64_t* idx_out, float* w_out,
                       float* score_out, int32_t* half_idx_out, pkmem_stream_t stream) {
  const char* fn = "mem_search_noalloc";
  int rc = check_search_shapes(fn, q, q_dt, subkeys, k_dt, T, H, n, S, k);
  if (rc) return rc;
  const size_t need = search_ws(nullptr, T, H, k).bytes;
  if (need > PKMEM_NOALLOC_SCRATCH_BYTES)
    return fail(PKMEM_ERR_UNSUPPORTED,
                "%s: T=%lld, H=%d, k=%d needs %zu bytes of scratch, more than its %zu "
                "(use mem_search with a workspace)",
                fn, (long long)T, H, k, need, (size_t)PKMEM_NOALLOC_SCRATCH_BYTES);
  if (T > 0 && (!idx_out || !w_out)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (T == 0) return PKMEM_OK;
  void* ws = nullptr;
  rc = scratch_on_current_device(fn, &ws);
  if (rc) return rc;
  return search_common(fn, q, q_dt, subkeys, k_dt, T, H, n, S, k, false, 0.f, 0, nullptr, false,
                       nullptr, 0, idx_out, w_out, score_out, half_idx_out, nullptr, nullptr, ws,
                       PKMEM_NOALLOC_SCRATCH_BYTES, stream);
}

int mem_search_qnorm(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                     int64_t T, int H, int n, int S, int k, float eps, int64_t* idx_out,
                     float* w_out, float* score_out, int32_t* half_idx_out, void* qhat_out,
                     float* stats_out, void* ws, size_t ws_bytes, pkmem_stream_t stream) {
  return search_common("mem_search_qnorm", q, q_dt, subkeys, k_dt, T, H, n, S, k, true, eps, 0,
                       nullptr, false, nullptr, 0, idx_out, w_out, score_out, half_idx_out, qhat_out, stats_out, ws,
                       ws_bytes, stream);
}

int mem_search_extra(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                     int64_t T, int H, int n, int S, int k, int r, const int64_t* extra_idx,
                     int64_t* idx_out, float* w_out, float* score_out, int32_t* half_idx_out,
                     void* ws, size_t ws_bytes, pkmem_stream_t stream) {
  return search_common("mem_search_extra", q, q_dt, subkeys, k_dt, T, H, n, S, k, false, 0.f, r,
                       extra_idx, false, nullptr, 0, idx_out, w_out, score_out, half_idx_out, nullptr,
                       nullptr, ws, ws_bytes, stream);
}

int mem_search_sink(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                    int64_t T, int H, int n, int S, int k, int r, const int64_t* extra_idx,
                    const void* sink_keys, int64_t sink_row0, int64_t* idx_out, float* w_out,
                    float* score_out, int32_t* half_idx_out, void* ws, size_t ws_bytes,
                    pkmem_stream_t stream) {
  return search_common("mem_search_sink", q, q_dt, subkeys, k_dt, T, H, n, S, k, false, 0.f, r,
                       extra_idx, true, sink_keys, sink_row0, idx_out, w_out, score_out,
                       half_idx_out, nullptr, nullptr, ws, ws_bytes, stream);
}

size_t mem_search_backward_workspace_size(int64_t T, int H, int S, int k) {
  (void)S;
  if (T < 0 || H < 1 || k < 1) return 0;
  // the sort and its inputs, then the queries' (mean, rstd) for the normalised variant
  return pk::search_backward_ws_bytes(T, H, k) + align256((size_t)T * H * sizeof(float2));
}

size_t mem_search_backward_sink_workspace_size(int64_t T, int H, int n, int S, int k) {
  (void)S;
  if (T < 0 || H < 1 || n < 2 || k < 1) return 0;
  // the sort and its inputs, then the per-chunk partial sums of grad_sink
  return pk::search_backward_ws_bytes(T, H, k) +
         align256((size_t)pk::sink_chunks(T) * H * n * sizeof(float));
}

// k: product-key slots per row.  With a sink the rows of idx and grad_scores
// hold k + 1 slots, the last the sink's.
static int search_backward_common(const char* fn, const void* q, pkmem_dtype q_dt,
                                  const void* subkeys, pkmem_dtype k_dt, int64_t T, int H, int n,
                                  int S, int k, bool qnorm, float eps, const int64_t* idx,
                                  const float* grad_scores, bool has_sink, const void* sink,
                                  float* grad_q, float* grad_subkeys, float* grad_sink, void* ws,
                                  size_t ws_bytes, pkmem_stream_t stream) {
  int rc = check_search_shapes(fn, q, q_dt, subkeys, k_dt, T, H, n, S, k, true);
  if (rc) return rc;
  if (k > PKMEM_KMAX - (has_sink ? 1 : 0))
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: more than %d slots per row", fn, PKMEM_KMAX);
  if (has_sink) {
    if (T > 0 && (grad_q || grad_sink) && !sink) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
    if (!aligned(sink, 16) || !aligned(grad_sink, 4))
      return fail(PKMEM_ERR_INVALID, "%s: sink_keys must be 16-byte and grad_sink 4-byte aligned", fn);
  }
  if (T > 0 && (!idx || !grad_scores)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (qnorm && !(eps >= 0.f && eps <= 3.0e38f))
    return fail(PKMEM_ERR_INVALID, "%s: eps must be finite and >= 0", fn);
  if (2 * T * (int64_t)H * k >= (int64_t(1) << 32))
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: 2*T*H*k must be < 2^32", fn);
  if (2 * (int64_t)H * S >= (int64_t(1) << 31))
    return fail(PKMEM_ERR_UNSUPPORTED, "%s: 2*H*S must be < 2^31", fn);
  if (!aligned(grad_subkeys, 16) || !aligned(grad_q, 4))
    return fail(PKMEM_ERR_INVALID, "%s: grad_subkeys must be 16-byte and grad_q 4-byte aligned", fn);
  const size_t need = has_sink ? mem_search_backward_sink_workspace_size(T, H, n, S, k)
                               : mem_search_backward_workspace_size(T, H, S, k);
  if (!ws || ws_bytes < need)
    return fail(PKMEM_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : (size_t)0);
  if (!aligned(ws, 256)) return fail(PKMEM_ERR_INVALID, "%s: workspace must be 256-byte aligned", fn);
  if (T == 0 || (!grad_q && !grad_subkeys && !grad_sink)) return PKMEM_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int kst = k + (has_sink ? 1 : 0);
  rc = check_indices_strided(fn, idx, T * H, k, kst, (int64_t)S * S, st);
  if (rc) return rc;
  const bool bf16 = q_dt == PKMEM_BF16;
  float2* qstats = nullptr;
  if (qnorm) {
    qstats = reinterpret_cast<float2*>(reinterpret_cast<char*>(ws) +
                                       pk::search_backward_ws_bytes(T, H, k));
    hipError_t e = pk::launch_qnorm(bf16, q, T * H, n, eps, qstats, nullptr, st);
    if (e != hipSuccess) return hip_status(e, fn);
  }
  float* sink_part = has_sink ? reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                                        pk::search_backward_ws_bytes(T, H, k))
                              : nullptr;
  hipError_t e = pk::launch_search_backward(bf16, q, subkeys, T, H, n, S, k, kst, idx, grad_scores,
                                            qstats, has_sink ? sink : nullptr, grad_q,
                                            grad_subkeys, has_sink ? grad_sink : nullptr,
                                            sink_part, ws, st);
  return hip_status(e, fn);
}

int mem_search_backward(const void* q, pkmem_dtype q_dt, const void* subkeys, pkmem_dtype k_dt,
                        int64_t T, int H, int n, int S, int k, const int64_t* idx,
                        const float* grad_scores, float* grad_q, float* grad_subkeys, void* ws,
                        size_t ws_bytes, pkmem_stream_t stream) {
  return search_backward_common("mem_search_backward", q, q_dt, subkeys, k_dt, T, H, n, S, k,
                                false, 0.f, idx, grad_scores, false, nullptr, grad_q, grad_subkeys,
                                nullptr, ws, ws_bytes, stream);
}

int mem_search_backward_sink(const void* q, pkmem_dtype q_dt, const void* subkeys,
                             pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k,
                             const int64_t* idx, const float* grad_scores, const void* sink_keys,
                             float* grad_q, float* grad_subkeys, float* grad_sink, void* ws,
                             size_t ws_bytes, pkmem_stream_t stream) {
  return search_backward_common("mem_search_backward_sink", q, q_dt, subkeys, k_dt, T, H, n, S, k,
                                false, 0.f, idx, grad_scores, true, sink_keys, grad_q,
                                grad_subkeys, grad_sink, ws, ws_bytes, stream);
}

int mem_search_backward_qnorm(const void* q, pkmem_dtype q_dt, const void* subkeys,
                              pkmem_dtype k_dt, int64_t T, int H, int n, int S, int k, float eps,
                              const int64_t* idx, const float* grad_scores, float* grad_q,
                              float* grad_subkeys, void* ws, size_t ws_bytes,
                              pkmem_stream_t stream) {
  return search_backward_common("mem_search_backward_qnorm", q, q_dt, subkeys, k_dt, T, H, n, S,
                                k, true, eps, idx, grad_scores, false, nullptr, grad_q,
                                grad_subkeys, nullptr, ws, ws_bytes, stream);
}

int mem_bag_forward(const void* values, pkmem_dtype v_dt, int64_t N, int D, const int64_t* idx,
                    const float* w, int64_t T, int bag, void* y_out, pkmem_stream_t stream) {
  const char* fn = "mem_bag_forward";
  int rc = check_bag_shapes(fn, v_dt, N, D, T, bag);
  if (rc) return rc;
  if (T > 0 && (!values || !idx || !w || !y_out)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(values, 16) || !aligned(y_out, 16)) return fail(PKMEM_ERR_INVALID, "%s: values and y_out must be 16-byte aligned", fn);
  if (T == 0) return PKMEM_OK;
  rc = check_indices(fn, idx, T * bag, N, reinterpret_cast<hipStream_t>(stream));
  if (rc) return rc;
  hipError_t e = pk::launch_bag_forward(v_dt == PKMEM_BF16, values, D, idx, w, T, bag, y_out, nullptr, nullptr,
                                        reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, fn);
}

int mem_bag_forward_gated(const void* values, pkmem_dtype v_dt, int64_t N, int D, const int64_t* idx,
                          const float* w, int64_t T, int bag, const void* gate, void* y_out,
                          void* out, pkmem_stream_t stream) {
  const char* fn = "mem_bag_forward_gated";
  int rc = check_bag_shapes(fn, v_dt, N, D, T, bag);
  if (rc) return rc;
  if (T > 0 && (!values || !idx || !w || !gate || !out)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(values, 16) || !aligned(gate, 16) || !aligned(out, 16) || !aligned(y_out, 16))
    return fail(PKMEM_ERR_INVALID, "%s: values, gate, y_out and out must be 16-byte aligned", fn);
  if (T == 0) return PKMEM_OK;
  rc = check_indices(fn, idx, T * bag, N, reinterpret_cast<hipStream_t>(stream));
  if (rc) return rc;
  hipError_t e = pk::launch_bag_forward(v_dt == PKMEM_BF16, values, D, idx, w, T, bag, out, gate,
                                        y_out, reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, fn);
}

int mem_gate_backward(const void* d_out, const void* gate, const void* y, pkmem_dtype v_dt, int64_t T,
                      int D, void* dy_out, float* grad_gate, pkmem_stream_t stream) {
  const char* fn = "mem_gate_backward";
  if (!dtype_ok(v_dt)) return fail(PKMEM_ERR_INVALID, "%s: unknown dtype %d", fn, (int)v_dt);
  if (T < 0) return fail(PKMEM_ERR_INVALID, "%s: T must be >= 0", fn);
  if (D < 8 || D % 8 != 0) return fail(PKMEM_ERR_UNSUPPORTED, "%s: D must be a positive multiple of 8 (got %d)", fn, D);
  if (T > 0 && (!d_out || !gate || !y || !dy_out || !grad_gate)) return fail(PKMEM_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(d_out, 16) || !aligned(gate, 16) || !aligned(y, 16) || !aligned(dy_out, 16) || !aligned(grad_gate, 16))
    return fail(PKMEM_ERR_INVALID, "%s: every buffer must be 16-byte aligned", fn);
  if (T == 0) return PKMEM_OK;
  hipError_t e = pk::launch_gate_backward(v_dt == PKMEM_BF16, d_out, gate, y, T, D, dy_out, grad_gate,
                                          reinterpret_cast<hipStream_t>(stream));
  return hip_status(e, fn);
}

size_t mem_bag_backward_workspace_size(int64_t T, int H, int k, int64_t N, int D, int mode) {
  (void)N;
  if (T < 0 || H < 1 || k < 1) return 0;
  return bwd_ws_bytes(T, H, k, D, resolve_mode(mode, D, T * H * (int64_t)k));
}

int mem_bag_backward(const void* dy, const void* values, pkmem_dtype v_dt, int64_t N, int D,
                     const int64_t* idx, const float* w, int64_t T, int H, int k,
                     float* grad_values, float* grad_w, float* grad_scores, int mode, void* ws,
                     size_t ws_bytes, pkmem_stream_t stream) {
  const char* fn = "mem_bag_backward";
  return bag_backward_common(fn, dy, values, v_dt, N, D, idx, w, T, H, k, grad_values, nullptr,
                             nullptr, 0, nullptr, grad_w, grad_scores, mode, ws, ws_bytes,
                             reinterpret_cast<hipStream_t>(stream));
}

int mem_bag_backward_sparse(const void* dy, const void* values, pkmem_dtype v_dt, int64_t N, int D,
                            const int64_t* idx, const float* w, int64_t T, int H, int k,
                            int64_t* rows_out, float* grad_rows_out, int64_t cap,
                            int64_t* num_rows_out, float* grad_w, float* grad_scores, void* ws,
                            size_t ws_bytes, pkmem_stream_t stream) {
  const char* fn = "mem_bag_backward_sparse";
  if (!rows_out || !grad_rows_out || !num_rows_out)
    return fail(PKMEM_ERR_INVALID, "%s: rows_out, grad_rows_out and num_rows_out are required", fn);
  return bag_backward_common(fn, dy, values, v_dt, N, D, idx, w, T, H, k, nullptr, rows_out,
                             grad_rows_out, cap, num_rows_out, grad_w, grad_scores,
                             PKMEM_BWD_SORTED, ws, ws_bytes, reinterpret_cast<hipStream_t>(stream));
}

}  // extern "C"
