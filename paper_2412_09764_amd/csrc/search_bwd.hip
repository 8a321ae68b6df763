// Search backward on gfx950: gradients of the selected scores into queries and
// sub-keys (the keys are trainable parameters, Sec. 3 of "Memory Layers at
// Scale"; the selection passes no gradient).  With the composed index
// i = i1*S + i2 of Sec. 3.1.1 the score of rank j is
//   z_j = q[:d] . K[h,0,i1_j] + q[d:] . K[h,1,i2_j],
// so grad_q[:d] = sum_j gz_j K[h,0,i1_j] and grad_K[h,0,i] += sum_{j: i1_j = i}
// gz_j q[:d] (same for half 1).
//
// grad_q: one wave per (token, head).  The k lookups sit one per lane; per
// half, each lane finds the leader of its sub-key group (lowest rank with the
// same sub-key index) and the group's summed gradient, in rank order; the wave
// reads each distinct sub-key row once.
//
// grad_K: every sub-key row is hot (only S rows per head and half), and fp32
// atomics, in global memory or in LDS, serialise on them.  Instead the same
// wave emits one (head, half, sub-key) sort key per group leader, with the
// group's gradient sum, at the front of its (token, head, half) row of k
// slots, and counts them; an exclusive scan of the counts places the leaders
// contiguously (in slot order), and the library's stable radix sort orders
// those pairs by key.  One wave per segment then sums gsum * q over the
// segment's tokens (in token order; each token's query half is read once) and
// adds the sum into the sub-key row with one plain read-modify-write: no
// atomics, bitwise deterministic.  A segment longer than 2048 pairs (a
// sub-key that thousands of tokens chose) goes to a workgroup of 16 waves
// instead, whose contiguous runs are added in run order.
#include "pk_device.h"
#include "pk_internal.h"

namespace pk {

// Per (token, head) wave, per half: lane j holds rank j's sub-key; each lane
// finds the ranks sharing its sub-key (one ballot per index bit), the lowest
// of them leads the group and adds the group's gradients in rank order.  Then
//   * grad_q (if wanted): the distinct sub-key rows are read QU at a time (all
//     loads in flight together), lane l owning elements 4l..4l+3;
//   * sort input (if wanted): row rp = (t*H + h)*2 + half gets its leaders'
//     keys (h*2 + half)*S + sub-key and group sums at slots rp*k + 0, 1, ...
//     (in rank order of the leaders) and their number at counts[rp].  Lookups
//     whose index lies outside [0, S*S) count as absent.
// idx and gz rows are kst >= k slots apart; with a sink (a fixed key-value
// pair per head scored as q . sink[h]) slot k of each row is the sink's and
// grad_q gains gz[sink slot] * sink[h] (its index is never read).
// With qstats (the forward normalised the queries, LayerNorm without affine)
// the two halves' gradients g with respect to the normalised query qhat stay
// in registers and grad_q = rstd * (g - mean(g) - xhat * mean(g * xhat)) over
// the query's n elements, xhat = (q - mean) * rstd in fp32 (the rounding of
// qhat to the query dtype passes the gradient unchanged).
#ifndef PK_SBWD_QU
#define PK_SBWD_QU 8
#endif
template <typename T>
__global__ __launch_bounds__(256) void k_search_bwd_q(const T* __restrict__ q,
                                                      const T* __restrict__ subkeys, int64_t ntok,
                                                      int H, int n, int S, int k, int kst,
                                                      const int64_t* __restrict__ idx,
                                                      const float* __restrict__ gz,
                                                      const T* __restrict__ sink,
                                                      const float2* __restrict__ qstats,
                                                      float* __restrict__ grad_q,
                                                      uint32_t* __restrict__ keys,
                                                      float* __restrict__ gvals,
                                                      uint32_t* __restrict__ counts) {
  constexpr int QU = PK_SBWD_QU;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = (int)(blockIdx.x % (unsigned)H);
  const int64_t t = (int64_t)(blockIdx.x / (unsigned)H) * 4 + wave;
  if (t >= ntok) return;
  const int d = n >> 1;
  const bool qlane = lane * 4 < d;
  const int ql = qlane ? lane * 4 : 0;
  const size_t r = (size_t)t * H + h;
  const int64_t ix = lane < k ? idx[r * kst + lane] : -1;
  const bool okl = ix >= 0 && ix < (int64_t)S * S;
  // the two sub-key indices (S * S <= 2^26: a 32-bit division)
  const int ix1 = okl ? (int)((uint32_t)ix / (uint32_t)S) : 0;
  const int ix2 = okl ? (int)((uint32_t)ix - (uint32_t)ix1 * (uint32_t)S) : 0;
  const float g = okl ? gz[r * kst + lane] : 0.f;
  const float gsink = sink ? gz[r * kst + k] : 0.f;
  const uint64_t below = (1ull << lane) - 1ull;
  const int nbits = S > 1 ? 32 - __builtin_clz((unsigned)(S - 1)) : 0;  // bits of a sub-key index
  float gh[2][4];  // with qstats: both halves' gradients with respect to qhat

#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int mine = okl ? (p == 0 ? ix1 : ix2) : -1;
    // the ranks sharing this lane's sub-key, as a mask over the wave's lanes:
    // one ballot per bit of the sub-key index
    uint64_t peers = __ballot(okl);
    for (int bt = 0; bt < nbits; ++bt) {
      const bool bit = (mine >> bt) & 1;
      const uint64_t set = __ballot(bit);
      peers &= bit ? set : ~set;
    }
    const bool leader = okl && (peers & below) == 0ull;
    // the leader's group sum, added in rank order; every lane takes part in
    // each exchange, the leaders keep what their own mask asks for
    float gsum = 0.f;
    uint64_t pm = leader ? peers : 0ull;
    while (__ballot(pm != 0ull) != 0ull) {
      const int j = pm != 0ull ? __builtin_ctzll(pm) : 0;
      const float v = __shfl(g, j, WAVE);
      if (pm != 0ull) {
        gsum += v;
        pm &= pm - 1ull;
      }
    }
    if (keys) {
      const uint64_t lm = __ballot(leader);
      const size_t rp = r * 2 + p;
      if (leader) {
        const size_t x = rp * k + __popcll(lm & below);
        keys[x] = (uint32_t)(h * 2 + p) * (uint32_t)S + (uint32_t)mine;
        gvals[x] = gsum;
      }
      if (lane == 0) counts[rp] = (uint32_t)__popcll(lm);
    }
    if (grad_q) {
      float acc[4] = {0.f, 0.f, 0.f, 0.f};
      const T* kh = subkeys + (size_t)(h * 2 + p) * S * d + ql;
      uint64_t m = __ballot(leader);
      while (m) {
        QQuad<T> kq[QU];
        float gg[QU];
        const int first = __builtin_ctzll(m);
#pragma unroll
        for (int j = 0; j < QU; ++j) {
          const bool has = m != 0;
          const int L = has ? __builtin_ctzll(m) : first;
          m = has ? (m & (m - 1)) : m;
          const int i = __builtin_amdgcn_readlane(mine, L);
          const float gj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gsum), L));
          gg[j] = has ? gj : 0.f;
          kq[j].load(kh + (size_t)i * d);
        }
#pragma unroll
        for (int j = 0; j < QU; ++j) kq[j].fma_into(gg[j], acc);
      }
      if (sink) {
        QQuad<T> sq;
        sq.load(sink + (size_t)h * n + (size_t)p * d + ql);
        sq.fma_into(gsink, acc);
      }
      if (qstats) {
#pragma unroll
        for (int i = 0; i < 4; ++i) gh[p][i] = qlane ? acc[i] : 0.f;
      } else if (qlane) {
        *reinterpret_cast<float4*>(grad_q + r * n + (size_t)p * d + ql) =
            make_float4(acc[0], acc[1], acc[2], acc[3]);
      }
    }
  }
  if (qstats && grad_q) {
    const float2 st = qstats[r];
    float xh[2][4];
    float sg = 0.f, sgx = 0.f;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      QQuad<T> xq;
      xq.load(q + r * n + (size_t)p * d + ql);
      float v[4];
      xq.to_f32(v);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xh[p][i] = qlane ? qn_apply(v[i], st.x, st.y) : 0.f;
        sg += gh[p][i];
        sgx = fmaf(gh[p][i], xh[p][i], sgx);
      }
    }
    sg = group_sum<WAVE>(sg);
    sgx = group_sum<WAVE>(sgx);
    const float mg = sg / (float)n, mgx = sgx / (float)n;
    if (qlane) {
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float o[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = st.y * (gh[p][i] - mg - xh[p][i] * mgx);
        *reinterpret_cast<float4*>(grad_q + r * n + (size_t)p * d + ql) =
            make_float4(o[0], o[1], o[2], o[3]);
      }
    }
  }
}

// The leaders of every row, packed: row rp's c = offs[rp+1] - offs[rp] keys
// move from slots rp*k .. rp*k + c - 1 to offs[rp] ..; the value is the slot.
__global__ __launch_bounds__(256) void k_sbwd_pack(const uint32_t* __restrict__ keys,
                                                   const uint32_t* __restrict__ offs, int64_t rows,
                                                   int k, uint32_t* __restrict__ keys_out,
                                                   uint32_t* __restrict__ slot_out) {
  const int64_t x = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (x >= rows * k) return;
  const int64_t rp = x / k;
  const uint32_t j = (uint32_t)(x - rp * k);
  const uint32_t o = offs[rp];
  if (j < offs[rp + 1] - o) {
    keys_out[o + j] = keys[x];
    slot_out[o + j] = (uint32_t)x;
  }
}

// Adds gsum * (query half as scored) of the sorted pairs [a, z) of one
// (head h, half) segment into acc, in pair order: the pairs are taken 64 at a
// time and consumed QU at a time, with their query-quad loads issued
// together; lane l owns elements 4l..4l+3 of the half (qh points at them).
template <typename T, bool QN>
__device__ __forceinline__ void sbwd_sum_run(const T* qh, int H, int n, int h, uint32_t hk2,
                                             const float2* __restrict__ qstats,
                                             const float* __restrict__ gvals,
                                             const uint32_t* __restrict__ vs, uint32_t a,
                                             uint32_t z, int lane, float* acc) {
  constexpr int QU = PK_SBWD_QU;
  for (uint32_t b0 = a; b0 < z; b0 += 64) {
    const uint32_t e = b0 + lane;
    const bool ok = e < z;
    const uint32_t x = ok ? vs[e] : 0u;
    const uint32_t t = x / hk2;
    const float gx = ok ? gvals[x] : 0.f;
    float2 st = make_float2(0.f, 1.f);
    if constexpr (QN) st = qstats[(size_t)t * H + h];
    const uint32_t cnt = (z - b0) < 64u ? (z - b0) : 64u;
    for (uint32_t j0 = 0; j0 < cnt; j0 += QU) {
      QQuad<T> qq[QU];
      float gg[QU], mj[QU], rj[QU];
#pragma unroll
      for (int j = 0; j < QU; ++j) {
        const bool has = j0 + j < cnt;
        const int L = has ? (int)(j0 + j) : (int)j0;
        const uint32_t tj = (uint32_t)__builtin_amdgcn_readlane((int)t, L);
        const float xj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gx), L));
        gg[j] = has ? xj : 0.f;
        if constexpr (QN) {
          mj[j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.x), L));
          rj[j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(st.y), L));
        }
        qq[j].load(qh + (size_t)tj * H * n);
      }
#pragma unroll
      for (int j = 0; j < QU; ++j) {
        if constexpr (QN) qq[j].fma_into_norm(gg[j], acc, mj[j], rj[j]);
        else qq[j].fma_into(gg[j], acc);
      }
    }
  }
}

// A segment of more than SBWD_LONG pairs (a sub-key chosen by that many
// tokens) is summed by k_sbwd_long instead of one wave.
constexpr uint32_t SBWD_LONG = 2048;
constexpr int SBWD_LWAVES = 16;
static int64_t sbwd_max_long(int64_t np) { return np / SBWD_LONG + 1; }

// One wave per segment (grid-stride) of the sorted pairs; a segment is one
// (head, half, sub-key) and holds at most one pair per token, in token order.
// Lane l owns elements 4l..4l+3 of the d-element row (d <= 256).  The sum is
// added into the sub-key row with one read-modify-write.
template <typename T, bool QN>
__global__ __launch_bounds__(256) void k_sbwd_segments(const T* __restrict__ q, int H, int n,
                                                       int S, int k,
                                                       const float2* __restrict__ qstats,
                                                       const float* __restrict__ gvals,
                                                       const uint32_t* __restrict__ ks,
                                                       const uint32_t* __restrict__ vs,
                                                       const uint32_t* __restrict__ seg,
                                                       const uint32_t* __restrict__ nseg_p,
                                                       float* __restrict__ grad_K) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t nseg = *nseg_p;
  const int d = n >> 1;
  const bool qlane = lane * 4 < d;
  const int ql = qlane ? lane * 4 : 0;
  const uint32_t nbins = (uint32_t)(2 * H) * (uint32_t)S;
  const uint32_t hk2 = 2u * (uint32_t)H * (uint32_t)k;  // slots per token
  for (uint32_t u = blockIdx.x * 4u + wave; u < nseg; u += gridDim.x * 4u) {
    const uint32_t s0 = seg[u], s1 = seg[u + 1];
    const uint32_t bin = ks[s0];
    if (bin >= nbins || s1 - s0 > SBWD_LONG) continue;
    const int hp = (int)(bin / (uint32_t)S);
    const int h = hp >> 1, p = hp & 1;
    const T* qh = q + (size_t)h * n + (size_t)p * d + ql;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    sbwd_sum_run<T, QN>(qh, H, n, h, hk2, qstats, gvals, vs, s0, s1, lane, acc);
    if (qlane) {
      float4* dst = reinterpret_cast<float4*>(grad_K + (size_t)bin * d + ql);
      float4 o = *dst;
      o.x += acc[0]; o.y += acc[1]; o.z += acc[2]; o.w += acc[3];
      *dst = o;
    }
  }
}

// The segments listed in long_list, one workgroup of SBWD_LWAVES waves per
// segment at a time: wave w sums the w-th contiguous run of the segment's
// pairs (in pair order) into a partial row; the partial rows meet in LDS and
// are added, in wave order, to the sub-key row with one read-modify-write.
template <typename T, bool QN>
__global__ __launch_bounds__(64 * SBWD_LWAVES) void k_sbwd_long(
    const T* __restrict__ q, int H, int n, int S, int k, const float2* __restrict__ qstats,
    const float* __restrict__ gvals, const uint32_t* __restrict__ ks,
    const uint32_t* __restrict__ vs, const uint32_t* __restrict__ seg,
    const uint32_t* __restrict__ long_list, const uint32_t* __restrict__ long_cnt,
    float* __restrict__ grad_K) {
  __shared__ float part[SBWD_LWAVES][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int d = n >> 1;
  const bool qlane = lane * 4 < d;
  const int ql = qlane ? lane * 4 : 0;
  const uint32_t nbins = (uint32_t)(2 * H) * (uint32_t)S;
  const uint32_t hk2 = 2u * (uint32_t)H * (uint32_t)k;
  const uint32_t nlong = *long_cnt;
  for (uint32_t it = blockIdx.x; it < nlong; it += gridDim.x) {
    const uint32_t u = long_list[it];
    const uint32_t s0 = seg[u], s1 = seg[u + 1];
    const uint32_t bin = ks[s0];
    if (bin >= nbins) continue;  // the same for every wave of the workgroup
    const int hp = (int)(bin / (uint32_t)S);
    const int h = hp >> 1, p = hp & 1;
    const T* qh = q + (size_t)h * n + (size_t)p * d + ql;
    const uint32_t len = s1 - s0;
    const uint32_t per = (len + SBWD_LWAVES - 1) / SBWD_LWAVES;
    uint32_t a = (uint32_t)wave * per, z = a + per;
    a = s0 + (a < len ? a : len);
    z = s0 + (z < len ? z : len);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    sbwd_sum_run<T, QN>(qh, H, n, h, hk2, qstats, gvals, vs, a, z, lane, acc);
    if (qlane) {
#pragma unroll
      for (int i = 0; i < 4; ++i) part[wave][ql + i] = acc[i];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < d; e += 64 * SBWD_LWAVES) {
      float sum = grad_K[(size_t)bin * d + e];
#pragma unroll
      for (int w = 0; w < SBWD_LWAVES; ++w) sum += part[w][e];
      grad_K[(size_t)bin * d + e] = sum;
    }
    __syncthreads();
  }
}

// grad_sink[h] += sum_t gz[t,h,sink slot] q[t,h], in two deterministic
// passes.  k_sink_partial: one workgroup per (chunk of SINK_TCH tokens, head);
// wave w takes the chunk's tokens w, w + 4, ... in order (SINK_U loads in
// flight), lane l owns elements 4l..4l+3 of each half; the four waves' sums
// are added in wave order into the chunk's partial row.  k_sink_reduce adds
// the partial rows in chunk order into grad_sink.
constexpr int SINK_TCH = 256;
constexpr int SINK_U = 8;
constexpr int SINK_NMAX = 512;  // n = 2d, d <= 256
int64_t sink_chunks(int64_t T) { return (T + SINK_TCH - 1) / SINK_TCH; }

template <typename T>
__global__ __launch_bounds__(256) void k_sink_partial(const T* __restrict__ q, int64_t ntok, int H,
                                                      int n, int kst, int k,
                                                      const float* __restrict__ gz,
                                                      float* __restrict__ part) {
  __shared__ float red[4][SINK_NMAX];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = (int)(blockIdx.x % (unsigned)H);
  const int64_t c = blockIdx.x / (unsigned)H;
  const int d = n >> 1;
  const bool qlane = lane * 4 < d;
  const int ql = qlane ? lane * 4 : 0;
  const int64_t t0 = c * SINK_TCH;
  const int64_t t1 = t0 + SINK_TCH < ntok ? t0 + SINK_TCH : ntok;
  float acc[2][4] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  for (int64_t tb = t0 + wave; tb < t1; tb += 4 * SINK_U) {
    QQuad<T> qa[SINK_U], qb[SINK_U];
    float g[SINK_U];
#pragma unroll
    for (int j = 0; j < SINK_U; ++j) {
      const int64_t t = tb + 4 * j;
      const bool has = t < t1;
      const size_t r = (size_t)(has ? t : tb) * H + h;
      g[j] = has ? gz[r * kst + k] : 0.f;
      qa[j].load(q + r * n + ql);
      qb[j].load(q + r * n + d + ql);
    }
#pragma unroll
    for (int j = 0; j < SINK_U; ++j) {
      qa[j].fma_into(g[j], acc[0]);
      qb[j].fma_into(g[j], acc[1]);
    }
  }
  if (qlane) {
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][p * d + ql + i] = acc[p][i];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < n; e += 256)
    part[((size_t)c * H + h) * n + e] = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
}

__global__ __launch_bounds__(256) void k_sink_reduce(const float* __restrict__ part, int64_t nch,
                                                     int Hn, float* __restrict__ grad_sink) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= Hn) return;
  float s = 0.f;
  for (int64_t c = 0; c < nch; ++c) s += part[(size_t)c * Hn + e];
  grad_sink[e] += s;
}

// Workspace: keys and group sums per slot (2*T*H*k each), the row counts
// (scanned in place into offsets, plus the total, plus the count of long
// segments), the scan's partials, the list of long segments, then the sort of
// up to 2*T*H*k pairs.
static size_t a256(size_t x) { return (x + 255) / 256 * 256; }
size_t search_backward_ws_bytes(int64_t T, int H, int k) {
  const int64_t rows = 2 * T * H;
  const int64_t np = rows * k;
  return 2 * a256((size_t)np * 4) + a256((size_t)(rows + 2) * 4) +
         a256(scan_scratch_u32(rows + 1) * 4) + a256((size_t)sbwd_max_long(np) * 4) +
         sorted_workspace_bytes(np);
}

template <typename T>
static hipError_t launch_sbwd(const void* q, const void* subkeys, int64_t T_, int H, int n, int S,
                              int k, int kst, const int64_t* idx, const float* gz,
                              const float2* qstats, const void* sink, float* grad_q, float* grad_K,
                              float* grad_sink, float* sink_part, void* ws, hipStream_t st) {
  LaunchTimer lt("search_backward", st);
  hipError_t e = hipSuccess;
  if (grad_sink) {
    const int64_t nch = sink_chunks(T_);
    hipLaunchKernelGGL(k_sink_partial<T>, dim3((unsigned)(nch * H)), dim3(256), 0, st, (const T*)q,
                       T_, H, n, kst, k, gz, sink_part);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int Hn = H * n;
    hipLaunchKernelGGL(k_sink_reduce, dim3((unsigned)((Hn + 255) / 256)), dim3(256), 0, st,
                       (const float*)sink_part, nch, Hn, grad_sink);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (!grad_q && !grad_K) return hipSuccess;
  const int64_t rows = 2 * T_ * H;
  const int64_t np = rows * k;
  char* p = reinterpret_cast<char*>(ws);
  uint32_t* keys = reinterpret_cast<uint32_t*>(p);
  p += a256((size_t)np * 4);
  float* gvals = reinterpret_cast<float*>(p);
  p += a256((size_t)np * 4);
  uint32_t* offs = reinterpret_cast<uint32_t*>(p);  // rows + 1, then the long count
  p += a256((size_t)(rows + 2) * 4);
  uint32_t* sums = reinterpret_cast<uint32_t*>(p);
  p += a256(scan_scratch_u32(rows + 1) * 4);
  uint32_t* long_list = reinterpret_cast<uint32_t*>(p);
  p += a256((size_t)sbwd_max_long(np) * 4);
  void* sort_ws = p;
  // the scan's last entry and the count of long segments
  if (grad_K) e = launch_fill_u32(offs + rows, 0u, 2, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_search_bwd_q<T>, dim3((unsigned)(((T_ + 3) / 4) * H)), dim3(256), 0, st,
                     (const T*)q, (const T*)subkeys, T_, H, n, S, k, kst, idx, gz,
                     grad_q ? (const T*)sink : nullptr, qstats, grad_q,
                     grad_K ? keys : nullptr, grad_K ? gvals : nullptr, grad_K ? offs : nullptr);
  e = hipGetLastError();
  if (e != hipSuccess || !grad_K) return e;
  // counts -> offsets; offs[rows] = number of leaders
  e = scan_exclusive_u32(offs, rows + 1, sums, st);
  if (e != hipSuccess) return e;
  uint32_t *kin, *vin;
  sort_u32_inputs(sort_ws, np, &kin, &vin);
  hipLaunchKernelGGL(k_sbwd_pack, dim3((unsigned)((np + 255) / 256)), dim3(256), 0, st, keys, offs,
                     rows, k, kin, vin);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const uint32_t nbins = (uint32_t)(2 * H) * (uint32_t)S;
  int key_bits = 1;
  while (key_bits < 32 && (uint64_t(1) << key_bits) < nbins) ++key_bits;
  const uint32_t *ks, *vs, *seg, *nseg;
  e = sort_u32_segments(np, offs + rows, key_bits, sort_ws, &ks, &vs, &seg, &nseg, st);
  if (e != hipSuccess) return e;
  int64_t maxseg = (int64_t)nbins < np ? (int64_t)nbins : np;
  uint32_t* long_cnt = offs + rows + 1;
  e = launch_list_long(seg, nseg, maxseg, SBWD_LONG, long_list, long_cnt, st);
  if (e != hipSuccess) return e;
  int64_t blocks = (maxseg + 3) / 4;
  if (blocks > 16384) blocks = 16384;
  int64_t lblocks = sbwd_max_long(np) < maxseg ? sbwd_max_long(np) : maxseg;
  if (lblocks > 256) lblocks = 256;
  if (qstats) {
    hipLaunchKernelGGL((k_sbwd_segments<T, true>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const T*)q, H, n, S, k, qstats, gvals, ks, vs, seg, nseg, grad_K);
    hipLaunchKernelGGL((k_sbwd_long<T, true>), dim3((unsigned)lblocks), dim3(64 * SBWD_LWAVES), 0,
                       st, (const T*)q, H, n, S, k, qstats, gvals, ks, vs, seg,
                       (const uint32_t*)long_list, (const uint32_t*)long_cnt, grad_K);
  } else {
    hipLaunchKernelGGL((k_sbwd_segments<T, false>), dim3((unsigned)blocks), dim3(256), 0, st,
                       (const T*)q, H, n, S, k, qstats, gvals, ks, vs, seg, nseg, grad_K);
    hipLaunchKernelGGL((k_sbwd_long<T, false>), dim3((unsigned)lblocks), dim3(64 * SBWD_LWAVES),
                       0, st, (const T*)q, H, n, S, k, qstats, gvals, ks, vs, seg,
                       (const uint32_t*)long_list, (const uint32_t*)long_cnt, grad_K);
  }
  return hipGetLastError();
}

hipError_t launch_search_backward(bool bf16, const void* q, const void* subkeys, int64_t T, int H,
                                  int n, int S, int k, int kst, const int64_t* idx, const float* gz,
                                  const float2* qstats, const void* sink, float* grad_q,
                                  float* grad_K, float* grad_sink, float* sink_part, void* ws,
                                  hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (bf16)
    return launch_sbwd<uint16_t>(q, subkeys, T, H, n, S, k, kst, idx, gz, qstats, sink, grad_q,
                                 grad_K, grad_sink, sink_part, ws, st);
  return launch_sbwd<float>(q, subkeys, T, H, n, S, k, kst, idx, gz, qstats, sink, grad_q, grad_K,
                            grad_sink, sink_part, ws, st);
}

}  // namespace pk
