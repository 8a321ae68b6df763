// Atomic-free EmbeddingBag backward on gfx950 ("reverse indices" of Sec. 3.1.4
// of "Memory Layers at Scale": invert the lookup -> row mapping so that each
// gradient row knows which lookups contribute to it).
//
//   1. Stable LSD radix sort of the L = T*H*k lookups by row: 8-bit digits,
//      per pass a tile histogram, a scan of each digit's tile counts (one
//      workgroup per digit), and a stable scatter: each wave ranks a
//      contiguous quarter of the tile with ballots, and the tile goes out
//      through LDS in sorted order.  Keys are rows (< 2^26), values lookup ids.
//   2. Segment heads (first lookup of each distinct row) -> seg_start[U + 1],
//      the head flags computed where they are counted and placed.
//   3. One lane group per touched row (two adjacent rows per iteration): read
//      the value row once, then take the contributing lookups in lookup order,
//      a few at a time with their dy rows loaded together, add w * dy into a
//      register accumulator and write grad_w = dy . V[row]; finally one
//      read-modify-write of the fp32 gradient row (dense) or one write of the
//      row's gradient (sparse).  Rows are visited in ascending order, so the
//      value and gradient tables are streamed nearly sequentially, and the
//      result is bitwise deterministic.
//   4. A row with more than LONG_SEG lookups would hold one lane group for
//      its whole length: k_list_long lists it, the per-row kernel skips it,
//      and a second kernel gives each listed row a workgroup whose lane
//      groups take contiguous runs of its lookups; their partial sums meet in
//      LDS and are added in group order (still deterministic).
#include "pk_device.h"
#include "pk_internal.h"

namespace pk {

constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;
constexpr int SORT_ITEMS = 16;                 // keys per thread per tile
constexpr int SORT_TILE = 256 * SORT_ITEMS;    // keys per workgroup tile
constexpr int SCAN_ITEMS = 8;
constexpr uint32_t LONG_SEG = 1024;  // lookups of a row beyond which it is split
constexpr uint32_t LONG_CHUNK = 1024;  // lookups of a long row per workgroup
constexpr int LONG_WAVES = 8;        // waves of the workgroup that takes a chunk
constexpr int SCAN_TILE = 256 * SCAN_ITEMS;

static inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// ------------------------------------------------------------------ scan ----
// Exclusive prefix sum of u32, any length, in three launches.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* wsum, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < WAVE; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, WAVE);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  uint32_t before = 0;
  for (int w = 0; w < wave; ++w) before += wsum[w];
  total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
  __syncthreads();
  return before + x - v;
}

__global__ __launch_bounds__(256) void k_scan_reduce(const uint32_t* __restrict__ in, int64_t n,
                                                     uint32_t* __restrict__ sums) {
  __shared__ uint32_t wsum[4];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i)
    if (base + i < n) s += in[base + i];
  uint32_t total;
  block_exclusive_scan(s, wsum, total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Single workgroup: exclusive scan of the tile sums, in place, any count.
__global__ __launch_bounds__(256) void k_scan_top(uint32_t* __restrict__ sums, int64_t nb) {
  __shared__ uint32_t wsum[4];
  uint32_t carry = 0;
  for (int64_t base = 0; base < nb; base += SCAN_TILE) {
    const int64_t b0 = base + threadIdx.x * SCAN_ITEMS;
    uint32_t v[SCAN_ITEMS];
    uint32_t s = 0;
#pragma unroll
    for (int i = 0; i < SCAN_ITEMS; ++i) {
      v[i] = (b0 + i < nb) ? sums[b0 + i] : 0u;
      s += v[i];
    }
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan(s, wsum, total);
#pragma unroll
    for (int i = 0; i < SCAN_ITEMS; ++i) {
      if (b0 + i < nb) sums[b0 + i] = run;
      run += v[i];
    }
    carry += total;
  }
}

__global__ __launch_bounds__(256) void k_scan_down(const uint32_t* __restrict__ in,
                                                   uint32_t* __restrict__ out, int64_t n,
                                                   const uint32_t* __restrict__ sums) {
  __shared__ uint32_t wsum[4];
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
  uint32_t v[SCAN_ITEMS];
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    v[i] = (base + i < n) ? in[base + i] : 0u;
    s += v[i];
  }
  uint32_t total;
  uint32_t run = sums[blockIdx.x] + block_exclusive_scan(s, wsum, total);
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    if (base + i < n) out[base + i] = run;
    run += v[i];
  }
}

static hipError_t exclusive_scan(uint32_t* data, int64_t n, uint32_t* sums, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t nb = cdiv(n, SCAN_TILE);
  hipLaunchKernelGGL(k_scan_reduce, dim3((unsigned)nb), dim3(256), 0, st, data, n, sums);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(256), 0, st, sums, nb);
  hipLaunchKernelGGL(k_scan_down, dim3((unsigned)nb), dim3(256), 0, st, data, data, n, sums);
  return hipGetLastError();
}

// Per digit d (one workgroup each) of a radix pass: exclusive scan, in place,
// of the tile counts hist[d*nblk .. (d+1)*nblk) (digit-major), and the digit's
// total in totals[d]; the scatter adds the digits' bases (a scan of totals).
__global__ __launch_bounds__(256) void k_scan_digits(uint32_t* __restrict__ hist, int64_t nblk,
                                                     uint32_t* __restrict__ totals) {
  __shared__ uint32_t wsum[4];
  uint32_t* h = hist + (int64_t)blockIdx.x * nblk;
  uint32_t carry = 0;
  for (int64_t base = 0; base < nblk; base += SCAN_TILE) {
    const int64_t i0 = base + (int64_t)threadIdx.x * SCAN_ITEMS;
    uint32_t v[SCAN_ITEMS];
    uint32_t sum = 0;
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
      v[j] = (i0 + j < nblk) ? h[i0 + j] : 0u;
      sum += v[j];
    }
    uint32_t total;
    uint32_t run = carry + block_exclusive_scan(sum, wsum, total);
#pragma unroll
    for (int j = 0; j < SCAN_ITEMS; ++j) {
      if (i0 + j < nblk) h[i0 + j] = run;
      run += v[j];
    }
    carry += total;
  }
  if (threadIdx.x == 0) totals[blockIdx.x] = carry;
}

// ----------------------------------------------------------- radix sort ----
// KM selects where a pass takes its items: SRC_I64 and SRC_U32 are first
// passes (keys from an int64 or u32 array, values = item positions), SRC_NEXT
// a later pass (keys and values from the previous pass's output).
constexpr int SRC_I64 = 0, SRC_U32 = 1, SRC_NEXT = 2;

template <int KM>
__device__ __forceinline__ uint32_t sort_key(const void* keys, int64_t i) {
  if constexpr (KM == SRC_I64) return (uint32_t)reinterpret_cast<const int64_t*>(keys)[i];
  else return reinterpret_cast<const uint32_t*>(keys)[i];
}

template <int KM>
__global__ __launch_bounds__(256) void k_radix_hist(const void* __restrict__ keys, int64_t Lmax,
                                                    const uint32_t* __restrict__ Ldev, int shift,
                                                    int bits, int64_t nblk,
                                                    uint32_t* __restrict__ hist) {
  const int64_t L = (Ldev && (int64_t)*Ldev < Lmax) ? (int64_t)*Ldev : Lmax;
  if ((int64_t)blockIdx.x * SORT_TILE >= L) {  // a tile past the count: empty
    hist[(int64_t)threadIdx.x * nblk + blockIdx.x] = 0u;
    return;
  }
  __shared__ uint32_t h[RADIX];
  h[threadIdx.x] = 0;
  __syncthreads();
  const uint32_t mask = (1u << bits) - 1u;
  const int64_t tile = (int64_t)blockIdx.x * SORT_TILE;
#pragma unroll 4
  for (int i = 0; i < SORT_ITEMS; ++i) {
    const int64_t pos = tile + i * 256 + threadIdx.x;
    if (pos < L) atomicAdd(&h[(sort_key<KM>(keys, pos) >> shift) & mask], 1u);
  }
  __syncthreads();
  hist[(int64_t)threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one radix pass.  Wave w of the workgroup ranks the w-th
// quarter of the tile (positions in order: 16 rounds of 64), each key's rank
// within its digit coming from ballots and the wave's own digit counters in
// LDS (a wave's LDS accesses stay in program order, so no barrier is needed
// between rounds).  One block scan then gives each digit's start in the tile
// and each wave's start within the digit; the tile is written to LDS in
// sorted order and from there to its digits' runs, consecutive threads
// writing consecutive addresses.  Keys of equal digit keep their order.
template <int KM>
__global__ __launch_bounds__(256) void k_radix_scatter(const void* __restrict__ keys_in,
                                                       const uint32_t* __restrict__ vals_in,
                                                       int64_t Lmax,
                                                       const uint32_t* __restrict__ Ldev, int shift,
                                                       int bits, int64_t nblk,
                                                       const uint32_t* __restrict__ offsets,
                                                       const uint32_t* __restrict__ totals,
                                                       uint32_t* __restrict__ keys_out,
                                                       uint32_t* __restrict__ vals_out) {
  constexpr int PER_WAVE = SORT_TILE / 4;  // contiguous keys ranked by one wave
  constexpr int ROUNDS = PER_WAVE / WAVE;
  const int64_t L = (Ldev && (int64_t)*Ldev < Lmax) ? (int64_t)*Ldev : Lmax;
  const int64_t tile = (int64_t)blockIdx.x * SORT_TILE;
  if (tile >= L) return;  // whole block: nothing to move
  __shared__ uint32_t run[RADIX];      // global start of each digit's run for this tile
  __shared__ uint32_t tstart[RADIX];   // start of each digit within the tile
  __shared__ uint32_t wcnt[4][RADIX];  // per-wave digit counts, then per-wave starts
  __shared__ uint32_t wsum[4];
  __shared__ uint32_t skey[SORT_TILE];
  __shared__ uint32_t sval[SORT_TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  {  // thread tid = digit: where the digit starts overall, plus this tile's offset in it
    uint32_t all;
    const uint32_t dbase = block_exclusive_scan(totals[tid], wsum, all);
    run[tid] = dbase + offsets[(int64_t)tid * nblk + blockIdx.x];
  }
#pragma unroll
  for (int w = 0; w < 4; ++w) wcnt[w][tid] = 0;
  __syncthreads();
  const uint32_t mask = (1u << bits) - 1u;
  const uint64_t below = (1ull << lane) - 1ull;
  const int64_t wbase = tile + (int64_t)wave * PER_WAVE;
  uint32_t key[ROUNDS], val[ROUNDS], rk[ROUNDS];
#pragma unroll
  for (int i = 0; i < ROUNDS; ++i) {
    const int64_t pos = wbase + i * WAVE + lane;
    const bool valid = pos < L;
    key[i] = valid ? sort_key<KM>(keys_in, pos) : 0u;
    val[i] = valid ? (KM != SRC_NEXT ? (uint32_t)pos : vals_in[pos]) : 0u;
    const uint32_t dig = (key[i] >> shift) & mask;
    uint64_t peers = __ballot(valid);
    for (int b = 0; b < bits; ++b) {
      const bool bit = (dig >> b) & 1u;
      const uint64_t set = __ballot(bit);
      peers &= bit ? set : ~set;
    }
    const uint32_t r = (uint32_t)__popcll(peers & below);
    rk[i] = wcnt[wave][dig] + r;  // keys of this digit in the wave's earlier rounds, then lanes
    if (valid && r == 0) wcnt[wave][dig] += (uint32_t)__popcll(peers);
  }
  __syncthreads();
  {  // thread tid = digit: the tile's digit starts and each wave's start within it
    const uint32_t c0 = wcnt[0][tid], c1 = wcnt[1][tid], c2 = wcnt[2][tid], c3 = wcnt[3][tid];
    uint32_t total;
    const uint32_t st = block_exclusive_scan(c0 + c1 + c2 + c3, wsum, total);
    tstart[tid] = st;
    wcnt[0][tid] = st;
    wcnt[1][tid] = st + c0;
    wcnt[2][tid] = st + c0 + c1;
    wcnt[3][tid] = st + c0 + c1 + c2;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < ROUNDS; ++i) {
    const int64_t pos = wbase + i * WAVE + lane;
    if (pos < L) {
      const uint32_t p = wcnt[wave][(key[i] >> shift) & mask] + rk[i];
      skey[p] = key[i];
      sval[p] = val[i];
    }
  }
  __syncthreads();
  const int64_t left = L - tile;
  const int n = left < SORT_TILE ? (int)left : SORT_TILE;
  for (int e = tid; e < n; e += 256) {
    const uint32_t kk = skey[e];
    const uint32_t dig = (kk >> shift) & mask;
    const uint32_t dst = run[dig] + (uint32_t)e - tstart[dig];
    keys_out[dst] = kk;
    vals_out[dst] = sval[e];
  }
}

// ------------------------------------------------------------- segments ----
// Segment heads of the sorted keys (i == 0 or keys[i] != keys[i-1]), counted
// per scan tile (thread: SCAN_ITEMS consecutive keys); k_scan_top then turns
// the counts into each tile's first segment number.
__global__ __launch_bounds__(256) void k_seg_count(const uint32_t* __restrict__ keys, int64_t Lmax,
                                                   const uint32_t* __restrict__ Ldev,
                                                   uint32_t* __restrict__ sums) {
  __shared__ uint32_t wsum[4];
  const int64_t L = (Ldev && (int64_t)*Ldev < Lmax) ? (int64_t)*Ldev : Lmax;
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
  uint32_t prev = (base > 0 && base <= L) ? keys[base - 1] : 0u;
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    const int64_t x = base + i;
    if (x < L) {
      const uint32_t kx = keys[x];
      s += (x == 0 || kx != prev) ? 1u : 0u;
      prev = kx;
    }
  }
  uint32_t total;
  block_exclusive_scan(s, wsum, total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Each head i, with u = the number of heads before it, writes seg_start[u] = i;
// the last item writes seg_start[U] = L and U (the number of segments).
__global__ __launch_bounds__(256) void k_seg_place(const uint32_t* __restrict__ keys, int64_t Lmax,
                                                   const uint32_t* __restrict__ Ldev,
                                                   const uint32_t* __restrict__ sums,
                                                   uint32_t* __restrict__ seg_start,
                                                   uint32_t* __restrict__ nseg) {
  __shared__ uint32_t wsum[4];
  const int64_t L = (Ldev && (int64_t)*Ldev < Lmax) ? (int64_t)*Ldev : Lmax;
  const int64_t base = (int64_t)blockIdx.x * SCAN_TILE + threadIdx.x * SCAN_ITEMS;
  uint32_t prev = (base > 0 && base <= L) ? keys[base - 1] : 0u;
  bool head[SCAN_ITEMS];
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    const int64_t x = base + i;
    head[i] = false;
    if (x < L) {
      const uint32_t kx = keys[x];
      head[i] = (x == 0 || kx != prev);
      prev = kx;
    }
    s += head[i] ? 1u : 0u;
  }
  uint32_t total;
  uint32_t run = sums[blockIdx.x] + block_exclusive_scan(s, wsum, total);
#pragma unroll
  for (int i = 0; i < SCAN_ITEMS; ++i) {
    const int64_t x = base + i;
    if (head[i]) seg_start[run] = (uint32_t)x;
    run += head[i] ? 1u : 0u;
    if (x == L - 1) {
      seg_start[run] = (uint32_t)L;
      *nseg = run;
    }
  }
}


// ------------------------------------------------------- per-row backward ----
// One lane group per touched row.  A row with more than LONG_SEG lookups is
// taken as empty here (its gradient row is written back unchanged, or as zero
// in the sparse form) and summed afterwards by k_bag_bwd_long, in stream
// order.  Value and gradient rows are streamed once
// per step with non-temporal accesses, so they do not push the re-read dy rows
// and metadata out of the caches.  A lane group takes SB adjacent segments per
// iteration (loads of all of them, then all of their gradient-row stores: one
// longer read burst and one contiguous write burst), with the next batch's
// bounds prefetched; the old gradient row is read into the accumulator
// together with the value row.
// Lookups of a segment taken together: more for narrow rows (fewer registers
// per dy row), capped by the lane group's width.
template <int NQ, int CL>
struct RowsBatch {
  static constexpr int raw = NQ >= 16 ? 1 : (NQ >= 8 ? 2 : (NQ >= 4 ? 4 : 8));
  static constexpr int value = raw < CL ? raw : CL;
};

template <typename V, int NQ, int CL, bool SPARSE, int SB>
__global__ __launch_bounds__(256) void k_bag_bwd_rows(
    const V* __restrict__ dy, const V* __restrict__ values, int D, const float* __restrict__ w,
    int bag, const uint32_t* __restrict__ rows_sorted, const uint32_t* __restrict__ lookups,
    const uint32_t* __restrict__ seg_start, const uint32_t* __restrict__ nseg,
    float* __restrict__ grad_values, int64_t* __restrict__ rows_out,
    float* __restrict__ grad_rows_out, float* __restrict__ grad_w) {
  using Q = Quad<V>;
  constexpr int G = WAVE / CL;
  constexpr int PB = RowsBatch<NQ, CL>::value;
  const int lane = threadIdx.x & 63;
  const int grp = lane / CL, cl = lane % CL;
  const int nquad = D / 4;
  const int64_t U = *nseg;
  const bool dense = !SPARSE && grad_values != nullptr;
  bool ok[NQ];
#pragma unroll
  for (int m = 0; m < NQ; ++m) ok[m] = (m * CL + cl) < nquad;

  const int64_t step = (int64_t)gridDim.x * 4 * G * SB;
  int64_t u0 = (((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * G + grp) * SB;
  uint32_t s0[SB], s1[SB];
  int64_t row[SB];
#pragma unroll
  for (int b = 0; b < SB; ++b) {
    const bool live = u0 + b < U;
    s0[b] = live ? seg_start[u0 + b] : 0;
    s1[b] = live ? seg_start[u0 + b + 1] : 0;
    if (s1[b] - s0[b] > LONG_SEG) s1[b] = s0[b];  // summed by k_bag_bwd_long
    row[b] = live ? (int64_t)rows_sorted[s0[b]] : 0;
  }
  while (u0 < U) {
    typename Q::raw vraw[SB][NQ];
    float acc[SB][NQ][4];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
      const bool live = u0 + b < U;
#pragma unroll
      for (int m = 0; m < NQ; ++m) {
        const size_t e0 = (size_t)(m * CL + cl) * 4;
        vraw[b][m] = (ok[m] && live) ? Q::load_nt(values + row[b] * D + e0) : Q::zero();
        const uint4 g = (ok[m] && dense && live)
                            ? ld16_hint<PK_GRAD_NT_LOAD>(grad_values + row[b] * D + e0)
                            : uint4{0, 0, 0, 0};
        acc[b][m][0] = __uint_as_float(g.x); acc[b][m][1] = __uint_as_float(g.y);
        acc[b][m][2] = __uint_as_float(g.z); acc[b][m][3] = __uint_as_float(g.w);
      }
    }
    const int64_t un = u0 + step;
    uint32_t s0n[SB], s1n[SB];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
      const bool live = un + b < U;
      s0n[b] = live ? seg_start[un + b] : 0;
      s1n[b] = live ? seg_start[un + b + 1] : 0;
      if (s1n[b] - s0n[b] > LONG_SEG) s1n[b] = s0n[b];
    }
#pragma unroll
    for (int b = 0; b < SB; ++b) {
      // The segment's lookups PB at a time: the group's lanes read PB lookup
      // ids and weights with one load each, then all PB dy rows are in flight
      // before the first is accumulated (lookup order is kept).
      // The next batch's lookup ids are loaded while this batch's dy rows are
      // in flight, so a long segment costs one dependent round trip per batch.
      uint32_t lid_next = (uint32_t)cl < s1[b] - s0[b] ? lookups[s0[b] + cl] : 0u;
      for (uint32_t s = s0[b]; s < s1[b]; s += PB) {
        const uint32_t nb = (s1[b] - s) < (uint32_t)PB ? (s1[b] - s) : (uint32_t)PB;
        const uint32_t lid = lid_next;
        const float wl = (uint32_t)cl < nb ? w[lid] : 0.f;
        lid_next = (uint32_t)cl + PB < s1[b] - s ? lookups[s + PB + cl] : 0u;
        typename Q::raw graw[PB][NQ];
        uint32_t lp[PB];
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) {
          lp[pp] = __shfl(lid, pp, CL);
          const int64_t t = lp[pp] / (uint32_t)bag;
#pragma unroll
          for (int m = 0; m < NQ; ++m)
            graw[pp][m] = (ok[m] && (uint32_t)pp < nb) ? Q::load(dy + t * D + (size_t)(m * CL + cl) * 4)
                                                       : Q::zero();
        }
        float part[PB];
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) {
          const float ww = __shfl(wl, pp, CL);
          part[pp] = 0.f;
#pragma unroll
          for (int m = 0; m < NQ; ++m) {
            float g[4], v[4];
            Q::unpack(graw[pp][m], g);
            Q::unpack(vraw[b][m], v);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              acc[b][m][e] = fmaf(ww, g[e], acc[b][m][e]);
              part[pp] = fmaf(g[e], v[e], part[pp]);
            }
          }
        }
#pragma unroll
        for (int pp = 0; pp < PB; ++pp) part[pp] = group_sum<CL>(part[pp]);
        float mine = part[0];
#pragma unroll
        for (int pp = 1; pp < PB; ++pp) mine = (cl == pp) ? part[pp] : mine;
        if ((uint32_t)cl < nb) grad_w[lid] = mine;
      }
    }
    int64_t rown[SB];
#pragma unroll
    for (int b = 0; b < SB; ++b) rown[b] = (un + b < U) ? (int64_t)rows_sorted[s0n[b]] : 0;
    if (SPARSE || dense) {
#pragma unroll
      for (int b = 0; b < SB; ++b) {
        if (u0 + b >= U) continue;
        float* dst = SPARSE ? grad_rows_out + (size_t)(u0 + b) * D : grad_values + row[b] * D;
#pragma unroll
        for (int m = 0; m < NQ; ++m)
          if (ok[m])
            st16_hint<PK_GRAD_NT_STORE>(dst + (size_t)(m * CL + cl) * 4,
                                        uint4{__float_as_uint(acc[b][m][0]), __float_as_uint(acc[b][m][1]),
                                              __float_as_uint(acc[b][m][2]), __float_as_uint(acc[b][m][3])});
      }
    }
    if (SPARSE && cl == 0) {
#pragma unroll
      for (int b = 0; b < SB; ++b)
        if (u0 + b < U) rows_out[u0 + b] = row[b];
    }
    u0 = un;
#pragma unroll
    for (int b = 0; b < SB; ++b) {
      s0[b] = s0n[b];
      s1[b] = s1n[b];
      row[b] = rown[b];
    }
  }
}

// -------------------------------------------------------------- launcher ----
struct SortedWs {
  uint32_t *keys_a, *vals_a, *keys_b, *vals_b, *hist, *sums, *seg, *misc, *long_list, *totals,
      *long_base;
};
static int64_t max_long(int64_t L) { return L / LONG_SEG + 1; }

static SortedWs carve(void* ws, int64_t L) {
  const int64_t nblk = cdiv(L, SORT_TILE);
  const int64_t hist_n = (int64_t)RADIX * nblk;
  const int64_t scan_n = (hist_n > L + 1 ? hist_n : L + 1);
  char* p = reinterpret_cast<char*>(ws);
  SortedWs w;
  auto take = [&](size_t bytes) { uint32_t* r = reinterpret_cast<uint32_t*>(p); p += align256(bytes); return r; };
  w.keys_a = take(4 * (size_t)L);
  w.vals_a = take(4 * (size_t)L);
  w.keys_b = take(4 * (size_t)L);
  w.vals_b = take(4 * (size_t)L);
  w.hist = take(4 * (size_t)scan_n);
  w.sums = take(4 * (size_t)(cdiv(scan_n, SCAN_TILE) + 1));
  w.seg = take(4 * (size_t)(L + 1));
  w.misc = take(256);  // [0] segments, [1] long rows listed
  w.long_list = take(4 * (size_t)max_long(L));
  w.totals = take(4 * (size_t)RADIX);  // a radix pass's count per digit
  w.long_base = take(4 * (size_t)(max_long(L) + 1));  // first chunk of each listed long row
  return w;
}

size_t sorted_workspace_bytes(int64_t L) {
  const int64_t nblk = cdiv(L, SORT_TILE);
  const int64_t hist_n = (int64_t)RADIX * nblk;
  const int64_t scan_n = (hist_n > L + 1 ? hist_n : L + 1);
  return 4 * align256(4 * (size_t)L) + align256(4 * (size_t)scan_n) +
         align256(4 * (size_t)(cdiv(scan_n, SCAN_TILE) + 1)) + align256(4 * (size_t)(L + 1)) + 256 +
         align256(4 * (size_t)max_long(L)) + align256(4 * (size_t)RADIX) +
         align256(4 * (size_t)(max_long(L) + 1));
}

// Partial rows of the long-row chunks: at most L / LONG_CHUNK + max_long(L)
// chunks of D fp32 each.
size_t long_partial_bytes(int64_t L, int D) {
  return align256((size_t)(L / LONG_CHUNK + max_long(L)) * (size_t)D * sizeof(float));
}

// Stable LSD radix sort of L keys (< 2^key_bits, from an int64 or a u32 array)
// with their positions as values, then the segment starts of equal keys:
// seg[0..U] in b.seg, U in b.misc[0].  *ks / *vs receive the sorted arrays.
// L is the item count, or its upper bound when Ldev (device memory) holds the
// count; vals_in, if given, are the first pass's values (else positions).
static hipError_t sort_segments(const void* keys, bool key64, int64_t L, int key_bits,
                                const SortedWs& b, const uint32_t** ks, const uint32_t** vs,
                                hipStream_t st, const uint32_t* vals_in = nullptr,
                                const uint32_t* Ldev = nullptr) {
  hipError_t e = hipSuccess;
  const int64_t nblk = cdiv(L, SORT_TILE);
  const void* kin = keys;
  const uint32_t* vin = vals_in;
  uint32_t *kout = b.keys_a, *vout = b.vals_a;
  for (int shift = 0, pass = 0; shift < key_bits; shift += RADIX_BITS, ++pass) {
    const int bits = (key_bits - shift) < RADIX_BITS ? (key_bits - shift) : RADIX_BITS;
    const dim3 g((unsigned)nblk), blk(256);
    if (pass > 0 || vals_in)
      hipLaunchKernelGGL(k_radix_hist<SRC_NEXT>, g, blk, 0, st, kin, L, Ldev, shift, bits, nblk, b.hist);
    else if (key64)
      hipLaunchKernelGGL(k_radix_hist<SRC_I64>, g, blk, 0, st, kin, L, Ldev, shift, bits, nblk, b.hist);
    else
      hipLaunchKernelGGL(k_radix_hist<SRC_U32>, g, blk, 0, st, kin, L, Ldev, shift, bits, nblk, b.hist);
    hipLaunchKernelGGL(k_scan_digits, dim3(RADIX), blk, 0, st, b.hist, nblk, b.totals);
    if (pass > 0 || vals_in)
      hipLaunchKernelGGL(k_radix_scatter<SRC_NEXT>, g, blk, 0, st, kin, vin, L, Ldev, shift, bits, nblk, b.hist, b.totals, kout, vout);
    else if (key64)
      hipLaunchKernelGGL(k_radix_scatter<SRC_I64>, g, blk, 0, st, kin, vin, L, Ldev, shift, bits, nblk, b.hist, b.totals, kout, vout);
    else
      hipLaunchKernelGGL(k_radix_scatter<SRC_U32>, g, blk, 0, st, kin, vin, L, Ldev, shift, bits, nblk, b.hist, b.totals, kout, vout);
    kin = kout;
    vin = vout;
    if (kout == b.keys_a) { kout = b.keys_b; vout = b.vals_b; }
    else { kout = b.keys_a; vout = b.vals_a; }
  }
  *ks = reinterpret_cast<const uint32_t*>(kin);
  *vs = vin;
  const int64_t nb = cdiv(L, SCAN_TILE);
  hipLaunchKernelGGL(k_seg_count, dim3((unsigned)nb), dim3(256), 0, st, *ks, L, Ldev, b.sums);
  hipLaunchKernelGGL(k_scan_top, dim3(1), dim3(256), 0, st, b.sums, nb);
  hipLaunchKernelGGL(k_seg_place, dim3((unsigned)nb), dim3(256), 0, st, *ks, L, Ldev, b.sums, b.seg,
                     b.misc);
  return hipGetLastError();
}

// Sort of u32 keys with u32 values for other kernels of the library: up to
// Lmax items, their count in device memory (*Ldev).  The input arrays must be
// the ones sort_u32_inputs returns for this workspace (the first radix pass
// reads them, the second overwrites them).
void sort_u32_inputs(void* ws, int64_t Lmax, uint32_t** keys_in, uint32_t** vals_in) {
  SortedWs b = carve(ws, Lmax);
  *keys_in = b.keys_b;
  *vals_in = b.vals_b;
}

hipError_t sort_u32_segments(int64_t Lmax, const uint32_t* Ldev, int key_bits, void* ws,
                             const uint32_t** ks, const uint32_t** vs, const uint32_t** seg,
                             const uint32_t** nseg, hipStream_t st) {
  SortedWs b = carve(ws, Lmax);
  *seg = b.seg;
  *nseg = b.misc;
  hipError_t e = launch_fill_u32(b.misc, 0u, 1, st);
  if (e != hipSuccess || Lmax == 0) return e;
  return sort_segments(b.keys_b, false, Lmax, key_bits, b, ks, vs, st, b.vals_b, Ldev);
}

// Exclusive prefix sum of n u32 in place; sums needs scan_scratch_u32(n) entries.
size_t scan_scratch_u32(int64_t n) { return (size_t)(cdiv(n, SCAN_TILE) + 1); }
hipError_t scan_exclusive_u32(uint32_t* data, int64_t n, uint32_t* sums, hipStream_t st) {
  return exclusive_scan(data, n, sums, st);
}

// Segments longer than LONG_SEG lookups, listed (in no particular order: each
// is then summed on its own) for k_bag_bwd_long; k_bag_bwd_rows skips them.
__global__ __launch_bounds__(256) void k_list_long(const uint32_t* __restrict__ seg_start,
                                                   const uint32_t* __restrict__ nseg,
                                                   uint32_t thresh,
                                                   uint32_t* __restrict__ long_list,
                                                   uint32_t* __restrict__ long_cnt) {
  const uint32_t U = *nseg;
  for (uint32_t u = blockIdx.x * 256 + threadIdx.x; u < U; u += gridDim.x * 256)
    if (seg_start[u + 1] - seg_start[u] > thresh) long_list[atomicAdd(long_cnt, 1u)] = u;
}

hipError_t launch_list_long(const uint32_t* seg_start, const uint32_t* nseg, int64_t max_seg,
                            uint32_t thresh, uint32_t* long_list, uint32_t* long_cnt,
                            hipStream_t st) {
  int64_t gb = cdiv(max_seg, 256);
  if (gb > 2048) gb = 2048;
  if (gb < 1) gb = 1;
  hipLaunchKernelGGL(k_list_long, dim3((unsigned)gb), dim3(256), 0, st, seg_start, nseg, thresh,
                     long_list, long_cnt);
  return hipGetLastError();
}

// Rows listed by k_list_long (more than LONG_SEG lookups) are cut into chunks
// of LONG_CHUNK consecutive lookups (in lookup order), and every chunk of
// every listed row is summed by a workgroup of its own, so a row chosen by a
// large share of the tokens is spread over many CUs:
//   k_long_bases    (one workgroup) the first chunk number of each listed row
//                   (an exclusive scan of the chunk counts, in list order),
//   k_bag_bwd_long  (persistent grid over the chunks) the chunk's lane groups
//                   take contiguous runs of its lookups, write their grad_w and
//                   sum w * dy into partial rows in LDS, added in group order
//                   into the chunk's partial row in the workspace,
//   k_long_reduce   (one workgroup per listed row) adds the row's partial rows
//                   in chunk order to the old gradient row (dense) or writes
//                   their sum as the row's gradient (sparse).
// The list's order varies from run to run, but a row's value depends only on
// its own chunks, summed in chunk order: bitwise deterministic.
__global__ __launch_bounds__(256) void k_long_bases(const uint32_t* __restrict__ seg_start,
                                                    const uint32_t* __restrict__ long_list,
                                                    const uint32_t* __restrict__ long_cnt,
                                                    uint32_t* __restrict__ long_base) {
  __shared__ uint32_t wsum[4];
  const uint32_t nlong = *long_cnt;
  uint32_t carry = 0;
  for (uint32_t i0 = 0; i0 < nlong; i0 += 256) {
    const uint32_t i = i0 + threadIdx.x;
    uint32_t nch = 0;
    if (i < nlong) {
      const uint32_t u = long_list[i];
      nch = (seg_start[u + 1] - seg_start[u] + LONG_CHUNK - 1) / LONG_CHUNK;
    }
    uint32_t total;
    const uint32_t before = block_exclusive_scan(nch, wsum, total);
    if (i < nlong) long_base[i] = carry + before;
    carry += total;
  }
  if (threadIdx.x == 0) long_base[nlong] = carry;
}

template <typename V, int NQ, int CL>
__global__ __launch_bounds__(64 * LONG_WAVES) void k_bag_bwd_long(
    const V* __restrict__ dy, const V* __restrict__ values, int D, const float* __restrict__ w,
    int bag, const uint32_t* __restrict__ rows_sorted, const uint32_t* __restrict__ lookups,
    const uint32_t* __restrict__ seg_start, const uint32_t* __restrict__ long_list,
    const uint32_t* __restrict__ long_cnt, const uint32_t* __restrict__ long_base,
    float* __restrict__ part, float* __restrict__ grad_w) {
  using Q = Quad<V>;
  constexpr int G = WAVE / CL;
  constexpr int PB = RowsBatch<NQ, CL>::value;
  extern __shared__ float lpart[];  // [ng][D]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = wave * G + lane / CL, cl = lane % CL;
  const int nquad = D / 4;
  int ng = LONG_WAVES * G;
  if (ng > 16384 / D) ng = 16384 / D;  // 64 KiB of partial rows
  const bool mine = grp < ng;
  bool ok[NQ];
#pragma unroll
  for (int m = 0; m < NQ; ++m) ok[m] = mine && (m * CL + cl) < nquad;
  const uint32_t nlong = *long_cnt;
  const uint32_t nchunk = long_base[nlong];
  for (uint32_t g = blockIdx.x; g < nchunk; g += gridDim.x) {
    // the listed row holding chunk g: long_base is ascending
    uint32_t lo = 0, hi = nlong;  // long_base[lo] <= g < long_base[hi]
    while (hi - lo > 1) {
      const uint32_t mid = (lo + hi) >> 1;
      if (long_base[mid] <= g) lo = mid;
      else hi = mid;
    }
    const uint32_t u = long_list[lo];
    const uint32_t c = g - long_base[lo];
    const uint32_t s_end = seg_start[u + 1];
    const uint32_t c0 = seg_start[u] + c * LONG_CHUNK;
    const uint32_t c1 = c0 + LONG_CHUNK < s_end ? c0 + LONG_CHUNK : s_end;
    const int64_t row = (int64_t)rows_sorted[c0];
    const uint32_t len = c1 - c0;
    const uint32_t per = (len + (uint32_t)ng - 1) / (uint32_t)ng;
    uint32_t a = mine ? (uint32_t)grp * per : len, z = mine ? (uint32_t)(grp + 1) * per : len;
    a = (a < len ? a : len) + c0;
    z = (z < len ? z : len) + c0;
    typename Q::raw vraw[NQ];
    float acc[NQ][4];
#pragma unroll
    for (int m = 0; m < NQ; ++m) {
      vraw[m] = ok[m] ? Q::load(values + row * D + (size_t)(m * CL + cl) * 4) : Q::zero();
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[m][e] = 0.f;
    }
    for (uint32_t s = a; s < z; s += PB) {
      const uint32_t nb = (z - s) < (uint32_t)PB ? (z - s) : (uint32_t)PB;
      const uint32_t lid = (uint32_t)cl < nb ? lookups[s + cl] : 0u;
      const float wl = (uint32_t)cl < nb ? w[lid] : 0.f;
      typename Q::raw graw[PB][NQ];
#pragma unroll
      for (int pp = 0; pp < PB; ++pp) {
        const uint32_t lp = __shfl(lid, pp, CL);
        const int64_t t = lp / (uint32_t)bag;
#pragma unroll
        for (int m = 0; m < NQ; ++m)
          graw[pp][m] = (ok[m] && (uint32_t)pp < nb) ? Q::load(dy + t * D + (size_t)(m * CL + cl) * 4)
                                                     : Q::zero();
      }
      float part_w[PB];
#pragma unroll
      for (int pp = 0; pp < PB; ++pp) {
        const float ww = __shfl(wl, pp, CL);
        part_w[pp] = 0.f;
#pragma unroll
        for (int m = 0; m < NQ; ++m) {
          float gg[4], v[4];
          Q::unpack(graw[pp][m], gg);
          Q::unpack(vraw[m], v);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[m][e] = fmaf(ww, gg[e], acc[m][e]);
            part_w[pp] = fmaf(gg[e], v[e], part_w[pp]);
          }
        }
      }
#pragma unroll
      for (int pp = 0; pp < PB; ++pp) part_w[pp] = group_sum<CL>(part_w[pp]);
      float gwv = part_w[0];
#pragma unroll
      for (int pp = 1; pp < PB; ++pp) gwv = (cl == pp) ? part_w[pp] : gwv;
      if ((uint32_t)cl < nb) grad_w[lid] = gwv;
    }
#pragma unroll
    for (int m = 0; m < NQ; ++m)
      if (ok[m]) {
        float* d = lpart + (size_t)grp * D + (size_t)(m * CL + cl) * 4;
        d[0] = acc[m][0]; d[1] = acc[m][1]; d[2] = acc[m][2]; d[3] = acc[m][3];
      }
    __syncthreads();
    for (int qd = threadIdx.x; qd < nquad; qd += blockDim.x) {
      float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int gi = 0; gi < ng; ++gi) {
        const float* sp = lpart + (size_t)gi * D + (size_t)qd * 4;
        tot.x += sp[0]; tot.y += sp[1]; tot.z += sp[2]; tot.w += sp[3];
      }
      *reinterpret_cast<float4*>(part + (size_t)g * D + (size_t)qd * 4) = tot;
    }
    __syncthreads();  // the LDS partial rows are reused for the next chunk
  }
}

template <bool SPARSE>
__global__ __launch_bounds__(256) void k_long_reduce(int D, const uint32_t* __restrict__ rows_sorted,
                                                     const uint32_t* __restrict__ seg_start,
                                                     const uint32_t* __restrict__ long_list,
                                                     const uint32_t* __restrict__ long_cnt,
                                                     const uint32_t* __restrict__ long_base,
                                                     const float* __restrict__ part,
                                                     float* __restrict__ grad_values,
                                                     int64_t* __restrict__ rows_out,
                                                     float* __restrict__ grad_rows_out) {
  const uint32_t nlong = *long_cnt;
  const int nquad = D / 4;
  const bool dense = !SPARSE && grad_values != nullptr;
  for (uint32_t i = blockIdx.x; i < nlong; i += gridDim.x) {
    const uint32_t u = long_list[i];
    const int64_t row = (int64_t)rows_sorted[seg_start[u]];
    const uint32_t b0 = long_base[i], b1 = long_base[i + 1];
    for (int qd = threadIdx.x; qd < nquad; qd += blockDim.x) {
      float4 tot = make_float4(0.f, 0.f, 0.f, 0.f);
      if (dense) tot = *reinterpret_cast<const float4*>(grad_values + row * D + (size_t)qd * 4);
      for (uint32_t g = b0; g < b1; ++g) {
        const float4 pv = *reinterpret_cast<const float4*>(part + (size_t)g * D + (size_t)qd * 4);
        tot.x += pv.x; tot.y += pv.y; tot.z += pv.z; tot.w += pv.w;
      }
      float* dst = SPARSE ? grad_rows_out + (size_t)u * D : grad_values + row * D;
      if (SPARSE || dense) *reinterpret_cast<float4*>(dst + (size_t)qd * 4) = tot;
    }
    if (SPARSE && threadIdx.x == 0) rows_out[u] = row;
  }
}

hipError_t launch_bag_backward_sorted(bool bf16, const void* dy, const void* values, int64_t N,
                                      int D, const int64_t* idx, const float* w, int64_t T,
                                      int bag, float* grad_values, int64_t* rows_out,
                                      float* grad_rows_out, float* grad_w, void* ws, float* part,
                                      uint32_t** num_rows_dev, hipStream_t st) {
  const int64_t L = T * bag;
  SortedWs b = carve(ws, L);
  if (num_rows_dev) *num_rows_dev = b.misc;
  hipError_t e = launch_fill_u32(b.misc, 0u, 2, st);
  if (e != hipSuccess || L == 0) return e;
  const uint32_t* ks = nullptr;
  const uint32_t* vs = nullptr;

  // 1. radix sort of (row, lookup) by row; 2. segments of equal rows
  {
    LaunchTimer lt_sort("sort_by_row", st);
    int key_bits = 1;
    while (key_bits < 32 && (int64_t(1) << key_bits) < N) ++key_bits;
    e = sort_segments(idx, true, L, key_bits, b, &ks, &vs, st);
    if (e != hipSuccess) return e;
  }

  // 3. one lane group per touched row
  const int nquad = D / 4;
  int64_t blocks = cdiv(L, 4 * PK_ROWS_BATCH);
  if (blocks > 16384) blocks = 16384;
  const dim3 grid((unsigned)blocks), block(256);
  const bool sparse = rows_out != nullptr;
  int64_t lblocks = L / LONG_CHUNK + max_long(L);  // chunks of long rows, at most
  if (lblocks > 1024) lblocks = 1024;
  int64_t rblocks = max_long(L);
  if (rblocks > 512) rblocks = 512;
  const int ngrp_cap = 16384 / D;  // partial rows that fit 64 KiB
  e = launch_list_long(b.seg, b.misc, L, (uint32_t)LONG_SEG, b.long_list, b.misc + 1, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_long_bases, dim3(1), dim3(256), 0, st, (const uint32_t*)b.seg,
                     (const uint32_t*)b.long_list, (const uint32_t*)(b.misc + 1), b.long_base);
  LaunchTimer lt("bag_backward_rows", st);
#define PK_ROWS_ONE(VT, NQ, CL, SP)                                                                \
  {                                                                                                \
    hipLaunchKernelGGL((k_bag_bwd_rows<VT, NQ, CL, SP, PK_ROWS_BATCH>), grid, block, 0, st,       \
                       (const VT*)dy, (const VT*)values, D, w, bag, ks, vs, b.seg, b.misc,         \
                       grad_values, rows_out, grad_rows_out, grad_w);                             \
    const int ng = (LONG_WAVES * (WAVE / CL)) < ngrp_cap ? LONG_WAVES * (WAVE / CL) : ngrp_cap;    \
    hipLaunchKernelGGL((k_bag_bwd_long<VT, NQ, CL>), dim3((unsigned)lblocks),                      \
                       dim3(64 * LONG_WAVES), (size_t)ng * D * sizeof(float), st, (const VT*)dy,   \
                       (const VT*)values, D, w, bag, ks, vs, b.seg, b.long_list, b.misc + 1,       \
                       b.long_base, part, grad_w);                                                \
    hipLaunchKernelGGL((k_long_reduce<SP>), dim3((unsigned)rblocks), dim3(256), 0, st, D, ks,      \
                       b.seg, b.long_list, b.misc + 1, b.long_base, part, grad_values, rows_out,   \
                       grad_rows_out);                                                             \
  }
#define PK_ROWS(NQ, CL)                                                                           \
  if (bf16) {                                                                                     \
    if (sparse) PK_ROWS_ONE(uint16_t, NQ, CL, true) else PK_ROWS_ONE(uint16_t, NQ, CL, false)     \
  } else {                                                                                        \
    if (sparse) PK_ROWS_ONE(float, NQ, CL, true) else PK_ROWS_ONE(float, NQ, CL, false)           \
  }
  if (nquad > 512) { PK_ROWS(16, 64); }
  else if (nquad > 256) { PK_ROWS(8, 64); }
  else if (nquad > 128) { PK_ROWS(4, 64); }
  else if (nquad > 64) { PK_ROWS(2, 64); }
  else if (nquad > 32) { PK_ROWS(1, 64); }
  else if (nquad > 16) { PK_ROWS(1, 32); }
  else if (nquad > 8) { PK_ROWS(1, 16); }
  else if (nquad > 4) { PK_ROWS(1, 8); }
  else if (nquad > 2) { PK_ROWS(1, 4); }
  else { PK_ROWS(1, 2); }
#undef PK_ROWS
#undef PK_ROWS_ONE
  return hipGetLastError();
}

}  // namespace pk
