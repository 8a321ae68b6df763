// Weighted EmbeddingBag on gfx950 (Sec. 3, Eq. (1) y = s V_I; Sec. 3.1.4 of
// "Memory Layers at Scale").
//
// Row mapping shared by the kernels here and in sorted.hip: a value row of D
// elements is cut into C = D * esize / 16 chunks of 16 bytes.  One wave owns
// one bag (a token's H*k lookups).  For C >= 64 each lane holds CPL = C / 64
// chunks i*64 + lane, so every load instruction of the wave reads 1 KiB of one
// row contiguously.  For C < 64 the wave splits into G = 64 / CL groups of CL
// lanes (CL = C rounded up to a power of two); group g takes the lookups
// j = g, g + G, ... and the groups are summed at the end.
#include "pk_device.h"
#include "pk_internal.h"

namespace pk {

// 16-byte vector <-> fp32 lanes for the two value dtypes.
template <typename V>
struct Row16;

template <>
struct Row16<uint16_t> {  // bf16
  static constexpr int N = 8;
  __device__ static __forceinline__ void unpack(const uint4& v, float (&f)[8]) {
    f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x); f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
    f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z); f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
  }
  __device__ static __forceinline__ uint4 pack(const float (&f)[8]) {
    return uint4{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                 pack_bf16x2(f[6], f[7])};
  }
};

template <>
struct Row16<float> {
  static constexpr int N = 4;
  __device__ static __forceinline__ void unpack(const uint4& v, float (&f)[4]) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  __device__ static __forceinline__ uint4 pack(const float (&f)[4]) {
    return uint4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                 __float_as_uint(f[3])};
  }
};


// The token's lookups are read 64 at a time, one per lane, with a single
// coalesced load; lookup j of the chunk is then taken from lane j (readlane
// into scalar registers when the whole wave works on one lookup, a lane
// shuffle when lane groups work on different lookups).
template <int G>
struct LookupChunk {
  uint32_t lo, hi;
  float w;
  __device__ __forceinline__ void load(const int64_t* ti, const float* tw, int c0, int nb, int lane) {
    const int64_t r = lane < nb ? ti[c0 + lane] : 0;
    lo = (uint32_t)r;
    hi = (uint32_t)((uint64_t)r >> 32);
    w = lane < nb ? tw[c0 + lane] : 0.f;
  }
  __device__ __forceinline__ void get(int j, int64_t& r, float& ww) const {
    if constexpr (G == 1) {
      const uint32_t a = __builtin_amdgcn_readlane(lo, j);
      const uint32_t b = __builtin_amdgcn_readlane(hi, j);
      r = (int64_t)(((uint64_t)b << 32) | a);
      ww = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w), j));
    } else {
      const uint32_t a = __shfl(lo, j, WAVE);
      const uint32_t b = __shfl(hi, j, WAVE);
      r = (int64_t)(((uint64_t)b << 32) | a);
      ww = __shfl(w, j, WAVE);
    }
  }
};

// y[t] = sum_j w[t,j] V[idx[t,j]]; fp32 accumulation, one rounding at the end.
// The output rows are stored non-temporal: a trickle of ordinary stores in the
// middle of the gather's random-read stream costs it about 12% on MI355X.
// Lookups go in groups of U per lane group through a two-deep register ring:
// the loads of group m+1 are in flight while group m is accumulated.  FULL
// means every lane owns CPL whole chunks (C == CPL * CL), so no chunk needs a
// per-lane predicate.
// SPLIT > 1 (full rows of 64-lane groups only) spreads a token over SPLIT
// waves, each owning CPL consecutive 1 KiB slabs of every row: more, smaller
// waves in flight.
// Memory+ epilogue (Sec. 3.1.4): with a gate [T, D] the kernel writes
// y = bag * silu(gate) instead of the bag, and the un-gated bag to y_plain
// when that is non-null; both from the fp32 accumulator, one rounding each.
template <typename V, int CPL, int CL, int U, bool FULL, int SPLIT>
__global__ __launch_bounds__(256) void k_bag_fwd(const V* __restrict__ values, int D,
                                                 const int64_t* __restrict__ idx,
                                                 const float* __restrict__ w, int64_t T, int bag,
                                                 V* __restrict__ y, const V* __restrict__ gate,
                                                 V* __restrict__ y_plain) {
  using R = Row16<V>;
  constexpr int G = WAVE / CL;
  static_assert(SPLIT == 1 || (FULL && CL == WAVE), "split waves need full 64-lane rows");
  const int lane = threadIdx.x & 63;
  const int C = D / R::N;
  const int64_t nwaves = (int64_t)gridDim.x * 4;
  for (int64_t gw = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); gw < T * SPLIT; gw += nwaves) {
  const int64_t t = gw / SPLIT;
  const int slab = (int)(gw % SPLIT);
  const int grp = lane / CL, cl = lane % CL + slab * CPL * CL;

  float acc[CPL][R::N];
#pragma unroll
  for (int i = 0; i < CPL; ++i)
#pragma unroll
    for (int e = 0; e < R::N; ++e) acc[i][e] = 0.f;

  bool ok[CPL];
#pragma unroll
  for (int i = 0; i < CPL; ++i) ok[i] = FULL || (i * CL + cl) < C;

  struct Group {
    uint4 v[U][CPL];
    float ww[U];
  };
  auto issue = [&](Group& g, const LookupChunk<G>& lk, int j0) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      int64_t r;
      lk.get(j0 + u * G, r, g.ww[u]);
      const V* row = values + r * D + (size_t)cl * R::N;
#pragma unroll
      for (int i = 0; i < CPL; ++i)
        g.v[u][i] = ok[i] ? ld16_nt(row + (size_t)i * CL * R::N) : uint4{0, 0, 0, 0};
    }
  };
  auto consume = [&](const Group& g) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        float f[R::N];
        R::unpack(g.v[u][i], f);
#pragma unroll
        for (int e = 0; e < R::N; ++e) acc[i][e] = fmaf(g.ww[u], f[e], acc[i][e]);
      }
  };

  const int64_t* ti = idx + t * bag;
  const float* tw = w + t * bag;
  for (int c0 = 0; c0 < bag; c0 += WAVE) {
    const int nb = (bag - c0) < WAVE ? (bag - c0) : WAVE;
    LookupChunk<G> lk;
    lk.load(ti, tw, c0, nb, lane);
    // Blocks of U*G lookups, then a tail; every lane group runs the same trip
    // counts (the shuffles in lk.get need the whole wave).
    const int full = nb / (U * G);
#if PK_FWD_RING
    if (full > 0) {
      Group ga, gb;
      issue(ga, lk, grp);
      for (int m = 0; m < full; m += 2) {
        if (m + 1 < full) issue(gb, lk, (m + 1) * U * G + grp);
        consume(ga);
        if (m + 1 < full) {
          if (m + 2 < full) issue(ga, lk, (m + 2) * U * G + grp);
          consume(gb);
        }
      }
    }
#else
    for (int m = 0; m < full; ++m) {
      Group ga;
      issue(ga, lk, m * U * G + grp);
      consume(ga);
    }
#endif
    const int base = full * U * G;
    const int tail = (nb - base + G - 1) / G;
    for (int q = 0; q < tail; ++q) {
      const int j = base + q * G + grp;
      const bool live = j < nb;
      int64_t r;
      float ww;
      lk.get(live ? j : base, r, ww);
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        if (!ok[i] || !live) continue;
        float f[R::N];
        R::unpack(ld16_nt(values + r * D + (size_t)(i * CL + cl) * R::N), f);
#pragma unroll
        for (int e = 0; e < R::N; ++e) acc[i][e] = fmaf(ww, f[e], acc[i][e]);
      }
    }
  }
  if (G > 1) {
#pragma unroll
    for (int m = CL; m < WAVE; m <<= 1)
#pragma unroll
      for (int i = 0; i < CPL; ++i)
#pragma unroll
        for (int e = 0; e < R::N; ++e) acc[i][e] += __shfl_xor(acc[i][e], m, WAVE);
  }
  if (grp == 0) {
    if (gate) {  // uniform
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        if (!ok[i]) continue;
        const size_t off = t * D + (size_t)(i * CL + cl) * R::N;
        float gv[R::N], o[R::N];
        R::unpack(ld16(gate + off), gv);
        if (y_plain) st16_nt(y_plain + off, R::pack(acc[i]));
#pragma unroll
        for (int e = 0; e < R::N; ++e) o[e] = acc[i][e] * silu_f32(gv[e]);
        st16_nt(y + off, R::pack(o));
      }
    } else {
#pragma unroll
      for (int i = 0; i < CPL; ++i)
        if (ok[i]) st16_nt(y + t * D + (size_t)(i * CL + cl) * R::N, R::pack(acc[i]));
    }
  }
  }
}

// Backward of the Memory+ epilogue, element-wise in 16-byte chunks:
//   dy = d_out * silu(g)                      (value dtype: the bag backward's dy)
//   grad_gate = d_out * y * silu'(g),  silu'(g) = sig(g) * (1 + g * (1 - sig(g)))
// with y the un-gated bag.  Grid-stride over the T*D/N chunks.
template <typename V>
__global__ __launch_bounds__(256) void k_gate_bwd(const V* __restrict__ d_out,
                                                  const V* __restrict__ gate,
                                                  const V* __restrict__ yb, int64_t nchunks,
                                                  V* __restrict__ dy, float* __restrict__ grad_gate) {
  using R = Row16<V>;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < nchunks;
       c += (int64_t)gridDim.x * 256) {
    float d[R::N], g[R::N], yy[R::N], o[R::N], dg[R::N];
    R::unpack(ld16_nt(d_out + c * R::N), d);
    R::unpack(ld16_nt(gate + c * R::N), g);
    R::unpack(ld16_nt(yb + c * R::N), yy);
#pragma unroll
    for (int e = 0; e < R::N; ++e) {
      const float sig = 1.f / (1.f + expf(-g[e]));
      o[e] = d[e] * (g[e] * sig);
      dg[e] = d[e] * yy[e] * (sig * (1.f + g[e] * (1.f - sig)));
    }
    st16_nt(dy + c * R::N, R::pack(o));
#pragma unroll
    for (int e = 0; e < R::N; e += 4)
      st16_nt(grad_gate + c * R::N + e,
              uint4{__float_as_uint(dg[e]), __float_as_uint(dg[e + 1]), __float_as_uint(dg[e + 2]),
                    __float_as_uint(dg[e + 3])});
  }
}

// Atomic strategy: per lookup, grad_w = dy . V[row] and grad_values[row] +=
// w * dy with fp32 atomic adds (no return) resolved in L2.  The dot product
// uses dy in the quad layout of the value loads (lane cl of a CL-lane group
// owns quads m*CL + cl); the atomics use a second, lane-strided copy of dy
// (element cl + CL*a in slot a), so each atomic instruction of a lane group
// covers CL consecutive floats.  A token's bag is cut into `split` contiguous
// parts of `per` lookups, one wave each (the token's dy row is then read by
// `split` waves, from L2), and a persistent grid strides over the T * split
// parts: small batches still fill the chip.
template <typename V, int NQ, int CL>
__global__ __launch_bounds__(256) void k_bag_bwd_atomic(const V* __restrict__ dy,
                                                        const V* __restrict__ values, int D,
                                                        const int64_t* __restrict__ idx,
                                                        const float* __restrict__ w, int64_t T,
                                                        int bag, int split, int per,
                                                        float* __restrict__ grad_values,
                                                        float* __restrict__ grad_w) {
  using Q = Quad<V>;
  constexpr int G = WAVE / CL;
  constexpr int AM = NQ * 4;  // strided elements per lane
  const int lane = threadIdx.x & 63;
  const int nquad = D / 4;
  const int grp = lane / CL, cl = lane % CL;
  bool ok[NQ];
#pragma unroll
  for (int m = 0; m < NQ; ++m) ok[m] = (m * CL + cl) < nquad;
  const int64_t units = T * split;
  for (int64_t u = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); u < units;
       u += (int64_t)gridDim.x * 4) {
    const int64_t t = u / split;
    const int j0 = (int)(u % split) * per;
    const int j1 = j0 + per < bag ? j0 + per : bag;
    const V* dyt = dy + t * D;
    float g[NQ][4];
#pragma unroll
    for (int m = 0; m < NQ; ++m) {
      const typename Q::raw r = ok[m] ? Q::load(dyt + (size_t)(m * CL + cl) * 4) : Q::zero();
      Q::unpack(r, g[m]);
    }
    float ga[AM];
#pragma unroll
    for (int a = 0; a < AM; ++a) {
      const int e = cl + CL * a;
      ga[a] = 0.f;
      if (e < D) {
        if constexpr (sizeof(V) == 2) ga[a] = bf16_to_f32(dyt[e]);
        else ga[a] = (float)dyt[e];
      }
    }
    const int64_t* ti = idx + t * bag;
    const float* tw = w + t * bag;
    for (int j = j0 + grp; j < j1; j += G) {
      const int64_t r = ti[j];
      const float ww = tw[j];
      float part = 0.f;
#pragma unroll
      for (int m = 0; m < NQ; ++m) {
        if (!ok[m]) continue;
        float f[4];
        Q::unpack(Q::load(values + r * D + (size_t)(m * CL + cl) * 4), f);
#pragma unroll
        for (int e = 0; e < 4; ++e) part = fmaf(g[m][e], f[e], part);
      }
      if (grad_values) {
        float* gr = grad_values + r * D;
#pragma unroll
        for (int a = 0; a < AM; ++a) {
          const int e = cl + CL * a;
          if (e < D) unsafeAtomicAdd(gr + e, ww * ga[a]);
        }
      }
      part = group_sum<CL>(part);
      if (cl == 0 && grad_w) grad_w[t * bag + j] = part;
    }
  }
}

// grad_scores = w * (grad_w - sum_j w_j grad_w_j) per (token, head) row of k.
// A row is handled by KG = k rounded up to a power of two lanes (coalesced).
template <int KG>
__global__ __launch_bounds__(256) void k_softmax_bwd(const float* __restrict__ w,
                                                     const float* __restrict__ gw, int64_t rows,
                                                     int k, float* __restrict__ gz) {
  constexpr int RPW = WAVE / KG;  // rows per wave
  const int lane = threadIdx.x & 63;
  const int64_t r = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW + lane / KG;
  const int j = lane % KG;
  const bool live = r < rows && j < k;
  const size_t o = (size_t)(live ? r : 0) * k + j;
  const float wv = live ? w[o] : 0.f;
  const float gv = live ? gw[o] : 0.f;
  const float inner = group_sum<KG>(wv * gv);
  if (live) gz[o] = wv * (gv - inner);
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint32_t value, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) p[i] = value;
}

hipError_t launch_fill_u32(uint32_t* p, uint32_t value, int64_t count, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_u32, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, st, p, value, count);
  return hipGetLastError();
}

hipError_t launch_softmax_backward(const float* w, const float* grad_w, int64_t rows, int k,
                                   float* grad_scores, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  LaunchTimer lt("softmax_backward", st);
  int kg = 1;
  while (kg < k) kg <<= 1;
  const int64_t rows_per_block = 4 * (WAVE / kg);
  const dim3 grid((unsigned)((rows + rows_per_block - 1) / rows_per_block)), block(256);
  switch (kg) {
    case 1: hipLaunchKernelGGL(k_softmax_bwd<1>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    case 2: hipLaunchKernelGGL(k_softmax_bwd<2>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    case 4: hipLaunchKernelGGL(k_softmax_bwd<4>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    case 8: hipLaunchKernelGGL(k_softmax_bwd<8>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    case 16: hipLaunchKernelGGL(k_softmax_bwd<16>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    case 32: hipLaunchKernelGGL(k_softmax_bwd<32>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
    default: hipLaunchKernelGGL(k_softmax_bwd<64>, grid, block, 0, st, w, grad_w, rows, k, grad_scores); break;
  }
  return hipGetLastError();
}

// Dispatch on (dtype, chunks per row): CPL in {1,2,4,8} for C >= 64, CL in
// {1..64} for C < 64.
#define PK_ROW_DISPATCH(C, MACRO)                    \
  do {                                               \
    if ((C) > 256) { MACRO(8, 64); }                 \
    else if ((C) > 128) { MACRO(4, 64); }            \
    else if ((C) > 64) { MACRO(2, 64); }             \
    else if ((C) > 32) { MACRO(1, 64); }             \
    else if ((C) > 16) { MACRO(1, 32); }             \
    else if ((C) > 8) { MACRO(1, 16); }              \
    else if ((C) > 4) { MACRO(1, 8); }               \
    else if ((C) > 2) { MACRO(1, 4); }               \
    else if ((C) > 1) { MACRO(1, 2); }               \
    else { MACRO(1, 1); }                            \
  } while (0)

// One wave per unit of work, or a persistent grid of PK_FWD_BLOCKS workgroups
// striding over the units.
static unsigned fwd_blocks(int64_t waves) {
  int64_t b = (waves + 3) / 4;
  if (PK_FWD_BLOCKS > 0 && b > PK_FWD_BLOCKS) b = PK_FWD_BLOCKS;
  return (unsigned)b;
}

hipError_t launch_bag_forward(bool bf16, const void* values, int D, const int64_t* idx,
                              const float* w, int64_t T, int bag, void* y, const void* gate,
                              void* y_plain, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  const int C = D * (bf16 ? 2 : 4) / 16;
  LaunchTimer lt("bag_forward", st);
  // Full rows of 4 or 8 slabs are split over PK_FWD_SPLIT waves per token.
  constexpr int SP = PK_FWD_SPLIT;
  if (C == 256 && (4 % SP) == 0) {
    const dim3 grid(fwd_blocks(T * SP)), block(256);
    if (bf16)
      hipLaunchKernelGGL((k_bag_fwd<uint16_t, 4 / SP, 64, PK_FWD_UNROLL, true, SP>), grid, block, 0,
                         st, (const uint16_t*)values, D, idx, w, T, bag, (uint16_t*)y, (const uint16_t*)gate, (uint16_t*)y_plain);
    else
      hipLaunchKernelGGL((k_bag_fwd<float, 4 / SP, 64, PK_FWD_UNROLL, true, SP>), grid, block, 0, st,
                         (const float*)values, D, idx, w, T, bag, (float*)y, (const float*)gate, (float*)y_plain);
    return hipGetLastError();
  }
  if (C == 512 && (8 % SP) == 0) {
    const dim3 grid(fwd_blocks(T * SP)), block(256);
    if (bf16)
      hipLaunchKernelGGL((k_bag_fwd<uint16_t, 8 / SP, 64, PK_FWD_UNROLL, true, SP>), grid, block, 0,
                         st, (const uint16_t*)values, D, idx, w, T, bag, (uint16_t*)y, (const uint16_t*)gate, (uint16_t*)y_plain);
    else
      hipLaunchKernelGGL((k_bag_fwd<float, 8 / SP, 64, PK_FWD_UNROLL, true, SP>), grid, block, 0, st,
                         (const float*)values, D, idx, w, T, bag, (float*)y, (const float*)gate, (float*)y_plain);
    return hipGetLastError();
  }
  const dim3 grid(fwd_blocks(T)), block(256);
#define PK_FWD(CPL, CL)                                                                              \
  if (C == (CPL) * (CL)) {                                                                           \
    if (bf16)                                                                                        \
      hipLaunchKernelGGL((k_bag_fwd<uint16_t, CPL, CL, PK_FWD_UNROLL, true, 1>), grid, block, 0, st,  \
                         (const uint16_t*)values, D, idx, w, T, bag, (uint16_t*)y, (const uint16_t*)gate, (uint16_t*)y_plain);                 \
    else                                                                                             \
      hipLaunchKernelGGL((k_bag_fwd<float, CPL, CL, PK_FWD_UNROLL, true, 1>), grid, block, 0, st,     \
                         (const float*)values, D, idx, w, T, bag, (float*)y, (const float*)gate, (float*)y_plain);                       \
  } else {                                                                                           \
    if (bf16)                                                                                        \
      hipLaunchKernelGGL((k_bag_fwd<uint16_t, CPL, CL, PK_FWD_UNROLL, false, 1>), grid, block, 0, st, \
                         (const uint16_t*)values, D, idx, w, T, bag, (uint16_t*)y, (const uint16_t*)gate, (uint16_t*)y_plain);                 \
    else                                                                                             \
      hipLaunchKernelGGL((k_bag_fwd<float, CPL, CL, PK_FWD_UNROLL, false, 1>), grid, block, 0, st,    \
                         (const float*)values, D, idx, w, T, bag, (float*)y, (const float*)gate, (float*)y_plain);                       \
  }
  PK_ROW_DISPATCH(C, PK_FWD);
#undef PK_FWD
  return hipGetLastError();
}

hipError_t launch_gate_backward(bool bf16, const void* d_out, const void* gate, const void* y,
                                int64_t T, int D, void* dy, float* grad_gate, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  const int64_t nchunks = T * D / (bf16 ? 8 : 4);
  int64_t blocks = (nchunks + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  LaunchTimer lt("gate_backward", st);
  if (bf16)
    hipLaunchKernelGGL(k_gate_bwd<uint16_t>, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const uint16_t*)d_out, (const uint16_t*)gate, (const uint16_t*)y, nchunks,
                       (uint16_t*)dy, grad_gate);
  else
    hipLaunchKernelGGL(k_gate_bwd<float>, dim3((unsigned)blocks), dim3(256), 0, st,
                       (const float*)d_out, (const float*)gate, (const float*)y, nchunks, (float*)dy,
                       grad_gate);
  return hipGetLastError();
}

// Debug check: *bad = 1 if any of the count indices lies outside [0, limit).
// Element i of the rows * cols checked is idx[(i / cols) * stride + i % cols].
__global__ __launch_bounds__(256) void k_check_indices(const int64_t* __restrict__ idx,
                                                       int64_t count, int cols, int stride,
                                                       int64_t limit, uint32_t* __restrict__ bad) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * 256) {
    const int64_t v = idx[(i / cols) * stride + i % cols];
    if (v < 0 || v >= limit) *bad = 1u;
  }
}

hipError_t launch_check_indices_strided(const int64_t* idx, int64_t rows, int cols, int stride,
                                        int64_t limit, uint32_t* bad, hipStream_t st) {
  hipError_t e = launch_fill_u32(bad, 0u, 1, st);
  const int64_t count = rows * cols;
  if (e != hipSuccess || count <= 0) return e;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(k_check_indices, dim3((unsigned)blocks), dim3(256), 0, st, idx, count, cols,
                     stride, limit, bad);
  return hipGetLastError();
}

hipError_t launch_check_indices(const int64_t* idx, int64_t count, int64_t limit, uint32_t* bad,
                                hipStream_t st) {
  return launch_check_indices_strided(idx, count, 1, 1, limit, bad, st);
}

constexpr int64_t ATOMIC_WAVES = 16384;  // waves the atomic backward aims for
constexpr int64_t ATOMIC_BLOCKS = 8192;  // its persistent grid, at most

hipError_t launch_bag_backward_atomic(bool bf16, const void* dy, const void* values, int D,
                                      const int64_t* idx, const float* w, int64_t T, int bag,
                                      float* grad_values, float* grad_w, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  // Parts per token: enough waves to fill the chip (ATOMIC_WAVES), each part
  // at least 4 lookups; then a persistent grid of at most ATOMIC_BLOCKS
  // workgroups of four waves.
  int split = 1;
  while ((int64_t)T * split < ATOMIC_WAVES && bag / (split * 2) >= 4) split *= 2;
  const int per = (bag + split - 1) / split;
  int64_t blocks = (T * split + 3) / 4;
  if (blocks > ATOMIC_BLOCKS) blocks = ATOMIC_BLOCKS;
  const dim3 grid((unsigned)blocks), block(256);
  LaunchTimer lt("bag_backward_atomic", st);
#define PK_BWD(NQ, CL)                                                                          \
  if (bf16)                                                                                     \
    hipLaunchKernelGGL((k_bag_bwd_atomic<uint16_t, NQ, CL>), grid, block, 0, st,                \
                       (const uint16_t*)dy, (const uint16_t*)values, D, idx, w, T, bag, split,   \
                       per, grad_values, grad_w);                                               \
  else                                                                                          \
    hipLaunchKernelGGL((k_bag_bwd_atomic<float, NQ, CL>), grid, block, 0, st, (const float*)dy,  \
                       (const float*)values, D, idx, w, T, bag, split, per, grad_values, grad_w);
  const int nquad = D / 4;
  if (nquad > 512) { PK_BWD(16, 64); }
  else if (nquad > 256) { PK_BWD(8, 64); }
  else if (nquad > 128) { PK_BWD(4, 64); }
  else if (nquad > 64) { PK_BWD(2, 64); }
  else if (nquad > 32) { PK_BWD(1, 64); }
  else if (nquad > 16) { PK_BWD(1, 32); }
  else if (nquad > 8) { PK_BWD(1, 16); }
  else if (nquad > 4) { PK_BWD(1, 8); }
  else if (nquad > 2) { PK_BWD(1, 4); }
  else { PK_BWD(1, 2); }
#undef PK_BWD
  return hipGetLastError();
}

}  // namespace pk
