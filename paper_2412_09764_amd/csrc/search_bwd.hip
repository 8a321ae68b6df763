// Search backward on gfx950: gradients of the selected scores into queries and
// sub-keys (the keys are trainable parameters, Sec. 3 of "Memory Layers at
// Scale"; the selection passes no gradient).  With the composed index
// i = i1*S + i2 of Sec. 3.1.1 the score of rank j is
//   z_j = q[:d] . K[h,0,i1_j] + q[d:] . K[h,1,i2_j],
// so grad_q[:d] = sum_j gz_j K[h,0,i1_j] and grad_K[h,0,i] += sum_{j: i1_j = i}
// gz_j q[:d] (same for half 1).
//
// One wave per (token, head).  The k lookups sit one per lane; per half, each
// lane finds the leader of its sub-key group (lowest rank with the same
// sub-key index) and the group's summed gradient, in rank order.  The wave then
// visits the distinct sub-keys only: it reads each needed sub-key row once for
// grad_q and adds g * q_half into the gradient row with lane-contiguous fp32
// atomics (no return).  Blocks are laid out so that consecutive blocks (which
// the dispatcher spreads over the XCDs) take different heads: each head's
// gradient table is then touched from as few XCDs as possible.
#include "pk_device.h"
#include "pk_internal.h"

namespace pk {

template <typename T>
__device__ __forceinline__ float elem_f32(const T* p);
template <>
__device__ __forceinline__ float elem_f32<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <>
__device__ __forceinline__ float elem_f32<float>(const float* p) { return *p; }

// NE = elements per lane per half = ceil(d / 64).
template <typename T, int NE>
__global__ __launch_bounds__(256) void k_search_bwd(const T* __restrict__ q,
                                                    const T* __restrict__ subkeys, int64_t ntok,
                                                    int H, int n, int S, int k,
                                                    const int64_t* __restrict__ idx,
                                                    const float* __restrict__ gz,
                                                    float* __restrict__ grad_q,
                                                    float* __restrict__ grad_K) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = (int)(blockIdx.x % (unsigned)H);
  const int64_t t = (int64_t)(blockIdx.x / (unsigned)H) * 4 + wave;
  if (t >= ntok) return;
  const int d = n >> 1;
  const size_t r = (size_t)t * H + h;
  const int64_t ix = lane < k ? idx[r * k + lane] : 0;
  const float g = lane < k ? gz[r * k + lane] : 0.f;
  const T* qrow = q + r * n;

#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const int mine = (int)(p == 0 ? ix / S : ix % S);
    // group sum in rank order; leader = first rank of the group
    float gsum = 0.f;
    bool leader = lane < k;
    for (int j = 0; j < k; ++j) {
      const int oi = __builtin_amdgcn_readlane(mine, j);
      const float og = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(g), j));
      if (oi == mine) {
        gsum += og;
        if (j < lane) leader = false;
      }
    }
    uint64_t lead = __ballot(leader);
    float qh[NE], dq[NE];
#pragma unroll
    for (int c = 0; c < NE; ++c) {
      const int e = lane + 64 * c;
      qh[c] = e < d ? elem_f32<T>(qrow + (size_t)p * d + e) : 0.f;
      dq[c] = 0.f;
    }
    const T* kh = subkeys + (size_t)(h * 2 + p) * S * d;
    float* gkh = grad_K ? grad_K + (size_t)(h * 2 + p) * S * d : nullptr;
    while (lead) {
      const int L = __builtin_ctzll(lead);
      lead &= lead - 1;
      const int i = __builtin_amdgcn_readlane(mine, L);
      const float gg = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(gsum), L));
      const T* krow = kh + (size_t)i * d;
#pragma unroll
      for (int c = 0; c < NE; ++c) {
        const int e = lane + 64 * c;
        if (e < d) {
          dq[c] = fmaf(gg, elem_f32<T>(krow + e), dq[c]);
          if (gkh) unsafeAtomicAdd(gkh + (size_t)i * d + e, gg * qh[c]);
        }
      }
    }
    if (grad_q) {
#pragma unroll
      for (int c = 0; c < NE; ++c) {
        const int e = lane + 64 * c;
        if (e < d) grad_q[r * n + (size_t)p * d + e] = dq[c];
      }
    }
  }
}

template <typename T>
static hipError_t launch_sbwd(const void* q, const void* subkeys, int64_t T_, int H, int n, int S,
                              int k, const int64_t* idx, const float* gz, float* grad_q,
                              float* grad_K, hipStream_t st) {
  const int d = n / 2;
  const int64_t blocks = ((T_ + 3) / 4) * H;
  const dim3 grid((unsigned)blocks), block(256);
  LaunchTimer lt("search_backward", st);
  const int ne = (d + 63) / 64;
#define PK_SB(NE)                                                                            \
  hipLaunchKernelGGL((k_search_bwd<T, NE>), grid, block, 0, st, (const T*)q, (const T*)subkeys, \
                     T_, H, n, S, k, idx, gz, grad_q, grad_K)
  if (ne <= 1) PK_SB(1);
  else if (ne <= 2) PK_SB(2);
  else PK_SB(4);
#undef PK_SB
  return hipGetLastError();
}

hipError_t launch_search_backward(bool bf16, const void* q, const void* subkeys, int64_t T, int H,
                                  int n, int S, int k, const int64_t* idx, const float* gz,
                                  float* grad_q, float* grad_K, hipStream_t st) {
  if (T <= 0) return hipSuccess;
  if (bf16) return launch_sbwd<uint16_t>(q, subkeys, T, H, n, S, k, idx, gz, grad_q, grad_K, st);
  return launch_sbwd<float>(q, subkeys, T, H, n, S, k, idx, gz, grad_q, grad_K, st);
}

}  // namespace pk
