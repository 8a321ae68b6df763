// Device helpers shared by the product-key memory kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pk {

constexpr int WAVE = 64;

// Tuning knobs (compile-time; the defaults are the measured best on MI355X).
#ifndef PK_FWD_UNROLL
#define PK_FWD_UNROLL 2  // lookups per group (two groups in flight) in the gather
#endif
#ifndef PK_FWD_RING
#define PK_FWD_RING 1    // two-deep register ring of lookup groups in the gather
#endif
#ifndef PK_FWD_BLOCKS
#define PK_FWD_BLOCKS 4096  // persistent grid of this many workgroups (0: one wave per token)
#endif
#ifndef PK_FWD_SPLIT
#define PK_FWD_SPLIT 1   // waves per token in the gather for 4 KiB / 8 KiB rows
#endif
#ifndef PK_ROWS_BATCH
#define PK_ROWS_BATCH 2  // adjacent touched rows per lane group per iteration (sorted backward)
#endif
#ifndef PK_STREAM_NT
#define PK_STREAM_NT 1   // non-temporal hints on value rows streamed once
#endif
#ifndef PK_GRAD_NT_LOAD
#define PK_GRAD_NT_LOAD 1   // non-temporal hint on the gradient-row read
#endif
#ifndef PK_GRAD_NT_STORE
#define PK_GRAD_NT_STORE 1  // non-temporal hint on the gradient-row write
#endif

// ------------------------------------------------------- 16-byte access ----
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }
// Non-temporal 16-byte load / store: for data streamed once per pass.
template <bool NT>
__device__ __forceinline__ uint4 ld16_hint(const void* p) {
  if constexpr (NT) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return uint4{v.x, v.y, v.z, v.w};
  } else {
    return ld16(p);
  }
}
template <bool NT>
__device__ __forceinline__ void st16_hint(void* p, uint4 v) {
  if constexpr (NT) {
    const u32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
  } else {
    *reinterpret_cast<uint4*>(p) = v;
  }
}
__device__ __forceinline__ uint4 ld16_nt(const void* p) {
#if PK_STREAM_NT
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return uint4{v.x, v.y, v.z, v.w};
#else
  return ld16(p);
#endif
}
__device__ __forceinline__ void st16_nt(void* p, uint4 v) {
#if PK_STREAM_NT
  const u32x4_t x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<u32x4_t*>(p));
#else
  *reinterpret_cast<uint4*>(p) = v;
#endif
}

// Direct global -> LDS copy of 16 bytes per lane (gfx950): lane i's bytes land
// at lds_base + 16 * i; lds_base must be the same for the whole wave.
__device__ __forceinline__ void lds_dma16(const void* gptr, void* lds_base) {
  __builtin_amdgcn_global_load_lds(gptr, (__attribute__((address_space(3))) void*)lds_base, 16, 0, 0);
}

// The same through a buffer resource (raw buffer of `bytes` bytes at base):
// lane i's 16 bytes from base + voff (per lane) + soff (uniform) land at
// lds_base + 16 * i.  Unlike the global form, the compiler tracks this copy
// as a vector-memory access only, so LDS reads of other buffers keep precise
// (partial) wait counts while the copy is in flight.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ void lds_dma16_buf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                              void* lds_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_base, 16,
                                           (int)voff, (int)soff, 0, 0);
}

// ---------------------------------------------------------------- bf16 ----
// silu(x) = x * sigmoid(x) = x / (1 + exp(-x)) (Memory+ gate, Sec. 3.1.4);
// for very negative x the denominator overflows to inf and the result is -0.
__device__ __forceinline__ float silu_f32(float x) { return x / (1.f + expf(-x)); }

__device__ __forceinline__ float bf16_lo(uint32_t two) { return __uint_as_float(two << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t two) { return __uint_as_float(two & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_bits(lo) | (f32_to_bf16_bits(hi) << 16);
}

// Query normalisation (LayerNorm without affine): (x - mean) * rstd in fp32.
// Every kernel that needs a normalised query element computes it with this
// one expression, so the forward and the backward see the same bits.
__device__ __forceinline__ float qn_apply(float x, float mean, float rstd) {
  return (x - mean) * rstd;
}
__device__ __forceinline__ float round_bf16_f32(float v) {
  return __uint_as_float(f32_to_bf16_bits(v) << 16);
}

// Four consecutive elements of a query or sub-key half row: bf16 (8 bytes) or
// fp32 (16 bytes).
template <typename T>
struct QQuad;
template <>
struct QQuad<uint16_t> {
  uint2 raw;
  __device__ __forceinline__ void load(const uint16_t* p) { raw = *reinterpret_cast<const uint2*>(p); }
  __device__ __forceinline__ void fma_into(float g, float* a) const {
    a[0] = fmaf(g, __uint_as_float(raw.x << 16), a[0]);
    a[1] = fmaf(g, __uint_as_float(raw.x & 0xffff0000u), a[1]);
    a[2] = fmaf(g, __uint_as_float(raw.y << 16), a[2]);
    a[3] = fmaf(g, __uint_as_float(raw.y & 0xffff0000u), a[3]);
  }
  __device__ __forceinline__ void to_f32(float* v) const {
    v[0] = __uint_as_float(raw.x << 16);
    v[1] = __uint_as_float(raw.x & 0xffff0000u);
    v[2] = __uint_as_float(raw.y << 16);
    v[3] = __uint_as_float(raw.y & 0xffff0000u);
  }
  // The same with the normalised query as scored (rounded to bf16).
  __device__ __forceinline__ void fma_into_norm(float g, float* a, float mean, float rstd) const {
    float v[4];
    to_f32(v);
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] = fmaf(g, round_bf16_f32(qn_apply(v[i], mean, rstd)), a[i]);
  }
};
template <>
struct QQuad<float> {
  float4 raw;
  __device__ __forceinline__ void load(const float* p) { raw = *reinterpret_cast<const float4*>(p); }
  __device__ __forceinline__ void fma_into(float g, float* a) const {
    a[0] = fmaf(g, raw.x, a[0]);
    a[1] = fmaf(g, raw.y, a[1]);
    a[2] = fmaf(g, raw.z, a[2]);
    a[3] = fmaf(g, raw.w, a[3]);
  }
  __device__ __forceinline__ void to_f32(float* v) const {
    v[0] = raw.x; v[1] = raw.y; v[2] = raw.z; v[3] = raw.w;
  }
  __device__ __forceinline__ void fma_into_norm(float g, float* a, float mean, float rstd) const {
    a[0] = fmaf(g, qn_apply(raw.x, mean, rstd), a[0]);
    a[1] = fmaf(g, qn_apply(raw.y, mean, rstd), a[1]);
    a[2] = fmaf(g, qn_apply(raw.z, mean, rstd), a[2]);
    a[3] = fmaf(g, qn_apply(raw.w, mean, rstd), a[3]);
  }
};

// Quad layout: a row of D elements is D/4 quads of 4 consecutive elements; the
// CL lanes of a group own quads q = m*CL + cl (m < NQ).  A bf16 quad is 8 bytes
// and an fp32 quad 16 bytes, so every instruction of a group reads or writes
// one contiguous span of the row, for the bf16 inputs and the fp32 gradient
// alike (no partial cache lines).  Used by the value-gradient kernels.
template <typename V>
struct Quad;
template <>
struct Quad<uint16_t> {
  __device__ static __forceinline__ uint2 load(const uint16_t* p) { return *reinterpret_cast<const uint2*>(p); }
  __device__ static __forceinline__ uint2 load_nt(const uint16_t* p) {
#if PK_STREAM_NT
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    return uint2{v.x, v.y};
#else
    return load(p);
#endif
  }
  __device__ static __forceinline__ void unpack(const uint2& v, float (&f)[4]) {
    f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x); f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  }
  using raw = uint2;
  __device__ static __forceinline__ raw zero() { return uint2{0, 0}; }
};
template <>
struct Quad<float> {
  __device__ static __forceinline__ uint4 load(const float* p) { return ld16(p); }
  __device__ static __forceinline__ uint4 load_nt(const float* p) { return ld16_nt(p); }
  __device__ static __forceinline__ void unpack(const uint4& v, float (&f)[4]) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  using raw = uint4;
  __device__ static __forceinline__ raw zero() { return uint4{0, 0, 0, 0}; }
};

// --------------------------------------------------- ordered 64-bit keys ----
// A selection key orders (score descending, index ascending) as one unsigned
// 64-bit integer, larger = better: the high word is the score mapped to an
// order-preserving unsigned value (-0 folded onto +0), the low word is the
// bitwise complement of the index.  Key 0 is never produced by a finite or
// infinite score and serves as "empty".
__device__ __forceinline__ uint32_t f32_to_ordered(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
// The smallest float above a finite x (-0 counts as +0): for finite z,
// z >= next_up(x) exactly when z > x.
__device__ __forceinline__ float next_up(float x) {
  uint32_t u = __float_as_uint(x);
  if (u == 0x80000000u) u = 0u;
  u = (u & 0x80000000u) ? u - 1u : u + 1u;
  return __uint_as_float(u);
}
__device__ __forceinline__ float ordered_to_f32(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t make_key(float score, uint32_t index) {
  return (uint64_t(f32_to_ordered(score)) << 32) | uint64_t(~index);
}
__device__ __forceinline__ float key_score(uint64_t key) { return ordered_to_f32(uint32_t(key >> 32)); }
__device__ __forceinline__ uint32_t key_index(uint64_t key) { return ~uint32_t(key); }

// ---------------------------------------------------------- shuffles ----
// Value of lane (lane ^ MASK) for a constant MASK.  Distances 1 and 2 are DPP
// quad permutations (a VALU operand modifier); 4 is two DPP row shifts, each
// writing the 4-lane banks that take it (+4 for banks 0 and 2, -4 for 1 and
// 3); 8 is a DPP rotation of each 16-lane row by 8; 16 is ds_swizzle in
// bit-mask mode (xor within 32 lanes: no address operand, no LDS access);
// only 32 takes a ds_bpermute.
template <int MASK>
__device__ __forceinline__ uint32_t xor_lane(uint32_t v) {
  static_assert(MASK > 0 && MASK < WAVE && (MASK & (MASK - 1)) == 0, "power-of-two lane distance");
  if constexpr (MASK == 1) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
  } else if constexpr (MASK == 2) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
  } else if constexpr (MASK == 4) {
    const int up = __builtin_amdgcn_update_dpp((int)v, (int)v, 0x104, 0xF, 0x5, false);  // row_shl:4
    return (uint32_t)__builtin_amdgcn_update_dpp(up, (int)v, 0x114, 0xF, 0xA, false);    // row_shr:4
  } else if constexpr (MASK == 8) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else if constexpr (MASK == 16) {
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (MASK << 10));  // and 0x1f, xor MASK
  } else {
    return __shfl_xor(v, MASK, WAVE);
  }
}
// The same for a run-time distance that unrolling turns into a constant.
__device__ __forceinline__ uint32_t xor_lane_rt(uint32_t v, int mask) {
  switch (mask) {
    case 1: return xor_lane<1>(v);
    case 2: return xor_lane<2>(v);
    case 4: return xor_lane<4>(v);
    case 8: return xor_lane<8>(v);
    case 16: return xor_lane<16>(v);
    default: return __shfl_xor(v, mask, WAVE);
  }
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  const uint32_t lo = xor_lane_rt(uint32_t(v), mask);
  const uint32_t hi = xor_lane_rt(uint32_t(v >> 32), mask);
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl(uint32_t(v), src, WAVE);
  uint32_t hi = __shfl(uint32_t(v >> 32), src, WAVE);
  return (uint64_t(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }

// Sum over groups of G consecutive lanes (G a power of two <= 64); every lane
// of a group ends with the group's sum.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int m = G / 2; m >= 1; m >>= 1) v += __shfl_xor(v, m, WAVE);
  return v;
}

// --------------------------------------------------- sorting networks ----
// max(a, b) and min(a, b) of finite or infinite floats as med3 against an
// infinity passed in a register: one instruction each, where fmaxf / fminf
// also quieten both inputs first.
__device__ __forceinline__ float max_med3(float a, float b, float pinf) {
  return __builtin_amdgcn_fmed3f(a, b, pinf);
}
__device__ __forceinline__ float min_med3(float a, float b, float ninf) {
  return __builtin_amdgcn_fmed3f(a, b, ninf);
}
// +inf and -inf in scalar registers, out of the compiler's sight (with a
// literal infinity med3 would be turned back into fmaxf / fminf).
__device__ __forceinline__ float opaque_pinf() {
  float x;
  asm("s_mov_b32 %0, 0x7f800000" : "=s"(x));
  return x;
}
__device__ __forceinline__ float opaque_ninf() {
  float x;
  asm("s_mov_b32 %0, 0xff800000" : "=s"(x));
  return x;
}

// Bitonic sort of a register array, descending (element 0 largest).
template <int N>
__device__ __forceinline__ void sort_desc_regs(float (&v)[N], float pinf, float ninf) {
#pragma unroll
  for (int size = 2; size <= N; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
      for (int i = 0; i < N; ++i) {
        const int j = i ^ stride;
        if (j > i) {
          const bool desc = (i & size) == 0;
          const float a = v[i], b = v[j];
          v[i] = desc ? max_med3(a, b, pinf) : min_med3(a, b, ninf);
          v[j] = desc ? min_med3(a, b, ninf) : max_med3(a, b, pinf);
        }
      }
    }
  }
}

// Bitonic merge of a register array that is already bitonic, descending.
template <int N>
__device__ __forceinline__ void merge_desc_regs(float (&v)[N], float pinf, float ninf) {
#pragma unroll
  for (int stride = N >> 1; stride > 0; stride >>= 1) {
#pragma unroll
    for (int i = 0; i < N; ++i) {
      const int j = i ^ stride;
      if (j > i) {
        const float a = v[i], b = v[j];
        v[i] = max_med3(a, b, pinf);
        v[j] = min_med3(a, b, ninf);
      }
    }
  }
}

// Lanes l with (l & m) == 0, for m a power of two up to 32.
__device__ __forceinline__ constexpr uint64_t lanes_bit_clear(int m) {
  return m == 1    ? 0x5555555555555555ull
         : m == 2  ? 0x3333333333333333ull
         : m == 4  ? 0x0F0F0F0F0F0F0F0Full
         : m == 8  ? 0x00FF00FF00FF00FFull
         : m == 16 ? 0x0000FFFF0000FFFFull
                   : 0x00000000FFFFFFFFull;
}
// Per-lane choice between a (bit clear) and b (bit set) by a lane mask held
// in scalar registers.
__device__ __forceinline__ uint32_t sel_lanes(uint32_t a, uint32_t b, uint64_t m) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "s"(m));
  return r;
}

// Bitonic sort, descending, of 64*E keys held by one wave: element
// e = r * 64 + lane lives in v[r] of that lane.  Afterwards element 0
// (lane 0, v[0]) is the largest.  A compare-exchange across lanes is one
// 64-bit compare into a lane mask, a scalar XNOR with the constant mask of
// lanes that keep the larger key, and two selects.  Every lane of the wave
// must be active.
template <int E>
__device__ __forceinline__ void wave_sort_desc(uint64_t (&v)[E], int lane) {
#pragma unroll
  for (int size = 2; size <= WAVE * E; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride >= WAVE) {
        const int rs = stride / WAVE;
#pragma unroll
        for (int r = 0; r < E; ++r) {
          const int r2 = r ^ rs;
          if (r2 > r) {
            const bool desc = ((r * WAVE + lane) & size) == 0;
            const uint64_t a = v[r], b = v[r2];
            const bool swap = desc ? (a < b) : (a > b);
            v[r] = swap ? b : a;
            v[r2] = swap ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < E; ++r) {
          const uint64_t p = shfl_xor_u64(v[r], stride);
          // lanes sorting their group of `size` descending; the lower lane of
          // each pair keeps the larger key there, the upper one elsewhere
          const uint64_t desc = size < WAVE ? lanes_bit_clear(size)
                                            : (((r * WAVE) & size) == 0 ? ~0ull : 0ull);
          const uint64_t keep_max = ~(lanes_bit_clear(stride) ^ desc);
          const uint64_t gt = __builtin_amdgcn_ballot_w64(v[r] > p);
          const uint64_t own = ~(gt ^ keep_max);
          const uint32_t lo = sel_lanes(uint32_t(p), uint32_t(v[r]), own);
          const uint32_t hi = sel_lanes(uint32_t(p >> 32), uint32_t(v[r] >> 32), own);
          v[r] = (uint64_t(hi) << 32) | lo;
        }
      }
    }
  }
}

}  // namespace pk
