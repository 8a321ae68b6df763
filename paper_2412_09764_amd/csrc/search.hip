// Product-key search on gfx950 (Sec. 3.1.1 of "Memory Layers at Scale";
// softmax of Sec. 3, Eq. (1)).
//
// Step 1, k_score_topk: for every (token, head, half) row, the top k of the S
// half-key scores s[i] = q_half . K_half[i], ordered (score desc, index asc).
//   * A workgroup owns SEARCH_TOK = 512 tokens (16 waves of 32, four per SIMD)
//     of one (head, half); the (head, half) index is blockIdx % (2H), so with
//     2H = 8 each XCD streams only its own sub-key table and keeps it in its
//     L2.  The kernel fits 128 registers, which is what four waves per SIMD
//     allow.
//   * Scores come from v_mfma_f32_32x32x16_bf16 (fp32 inputs: 32x32x2 f32) with
//     sub-keys as the A operand (M = 32 sub-keys) and the wave's 32 queries as
//     the register-resident B operand (N = 32 tokens); sub-key chunks of 64 rows
//     are copied into LDS by buffer LDS-DMA, double buffered, and read as
//     fragments one MFMA step ahead of their use.  Scores never leave
//     registers.  A 32-row tile is one chain of dependent MFMAs, then the
//     pass works on its 16 accumulator slots per lane; half of the waves on
//     each SIMD run one tile behind the others, so one half's vector work
//     meets the other half's matrix work.
//   * Threshold: per token, the maximum of each of 64 interleaved groups of
//     sub-keys (group = row mod 64), kept as 16-bit floats rounded toward
//     zero, two per register; the k-th largest of those maxima, one 16-bit
//     step down, has at least k distinct scores at or above it, so no score
//     below it can be selected.  It is found by sorting each lane's 32
//     maxima and a binary search for the split between the two lanes'
//     sorted runs (left in LDS).
//   * Sweeps: the first P1 chunks of rows give group maxima and a first
//     threshold; the rest, in doubling segments, are filtered against the
//     current threshold while the maxima are completed (a new threshold
//     after each segment, the last from all rows); the first P1 chunks are
//     then filtered against the final one (their products recomputed bitwise
//     alike).  P1 is half of the chunks (1.5 sweeps in all), a quarter from
//     32 chunks and an eighth from SPLIT8 chunks up.  Every score at or above
//     its threshold goes, as a raw 64-bit (row | lane << 16, score) record,
//     to the wave's candidate run (about 96 per row of 2048 at k = 32).  A
//     tile's candidates are found with one compare per slot into a per-lane
//     mask and taken out in rounds (each lane its two lowest remaining slots
//     per round, the scores read back from a per-wave LDS scratch), a
//     round's records packed across lanes, so a tile costs about as many
//     stores as the most candidates any lane has in it, and the run is
//     written in whole lines.
//     A lane holding k records taken against the current threshold (within
//     one pass over increasing rows) takes only scores above the lowest of
//     them from then on (lower indices win ties), so rows of tied scores stay
//     within bounds.
//   * Pass 3, k_topk_sort, a kernel of its own (a sort needs few registers, so
//     it runs at far higher occupancy than the scoring kernel): per wave run
//     the records below their row's final threshold are dropped, the rest
//     bucketed by token in LDS, and each token's sorted by one wave, the
//     first k written.  A run past its capacity, or a token with more than
//     256 records at its threshold, is listed for k_topk_fallback, which
//     rescans the row exactly.
//   * With query normalisation (qk-normalisation, Sec. 3.1.4) k_qnorm first
//     computes each (token, head) query's mean and rstd = 1/sqrt(var + eps)
//     (LayerNorm without affine, fp32, centred second pass); the scoring
//     kernel normalises its query fragments as it loads them and rounds them
//     to the query dtype, so the normalised queries never go through memory.
//   * With a sink (a fixed key per head), the kernel's prologue also forms
//     each half's part of q . sink[h] from the query fragments in registers.
// Step 2, k_cartesian: per (token, head) the top k of the sums s1[a] + s2[b]
//   over rank pairs with (a+1)(b+1) <= k (every other pair is beaten by at
//   least k pairs), ordered (sum desc, composed index i1*S + i2 asc), then the
//   softmax over the k selected sums (and over any extra key-value pairs the
//   caller adds, scored in the same kernel, and the sink's score).
#include "pk_device.h"
#include "pk_internal.h"

namespace pk {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(16))) float f32x16_t;

constexpr int CHUNK_ROWS = 64;  // sub-keys per LDS chunk = two MFMA tiles
#ifndef PK_SCORE_SPLIT8
#define PK_SCORE_SPLIT8 128  // chunks from which the first threshold takes an eighth of them
#endif
constexpr int SPLIT8 = PK_SCORE_SPLIT8;

// Lambdas of the scoring kernel are always inlined: register arrays indexed
// by their arguments must see those arguments as constants.
#define PK_INLINE __attribute__((always_inline))

#ifndef PK_SCORE_PREFETCH
#define PK_SCORE_PREFETCH 1  // LDS fragments read this many MFMA steps ahead (0: none)
#endif

template <typename T>
struct MfmaOp;

template <>
struct MfmaOp<uint16_t> {  // bf16 storage
  static constexpr int KSTEP = 16;  // reduction elements per instruction
  static constexpr int LANE_K = 8;  // reduction elements supplied per lane
  static constexpr int ESIZE = 2;
  using frag = bf16x8_t;
  __device__ static __forceinline__ f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ frag load(const void* p) {
    return __builtin_bit_cast(frag, *reinterpret_cast<const uint4*>(p));
  }
  __device__ static __forceinline__ frag zero() { return __builtin_bit_cast(frag, uint4{0, 0, 0, 0}); }
  __device__ static __forceinline__ float to_f32(uint16_t v) { return bf16_to_f32(v); }
  __device__ static __forceinline__ float stored(float v) { return round_bf16_f32(v); }
  // sum over the fragment's 8 elements of f[i] * s[i] (s: 8 bf16, 16-byte aligned)
  __device__ static __forceinline__ float dot(frag f, const uint16_t* s) {
    const uint4 u = __builtin_bit_cast(uint4, f);
    const uint4 v = *reinterpret_cast<const uint4*>(s);
    float a = bf16_lo(u.x) * bf16_lo(v.x);
    a = fmaf(bf16_hi(u.x), bf16_hi(v.x), a);
    a = fmaf(bf16_lo(u.y), bf16_lo(v.y), a);
    a = fmaf(bf16_hi(u.y), bf16_hi(v.y), a);
    a = fmaf(bf16_lo(u.z), bf16_lo(v.z), a);
    a = fmaf(bf16_hi(u.z), bf16_hi(v.z), a);
    a = fmaf(bf16_lo(u.w), bf16_lo(v.w), a);
    return fmaf(bf16_hi(u.w), bf16_hi(v.w), a);
  }
  // Normalised fragment, rounded to bf16 (nearest, ties to even).
  __device__ static __forceinline__ frag normalize(frag f, float mean, float rstd) {
    uint4 u = __builtin_bit_cast(uint4, f);
    u.x = pack_bf16x2(qn_apply(bf16_lo(u.x), mean, rstd), qn_apply(bf16_hi(u.x), mean, rstd));
    u.y = pack_bf16x2(qn_apply(bf16_lo(u.y), mean, rstd), qn_apply(bf16_hi(u.y), mean, rstd));
    u.z = pack_bf16x2(qn_apply(bf16_lo(u.z), mean, rstd), qn_apply(bf16_hi(u.z), mean, rstd));
    u.w = pack_bf16x2(qn_apply(bf16_lo(u.w), mean, rstd), qn_apply(bf16_hi(u.w), mean, rstd));
    return __builtin_bit_cast(frag, u);
  }
};

template <>
struct MfmaOp<float> {
  static constexpr int KSTEP = 2;
  static constexpr int LANE_K = 1;
  static constexpr int ESIZE = 4;
  using frag = float;
  __device__ static __forceinline__ f32x16_t mma(frag a, frag b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ frag load(const void* p) { return *reinterpret_cast<const float*>(p); }
  __device__ static __forceinline__ frag zero() { return 0.f; }
  __device__ static __forceinline__ float to_f32(float v) { return v; }
  __device__ static __forceinline__ float stored(float v) { return v; }
  __device__ static __forceinline__ frag normalize(frag f, float mean, float rstd) {
    return qn_apply(f, mean, rstd);
  }
};

// Per (token, head) query of n elements (n * esize <= 1 KiB): mean and
// rstd = 1 / sqrt(var + eps) of LayerNorm without affine (biased variance,
// fp32, centred second pass; rstd = 0 where var + eps == 0), one wave per
// four queries (their loads issued together), lane l holding the 16-byte
// chunk l of each.  qhat (optional) receives the
// normalised query rounded to the query dtype, exactly as the scoring uses it.
constexpr int QNORM_ROWS = 4;  // query rows per wave

template <typename T>
__global__ __launch_bounds__(256) void k_qnorm(const T* __restrict__ q, int64_t rows, int n,
                                               float eps, float2* __restrict__ stats,
                                               T* __restrict__ qhat) {
  constexpr int EPL = 16 / (int)sizeof(T);
  using M = MfmaOp<T>;
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * QNORM_ROWS;
  if (r0 >= rows) return;  // whole wave
  const bool has = lane * EPL < n;
  // the wave's rows loaded together, then each reduced on its own
  float x[QNORM_ROWS][EPL];
#pragma unroll
  for (int j = 0; j < QNORM_ROWS; ++j) {
    const int64_t r = r0 + j;
    const uint4 raw = (has && r < rows) ? ld16(q + r * n + lane * EPL) : uint4{0, 0, 0, 0};
    const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int i = 0; i < EPL; ++i) x[j][i] = M::to_f32(e[i]);
  }
#pragma unroll
  for (int j = 0; j < QNORM_ROWS; ++j) {
    const int64_t r = r0 + j;
    if (r >= rows) break;  // the same for the whole wave
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < EPL; ++i) sum += x[j][i];
    sum = group_sum<WAVE>(sum);
    const float mean = sum / (float)n;
    float sq = 0.f;
    if (has) {
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const float c = x[j][i] - mean;
        sq = fmaf(c, c, sq);
      }
    }
    sq = group_sum<WAVE>(sq);
    const float ve = sq / (float)n + eps;
    const float rstd = ve > 0.f ? 1.f / sqrtf(ve) : 0.f;
    if (lane == 0) stats[r] = make_float2(mean, rstd);
    if (qhat && has) {
      uint4 o;
      T* e = reinterpret_cast<T*>(&o);
#pragma unroll
      for (int i = 0; i < EPL; ++i) {
        const float v = M::stored(qn_apply(x[j][i], mean, rstd));
        if constexpr (sizeof(T) == 2) e[i] = (T)(__float_as_uint(v) >> 16);
        else e[i] = v;
      }
      *reinterpret_cast<uint4*>(qhat + r * n + lane * EPL) = o;
    }
  }
}

// Row of the 32x32 MFMA result held in accumulator slot j of a lane whose
// upper-half bit is kh (columns are lane & 31).
__device__ __forceinline__ int acc_row(int j, int kh) { return 8 * (j >> 2) + 4 * kh + (j & 3); }

typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Group maxima of the scoring kernel: pairs of 16-bit floats rounded toward
// zero from fp32 scores (two groups per register).
typedef _Float16 h16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ h16x2_t pk_rtz(float lo, float hi) {
  return __builtin_bit_cast(h16x2_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
}
// Element-wise maximum of two pairs (the inputs are never signalling NaNs, so
// the instruction needs none of the quieting that maxnum would add).
__device__ __forceinline__ void pk_max_into(h16x2_t& a, h16x2_t b) {
  asm("v_pk_max_f16 %0, %0, %1" : "+v"(a) : "v"(b));
}
__device__ __forceinline__ h16x2_t pk_max2(h16x2_t a, h16x2_t b) {
  h16x2_t r;
  asm("v_pk_max_f16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ h16x2_t pk_min2(h16x2_t a, h16x2_t b) {
  h16x2_t r;
  asm("v_pk_min_f16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// (max(a.lo, b.hi), max(a.hi, b.lo)) and the same with min: b's halves
// crossed by the operand selects.
__device__ __forceinline__ h16x2_t pk_max_x(h16x2_t a, h16x2_t b) {
  h16x2_t r;
  asm("v_pk_max_f16 %0, %1, %2 op_sel:[0,1] op_sel_hi:[1,0]" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ h16x2_t pk_min_x(h16x2_t a, h16x2_t b) {
  h16x2_t r;
  asm("v_pk_min_f16 %0, %1, %2 op_sel:[0,1] op_sel_hi:[1,0]" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// (a.lo, b.lo)
__device__ __forceinline__ h16x2_t pk_pack_lo(h16x2_t a, h16x2_t b) {
  h16x2_t r;
  asm("v_pack_b32_f16 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Sorts the 32 16-bit floats of r descending, in place: afterwards r[m] holds
// elements 2m (low half) and 2m + 1 (high half) of the order.  Two operations
// per pair of compare-exchanges: the low halves and the high halves are
// first sorted as two sequences of 16 by one bitonic network applied to both
// at once; X (the low halves) followed by Y (the high halves) reversed is
// then a bitonic sequence whose mirror pairs (element j, element 31 - j) are
// exactly the registers (X[j], Y[j]).  Each half-cleaner step of its merge
// keeps that form for the two halves it produces (one max and one min with
// the second register's halves crossed per pair of registers), down to
// groups of two, which are ordered within their register.  272 instructions
// in all, no conversion to 32-bit floats.
__device__ __forceinline__ void sort_desc_f16x32(h16x2_t (&r)[16]) {
#pragma unroll
  for (int size = 2; size <= 16; size <<= 1) {
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int j = i ^ stride;
        if (j > i) {
          const h16x2_t mx = pk_max2(r[i], r[j]), mn = pk_min2(r[i], r[j]);
          const bool desc = (i & size) == 0;
          r[i] = desc ? mx : mn;
          r[j] = desc ? mn : mx;
        }
      }
    }
  }
  // merge: groups of G elements held as G / 2 mirror-pair registers
  // (element j, element G - 1 - j), group g at registers g * G / 2 ...
#pragma unroll
  for (int G = 32; G > 2; G >>= 1) {
    h16x2_t n[16];
#pragma unroll
    for (int g = 0; g < 32 / G; ++g) {
#pragma unroll
      for (int j = 0; j < G / 4; ++j) {
        const h16x2_t a = r[g * (G / 2) + j], b = r[g * (G / 2) + G / 2 - 1 - j];
        n[(2 * g) * (G / 4) + j] = pk_max_x(a, b);      // the larger half of the group
        n[(2 * g + 1) * (G / 4) + j] = pk_min_x(a, b);  // the smaller half
      }
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) r[i] = n[i];
  }
#pragma unroll
  for (int m = 0; m < 16; ++m) r[m] = pk_pack_lo(pk_max_x(r[m], r[m]), pk_min_x(r[m], r[m]));
}
// The next 16-bit float below t (t holds a 16-bit float value exactly; -inf
// stays -inf).
__device__ __forceinline__ float f16_step_down(float t) {
  const uint32_t hb = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)t);
  uint32_t r = (hb & 0x8000u) ? hb + 1u : hb - 1u;  // negative (and -0): one step more negative;
                                                     // positive: one step toward zero
  r = hb == 0x0000u ? 0x8001u : r;                   // +0: the smallest negative value
  r = hb == 0xFC00u ? hb : r;                        // -inf stays
  return (float)__builtin_bit_cast(_Float16, (uint16_t)r);
}

// Bit j of the result is acc[j] >= b. Sixteen compares into three rotating
// SGPR pairs, each consumed by an add with carry (m + m + c) two VALU
// instructions after it was written: the hardware's wait states between a
// VALU write of an SGPR and a VALU read of it are covered by independent work
// instead of s_nop.
__device__ __forceinline__ uint32_t mask16(const f32x16_t& acc, float b) {
  uint32_t m;
  uint64_t c0, c1, c2;
  asm(
      "v_cmp_ge_f32_e64 %[c0], %[z15], %[b]\n\t"
      "v_cmp_ge_f32_e64 %[c1], %[z14], %[b]\n\t"
      "v_cmp_ge_f32_e64 %[c2], %[z13], %[b]\n\t"
      "v_cndmask_b32_e64 %[m], 0, 1, %[c0]\n\t"
      "v_cmp_ge_f32_e64 %[c0], %[z12], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c1]\n\t"
      "v_cmp_ge_f32_e64 %[c1], %[z11], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c2]\n\t"
      "v_cmp_ge_f32_e64 %[c2], %[z10], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c0]\n\t"
      "v_cmp_ge_f32_e64 %[c0], %[z9], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c1]\n\t"
      "v_cmp_ge_f32_e64 %[c1], %[z8], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c2]\n\t"
      "v_cmp_ge_f32_e64 %[c2], %[z7], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c0]\n\t"
      "v_cmp_ge_f32_e64 %[c0], %[z6], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c1]\n\t"
      "v_cmp_ge_f32_e64 %[c1], %[z5], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c2]\n\t"
      "v_cmp_ge_f32_e64 %[c2], %[z4], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c0]\n\t"
      "v_cmp_ge_f32_e64 %[c0], %[z3], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c1]\n\t"
      "v_cmp_ge_f32_e64 %[c1], %[z2], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c2]\n\t"
      "v_cmp_ge_f32_e64 %[c2], %[z1], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c0]\n\t"
      "v_cmp_ge_f32_e64 %[c0], %[z0], %[b]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c1]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c2]\n\t"
      "v_addc_co_u32_e64 %[m], vcc, %[m], %[m], %[c0]"
      : [m] "=&v"(m), [c0] "=&s"(c0), [c1] "=&s"(c1), [c2] "=&s"(c2)
      : [b] "v"(b),
        [z0] "v"(acc[0]), [z1] "v"(acc[1]), [z2] "v"(acc[2]), [z3] "v"(acc[3]), [z4] "v"(acc[4]), [z5] "v"(acc[5]), [z6] "v"(acc[6]), [z7] "v"(acc[7]), [z8] "v"(acc[8]), [z9] "v"(acc[9]), [z10] "v"(acc[10]), [z11] "v"(acc[11]), [z12] "v"(acc[12]), [z13] "v"(acc[13]), [z14] "v"(acc[14]), [z15] "v"(acc[15])
      : "vcc");
  return m;
}

// KBIG (k > 32): the threshold comes from all rows (P = all chunks: no second
// sweep).
template <typename T, int NSTEP, bool KBIG>
__global__ __launch_bounds__(64 * SEARCH_WAVES, 4) void k_score_topk(
    const T* __restrict__ q, const T* __restrict__ subkeys, int64_t ntok, int H, int n, int S,
    int k, const float2* __restrict__ qstats, const T* __restrict__ sink,
    float* __restrict__ sink_part, uint64_t* __restrict__ cand, uint32_t* __restrict__ cnts,
    float* __restrict__ thr) {
  using M = MfmaOp<T>;
  constexpr int DPAD = NSTEP * M::KSTEP;      // padded half dim
  constexpr int RB = DPAD * M::ESIZE;         // bytes of a sub-key row
  constexpr int NCOL = RB / 16;               // 16-byte segments per row
  constexpr int NSLOT = NCOL + 1;             // 16-byte slots per row in LDS (one spare)
  constexpr int RBP = NSLOT * 16;             // row pitch in LDS
  constexpr int EPS = 16 / M::ESIZE;          // elements per segment
  constexpr int CBYTES = CHUNK_ROWS * RBP;
  constexpr int NDMA = (NSLOT + SEARCH_WAVES - 1) / SEARCH_WAVES;  // loads per wave and chunk, at most

  // Sub-key chunks of 64 rows, double buffered, each row followed by a spare
  // 16-byte slot: with a pitch of an odd number of 16-byte slots, the 16
  // consecutive rows that one fragment read touches start in 16 different
  // bank groups, and a fragment's address is the lane's row address plus a
  // constant per step (the instruction's offset field: no address arithmetic
  // in the product loop).  The direct global -> LDS loads fill 64 consecutive
  // slots each, spare ones included (they receive a copy of the row's last
  // segment, never read).  The two buffers are statically named arrays, so
  // LDS accesses elsewhere never wait on the copies in flight.  Each wave
  // also has a scratch for taking candidates out of a tile (64 lanes x 16
  // fp32 scores), which between sweeps holds each lane's sorted group maxima
  // (32 16-bit floats) for the threshold, and a table of its lanes' source
  // offsets for the loads.
  constexpr int XS_WAVE = WAVE * 16 * 4;
  __shared__ __align__(1024) unsigned char kbuf0[CBYTES];
  __shared__ __align__(1024) unsigned char kbuf1[CBYTES];
  __shared__ __align__(16) unsigned char xsmem[SEARCH_WAVES * XS_WAVE];
  __shared__ uint32_t dtab[NDMA * SEARCH_WAVES * WAVE];

  const int d = n >> 1;
  const int HP = 2 * H;
  const int hp = blockIdx.x % HP;
  const int64_t tile = blockIdx.x / HP;
  const int h = hp >> 1, p = hp & 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kh = lane >> 5;
  const int col = lane & 31;
  const int64_t tok = tile * SEARCH_TOK + wave * 32 + col;
  const bool tok_ok = tok < ntok;
  const T* kbase = subkeys + (size_t)hp * S * d;

  // Queries of this lane's token, as B fragments: lane supplies reduction
  // elements [s*KSTEP + kh*LANE_K, +LANE_K) of column `col`; normalised here
  // when qstats holds the queries' (mean, rstd).
  typename M::frag bq[NSTEP];
  {
    const size_t qr = (size_t)(tok_ok ? tok : 0) * H + h;
    const T* qrow = q + qr * n + (size_t)p * d;
    const float2 qs = (qstats && tok_ok) ? qstats[qr] : make_float2(0.f, 1.f);
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      const int e0 = s * M::KSTEP + kh * M::LANE_K;
      const bool ld = tok_ok && e0 + M::LANE_K <= d;
      typename M::frag f = ld ? M::load(qrow + e0) : M::zero();
      if (qstats && ld) f = M::normalize(f, qs.x, qs.y);
      bq[s] = f;
    }
  }
  // With a sink (a fixed key per head scored like any full key): this half's
  // part of q . sink[h], from the fragments already in registers; the token's
  // two lanes add their parts, and k_cartesian adds the two halves.
  if (sink) {
    const T* srow = sink + (size_t)h * n + (size_t)p * d;
    float part = 0.f;
    if constexpr (M::LANE_K > 1) {  // bf16: the fragments in registers
#pragma unroll
      for (int s = 0; s < NSTEP; ++s) {
        const int e0 = s * M::KSTEP + kh * M::LANE_K;
        if (e0 + M::LANE_K <= d) part += M::dot(bq[s], srow + e0);
      }
    } else {  // fp32: one element per fragment, read again (cached) to spare registers
      const T* qrow = q + ((size_t)(tok_ok ? tok : 0) * H + h) * n + (size_t)p * d;
#pragma unroll 8
      for (int e = kh; e < d; e += 2) part = fmaf(M::to_f32(qrow[e]), M::to_f32(srow[e]), part);
    }
    part += __shfl_xor(part, 32, WAVE);
    if (kh == 0 && tok_ok) sink_part[((size_t)tok * H + h) * 2 + p] = part;
  }

  // Chunk c into buffer b: 64*NSLOT slots, 64 per wave instruction, each
  // lane's 16 bytes going to LDS at base + 16*lane.  Padded columns read a
  // valid (finite) sub-key element instead (they meet zero query entries);
  // the last, partial chunk reads row S - 1 in place of rows past S (masked
  // out later).
  // The (head, half) table as a raw buffer: S rows of d elements.
  const __amdgpu_buffer_rsrc_t ktab = raw_buffer(kbase, (uint32_t)((size_t)S * d * M::ESIZE));
  // Offset in a chunk of the sub-key bytes for slot t (row t / NSLOT, spare
  // slots repeating the row's last segment).
  auto slot_src = [&](int t, int& r) PK_INLINE {
    r = t / NSLOT;
    int g = t - r * NSLOT;
    g = g < NCOL ? g : NCOL - 1;
    int e0 = g * EPS;
    e0 = e0 < d ? e0 : 0;
    return e0 * M::ESIZE;
  };
  // The lane's source offsets within a chunk are the same for every chunk:
  // computed once into the table in LDS (read back by the lane itself), so a
  // chunk whose rows all exist costs one LDS read per load and no vector
  // arithmetic.
#pragma unroll
  for (int j = 0; j < NDMA; ++j) {
    const int i = wave + j * SEARCH_WAVES;
    if (i < NSLOT) {
      int r;
      const int eb = slot_src(i * WAVE + lane, r);
      dtab[j * SEARCH_WAVES * WAVE + tid] = (uint32_t)(r * d * M::ESIZE + eb);
    }
  }
  const int nfull_rows = S / CHUNK_ROWS;  // chunks whose 64 rows all exist
  auto issue_chunk = [&](int c, unsigned char* buf) PK_INLINE {
    if (c < nfull_rows) {
      const uint32_t cb = (uint32_t)((size_t)c * CHUNK_ROWS * d * M::ESIZE);
#pragma unroll
      for (int j = 0; j < NDMA; ++j) {
        const int i = wave + j * SEARCH_WAVES;
        if (NSLOT % SEARCH_WAVES == 0 || i < NSLOT)
          lds_dma16_buf(ktab, dtab[j * SEARCH_WAVES * WAVE + tid], cb, &buf[i * WAVE * 16]);
      }
      return;
    }
    for (int i = wave; i < NSLOT; i += SEARCH_WAVES) {
      int r;
      const int eb = slot_src(i * WAVE + lane, r);
      int row = c * CHUNK_ROWS + r;
      row = row < S ? row : S - 1;
      lds_dma16_buf(ktab, (uint32_t)((size_t)row * d * M::ESIZE + eb), 0u, &buf[i * WAVE * 16]);
    }
  };
  // ---- the sweeps -----------------------------------------------------------
  // A sweep visits every 32-row tile once, in row order.  Tile t is one chain
  // of NSTEP dependent MFMAs into the accumulator (fragments read from LDS
  // LEAD steps ahead of their use), then the pass filters its 16 slots per
  // lane.  Four waves share each SIMD (one 16-wave workgroup per CU), so one
  // wave's filtering and waits run while the others' products occupy the
  // matrix pipe.  Chunks of two tiles alternate between the two LDS buffers
  // (unrolled by two so every access names its buffer statically).
  // The lane's fragment of step s: row col of the tile, reduction elements
  // from s * KSTEP + kh * LANE_K, at lane_addr + s * KSTEP * ESIZE.
  const uint32_t lane_addr = (uint32_t)(col * RBP + kh * M::LANE_K * M::ESIZE);
  constexpr int LEAD = PK_SCORE_PREFETCH > 0 ? PK_SCORE_PREFETCH : 1;
  const int nch = (S + CHUNK_ROWS - 1) / CHUNK_ROWS;
  const int nfull = S / CHUNK_ROWS;  // chunks with all 64 rows valid

  // Rows half*32 .. half*32 + 31 of the chunk in buf into acc.
  auto run_tile = [&](const unsigned char* buf, int half, f32x16_t& acc) PK_INLINE {
    const unsigned char* rp = buf + half * 32 * RBP + lane_addr;
    acc = f32x16_t{};
    typename M::frag ring[LEAD + 1];
#pragma unroll
    for (int s = 0; s < LEAD && s < NSTEP; ++s) ring[s] = M::load(rp + s * M::KSTEP * M::ESIZE);
#pragma unroll
    for (int s = 0; s < NSTEP; ++s) {
      if (s + LEAD < NSTEP) ring[(s + LEAD) % (LEAD + 1)] = M::load(rp + (s + LEAD) * M::KSTEP * M::ESIZE);
      __builtin_amdgcn_sched_barrier(0);  // reads stay LEAD steps ahead of their use
      acc = M::mma(ring[s % (LEAD + 1)], bq[s], acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // Rows past S (the last chunk only) score -inf: no group maximum takes
  // them, and the candidate path checks the row as well.
  auto mask_tail = [&](f32x16_t& acc, int c, int half) PK_INLINE {
    const int r0 = c * CHUNK_ROWS + half * 32;
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = r0 + acc_row(j, kh) < S ? acc[j] : -INFINITY;
  };
  // Chunks [cb, ce) in order (any range; the two LDS buffers alternate);
  // tile(acc, c, half) consumes each tile.  Half of the waves on each SIMD
  // (waves 4-7 and 12-15, with wave w on SIMD w mod 4) lag by one tile: they
  // consume a chunk's second tile at the start of the next chunk, so their
  // filtering (vector ALU) runs while the other waves' products occupy the
  // matrix pipe, and the other way round.
  const bool lag = ((wave >> 2) & 1) != 0;
  // Chunk cb must already be on its way into kbuf0 (issued once both buffers
  // were free): the caller issues it before forming a threshold, so the load
  // runs under that work.
  auto sweep = [&](int cb, int ce, auto&& tile_fn) PK_INLINE {
    f32x16_t acc;
    int pc = -1;  // lagging waves: chunk whose second tile (in acc) is pending
    auto chunk = [&](const unsigned char* buf, int c) PK_INLINE {
      if (lag) {
        if (pc >= 0) tile_fn(acc, pc, 1);
        run_tile(buf, 0, acc);
        if (__builtin_expect(c >= nfull, 0)) mask_tail(acc, c, 0);
        tile_fn(acc, c, 0);
        run_tile(buf, 1, acc);
        if (__builtin_expect(c >= nfull, 0)) mask_tail(acc, c, 1);
        pc = c;
      } else {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          run_tile(buf, half, acc);
          if (__builtin_expect(c >= nfull, 0)) mask_tail(acc, c, half);
          tile_fn(acc, c, half);
        }
      }
    };
    for (int c = cb; c < ce; c += 2) {
      __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of chunk c have landed
      __syncthreads();                // ... and every wave's; kbuf1 is free
      if (c + 1 < ce) issue_chunk(c + 1, kbuf1);
      chunk(kbuf0, c);
      if (c + 1 < ce) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (c + 2 < ce) issue_chunk(c + 2, kbuf0);
        chunk(kbuf1, c + 1);
      }
    }
    if (pc >= 0) tile_fn(acc, pc, 1);
    __syncthreads();  // every wave is done with both buffers
  };

  // ---- group maxima and the threshold ---------------------------------------
  // 64 interleaved groups per token (group = row mod 64): 32 maxima in this
  // lane, 32 in lane ^ 32, kept as 16-bit floats rounded toward zero, two
  // groups per register (slots 2i and 2i + 1 of a tile are adjacent rows).
  const float pinf = opaque_pinf(), ninf = opaque_ninf();
  h16x2_t mxp[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) mxp[i] = h16x2_t{(_Float16)-INFINITY, (_Float16)-INFINITY};
  auto max_tile = [&](const f32x16_t& acc, int, int half) PK_INLINE {
#pragma unroll
    for (int i = 0; i < 8; ++i) pk_max_into(mxp[half * 8 + i], pk_rtz(acc[2 * i], acc[2 * i + 1]));
  };
  // The k-th largest of the token's 64 rounded maxima, one 16-bit step down:
  // at least k distinct scores lie at or above the result (each of the k
  // groups whose rounded maximum reaches the k-th largest holds a score above
  // the value one step below it, whichever way the rounding toward zero
  // went).  Each lane sorts its 32 in place (as 16-bit floats, two per
  // instruction) and leaves them in LDS; the k-th largest of the two sorted
  // runs (this lane's and lane ^ 32's) is then found by a binary search for
  // the split between them.  Sorting moves maxima between groups, but later
  // updates keep every value the maximum over rows of its own (each old
  // maximum and each new row goes to exactly one register half), so the
  // bound stays valid when the sweep continues afterwards.  Runs between
  // sweeps, when the chunk buffers are free.
  auto kth_of_maxima = [&]() PK_INLINE -> float {
    sort_desc_f16x32(mxp);
    uint16_t* const runs = reinterpret_cast<uint16_t*>(xsmem);  // [64 * SEARCH_WAVES][32]
    uint4* const mine = reinterpret_cast<uint4*>(runs + tid * 32);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      mine[i] = uint4{__builtin_bit_cast(uint32_t, mxp[4 * i]), __builtin_bit_cast(uint32_t, mxp[4 * i + 1]),
                      __builtin_bit_cast(uint32_t, mxp[4 * i + 2]), __builtin_bit_cast(uint32_t, mxp[4 * i + 3])};
    const uint16_t* const ra = runs + tid * 32;          // this lane's run, descending
    const uint16_t* const rb = runs + (tid ^ 32) * 32;   // the partner's
    auto at = [](const uint16_t* r, int i) PK_INLINE {
      return (float)__builtin_bit_cast(_Float16, r[i]);
    };
    // i from this run and k - i from the other: the smallest i in
    // [max(0, k - 32), min(k, 32)] at which taking one more from this run
    // would not beat the last one taken from the other.
    int lo = k > 32 ? k - 32 : 0, hi = k < 32 ? k : 32;
#pragma unroll
    for (int it = 0; it < 6; ++it) {
      if (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (at(ra, mid) > at(rb, k - 1 - mid)) lo = mid + 1;  // mid < 32 and k - mid > 0 here
        else hi = mid;
      }
    }
    const int j = k - lo;
    const float a = lo > 0 ? at(ra, lo > 0 ? lo - 1 : 0) : INFINITY;
    const float b = j > 0 ? at(rb, j > 0 ? j - 1 : 0) : INFINITY;
    return f16_step_down(a < b ? a : b);
  };

  // ---- candidate collection ---------------------------------------------------
  // A lane's candidates in a tile are the slots whose score is >= bound: one
  // compare per slot builds the lane's 16-bit candidate mask.  When any lane
  // has one, the lane's 16 scores go to its scratch in LDS and the wave takes
  // the candidates out in rounds, each lane its lowest remaining slot per
  // round (index from the mask, score read back from LDS): a tile costs a
  // compare per slot and as many stores as the most candidates any lane of
  // the wave has in it, not work per slot.  Each round's records go to the
  // wave's run packed across lanes (a lane's place is the number of lanes
  // below it with a record), so the run is written in whole lines; a record
  // is (row | lane << 16, raw fp32 score bits).  The run holds 32 * CAND_CAP
  // records; past that the buffer bound drops stores, the count goes on and
  // the wave's rows are rescanned exactly later.
  //
  // A lane meets the rows of one sweep in increasing index order, tile by
  // tile.  Once it holds k records taken against the current threshold, the
  // lowest of them, lo, is a bound of its own: a later score at or below lo
  // is beaten by all k of them (by score, or on a tie by their lower index),
  // so it cannot be selected, and the lane takes only scores above lo from
  // then on; this holds across the segments of one pass, whose rows keep
  // increasing.  Heavily tied rows (equal sub-keys) thus stay within bounds
  // (at most k + 15 records per lane and pass); the test runs once per tile.
  constexpr uint32_t RUN = 32 * CAND_CAP;  // records per wave run
  const size_t rid = ((size_t)(tok_ok ? tok : 0) * H + h) * 2 + p;
  // this wave's run (the wave index taken as uniform, so the run's buffer
  // resource lives in scalar registers as the store instruction needs)
  const size_t wr = (((size_t)tile * SEARCH_WAVES + __builtin_amdgcn_readfirstlane(wave)) * H + h) * 2 + p;
  uint32_t taken = 0;   // records of this lane since the last restart
  uint32_t wcnt = 0;    // records of the wave (uniform)
  float bound = INFINITY;
  float lo = INFINITY;  // lowest record taken against the current threshold
  const __amdgpu_buffer_rsrc_t crs = raw_buffer(cand + wr * RUN, RUN * (uint32_t)sizeof(uint64_t));
  // This wave's scratch: slot j of lane l at float j * 64 + l (each slot's
  // write and each round's read are one conflict-free access).
  float* const xs = reinterpret_cast<float*>(xsmem + wave * XS_WAVE);
  // The last threshold set is the row's final one (what the sort keeps).
  // The records behind lo stay valid while the rows go on increasing (the
  // segments of one pass); restart when the next sweep begins again at row 0.
  auto set_threshold = [&](float t, bool restart) PK_INLINE {
    if (restart) {
      lo = INFINITY;
      taken = 0;
    }
    const float tb = tok_ok ? t : INFINITY;  // scores are finite
    bound = taken >= (uint32_t)k ? fmaxf(tb, next_up(lo)) : tb;
    if (tok_ok && kh == 0) thr[rid] = t;
  };
  auto collect_tile = [&](const f32x16_t& acc, int c, int half) PK_INLINE {
    const uint32_t r0 = (uint32_t)(c * CHUNK_ROWS + half * 32 + 4 * kh) | ((uint32_t)lane << 16);
    uint32_t msk = 0;  // bit j: slot j is a candidate
    if (c < nfull) {
      msk = mask16(acc, bound);
    } else {  // rows past S are no candidates
#pragma unroll
      for (int j = 15; j >= 0; --j)
        msk = msk * 2u + (uint32_t)(acc[j] >= bound && (r0 & 0xFFFFu) + acc_row(j, 0) < (uint32_t)S);
    }
    uint64_t m = __builtin_amdgcn_ballot_w64(msk != 0);
    if (m != 0) {  // uniform
      taken += (uint32_t)__builtin_popcount(msk);  // every candidate becomes a record
#pragma unroll
      for (int j = 0; j < 16; ++j) xs[j * WAVE + lane] = acc[j];
      do {  // two candidates per lane and round: their LDS reads in flight together
        const uint32_t m1 = msk & (msk - 1u);
        const uint32_t j0 = (uint32_t)__builtin_ctz(msk | 0x8000u);  // any slot when none
        const uint32_t j1 = (uint32_t)__builtin_ctz(m1 | 0x8000u);
        const float z0 = xs[j0 * WAVE + lane];
        const float z1 = xs[j1 * WAVE + lane];
        const uint64_t m2 = __builtin_amdgcn_ballot_w64(m1 != 0);  // lanes with a second one
        // records of the lanes below: one per lane with a candidate, one more
        // per lane with a second
        const uint32_t below =
            __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u)) +
            __builtin_amdgcn_mbcnt_hi((uint32_t)(m2 >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m2, 0u));
        const uint32_t at = (wcnt + below) * 8u;
        asm volatile("" ::"v"(z0), "v"(z1));  // both reads issued before either store
        if (msk != 0) {
          __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{r0 + j0 + (j0 & 12u), __float_as_uint(z0)}, crs, at,
                                                0, 0);
          lo = min_med3(lo, z0, ninf);
        }
        if (m1 != 0) {
          __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{r0 + j1 + (j1 & 12u), __float_as_uint(z1)}, crs,
                                                at + 8u, 0, 0);
          lo = min_med3(lo, z1, ninf);
        }
        wcnt += (uint32_t)(__popcll(m) + __popcll(m2));
        msk = m1 & (m1 - 1u);
        m = __builtin_amdgcn_ballot_w64(msk != 0);
      } while (m != 0);
    }
    bound = taken >= (uint32_t)k ? fmaxf(bound, next_up(lo)) : bound;
  };

  // ---- the sweeps ------------------------------------------------------------
  // 1. Chunks [0, P1): group maxima only; their k-th largest is a first
  //    threshold.  2. The rest in segments that double, [P1, 2 P1),
  //    [2 P1, 4 P1), ...: candidates against the current threshold, maxima
  //    still updated, then a new threshold from the maxima so far (after the
  //    last segment, the final one from all rows).  3. Chunks [0, P1) again:
  //    candidates against the final threshold.  Every score of the top k is
  //    at or above each threshold, so every one is collected; the products
  //    over [0, P1) are computed twice, bitwise alike.  P1 = half of the
  //    chunks (1.5 sweeps) below 32 chunks, a quarter (1.25) from 32 and an
  //    eighth (1.125) from SPLIT8 chunks up: with fewer chunks the looser
  //    early thresholds and the extra ones cost more than the shorter first
  //    sweep saves, counting the candidate sort's share (measured).  With k > 32 P1 = all of them (one threshold
  //    from all rows, then one filtering sweep).
  const int P1 = KBIG ? nch : nch >= SPLIT8 ? (nch + 7) / 8 : nch >= 32 ? (nch + 3) / 4 : (nch + 1) / 2;
  auto max_collect = [&](const f32x16_t& acc, int c, int half) PK_INLINE {
    max_tile(acc, c, half);
    collect_tile(acc, c, half);
  };
  issue_chunk(0, kbuf0);
  sweep(0, P1, max_tile);
  issue_chunk(P1 < nch ? P1 : 0, kbuf0);  // the next sweep's first chunk, under the threshold
  set_threshold(kth_of_maxima(), true);
  for (int lo_c = P1; lo_c < nch;) {
    const int hi_c = 2 * lo_c < nch ? 2 * lo_c : nch;
    sweep(lo_c, hi_c, max_collect);
    issue_chunk(hi_c < nch ? hi_c : 0, kbuf0);
    set_threshold(kth_of_maxima(), hi_c >= nch);  // the last: sweep 3 restarts at row 0
    lo_c = hi_c;
  }
  sweep(0, P1, collect_tile);
  if (lane == 0) cnts[wr] = wcnt;
}

// Pass 3 as a kernel of its own: one workgroup per wave run (32 tokens of one
// head and half).  Its records are read in order, those below their row's
// final threshold (taken against a looser one) dropped, and the places of the
// rest gathered into per-token buckets in LDS (16-bit record numbers, so the
// buckets stay small and many workgroups share a CU); then each wave takes
// tokens in turn, reads its records again (from L2), sorts them as
// (score desc, index asc) keys and writes the first k.  A run past
// its capacity, or a token with more than BCAP records at or above its
// threshold, goes to the rescan list.
constexpr int SORT_BCAP = 4 * WAVE;  // records a token may keep for the sort
__global__ __launch_bounds__(256) void k_topk_sort(const uint64_t* __restrict__ cand,
                                                   const uint32_t* __restrict__ cnts,
                                                   const float* __restrict__ thr,
                                                   int64_t ntok, int H, int k,
                                                   int32_t* __restrict__ half_idx,
                                                   float* __restrict__ half_score,
                                                   uint32_t* __restrict__ ovf) {
  constexpr uint32_t RUN = 32 * CAND_CAP;
  __shared__ uint16_t bucket[32][SORT_BCAP];
  __shared__ uint32_t bcnt[32];
  __shared__ float bthr[32];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t nruns = (ntok + 31) / 32 * H * 2;
  for (int64_t wr = blockIdx.x; wr < nruns; wr += gridDim.x) {
    const int p = (int)(wr & 1);
    const int h = (int)((wr >> 1) % H);
    const int64_t tok0 = (wr >> 1) / H * 32;
    if (tid < 32) {
      const int64_t t = tok0 + tid;
      bcnt[tid] = 0;
      bthr[tid] = t < ntok ? thr[((size_t)t * H + h) * 2 + p] : INFINITY;
    }
    __syncthreads();
    const uint32_t c = cnts[wr];
    const uint64_t* run = cand + (size_t)wr * RUN;
    if (c <= RUN) {
      // four records per thread and pass, their loads in flight together
      for (uint32_t i0 = tid; i0 < c; i0 += 4 * 256) {
        uint64_t rec[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t i = i0 + (uint32_t)u * 256u;
          rec[u] = i < c ? run[i] : 0ull;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t i = i0 + (uint32_t)u * 256u;
          const uint32_t col = (uint32_t)(rec[u] >> 16) & 31u;
          const float z = __uint_as_float(uint32_t(rec[u] >> 32));
          if (i < c && z >= bthr[col]) {
            const uint32_t slot = atomicAdd(&bcnt[col], 1u);
            if (slot < (uint32_t)SORT_BCAP) bucket[col][slot] = (uint16_t)i;
          }
        }
      }
    }
    __syncthreads();
    auto key_at = [&](int col, uint32_t n, uint32_t x) PK_INLINE -> uint64_t {
      if (x >= n) return 0ull;
      const uint64_t rec = run[bucket[col][x]];
      return make_key(__uint_as_float(uint32_t(rec >> 32)), (uint32_t)rec & 0xFFFFu);
    };
    auto write_top = [&](size_t r, uint64_t top) PK_INLINE {
      if (lane < k) {
        half_idx[r * k + lane] = (int32_t)key_index(top);
        half_score[r * k + lane] = key_score(top);
      }
    };
    auto row_of = [&](int col) PK_INLINE { return ((size_t)(tok0 + col) * H + h) * 2 + p; };
    // one token: its records sorted 64, 128 or 256 wide, or the rescan list
    auto one = [&](int col) PK_INLINE {
      const size_t r = row_of(col);
      const uint32_t n = bcnt[col];
      if (c > RUN || n > (uint32_t)SORT_BCAP) {
        if (lane == 0) {
          const uint32_t slot = atomicAdd(&ovf[0], 1u);
          ovf[1 + slot] = (uint32_t)r;
        }
        return;
      }
      if (n <= (uint32_t)WAVE) {
        uint64_t v[1] = {key_at(col, n, (uint32_t)lane)};
        wave_sort_desc<1>(v, lane);
        write_top(r, v[0]);
      } else if (n <= 2u * WAVE) {
        uint64_t v[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) v[e] = key_at(col, n, (uint32_t)(lane + e * WAVE));
        wave_sort_desc<2>(v, lane);
        write_top(r, v[0]);
      } else {
        uint64_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = key_at(col, n, (uint32_t)(lane + e * WAVE));
        wave_sort_desc<4>(v, lane);
        write_top(r, v[0]);
      }
    };
    // Tokens col and col + 4 per pass: when both keep at most 64 records (the
    // usual case), their reads and their two sorts run side by side.
    for (int col = wave; col < 32; col += 8) {
      if (tok0 + col >= ntok) break;  // the same for the whole wave
      const int colB = col + 4;
      const bool hasB = tok0 + colB < ntok;
      const uint32_t nA = bcnt[col], nB = hasB ? bcnt[colB] : 0u;
      if (c <= RUN && hasB && nA <= (uint32_t)WAVE && nB <= (uint32_t)WAVE) {
        uint64_t va[1] = {key_at(col, nA, (uint32_t)lane)};
        uint64_t vb[1] = {key_at(colB, nB, (uint32_t)lane)};
        wave_sort_desc<1>(va, lane);
        wave_sort_desc<1>(vb, lane);
        write_top(row_of(col), va[0]);
        write_top(row_of(colB), vb[0]);
      } else {
        one(col);
        if (hasB) one(colB);
      }
    }
    __syncthreads();  // the buckets are reused by the next run
  }
}

// Exact rescan of rows whose candidate list overflowed: all S scores of the row
// in LDS, then k rounds of workgroup arg-max over the (score, index) keys, each
// round restricted to keys below the previous winner (keys are distinct).
template <typename T>
__global__ __launch_bounds__(256) void k_topk_fallback(const T* __restrict__ q,
                                                       const T* __restrict__ subkeys, int H, int n,
                                                       int S, int k,
                                                       const float2* __restrict__ qstats,
                                                       const uint32_t* __restrict__ ovf,
                                                       int32_t* __restrict__ half_idx,
                                                       float* __restrict__ half_score) {
  extern __shared__ float sc[];  // S scores
  __shared__ uint64_t red[4];
  __shared__ float qv[256];      // the row's query half as scored (d <= 256)
  using M = MfmaOp<T>;
  const int d = n >> 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t count = ovf[0];
  for (uint32_t it = blockIdx.x; it < count; it += gridDim.x) {
    const size_t r = ovf[1 + it];
    const int p = (int)(r & 1);
    const int h = (int)((r >> 1) % (size_t)H);
    const size_t t = (r >> 1) / (size_t)H;
    const T* qrow = q + (t * H + h) * (size_t)n + (size_t)p * d;
    const T* kb = subkeys + (size_t)(h * 2 + p) * S * d;
    if (tid < d) {
      float v = M::to_f32(qrow[tid]);
      if (qstats) {
        const float2 qs = qstats[t * H + h];
        v = M::stored(qn_apply(v, qs.x, qs.y));
      }
      qv[tid] = v;
    }
    __syncthreads();
    for (int s = tid; s < S; s += 256) {
      float acc = 0.f;
      for (int e = 0; e < d; ++e) acc = fmaf(qv[e], M::to_f32(kb[(size_t)s * d + e]), acc);
      sc[s] = acc;
    }
    __syncthreads();
    uint64_t prev = ~0ull;
    for (int kk = 0; kk < k; ++kk) {
      uint64_t best = 0;
      for (int s = tid; s < S; s += 256) {
        const uint64_t key = make_key(sc[s], (uint32_t)s);
        if (key < prev) best = umax64(best, key);
      }
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) best = umax64(best, shfl_xor_u64(best, m));
      if (lane == 0) red[wave] = best;
      __syncthreads();
      best = umax64(umax64(red[0], red[1]), umax64(red[2], red[3]));
      if (tid == 0) {
        half_idx[r * k + kk] = (int32_t)key_index(best);
        half_score[r * k + kk] = key_score(best);
      }
      prev = best;
      __syncthreads();
    }
  }
}

// Extra key-value pairs (EXTRA): the row's nex caller-given composed indices
// are scored like any full key, q1 . K1[i1] + q2 . K2[i2] (lane l holds
// elements 4l..4l+3 of each half, fp32 products summed over the wave), and
// occupy slots k .. k + nex - 1 after the selected ones; the softmax runs over
// all k + nex.  An index outside [0, S*S) is read as 0 (no out-of-bounds
// access) and written out as given.  With a sink (a fixed key-value pair per
// head), one more slot follows: its score is the sum of the two halves' parts
// of q . sink[h] that the scoring kernel left in sink_part, and its index is
// sink_row0 + h.
// MODE: 0 = the k selected only, 1 = extra pairs (and the sink, if given),
// 2 = the sink only.
template <int E, typename T, int MODE>
__global__ __launch_bounds__(256) void k_cartesian(const int32_t* __restrict__ half_idx,
                                                   const float* __restrict__ half_score,
                                                   int64_t rows, int S, int k, int npairs,
                                                   const T* __restrict__ q,
                                                   const T* __restrict__ subkeys, int H, int n,
                                                   const int64_t* __restrict__ ex_idx, int nex,
                                                   const float* __restrict__ sink_part,
                                                   int64_t sink_row0,
                                                   int64_t* __restrict__ idx_out,
                                                   float* __restrict__ w_out,
                                                   float* __restrict__ score_out) {
  __shared__ uint32_t pairs[WAVE * E];
  if (threadIdx.x == 0) {
    int m = 0;
    for (int a = 0; a < k; ++a)
      for (int b = 0; b < k / (a + 1); ++b) pairs[m++] = (uint32_t(a) << 16) | uint32_t(b);
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr bool EXTRA = MODE != 0;
  const int nsc = EXTRA ? nex + (sink_part ? 1 : 0) : 0;  // full keys scored per row
  const int kk = k + nsc;                             // slots per row
  if constexpr (!EXTRA) {
    // Two rows per pass (this wave's next grid-stride row beside it): their
    // loads, their candidate keys and their two sorts run side by side.
    auto build = [&](int64_t row, uint64_t (&v)[E]) PK_INLINE {
      const int32_t* i1 = half_idx + (size_t)row * 2 * k;
      const float* s1 = half_score + (size_t)row * 2 * k;
      const float s1v = lane < k ? s1[lane] : 0.f;
      const float s2v = lane < k ? s1[k + lane] : 0.f;
      const int i1v = lane < k ? i1[lane] : 0;
      const int i2v = lane < k ? i1[k + lane] : 0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int m = e * WAVE + lane;
        const uint32_t pr = pairs[m < npairs ? m : 0];
        const int a = (int)(pr >> 16), b = (int)(pr & 0xFFFFu);
        const float sa = __shfl(s1v, a, WAVE), sb = __shfl(s2v, b, WAVE);
        const int ia = __shfl(i1v, a, WAVE), ib = __shfl(i2v, b, WAVE);
        v[e] = m < npairs ? make_key(sa + sb, (uint32_t)ia * (uint32_t)S + (uint32_t)ib) : 0ull;
      }
    };
    auto finish = [&](int64_t row, const uint64_t (&v)[E]) PK_INLINE {
      const float z = key_score(v[0]);
      const int64_t ci = (int64_t)key_index(v[0]);
      const float zmax = __shfl(z, 0, WAVE);
      const float ex = lane < k ? expf(z - zmax) : 0.f;
      const float sum = group_sum<WAVE>(ex);
      if (lane < k) {
        const size_t o = (size_t)row * k + lane;
        idx_out[o] = ci;
        w_out[o] = ex / sum;
        if (score_out) score_out[o] = z;
      }
    };
    const int64_t stride = (int64_t)gridDim.x * 4;
    for (int64_t row = (int64_t)blockIdx.x * 4 + wave; row < rows; row += 2 * stride) {
      const bool two = row + stride < rows;             // the same for the whole wave
      const int64_t row2 = two ? row + stride : row;  // a repeated row is sorted, not written
      uint64_t va[E], vb[E];
      build(row, va);
      build(row2, vb);
      wave_sort_desc<E>(va, lane);
      wave_sort_desc<E>(vb, lane);
      finish(row, va);
      if (two) finish(row2, vb);
    }
    return;
  }
  for (int64_t row = (int64_t)blockIdx.x * 4 + wave; row < rows; row += (int64_t)gridDim.x * 4) {
    // extra pairs first: their loads overlap the candidate sort below
    float ex_score = 0.f;
    int64_t ex_given = 0;
    if constexpr (EXTRA) {
      const int h = (int)(row % H);
      const int64_t N = (int64_t)S * S;
      ex_given = lane < nex ? ex_idx[(size_t)row * nex + lane] : (lane == nex ? sink_row0 + h : 0);
      if (MODE == 1 && nex > 0) {
        const int d = n >> 1;
        const bool ql = lane * 4 < d;
        const int qo = ql ? lane * 4 : 0;
        float fa[4], fb[4];
        {
          QQuad<T> qa, qb;
          qa.load(q + (size_t)row * n + qo);
          qb.load(q + (size_t)row * n + d + qo);
          qa.to_f32(fa);
          qb.to_f32(fb);
        }
        const int64_t ex_safe = (ex_given >= 0 && ex_given < N) ? ex_given : 0;
        // each lane splits its own extra index once (S * S <= 2^26 fits 32 bits)
        const uint32_t exu = (uint32_t)ex_safe;
        const uint32_t ex1 = exu / (uint32_t)S, ex2 = exu - ex1 * (uint32_t)S;
        const T* k1 = subkeys + (size_t)(h * 2) * S * d + qo;
        const T* k2 = k1 + (size_t)S * d;
        // eight extras at a time: their sub-key loads in flight together, then
        // one transposed butterfly (4 + 2 + 1 + 3 exchanges) leaves extra j's
        // sum in lanes 8j .. 8j + 7
        for (int e0 = 0; e0 < nex; e0 += 8) {
          QQuad<T> ka[8], kb[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int e = e0 + j < nex ? e0 + j : nex - 1;
            const int i1 = __builtin_amdgcn_readlane((int)ex1, e), i2 = __builtin_amdgcn_readlane((int)ex2, e);
            ka[j].load(k1 + (size_t)i1 * d);
            kb[j].load(k2 + (size_t)i2 * d);
          }
          float p[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            float va[4], vb[4];
            ka[j].to_f32(va);
            kb[j].to_f32(vb);
            float a = 0.f;
#pragma unroll
            for (int i = 0; i < 4; ++i) a = fmaf(fa[i], va[i], a);
#pragma unroll
            for (int i = 0; i < 4; ++i) a = fmaf(fb[i], vb[i], a);
            p[j] = ql ? a : 0.f;
          }
          const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
          float p4[4], p2[2];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float send = b5 ? p[i] : p[i + 4];
            p4[i] = (b5 ? p[i + 4] : p[i]) + __shfl_xor(send, 32, WAVE);
          }
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            const float send = b4 ? p4[i] : p4[i + 2];
            p2[i] = (b4 ? p4[i + 2] : p4[i]) + __shfl_xor(send, 16, WAVE);
          }
          float t1;
          {
            const float send = b3 ? p2[0] : p2[1];
            t1 = (b3 ? p2[1] : p2[0]) + __shfl_xor(send, 8, WAVE);
          }
          t1 = group_sum<8>(t1);
          const int src = (lane - e0) * 8;
          const float got = __shfl(t1, src >= 0 && src < WAVE ? src : 0, WAVE);
          if (lane >= e0 && lane < e0 + 8) ex_score = got;
        }
      }
      if (sink_part && lane == nex) ex_score = sink_part[(size_t)row * 2] + sink_part[(size_t)row * 2 + 1];
    }
    const int32_t* i1 = half_idx + (size_t)row * 2 * k;
    const int32_t* i2 = i1 + k;
    const float* s1 = half_score + (size_t)row * 2 * k;
    const float* s2 = s1 + k;
    const float s1v = lane < k ? s1[lane] : 0.f;
    const float s2v = lane < k ? s2[lane] : 0.f;
    const int i1v = lane < k ? i1[lane] : 0;
    const int i2v = lane < k ? i2[lane] : 0;
    uint64_t v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int m = e * WAVE + lane;
      const uint32_t pr = pairs[m < npairs ? m : 0];
      const int a = (int)(pr >> 16), b = (int)(pr & 0xFFFFu);
      const float sa = __shfl(s1v, a, WAVE), sb = __shfl(s2v, b, WAVE);
      const int ia = __shfl(i1v, a, WAVE), ib = __shfl(i2v, b, WAVE);
      v[e] = m < npairs ? make_key(sa + sb, (uint32_t)ia * (uint32_t)S + (uint32_t)ib) : 0ull;
    }
    wave_sort_desc<E>(v, lane);
    float z = key_score(v[0]);
    int64_t ci = (int64_t)key_index(v[0]);
    float zmax;
    if constexpr (EXTRA) {
      const int src = lane >= k ? lane - k : 0;
      const float zx = __shfl(ex_score, src, WAVE);
      const int64_t ix = (int64_t)(((uint64_t)(uint32_t)__shfl((int)(ex_given >> 32), src, WAVE) << 32) |
                                   (uint32_t)__shfl((int)(uint32_t)ex_given, src, WAVE));
      if (lane >= k) { z = zx; ci = ix; }
      float m = lane < kk ? z : -INFINITY;
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, WAVE));
      zmax = m;
    } else {
      zmax = __shfl(z, 0, WAVE);
    }
    const float ex = lane < kk ? expf(z - zmax) : 0.f;
    const float sum = group_sum<WAVE>(ex);
    if (lane < kk) {
      const size_t o = (size_t)row * kk + lane;
      idx_out[o] = ci;
      w_out[o] = ex / sum;
      if (score_out) score_out[o] = z;
    }
  }
}

int cartesian_pairs(int k) {
  int m = 0;
  for (int a = 0; a < k; ++a) m += k / (a + 1);
  return m;
}

template <typename T, int NSTEP>
static hipError_t launch_score(const void* q, const void* subkeys, int64_t T_, int H, int n, int S,
                               int k, const float2* qstats, const void* sink, float* sink_part,
                               uint64_t* cand, uint32_t* cnts, float* thr,
                               int32_t* half_idx, float* half_score, uint32_t* ovf,
                               hipStream_t st) {
  const int64_t tiles = (T_ + SEARCH_TOK - 1) / SEARCH_TOK;
  const int64_t blocks = tiles * 2 * H;
  {
    LaunchTimer lt("score_topk", st);
    if (k > 32)
      hipLaunchKernelGGL((k_score_topk<T, NSTEP, true>), dim3((unsigned)blocks), dim3(64 * SEARCH_WAVES),
                         0, st, (const T*)q, (const T*)subkeys, T_, H, n, S, k, qstats,
                         (const T*)sink, sink_part, cand, cnts, thr);
    else
      hipLaunchKernelGGL((k_score_topk<T, NSTEP, false>), dim3((unsigned)blocks), dim3(64 * SEARCH_WAVES),
                         0, st, (const T*)q, (const T*)subkeys, T_, H, n, S, k, qstats,
                         (const T*)sink, sink_part, cand, cnts, thr);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    int64_t sb = (T_ + 31) / 32 * H * 2;  // one workgroup per wave run
    if (sb > 16384) sb = 16384;
    LaunchTimer lt("topk_sort", st);
    hipLaunchKernelGGL(k_topk_sort, dim3((unsigned)sb), dim3(256), 0, st, (const uint64_t*)cand,
                       (const uint32_t*)cnts, (const float*)thr, T_, H, k, half_idx, half_score, ovf);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t lds = (size_t)S * sizeof(float);
  hipLaunchKernelGGL((k_topk_fallback<T>), dim3(256), dim3(256), lds, st, (const T*)q,
                     (const T*)subkeys, H, n, S, k, qstats, (const uint32_t*)ovf, half_idx, half_score);
  return hipGetLastError();
}

hipError_t launch_qnorm(bool bf16, const void* q, int64_t rows, int n, float eps, float2* stats,
                       void* qhat, hipStream_t st) {
  if (rows <= 0) return hipSuccess;
  LaunchTimer lt("qnorm", st);
  const dim3 g((unsigned)((rows + 4 * QNORM_ROWS - 1) / (4 * QNORM_ROWS))), b(256);
  if (bf16)
    hipLaunchKernelGGL(k_qnorm<uint16_t>, g, b, 0, st, (const uint16_t*)q, rows, n, eps, stats,
                       (uint16_t*)qhat);
  else
    hipLaunchKernelGGL(k_qnorm<float>, g, b, 0, st, (const float*)q, rows, n, eps, stats,
                       (float*)qhat);
  return hipGetLastError();
}

hipError_t launch_search_half(bool bf16, const void* q, const void* subkeys, int64_t T_, int H,
                              int n, int S, int k, const float2* qstats, const void* sink,
                              float* sink_part, uint64_t* cand, uint32_t* cnts, float* thr,
                              int32_t* half_idx, float* half_score, uint32_t* ovf,
                              hipStream_t st) {
  hipError_t e = launch_fill_u32(ovf, 0u, 1, st);
  if (e != hipSuccess) return e;
  const int d = n / 2;
  if (bf16) {
    const int steps = (d + 15) / 16;
    if (steps <= 1) return launch_score<uint16_t, 1>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
    if (steps <= 2) return launch_score<uint16_t, 2>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
    if (steps <= 4) return launch_score<uint16_t, 4>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
    if (steps <= 8) return launch_score<uint16_t, 8>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
    return launch_score<uint16_t, 16>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
  }
  const int steps = (d + 1) / 2;
  if (steps <= 2) return launch_score<float, 2>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
  if (steps <= 4) return launch_score<float, 4>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
  if (steps <= 8) return launch_score<float, 8>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
  if (steps <= 16) return launch_score<float, 16>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
  return launch_score<float, 32>(q, subkeys, T_, H, n, S, k, qstats, sink, sink_part, cand, cnts, thr, half_idx, half_score, ovf, st);
}

template <int E>
static void cart_launch(dim3 g, dim3 b, hipStream_t st, const int32_t* half_idx,
                        const float* half_score, int64_t rows, int S, int k, int np, bool bf16,
                        const void* q, const void* subkeys, int H, int n, const int64_t* ex_idx,
                        int nex, const float* sink_part, int64_t sink_row0, int64_t* idx_out,
                        float* w_out, float* score_out) {
  if (nex == 0 && !sink_part)
    hipLaunchKernelGGL((k_cartesian<E, uint16_t, 0>), g, b, 0, st, half_idx, half_score, rows,
                       S, k, np, (const uint16_t*)nullptr, (const uint16_t*)nullptr, H, n,
                       (const int64_t*)nullptr, 0, (const float*)nullptr, (int64_t)0, idx_out,
                       w_out, score_out);
  else if (nex == 0)
    hipLaunchKernelGGL((k_cartesian<E, uint16_t, 2>), g, b, 0, st, half_idx, half_score, rows,
                       S, k, np, (const uint16_t*)nullptr, (const uint16_t*)nullptr, H, n,
                       (const int64_t*)nullptr, 0, sink_part, sink_row0, idx_out, w_out,
                       score_out);
  else if (bf16)
    hipLaunchKernelGGL((k_cartesian<E, uint16_t, 1>), g, b, 0, st, half_idx, half_score, rows, S,
                       k, np, (const uint16_t*)q, (const uint16_t*)subkeys, H, n, ex_idx, nex,
                       sink_part, sink_row0, idx_out, w_out, score_out);
  else
    hipLaunchKernelGGL((k_cartesian<E, float, 1>), g, b, 0, st, half_idx, half_score, rows, S, k,
                       np, (const float*)q, (const float*)subkeys, H, n, ex_idx, nex,
                       sink_part, sink_row0, idx_out, w_out, score_out);
}

hipError_t launch_cartesian(const int32_t* half_idx, const float* half_score, int64_t T_, int H,
                            int S, int k, bool bf16, const void* q, const void* subkeys, int n,
                            const int64_t* ex_idx, int nex, const float* sink_part,
                            int64_t sink_row0, int64_t* idx_out, float* w_out, float* score_out,
                            hipStream_t st) {
  const int64_t rows = T_ * H;
  const int np = cartesian_pairs(k);
  int64_t blocks = (rows + 3) / 4;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  const dim3 g((unsigned)blocks), b(256);
  LaunchTimer lt("cartesian", st);
  if (np <= 64) cart_launch<1>(g, b, st, half_idx, half_score, rows, S, k, np, bf16, q, subkeys, H, n, ex_idx, nex, sink_part, sink_row0, idx_out, w_out, score_out);
  else if (np <= 128) cart_launch<2>(g, b, st, half_idx, half_score, rows, S, k, np, bf16, q, subkeys, H, n, ex_idx, nex, sink_part, sink_row0, idx_out, w_out, score_out);
  else if (np <= 256) cart_launch<4>(g, b, st, half_idx, half_score, rows, S, k, np, bf16, q, subkeys, H, n, ex_idx, nex, sink_part, sink_row0, idx_out, w_out, score_out);
  else cart_launch<8>(g, b, st, half_idx, half_score, rows, S, k, np, bf16, q, subkeys, H, n, ex_idx, nex, sink_part, sink_row0, idx_out, w_out, score_out);
  return hipGetLastError();
}

}  // namespace pk
