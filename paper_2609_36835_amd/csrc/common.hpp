// Shared device helpers for the gfx950 ARC-KV kernels: element types, MFMA
// fragments, bf16 splitting, and the XCD-aware tile mapping.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "arckv.h"

namespace arckv {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2;
typedef _Float16 f16;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4;
typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;

constexpr int kHeadDim = 128;
constexpr int kHidden = 64;
constexpr int kPad = 256;      // every padded workspace dimension is a multiple of this
constexpr int kNumXcd = 8;     // MI355X: 8 XCDs, workgroups dispatched round-robin
// Response profiles of bf16 inputs are stored in fp16 scaled by 2^15: values
// in (0, 1] land in [2^-9, 2^15], the fp16 normal range covers E >= 2^-29, and
// the scale (a power of two) changes no rounding.
constexpr int kProfLog2Scale = 15;
constexpr float kProfScale = 32768.0f;
constexpr float kProfInvScale = 1.0f / 32768.0f;

__host__ __device__ inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- MFMA fragments
// A 32x32 output tile lives in a f32x16 accumulator: lane l holds column
// (l % 32) and rows 8*(v/4) + 4*(l/32) + (v%4) for v = 0..15.  The A operand
// (32 x K) gives lane l row (l % 32) and KPL consecutive k starting at
// KPL*(l/32); the B operand (K x 32) gives lane l column (l % 32) with the same
// k range.  A k-step therefore covers 2*KPL values of k.
template <typename T> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int KPL = 8;           // k values per lane
  static constexpr int KSTEP = 16;        // k values per instruction
  typedef bf16x8 frag;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const bf16 *p) { return *reinterpret_cast<const bf16x8 *>(p); }
  __device__ static inline frag zero() { frag f; for (int e = 0; e < 8; ++e) f[e] = (bf16)0.0f; return f; }
};

template <> struct Mfma<float> {
  static constexpr int KPL = 1;
  static constexpr int KSTEP = 2;
  typedef float frag;
  __device__ static inline f32x16 mma(frag a, frag b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static inline frag load(const float *p) { return *p; }
  __device__ static inline frag zero() { return 0.0f; }
};

// 32x32x16 MFMA on raw 16-byte fragments holding eight bf16 or eight fp16
// values (E selects the instruction); products are exact in fp32.
template <typename E>
__device__ inline f32x16 mma16(bf16x8 a, bf16x8 b, f32x16 c) {
  if constexpr (sizeof(E) == 2 && !__is_same(E, bf16))
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline int acc_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

__device__ inline f32x16 zero16() {
  f32x16 z;
  for (int v = 0; v < 16; ++v) z[v] = 0.0f;
  return z;
}

// ---------------------------------------------------------------- conversions
__device__ inline bf16 to_bf16(float x) { return (bf16)x; }       // round to nearest even
__device__ inline float from_bf16(bf16 x) { return (float)x; }
// x = hi + lo with hi = bf16(x), lo = bf16(x - hi): ~16 significant bits.
__device__ inline void split_bf16(float x, bf16 &hi, bf16 &lo) {
  hi = (bf16)x;
  lo = (bf16)(x - (float)hi);
}
template <typename T> __device__ inline float to_f(T x) { return (float)x; }

// Order-preserving map from float scores to uint32 keys: larger score, larger
// key; -0 equals +0; NaN maps to 0, below every number (-inf maps to 0x007FFFFF).
__device__ inline uint32_t score_key(float f) {
  if (f != f) return 0u;
  if (f == 0.0f) f = 0.0f;
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---------------------------------------------------------------- top-3 partials
// The three largest similarities (all >= 0) of a set of anchors for one key:
// the best two as packed 64-bit keys (float bits << 32 | ~r, so the larger
// similarity wins and equal similarities go to the lower r; 0 = empty) and
// the third as float bits only (0 = empty).  A later stage uses the third to
// tell whether a set may hold more candidates than its two best.
struct Top3 {
  float v1, v2, v3;
  uint32_t r1, r2;
  __device__ inline void init() {
    v1 = v2 = v3 = -1.0f;
    r1 = r2 = 0u;
  }
  // values must arrive in ascending r for the lower-r rule within one set
  __device__ inline void add(float v, uint32_t r, bool valid) {
    const bool c1 = valid && v > v1, c2 = valid && v > v2, c3 = valid && v > v3;
    v3 = c2 ? v2 : (c3 ? v : v3);
    const float nv2 = c1 ? v1 : (c2 ? v : v2);
    const uint32_t nr2 = c1 ? r1 : (c2 ? r : r2);
    v1 = c1 ? v : v1;
    r1 = c1 ? r : r1;
    v2 = nv2;
    r2 = nr2;
  }
};
// Median of three (the compiler forms v_med3_u32 from this pattern).
__device__ inline uint32_t med3u(uint32_t a, uint32_t b, uint32_t c) { return max(min(a, b), min(max(a, b), c)); }
__device__ inline uint64_t pack_sim(float v, uint32_t r) {
  return v < 0.0f ? 0ull : (((uint64_t)__float_as_uint(v) << 32) | (uint64_t)(0xFFFFFFFFu - r));
}
__device__ inline float packed_sim(uint64_t k) { return __uint_as_float((uint32_t)(k >> 32)); }
__device__ inline uint32_t packed_r(uint64_t k) { return 0xFFFFFFFFu - (uint32_t)(k & 0xFFFFFFFFull); }
// Merge two packed top-3 lists (a1 >= a2 >= a3, b1 >= b2 >= b3) in place into (a1, a2, a3).
__device__ inline void merge_top3(uint64_t &a1, uint64_t &a2, uint32_t &a3, uint64_t b1, uint64_t b2, uint32_t b3) {
  const uint32_t c1 = min((uint32_t)(a1 >> 32), (uint32_t)(b2 >> 32));
  const uint32_t c2 = min((uint32_t)(a2 >> 32), (uint32_t)(b1 >> 32));
  const uint32_t n3 = max(max(a3, b3), max(c1, c2));
  const uint64_t n2 = max(min(a1, b1), max(a2, b2));
  a1 = max(a1, b1);
  a2 = n2;
  a3 = n3;
}

// ---------------------------------------------------------------- wave helpers
__device__ inline float shfl_xor(float v, int mask) { return __shfl_xor(v, mask, 64); }
__device__ inline double shfl_xor(double v, int mask) { return __shfl_xor(v, mask, 64); }

__device__ inline float wave_sum(float v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ inline double wave_sum(double v) {
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ inline float wave_max(float v) {
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}

// ---------------------------------------------------------------- tile mapping
// Workgroups are handed to the 8 XCDs round-robin.  Remap the linear block id
// so that each XCD receives one contiguous range of logical tiles; tiles that
// share operands then run on the same XCD and share its L2.
__device__ inline int64_t xcd_remap(int64_t bid, int64_t nblocks) {
  int64_t per = (nblocks + kNumXcd - 1) / kNumXcd;
  int64_t xcd = bid % kNumXcd, slot = bid / kNumXcd;
  int64_t full = nblocks % kNumXcd == 0 ? kNumXcd : nblocks % kNumXcd;  // XCDs with `per` blocks
  // XCD x owns logical range [start_x, start_x + cnt_x)
  int64_t start = xcd < full ? xcd * per : full * per + (xcd - full) * (per - 1);
  return start + slot;
}

}  // namespace arckv
