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

constexpr int kHeadDim = 128;
constexpr int kHidden = 64;
constexpr int kPad = 256;      // every padded workspace dimension is a multiple of this
constexpr int kNumXcd = 8;     // MI355X: 8 XCDs, workgroups dispatched round-robin

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
