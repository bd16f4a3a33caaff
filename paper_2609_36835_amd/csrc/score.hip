// Token scoring: one logit per cached token from the 2-layer MLP
// I_j = w2 . GELU(W1 [k_j; v_j] + b1) + b2 (erf GELU).  This is the
// query-independent scorer whose root-mean-square pooling (eq. indexer_pooling)
// is a monotone map of I, so the top-t anchors are the top-t of I (Section 3.3).
//
// HBM-bound: each token's key and value (2 x 128 elements) are read once.
#include "common.hpp"

namespace arckv {

namespace {
constexpr int kScoreWaves = 4;
constexpr int kScoreSlab = 32 * kScoreWaves;   // tokens per workgroup iteration (32 per wave)
constexpr int kScoreIters = 8;                  // slabs per workgroup: W1 is staged once per 1024 tokens
constexpr int kW1Stride = 2 * kHeadDim + 8;     // LDS row stride (elements), padded

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

// GELU(x) = x Phi(x) = max(x, 0) - |x|/2 erfc(|x|/sqrt 2), with erfc(u) from the
// rational approximation of Abramowitz & Stegun, Handbook of Mathematical
// Functions, formula 7.1.26: erfc(u) = t (a1 + t (a2 + ... + t a5)) e^{-u^2},
// t = 1 / (1 + p u), absolute error at most 1.5e-7 for u >= 0.
//
// It is evaluated on y = c x with c = sqrt(log2(e) / 2), so e^{-x^2/2} is the
// hardware base-2 exponential of -y^2, and returns GELU(x) * c:
//   c GELU(x) = max(y, 0) - |y| t P(t) 2^{-y^2},  t = 1 / (1 + p |y| / (sqrt 2 c)),
// with the halving folded into P.  The caller multiplies by w2 / c.  One
// reciprocal, one exponential and no branches; in fp32 the result differs from
// the exact GELU by at most about 3.3e-7.
constexpr float kGeluC = 0.8493218002880191f;        // sqrt(log2(e) / 2)
__device__ inline float gelu_scaled(float y) {
  const float ay = fabsf(y);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.2727374808792225f, ay, 1.0f));   // p / (sqrt 2 c)
  float P = fmaf(0.5f * 1.061405429f, t, 0.5f * -1.453152027f);
  P = fmaf(P, t, 0.5f * 1.421413741f);
  P = fmaf(P, t, 0.5f * -0.284496736f);
  P = fmaf(P, t, 0.5f * 0.254829592f);
  const float e = __builtin_amdgcn_exp2f(-y * y);
  return fmaf(-P * (t * ay), e, fmaxf(y, 0.0f));
}
}  // namespace

// bf16: a workgroup of 4 waves streams kScoreIters slabs of 128 tokens of one
// pair.  The hidden layer runs on MFMA 32x32x16 as D[hidden][token] = W1 X^T
// with W1 (64 x 256) in LDS, so each lane owns one token column.  Each wave
// holds one slab of its 32 tokens' features in registers; the loads of the next
// slab are issued as soon as the MFMAs have consumed the current one, and the
// GELU epilogue runs while they are in flight.
__global__ void __launch_bounds__(256) k_score_bf16(const bf16 *__restrict__ K, const bf16 *__restrict__ V,
                                                     const bf16 *__restrict__ W1, const float *__restrict__ b1,
                                                     const float *__restrict__ w2, const float *__restrict__ b2,
                                                     float *__restrict__ scores, int T) {
  __shared__ bf16 sW[kHidden * kW1Stride];
  __shared__ f32x4 sBW[2][kHidden / 4];   // c b1, w2 / c in groups of 4 hidden rows
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int tok0 = blockIdx.x * (kScoreSlab * kScoreIters) + wave * 32 + col;
  const bf16 *Kb = K + (size_t)b * T * kHeadDim + 8 * h, *Vb = V + (size_t)b * T * kHeadDim + 8 * h;
  // B fragments: token `tok`, features 16*ks + 8*h .. +7 (ks < 8 from K, else V)
  bf16x8 xb[16];
  auto load_slab = [&](int it) {
    const int tok = tok0 + it * kScoreSlab;
    const size_t ro = (size_t)(tok < T ? tok : 0) * kHeadDim;
#pragma unroll
    for (int ks = 0; ks < 16; ++ks)
      xb[ks] = *reinterpret_cast<const bf16x8 *>((ks < 8 ? Kb : Vb) + ro + (ks & 7) * 16);
  };
  load_slab(0);
  // stage W1 (64 x 256 bf16 = 2048 chunks of 16 B), b1 and w2 into LDS
  const bf16 *W1b = W1 + (size_t)b * kHidden * 2 * kHeadDim;
  for (int c = tid; c < kHidden * 2 * kHeadDim / 8; c += 256) {
    const int row = c / 32, cc = (c % 32) * 8;
    *reinterpret_cast<bf16x8 *>(&sW[row * kW1Stride + cc]) = *reinterpret_cast<const bf16x8 *>(&W1b[row * 256 + cc]);
  }
  // the GELU runs on c (acc + b1): store c b1 and w2 / c
  if (tid < kHidden) reinterpret_cast<float *>(sBW[0])[tid] = kGeluC * b1[b * kHidden + tid];
  else if (tid < 2 * kHidden)
    reinterpret_cast<float *>(sBW[1])[tid - kHidden] = w2[b * kHidden + tid - kHidden] / kGeluC;
  const float bias2 = b2[b];
  __syncthreads();
#pragma unroll 1
  for (int it = 0; it < kScoreIters; ++it) {
    // W1 fragments are re-read from LDS every slab (kept out of registers so
    // three waves fit per SIMD)
    asm volatile("" ::: "memory");
    f32x16 acc0 = zero16(), acc1 = zero16();
#pragma unroll
    for (int ks = 0; ks < 16; ++ks) {
      const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(&sW[col * kW1Stride + ks * 16 + 8 * h]);
      const bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(&sW[(32 + col) * kW1Stride + ks * 16 + 8 * h]);
      acc0 = Mfma<bf16>::mma(a0, xb[ks], acc0);
      acc1 = Mfma<bf16>::mma(a1, xb[ks], acc1);
    }
    if (it + 1 < kScoreIters) load_slab(it + 1);
    // lane holds hidden rows 8g + 4h + e (e < 4) of both 32-row tiles
    float part = 0.0f;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 bA = sBW[0][2 * g + h], wA = sBW[1][2 * g + h], bB = sBW[0][8 + 2 * g + h], wB = sBW[1][8 + 2 * g + h];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        part = fmaf(wA[e], gelu_scaled(fmaf(acc0[4 * g + e], kGeluC, bA[e])), part);
        part = fmaf(wB[e], gelu_scaled(fmaf(acc1[4 * g + e], kGeluC, bB[e])), part);
      }
    }
    part += __shfl_xor(part, 32, 64);
    const int tok = tok0 + it * kScoreSlab;
    if (h == 0 && tok < T) scores[(size_t)b * T + tok] = part + bias2;
  }
}

// fp32 inputs: one thread per token, W1 (64 x 256 fp32) staged through LDS.
__global__ void __launch_bounds__(256) k_score_f32(const float *__restrict__ K, const float *__restrict__ V,
                                                    const float *__restrict__ W1, const float *__restrict__ b1,
                                                    const float *__restrict__ w2, const float *__restrict__ b2,
                                                    float *__restrict__ scores, int T) {
  __shared__ float sW[kHidden * 2 * kHeadDim];
  const int b = blockIdx.y, tid = threadIdx.x;
  const float *W1b = W1 + (size_t)b * kHidden * 2 * kHeadDim;
  for (int c = tid; c < kHidden * 2 * kHeadDim; c += 256) sW[c] = W1b[c];
  __syncthreads();
  const int tok = blockIdx.x * 256 + tid;
  if (tok >= T) return;
  const float *k = K + ((size_t)b * T + tok) * kHeadDim;
  const float *v = V + ((size_t)b * T + tok) * kHeadDim;
  float acc = 0.0f;
  for (int a = 0; a < kHidden; ++a) {
    const float *w = sW + a * 2 * kHeadDim;
    float pre = b1[b * kHidden + a];
    for (int c = 0; c < kHeadDim; ++c) pre = fmaf(w[c], k[c], pre);
    for (int c = 0; c < kHeadDim; ++c) pre = fmaf(w[kHeadDim + c], v[c], pre);
    acc = fmaf(w2[b * kHidden + a], gelu_erf(pre), acc);
  }
  scores[(size_t)b * T + tok] = acc + b2[b];
}

hipError_t launch_score(int dtype, const void *K, const void *V, const void *W1, const float *b1,
                        const float *w2, const float *b2, float *scores, int B, int T, hipStream_t s) {
  if (dtype == ARCKV_BF16) {
    const int per_wg = kScoreSlab * kScoreIters;
    dim3 grid((T + per_wg - 1) / per_wg, B);
    hipLaunchKernelGGL(k_score_bf16, grid, dim3(256), 0, s, (const bf16 *)K, (const bf16 *)V, (const bf16 *)W1,
                       b1, w2, b2, scores, T);
  } else {
    dim3 grid((T + 255) / 256, B);
    hipLaunchKernelGGL(k_score_f32, grid, dim3(256), 0, s, (const float *)K, (const float *)V, (const float *)W1,
                       b1, w2, b2, scores, T);
  }
  return hipGetLastError();
}

}  // namespace arckv
