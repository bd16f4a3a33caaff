// Token scoring: one logit per cached token from the 2-layer MLP
// I_j = w2 . GELU(W1 [k_j; v_j] + b1) + b2 (exact erf GELU).  This is the
// query-independent scorer whose root-mean-square pooling (eq. indexer_pooling)
// is a monotone map of I, so the top-t anchors are the top-t of I (Section 3.3).
//
// HBM-bound: each token's key and value (2 x 128 elements) are read once.
// bf16: the 64 x 256 weight matrix sits in LDS and the hidden layer runs on
// MFMA 32x32x16 with D[hidden][token] = W1 . X^T, so each lane ends up owning
// one token column and reduces its hidden units in registers.
#include "common.hpp"

namespace arckv {

namespace {
constexpr int kScoreTokensPerBlock = 128;   // 4 waves x 32 tokens
constexpr int kW1Stride = 2 * kHeadDim + 8; // LDS row stride (elements), padded

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }
}  // namespace

__global__ void __launch_bounds__(256) k_score_bf16(const bf16 *__restrict__ K, const bf16 *__restrict__ V,
                                                     const bf16 *__restrict__ W1, const float *__restrict__ b1,
                                                     const float *__restrict__ w2, const float *__restrict__ b2,
                                                     float *__restrict__ scores, int T) {
  __shared__ bf16 sW[kHidden * kW1Stride];
  const int b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bf16 *W1b = W1 + (size_t)b * kHidden * 2 * kHeadDim;
  // stage W1 (64 x 256 bf16 = 2048 chunks of 16 B) into LDS
  for (int c = tid; c < kHidden * 2 * kHeadDim / 8; c += 256) {
    int row = c / 32, col = (c % 32) * 8;
    *reinterpret_cast<bf16x8 *>(&sW[row * kW1Stride + col]) = *reinterpret_cast<const bf16x8 *>(&W1b[row * 256 + col]);
  }
  const int h = lane >> 5, col = lane & 31;
  const int tok = blockIdx.x * kScoreTokensPerBlock + wave * 32 + col;
  const bool valid = tok < T;
  const size_t row_off = ((size_t)b * T + (valid ? tok : 0)) * kHeadDim;
  // B fragments: token `tok`, features 16*ks + 8*h .. +7 (ks < 8 from K, else V)
  bf16x8 xb[16];
  #pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    const bf16 *src = (ks < 8 ? K : V) + row_off + (ks & 7) * 16 + 8 * h;
    xb[ks] = valid ? *reinterpret_cast<const bf16x8 *>(src) : Mfma<bf16>::zero();
  }
  __syncthreads();
  f32x16 acc0 = zero16(), acc1 = zero16();
  #pragma unroll
  for (int ks = 0; ks < 16; ++ks) {
    bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(&sW[col * kW1Stride + ks * 16 + 8 * h]);
    bf16x8 a1 = *reinterpret_cast<const bf16x8 *>(&sW[(32 + col) * kW1Stride + ks * 16 + 8 * h]);
    acc0 = Mfma<bf16>::mma(a0, xb[ks], acc0);
    acc1 = Mfma<bf16>::mma(a1, xb[ks], acc1);
  }
  const float *b1b = b1 + b * kHidden, *w2b = w2 + b * kHidden;
  float part = 0.0f;
  #pragma unroll
  for (int v = 0; v < 16; ++v) {
    int m0 = acc_row(v, lane);
    part += w2b[m0] * gelu_erf(acc0[v] + b1b[m0]);
    part += w2b[m0 + 32] * gelu_erf(acc1[v] + b1b[m0 + 32]);
  }
  part += __shfl_xor(part, 32, 64);
  if (h == 0 && valid) scores[(size_t)b * T + tok] = part + b2[b];
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
    dim3 grid((T + kScoreTokensPerBlock - 1) / kScoreTokensPerBlock, B);
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
