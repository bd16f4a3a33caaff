// Small copy/padding kernels used by the host sequencing.
#include "common.hpp"

namespace arckv {

// User compact keys [P][t][128] fp32 -> padded operand copy: bf16 hi/lo planes
// [P][2][tp][128] (bf16 problems) or fp32 [P][tp][128]; rows r >= t are zero.
template <bool SPLIT>
__global__ void __launch_bounds__(256) k_pad_ck(const float *__restrict__ Ck, int t, int64_t tp, void *__restrict__ out) {
  const int b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= tp * kHeadDim) return;
  const int64_t r = e / kHeadDim;
  const float v = r < t ? Ck[(size_t)b * t * kHeadDim + e] : 0.0f;
  if constexpr (SPLIT) {
    bf16 *o = reinterpret_cast<bf16 *>(out) + (size_t)b * 2 * tp * kHeadDim + e;
    split_bf16(v, o[0], o[tp * kHeadDim]);
  } else {
    reinterpret_cast<float *>(out)[(size_t)b * tp * kHeadDim + e] = v;
  }
}

__global__ void __launch_bounds__(256) k_pad_beta(const float *__restrict__ beta, int t, int64_t tp,
                                                  float *__restrict__ out) {
  const int b = blockIdx.y;
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= tp) return;
  out[(size_t)b * tp + r] = r < t ? beta[(size_t)b * t + r] : 0.0f;
}

__global__ void __launch_bounds__(256) k_copy_info(const int32_t *__restrict__ a, const int32_t *__restrict__ b2,
                                                   int B, int32_t *__restrict__ info) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B) return;
  if (b2) {
    info[2 * i] = a[i];
    info[2 * i + 1] = b2[i];
  } else {
    info[i] = a[i];
  }
}

__global__ void __launch_bounds__(256) k_copy_f32(const float *__restrict__ src, float *__restrict__ dst, int B) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < B) dst[i] = src[i];
}

hipError_t launch_pad_ck(int dtype, const float *Ck, int P, int t, int64_t tp, void *Ckp, hipStream_t s) {
  dim3 grid((unsigned)((tp * kHeadDim + 255) / 256), P);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_pad_ck<true>, grid, dim3(256), 0, s, Ck, t, tp, Ckp);
  else
    hipLaunchKernelGGL(k_pad_ck<false>, grid, dim3(256), 0, s, Ck, t, tp, Ckp);
  return hipGetLastError();
}

hipError_t launch_pad_beta(const float *beta, int P, int t, int64_t tp, float *beta_ws, hipStream_t s) {
  hipLaunchKernelGGL(k_pad_beta, dim3((unsigned)((tp + 255) / 256), P), dim3(256), 0, s, beta, t, tp, beta_ws);
  return hipGetLastError();
}

hipError_t launch_copy_info(const int32_t *a, const int32_t *b, int B, int32_t *info, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_info, dim3((B + 255) / 256), dim3(256), 0, s, a, b, B, info);
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float *src, float *dst, int B, hipStream_t s) {
  hipLaunchKernelGGL(k_copy_f32, dim3((B + 255) / 256), dim3(256), 0, s, src, dst, B);
  return hipGetLastError();
}

}  // namespace arckv
