// Full-cache row statistics (Appendix A.9): for every reference query q_i,
//   z_i = max_j s q_i.k_j,   m_i = sum_j exp(s q_i.k_j - z_i),   Y_i = sum_j exp(.) v_j / m_i.
// z are the row maxima that shift Phi_K and Phi_C, m = Phi_K 1 are the mass
// targets of the bias fit, Y the full-attention outputs the value fit matches.
//
// Flash-style single pass over the keys with an online maximum.  Each wave
// owns 32 queries and computes D[key][query] = K Q^T, so every lane holds one
// query column: its running max/sum live in registers.  The probabilities are
// fed back as the B operand of Y^T[c][q] += V^T[c][key] P^T[key][q]; the MFMA
// k-slots are permuted to match the accumulator layout, and V^T is staged in
// LDS with the same key order.
#include "common.hpp"

namespace arckv {

template <typename T> struct RowstatsCfg;
template <> struct RowstatsCfg<bf16> { static constexpr int NSUB = 2; };   // 64 keys per tile
template <> struct RowstatsCfg<float> { static constexpr int NSUB = 1; };  // 32 keys per tile

template <typename T>
__global__ void __launch_bounds__(256) k_rowstats(const T *__restrict__ K, const T *__restrict__ V,
                                                  const T *__restrict__ Q, float *__restrict__ z,
                                                  float *__restrict__ m, float *__restrict__ Y, int Tn, int n,
                                                  float scale) {
  using M = Mfma<T>;
  constexpr int KPL = M::KPL, KSTEP = M::KSTEP;
  constexpr int NSUB = RowstatsCfg<T>::NSUB, KB = 32 * NSUB;
  constexpr int EPC = 16 / sizeof(T);                   // elements per 16-byte chunk
  constexpr int SK = kHeadDim + EPC;                    // padded LDS strides (elements)
  constexpr int SV = KB + EPC;
  __shared__ __attribute__((aligned(16))) T sK[KB * SK];
  __shared__ __attribute__((aligned(16))) T sVt[kHeadDim * SV];

  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int q = blockIdx.x * 128 + wave * 32 + col;
  const bool qvalid = q < n;
  const T *Kb = K + (size_t)b * Tn * kHeadDim;
  const T *Vb = V + (size_t)b * Tn * kHeadDim;

  typename M::frag qf[kHeadDim / KSTEP];
  {
    const T *qrow = Q + ((size_t)b * n + (qvalid ? q : 0)) * kHeadDim;
    #pragma unroll
    for (int ks = 0; ks < kHeadDim / KSTEP; ++ks)
      qf[ks] = qvalid ? M::load(qrow + ks * KSTEP + KPL * h) : M::zero();
  }
  const float c2 = scale * 1.4426950408889634f;   // exp(s x) = exp2(c2 x)
  float run_max = -INFINITY, run_sum = 0.0f;
  f32x16 accY[4];
  #pragma unroll
  for (int cs = 0; cs < 4; ++cs) accY[cs] = zero16();

  for (int k0 = 0; k0 < Tn; k0 += KB) {
    // stage K rows [k0, k0+KB) and V^T into LDS (rows past T are zero)
    for (int c = tid; c < KB * (kHeadDim / EPC); c += 256) {
      int r = c / (kHeadDim / EPC), cc = (c % (kHeadDim / EPC)) * EPC;
      int key = k0 + r;
      f32x4 kv, vv;
      if (key < Tn) {
        kv = *reinterpret_cast<const f32x4 *>(Kb + (size_t)key * kHeadDim + cc);
        vv = *reinterpret_cast<const f32x4 *>(Vb + (size_t)key * kHeadDim + cc);
      } else {
        kv = f32x4{0.f, 0.f, 0.f, 0.f};
        vv = kv;
      }
      *reinterpret_cast<f32x4 *>(&sK[r * SK + cc]) = kv;
      const T *ve = reinterpret_cast<const T *>(&vv);
      #pragma unroll
      for (int e = 0; e < EPC; ++e) sVt[(cc + e) * SV + r] = ve[e];
    }
    __syncthreads();
    f32x16 accS[NSUB];
    #pragma unroll
    for (int ms = 0; ms < NSUB; ++ms) {
      accS[ms] = zero16();
      const T *arow = &sK[(32 * ms + col) * SK + KPL * h];
      #pragma unroll
      for (int ks = 0; ks < kHeadDim / KSTEP; ++ks) accS[ms] = M::mma(M::load(arow + ks * KSTEP), qf[ks], accS[ms]);
    }
    float bmax = -INFINITY;
    #pragma unroll
    for (int ms = 0; ms < NSUB; ++ms)
      #pragma unroll
      for (int v = 0; v < 16; ++v) {
        if (k0 + 32 * ms + acc_row(v, lane) >= Tn) accS[ms][v] = -INFINITY;
        bmax = fmaxf(bmax, accS[ms][v]);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float new_max = fmaxf(run_max, bmax);
    const float alpha = exp2f((run_max - new_max) * c2);
    run_max = new_max;
    float psum = 0.0f;
    #pragma unroll
    for (int ms = 0; ms < NSUB; ++ms)
      #pragma unroll
      for (int v = 0; v < 16; ++v) {
        float p = exp2f((accS[ms][v] - new_max) * c2);
        accS[ms][v] = p;
        psum += p;
      }
    run_sum = run_sum * alpha + psum;
    #pragma unroll
    for (int cs = 0; cs < 4; ++cs)
      #pragma unroll
      for (int v = 0; v < 16; ++v) accY[cs][v] *= alpha;
    // Y^T += V^T P^T over this tile's keys, k-slots permuted to the accumulator layout
    #pragma unroll
    for (int kk = 0; kk < KB / KSTEP; ++kk) {
      typename M::frag pf;
      int keys[KPL];
      #pragma unroll
      for (int e = 0; e < KPL; ++e) {
        int vv = kk * KPL + e, ms = vv >> 4, v = vv & 15;
        keys[e] = 32 * ms + acc_row(v, lane);
        if constexpr (KPL == 1) pf = (T)accS[ms][v];
        else pf[e] = (T)accS[ms][v];
      }
      #pragma unroll
      for (int cs = 0; cs < 4; ++cs) {
        const T *vrow = &sVt[(32 * cs + col) * SV];
        typename M::frag vf;
        if constexpr (KPL == 1) vf = vrow[keys[0]];
        else
          #pragma unroll
          for (int e = 0; e < KPL; ++e) vf[e] = vrow[keys[e]];
        accY[cs] = M::mma(vf, pf, accY[cs]);
      }
    }
    __syncthreads();
  }
  run_sum += __shfl_xor(run_sum, 32, 64);
  if (!qvalid) return;
  const float inv = 1.0f / run_sum;
  float *yrow = Y + ((size_t)b * n + q) * kHeadDim;
  #pragma unroll
  for (int cs = 0; cs < 4; ++cs)
    #pragma unroll
    for (int g = 0; g < 4; ++g) {
      f32x4 o = {accY[cs][4 * g] * inv, accY[cs][4 * g + 1] * inv, accY[cs][4 * g + 2] * inv,
                 accY[cs][4 * g + 3] * inv};
      *reinterpret_cast<f32x4 *>(yrow + 32 * cs + 8 * g + 4 * h) = o;
    }
  if (h == 0) {
    z[(size_t)b * n + q] = run_max * scale;
    m[(size_t)b * n + q] = run_sum;
  }
}

hipError_t launch_rowstats(int dtype, const void *K, const void *V, const void *Q, float *z, float *m, float *Y,
                           int B, int T, int n, float scale, hipStream_t s) {
  dim3 grid((n + 127) / 128, B);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_rowstats<bf16>, grid, dim3(256), 0, s, (const bf16 *)K, (const bf16 *)V, (const bf16 *)Q,
                       z, m, Y, T, n, scale);
  else
    hipLaunchKernelGGL(k_rowstats<float>, grid, dim3(256), 0, s, (const float *)K, (const float *)V,
                       (const float *)Q, z, m, Y, T, n, scale);
  return hipGetLastError();
}

}  // namespace arckv
