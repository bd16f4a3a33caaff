// Full-cache row statistics (Appendix A.9): for every reference query q_i,
//   z_i = max_j s q_i.k_j,   m_i = sum_j exp(s q_i.k_j - z_i),   Y_i = sum_j exp(.) v_j / m_i.
// z are the row maxima that shift Phi_K and Phi_C, m = Phi_K 1 are the mass
// targets of the bias fit, Y the full-attention outputs the value fit matches.
//
// Flash-style single pass over the keys with an online maximum.  Each wave
// owns 32 queries and computes D[key][query] = K Q^T, so every lane holds one
// query column: its running max/sum live in registers.  The probabilities are
// fed back as the B operand of Y^T[c][q] += V^T[c][key] P^T[key][q].
// fp32 inputs: the MFMA k-slots are permuted to match the accumulator layout,
// and V^T is staged in LDS with the same key order (k_rowstats<float>).
// bf16 inputs: see k_rowstats_bf16 below.
#include "common.hpp"

namespace arckv {

template <typename T> struct RowstatsCfg;
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


// ---------------------------------------------------------------- bf16 path
// 256 queries per workgroup (8 waves x 32), 64-key tiles in two LDS stages.
// K tiles arrive with the direct-to-LDS loads, rows of 256 bytes with their
// 16-byte chunks XOR-swizzled by (row & 15), so the fragment reads of 16
// consecutive rows hit distinct banks.  V tiles are transposed on the way in
// (each thread loads a column pair of 8 keys and writes two 16-byte runs) into
// V^T[c][key] rows of 128 bytes, chunk-swizzled by ((c >> 1) & 7).
// P^T is the B operand of Y^T += V^T P^T with k-slot e of lane half h standing
// for key 8h + e of the 16-key step; the accumulator layout of S leaves half of
// those keys in the other half-wave, so four bf16 values are exchanged with a
// cross-half shuffle per k-step.  Workgroups are remapped so the query tiles of
// one pair share an XCD (and its L2 copy of that pair's keys and values).
constexpr int kRsQ = 256, kRsK = 64;
constexpr int kRsKBytes = kRsK * kHeadDim * 2;            // 16 KB
constexpr int kRsStage = 2 * kRsKBytes;                   // K tile + V^T tile

typedef __attribute__((address_space(3))) void rs_lds_t;

__global__ void __launch_bounds__(512, 1) k_rowstats_bf16(const bf16 *__restrict__ K, const bf16 *__restrict__ V,
                                                          const bf16 *__restrict__ Q, float *__restrict__ z,
                                                          float *__restrict__ m, float *__restrict__ Y, int Tn, int n,
                                                          float scale, int qtiles) {
  __shared__ __attribute__((aligned(1024))) char sbuf[2 * kRsStage];
  const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(tile / qtiles), qt = (int)(tile % qtiles);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int q = qt * kRsQ + wave * 32 + col;
  const bool qvalid = q < n;
  const bf16 *Kb = K + (size_t)b * Tn * kHeadDim;
  const bf16 *Vb = V + (size_t)b * Tn * kHeadDim;

  bf16x8 qf[kHeadDim / 16];
  {
    const bf16 *qrow = Q + ((size_t)b * n + (qvalid ? q : 0)) * kHeadDim;
#pragma unroll
    for (int ks = 0; ks < kHeadDim / 16; ++ks)
      qf[ks] = qvalid ? *reinterpret_cast<const bf16x8 *>(qrow + ks * 16 + 8 * h) : Mfma<bf16>::zero();
  }
  // K: run gi (2 per wave) covers rows 4 gi .. 4 gi + 3; lane l fills physical
  // chunk l % 16 of row 4 gi + l / 16 with logical chunk (l % 16) ^ row.
  int koff[2], krow[2];
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int gi = wave * 2 + u, row = 4 * gi + lane / 16;
    krow[u] = row;
    koff[u] = 8 * ((lane % 16) ^ (row & 15));
  }
  auto issue_k = [&](int k0, int st) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int key = min(k0 + krow[u], Tn - 1);
      __builtin_amdgcn_global_load_lds((const void *)(Kb + (size_t)key * kHeadDim + koff[u]),
                                       (rs_lds_t *)(sbuf + st * kRsStage + (wave * 2 + u) * 1024), 16, 0, 0);
    }
  };
  // V: thread -> column pair cp (c = 2 cp) and key group kg (keys 8 kg .. 8 kg + 7)
  const int cp = tid & 63, kg = tid >> 6;
  uint32_t vr[8];
  auto load_v = [&](int k0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = min(k0 + 8 * kg + e, Tn - 1);
      vr[e] = *reinterpret_cast<const uint32_t *>(Vb + (size_t)key * kHeadDim + 2 * cp);
    }
  };
  auto store_vt = [&](int st) {
    char *vt = sbuf + st * kRsStage + kRsKBytes;
    const int c = 2 * cp, ph = kg ^ ((c >> 1) & 7);
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = (vr[2 * e] & 0xFFFFu) | (vr[2 * e + 1] << 16);
      hi[e] = (vr[2 * e] >> 16) | (vr[2 * e + 1] & 0xFFFF0000u);
    }
    *reinterpret_cast<uint4 *>(vt + c * 128 + 16 * ph) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
    *reinterpret_cast<uint4 *>(vt + (c + 1) * 128 + 16 * ph) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
  };

  const float c2 = scale * 1.4426950408889634f;   // exp(s x) = exp2(c2 x)
  float run_max = -INFINITY, run_sum = 0.0f;
  f32x16 accY[4];
#pragma unroll
  for (int cs = 0; cs < 4; ++cs) accY[cs] = zero16();

  const int nt = (Tn + kRsK - 1) / kRsK;
  // S = K Q^T for the 64 keys in the K part of LDS stage st
  auto scores = [&](int st, f32x16 (&S)[2]) {
    const char *sk = sbuf + st * kRsStage;
#pragma unroll
    for (int ms = 0; ms < 2; ++ms) {
      S[ms] = zero16();
      const int row = 32 * ms + col;
#pragma unroll
      for (int ks = 0; ks < kHeadDim / 16; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(sk + row * 256 + 16 * ((2 * ks + h) ^ (row & 15)));
        S[ms] = Mfma<bf16>::mma(a, qf[ks], S[ms]);
      }
    }
  };
  // Tile i: the online softmax of its scores S and Y^T += V^T P^T from the V
  // part of stage i & 1.  The scores of tile i + 1 (K part of stage (i + 1) & 1)
  // go to Sn in the same basic block as the exponentials, so the matrix cores
  // work on them while the VALUs run the softmax (in the last tile they read a
  // stale stage and are discarded).  Keys therefore run one tile ahead of
  // values: on entry stage (i + 1) & 1 holds K tile i + 1 and stage i & 1
  // holds V^T tile i; V tile i + 1 is in registers.
  auto body = [&](int i, f32x16 (&S)[2], f32x16 (&Sn)[2]) {
    const int k0 = i * kRsK, st = i & 1;
    if (i + 1 < nt) store_vt(st ^ 1);
    if (i + 2 < nt) {   // stage st: its K tile was read in tile i - 1, before the last barrier
      issue_k(k0 + 2 * kRsK, st);
      load_v(k0 + 2 * kRsK);
    }
    if (k0 + kRsK > Tn) {   // last tile: keys past Tn get no weight
#pragma unroll
      for (int ms = 0; ms < 2; ++ms)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (k0 + 32 * ms + acc_row(v, lane) >= Tn) S[ms][v] = -INFINITY;
    }
    float bmax = -INFINITY;
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int v = 0; v < 16; ++v) bmax = fmaxf(bmax, S[ms][v]);
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
    const float new_max = fmaxf(run_max, bmax);
    // The accumulators are rescaled only when some row's maximum grew (rare
    // after the first tiles); unchanged rows take alpha = 1.  The exponentials
    // are the hardware base-2 ones: arguments are <= 0 and a result below the
    // smallest normal float is negligible next to the running sum (>= 1).
    if (__ballot(new_max > run_max)) {
      const float alpha = __builtin_amdgcn_exp2f((run_max - new_max) * c2);
      run_sum *= alpha;
#pragma unroll
      for (int cs = 0; cs < 4; ++cs)
#pragma unroll
        for (int v = 0; v < 16; ++v) accY[cs][v] *= alpha;
    }
    run_max = new_max;
    scores(st ^ 1, Sn);
    const float mc2 = new_max * c2;
    float psum = 0.0f;
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(S[ms][v], c2, -mc2));
        S[ms][v] = p;
        psum += p;
      }
    run_sum += psum;
    const char *svt = sbuf + st * kRsStage + kRsKBytes;
#pragma unroll
    for (int kk = 0; kk < kRsK / 16; ++kk) {
      const int ms = kk >> 1, base = 8 * (kk & 1);
      uint32_t pk[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bf16x2 x = {(bf16)S[ms][base + 2 * e], (bf16)S[ms][base + 2 * e + 1]};
        pk[e] = __builtin_bit_cast(uint32_t, x);
      }
      // pk[0..1]: own keys 4h + 0..3, pk[2..3]: own keys 8 + 4h + 0..3 (of this
      // 16-key step).  The half-wave swap exchanges the upper half-wave's
      // pk[0..1] with the lower half-wave's pk[2..3], so that every lane then
      // holds keys 8h + 0..7 of its query in order.
      const auto x02 = __builtin_amdgcn_permlane32_swap(pk[0], pk[2], false, false);
      const auto x13 = __builtin_amdgcn_permlane32_swap(pk[1], pk[3], false, false);
      uint32_t bw[4];
      bw[0] = x02[0];
      bw[1] = x13[0];
      bw[2] = x02[1];
      bw[3] = x13[1];
      bf16x8 pf;
      __builtin_memcpy(&pf, bw, 16);
#pragma unroll
      for (int cs = 0; cs < 4; ++cs) {
        const int c = 32 * cs + col;
        const bf16x8 vf = *reinterpret_cast<const bf16x8 *>(svt + c * 128 + 16 * ((2 * kk + h) ^ ((c >> 1) & 7)));
        accY[cs] = Mfma<bf16>::mma(vf, pf, accY[cs]);
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };

  issue_k(0, 0);
  if (nt > 1) issue_k(kRsK, 1);
  load_v(0);
  __builtin_amdgcn_s_waitcnt(0);
  store_vt(0);
  if (nt > 1) load_v(kRsK);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  f32x16 Sa[2], Sb[2];
  scores(0, Sa);
  int i = 0;
  for (; i + 1 < nt; i += 2) {
    body(i, Sa, Sb);
    body(i + 1, Sb, Sa);
  }
  if (i < nt) body(i, Sa, Sb);
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
  if (dtype == ARCKV_BF16) {
    const int qtiles = (n + kRsQ - 1) / kRsQ;
    hipLaunchKernelGGL(k_rowstats_bf16, dim3((unsigned)(qtiles * B)), dim3(512), 0, s, (const bf16 *)K,
                       (const bf16 *)V, (const bf16 *)Q, z, m, Y, T, n, scale, qtiles);
    return hipGetLastError();
  }
  dim3 grid((n + 127) / 128, B);
  hipLaunchKernelGGL(k_rowstats<float>, grid, dim3(256), 0, s, (const float *)K, (const float *)V, (const float *)Q, z,
                     m, Y, T, n, scale);
  return hipGetLastError();
}

}  // namespace arckv
