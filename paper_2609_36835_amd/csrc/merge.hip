// Convex key merge (Section 3.4).
//
//  k_zmax            z_merge = max_i z_i (the global logit maximum equals the
//                    largest full-cache row maximum, eq. response_profile)
//  (the assignment itself, kappa, is in assign.hip)
//  k_group_sort      stable counting sort of positions by group (deterministic)
//  k_group_merge     c_r = sum_j alpha_rj k_j with alpha_rj = lambda phi_j / sum_G phi
//                    + (1 - lambda)[j = s_r], renormalised to sum exactly to 1
//                    in float (eq. mass_centroid, eq. key_merge)
#include "common.hpp"

namespace arckv {

__global__ void __launch_bounds__(256) k_zmax(const float *__restrict__ z, int n, float *__restrict__ zmax) {
  __shared__ float red[4];
  const int b = blockIdx.x, tid = threadIdx.x;
  float v = -INFINITY;
  for (int i = tid; i < n; i += 256) v = fmaxf(v, z[(size_t)b * n + i]);
  v = wave_max(v);
  if ((tid & 63) == 0) red[tid >> 6] = v;
  __syncthreads();
  if (tid == 0) zmax[b] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

// Groups whose cursors fit in LDS (64 KB) take the LDS variant.
constexpr int kSortLdsGroups = 16384;

// One workgroup per pair.  Produces offsets [t+1] and perm [T] (positions
// grouped by kappa, ascending position within each group).  The cursors live
// in LDS (kLds, t <= kSortLdsGroups) or in cursor [B][t] (global scratch).
// Four waves clear and count; wave 0 alone scans and places, one 64-position
// chunk at a time in order, which keeps every group in ascending position.
template <bool kLds>
__global__ void __launch_bounds__(256) k_group_sort(const int32_t *__restrict__ kappa, int T, int t,
                                                    int32_t *__restrict__ offsets, int32_t *__restrict__ cursor,
                                                    int32_t *__restrict__ perm) {
  __shared__ int32_t lcur[kLds ? kSortLdsGroups : 1];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int32_t *kp = kappa + (size_t)b * T;
  int32_t *off = offsets + (size_t)b * (t + 1);
  int32_t *cur = kLds ? lcur : cursor + (size_t)b * t;
  int32_t *pm = perm + (size_t)b * T;
  // every access to cur[] is an atomic, fenced between phases
  for (int r = tid; r < t; r += 256) atomicExch(&cur[r], 0);
  if (!kLds) __threadfence();
  __syncthreads();
  for (int j = tid; j < T; j += 256) atomicAdd(&cur[kp[j]], 1);
  if (!kLds) __threadfence();
  __syncthreads();
  if (tid >= 64) return;
  // exclusive scan of the counts
  int32_t carry = 0;
  for (int r0 = 0; r0 < t; r0 += 64) {
    const int r = r0 + lane;
    int32_t c = r < t ? atomicAdd(&cur[r], 0) : 0;
    int32_t x = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      int32_t y = __shfl_up(x, d, 64);
      if (lane >= d) x += y;
    }
    if (r < t) {
      off[r] = carry + x - c;
      atomicExch(&cur[r], carry + x - c);
    }
    carry += __shfl(x, 63, 64);
  }
  if (lane == 0) off[t] = carry;
  if (!kLds) __threadfence();
  int nbits = 1;
  while ((1 << nbits) < t) ++nbits;
  const uint64_t lanemask = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int j0 = 0; j0 < T; j0 += 64) {
    const int j = j0 + lane;
    const bool in = j < T;
    const int32_t r = in ? kp[j] : 0;
    uint64_t match = __ballot(in);
    for (int bit = 0; bit < nbits; ++bit) {
      uint64_t bal = __ballot(in && ((r >> bit) & 1));
      match &= ((r >> bit) & 1) ? bal : ~bal;
    }
    const int rank = __popcll(match & lanemask);
    const int leader = __ffsll((long long)match) - 1;
    int32_t base = 0;
    if (in && lane == leader) base = atomicAdd(&cur[r], __popcll(match));
    base = __shfl(base, leader < 0 ? 0 : leader, 64);
    if (in && base + rank < T) pm[base + rank] = j;
  }
}

// One wave per compact key r (rows r >= t of the padded copies are zeroed).
// Outputs: C_k [B][t][d] fp32 and the padded operand copy used by Phi_C:
// bf16 hi/lo planes [B][2][tp][d] (bf16 inputs) or fp32 [B][tp][d].
template <typename E>
__global__ void __launch_bounds__(256) k_group_merge(const E *__restrict__ K, const float *__restrict__ phi,
                                                     const int32_t *__restrict__ offsets,
                                                     const int32_t *__restrict__ perm,
                                                     const int32_t *__restrict__ anchors, int T, int t,
                                                     int64_t tp, float lambda, float *__restrict__ Ck,
                                                     void *__restrict__ Ckp) {
  // One wave per group r.  The group mass is a wave reduction over its members;
  // the weighted sum takes four members at a time, lane (kq, dl) = (lane / 16,
  // lane % 16) owning member beg + kq + 4 i and dims 8 dl .. 8 dl + 7 (16-byte
  // rows for bf16), and the four partial sums meet in two shuffles.  Every sum
  // runs in a fixed order, so results are deterministic.
  const int b = blockIdx.y, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= tp) return;
  const int kq = lane >> 4, d0 = 8 * (lane & 15);
  float c[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) c[e] = 0.0f;
  if (r < t) {
    const int32_t beg = offsets[(size_t)b * (t + 1) + r], end = offsets[(size_t)b * (t + 1) + r + 1];
    const int32_t *pm = perm + (size_t)b * T;
    const float *ph = phi + (size_t)b * T;
    const int32_t s = anchors[(size_t)b * t + r];
    float mass = 0.0f;
    for (int32_t q = beg + lane; q < end; q += 64) mass += ph[pm[q]];
    mass = wave_sum(mass);
    const E *Kb = K + (size_t)b * T * kHeadDim + d0;
    float wsum = 0.0f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
    for (int32_t q = beg + kq; q < end; q += 4) {
      const int32_t j = pm[q];
      float alpha = (mass > 0.0f) ? lambda * (ph[j] / mass) : 0.0f;
      if (j == s) alpha += (mass > 0.0f) ? (1.0f - lambda) : 1.0f;
      wsum += alpha;
      const E *kr = Kb + (size_t)j * kHeadDim;
      float kv[8];
      if constexpr (sizeof(E) == 2) {
        const bf16x8 v = *reinterpret_cast<const bf16x8 *>(kr);
#pragma unroll
        for (int e = 0; e < 8; ++e) kv[e] = (float)v[e];
      } else {
        const f32x4 v0 = *reinterpret_cast<const f32x4 *>(kr), v1 = *reinterpret_cast<const f32x4 *>(kr + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          kv[e] = v0[e];
          kv[4 + e] = v1[e];
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(alpha, kv[e], acc[e]);
    }
    wsum += __shfl_xor(wsum, 16, 64);
    wsum += __shfl_xor(wsum, 32, 64);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[e] += __shfl_xor(acc[e], 16, 64);
      acc[e] += __shfl_xor(acc[e], 32, 64);
      c[e] = acc[e] / wsum;
    }
    if (kq == 0) {
      float *o = Ck + ((size_t)b * t + r) * kHeadDim + d0;
      *reinterpret_cast<f32x4 *>(o) = f32x4{c[0], c[1], c[2], c[3]};
      *reinterpret_cast<f32x4 *>(o + 4) = f32x4{c[4], c[5], c[6], c[7]};
    }
  }
  if (kq != 0) return;
  if constexpr (sizeof(E) == 2) {
    bf16 *hi = reinterpret_cast<bf16 *>(Ckp) + ((size_t)b * 2 * tp + r) * kHeadDim + d0;
    bf16 *lo = hi + tp * kHeadDim;
    bf16x8 vh, vl;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      bf16 h, l;
      split_bf16(c[e], h, l);
      vh[e] = h;
      vl[e] = l;
    }
    *reinterpret_cast<bf16x8 *>(hi) = vh;
    *reinterpret_cast<bf16x8 *>(lo) = vl;
  } else {
    float *o = reinterpret_cast<float *>(Ckp) + ((size_t)b * tp + r) * kHeadDim + d0;
    *reinterpret_cast<f32x4 *>(o) = f32x4{c[0], c[1], c[2], c[3]};
    *reinterpret_cast<f32x4 *>(o + 4) = f32x4{c[4], c[5], c[6], c[7]};
  }
}

// ------------------------------------------------------------------ launchers
hipError_t launch_zmax(const float *z, int B, int n, float *zmax, hipStream_t s) {
  hipLaunchKernelGGL(k_zmax, dim3(B), dim3(256), 0, s, z, n, zmax);
  return hipGetLastError();
}


hipError_t launch_group_merge(int dtype, const void *K, const float *phi, const int32_t *kappa,
                              const int32_t *anchors, int B, int T, int t, int64_t tp, float lambda,
                              int32_t *offsets, int32_t *cursor, int32_t *perm, float *Ck, void *Ckp,
                              hipStream_t s) {
  if (t <= kSortLdsGroups)
    hipLaunchKernelGGL(k_group_sort<true>, dim3(B), dim3(256), 0, s, kappa, T, t, offsets, cursor, perm);
  else
    hipLaunchKernelGGL(k_group_sort<false>, dim3(B), dim3(256), 0, s, kappa, T, t, offsets, cursor, perm);
  dim3 grid((unsigned)(tp / 4), B);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_group_merge<bf16>, grid, dim3(256), 0, s, (const bf16 *)K, phi, offsets, perm, anchors, T,
                       t, tp, lambda, Ck, Ckp);
  else
    hipLaunchKernelGGL(k_group_merge<float>, grid, dim3(256), 0, s, (const float *)K, phi, offsets, perm, anchors,
                       T, t, tp, lambda, Ck, Ckp);
  return hipGetLastError();
}

}  // namespace arckv
