// Key-to-anchor assignment with a certified argmax (Section 3.4,
// eq. anchor_assignment; ties to the lowest r).
//
// The bulk similarity contraction S[r][j] = sum_i U_S[i][r] E[i][j] runs on
// fp16 (bf16 inputs) or fp32 (fp32 inputs) operands; rounding the operands can
// reorder two anchors whose similarities to a key are close.  Every key is
// therefore decided in up to three passes, each a certified filter for the next:
//
//  A  the contraction keeps, per (anchor tile, key), the two best similarities
//     and the third value (EpiArgmax*).  With eta the relative and alpha the
//     absolute error bound of one similarity, no anchor r with
//     S_A(r) < (S_A(best) - alpha)(1 - eta)/(1 + eta) - alpha can be the argmax.
//     A key with exactly one anchor above that threshold is decided; the others
//     are flagged, with the best two of each tile above the threshold, or the
//     whole tile where its third value reaches it, as candidates
//     (k_assign_finalize).
//  C  flagged keys are re-scored against their candidates' fp32 profiles
//     (k_prof_anchor_*): for bf16 inputs the key's logits come from MFMA with
//     one fp32 accumulator per 16-wide slice of the head dimension, the eight
//     slices summed in fp32 (logit error at most gamma_23 s ||q|| ||k||), the
//     exponentials from v_exp_f32 (exp32_err), and each dot product from fp32
//     products summed four at a time, then in float64 (for fp32 inputs, float64
//     logits).  Keys that still have more than one survivor go on
//     (k_assign_refine).
//  D  float64 throughout: logits, exponentials, norms and dot products
//     (k_assign_exact).  Equal float64 similarities go to the lower r.
//
// The bounds are stated on the functions that use them.
#include <type_traits>

#include "assign.hpp"
#include "common.hpp"

namespace arckv {
typedef __attribute__((__vector_size__(4 * sizeof(double)))) double f64x4;

constexpr double kU32 = 5.9604644775390625e-08;   // 2^-24, unit roundoff of fp32
constexpr double kU16 = 4.8828125e-04;            // 2^-11, unit roundoff of fp16

__device__ inline double gamma_m(double m) { return m * kU32 / (1.0 - m * kU32); }

// Per-pair constants of the error bounds.
struct AssignPair {
  double qmax;   // max_i ||q_i||_2
  double amax;   // max_r ||k_{s_r}||_2
};

// A fixed grid of nx workgroups per pair, remapped so that each XCD receives a
// contiguous range of (pair, x): all workgroups of a pair share one L2 (the
// pair's queries and anchor profiles are read by each of them).
__device__ inline void pair_block(int nx, int P, int &x, int &b) {
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  const int64_t tile = xcd_remap(lin, (int64_t)nx * P);
  b = (int)(tile / nx);
  x = (int)(tile % nx);
}

// ---------------------------------------------------------------- norms
// pn[b] = {max_i ||q_i||, max_r ||k_{s_r}||}, in float64, rounded up by one part
// in 1e12 so that the bounds built on them stay upper bounds.
template <typename E>
__global__ void __launch_bounds__(256) k_pair_norms(const E *__restrict__ Q, const E *__restrict__ K,
                                                    const int32_t *__restrict__ anchors, int n, int T, int t,
                                                    AssignPair *__restrict__ pn) {
  __shared__ double red[2][4];
  const int b = blockIdx.x, tid = threadIdx.x;
  double mq = 0.0, ma = 0.0;
  for (int i = tid; i < n; i += 256) {
    const E *q = Q + ((size_t)b * n + i) * kHeadDim;
    double ss = 0.0;
    for (int k = 0; k < kHeadDim; ++k) {
      const double v = (double)(float)q[k];
      ss = fma(v, v, ss);
    }
    mq = fmax(mq, ss);
  }
  for (int r = tid; r < t; r += 256) {
    const E *kr = K + ((size_t)b * T + anchors[(size_t)b * t + r]) * kHeadDim;
    double ss = 0.0;
    for (int k = 0; k < kHeadDim; ++k) {
      const double v = (double)(float)kr[k];
      ss = fma(v, v, ss);
    }
    ma = fmax(ma, ss);
  }
  for (int m = 32; m >= 1; m >>= 1) {
    mq = fmax(mq, __shfl_xor(mq, m, 64));
    ma = fmax(ma, __shfl_xor(ma, m, 64));
  }
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = mq;
    red[1][tid >> 6] = ma;
  }
  __syncthreads();
  if (tid == 0) {
    double a = 0.0, c = 0.0;
    for (int w = 0; w < 4; ++w) {
      a = fmax(a, red[0][w]);
      c = fmax(c, red[1][w]);
    }
    pn[b].qmax = sqrt(a) * (1.0 + 1e-12);
    pn[b].amax = sqrt(c) * (1.0 + 1e-12);
  }
}

// Logit of one (query, key) element from the eight 16-wide slices of the head
// dimension: each slice is one MFMA into a zero accumulator (products of bf16
// values are exact in fp32, so a slice sum is within gamma_16 of the sum of its
// |products|), and the eight slice sums are added in fp32 in a fixed order, so
// the logit is within gamma_23 s sum_k |q_k k_k| <= gamma_23 s ||q|| ||k|| of exact.
constexpr double kSliceTerms = 23.0;

// Relative error bound of exp(s l - z) evaluated as 2^(l c2 - z2) with c2 = s
// log2(e) and z2 = z log2(e) rounded to fp32, one fp32 fma and v_exp_f32 (1 ulp):
// the exponent's absolute error is at most u (2 |l c2| + 2 |z2| + |result|)
// and |result| <= |l c2| + |z2|.  A bounds |l c2|, Z bounds |z2|.
__device__ inline double exp32_err(double A, double Z) {
  return 0.6931471805599453 * kU32 * (3.0 * A + 3.0 * Z) + 2.0 * kU32;
}

// ---------------------------------------------------------------- anchor profiles
// Precise anchor profiles e_ir = exp(s q_i.k_{s_r} - z_merge) for bf16 inputs:
// logits from eight MFMA slices added in a fixed order (kSliceTerms), the
// exponential in fp32 (exp32_err).  Ua [P][tp][np] float32 (zero for i >= n),
// anorm [P][tp] = ||e_r||_2, accumulated in float64.  A workgroup
// owns 128 anchors (32 per wave, kept as MFMA B fragments) and sweeps all
// queries in tiles of 64.
__global__ void __launch_bounds__(256) k_prof_anchor_bf16(const bf16 *__restrict__ Q, const bf16 *__restrict__ K,
                                                          const int32_t *__restrict__ anchors,
                                                          const float *__restrict__ zmerge, int n, int T, int t,
                                                          int64_t tp, int64_t np_, double scale,
                                                          float *__restrict__ Ua, double *__restrict__ anorm) {
  constexpr int SQ = kHeadDim + 8;
  __shared__ __attribute__((aligned(16))) bf16 sQ[64 * SQ];
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int r = blockIdx.x * 128 + wave * 32 + col;
  const bool rvalid = r < t;
  bf16x8 bfr[8];
  const bf16 *kr = K + ((size_t)b * T + (rvalid ? anchors[(size_t)b * t + r] : 0)) * kHeadDim;
#pragma unroll
  for (int ks = 0; ks < 8; ++ks)
    bfr[ks] = rvalid ? *reinterpret_cast<const bf16x8 *>(kr + ks * 16 + 8 * h) : Mfma<bf16>::zero();
  const float c2 = (float)(scale * 1.4426950408889634), zs2 = zmerge[b] * 1.4426950408889634f;
  const bf16 *Qb = Q + (size_t)b * n * kHeadDim;
  float *urow = Ua + ((size_t)b * tp + (rvalid ? r : 0)) * np_;
  double ss = 0.0;
  // the next 64-query tile is loaded into registers while this one is processed
  f32x4 qn[4];
  auto fetch_q = [&](int j0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u, rr = c / 16, cc = (c % 16) * 8;
      qn[u] = j0 + rr < n ? *reinterpret_cast<const f32x4 *>(Qb + (size_t)(j0 + rr) * kHeadDim + cc)
                          : f32x4{0.f, 0.f, 0.f, 0.f};
    }
  };
  fetch_q(0);
  for (int i0 = 0; i0 < np_; i0 += 64) {
    __syncthreads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u, rr = c / 16, cc = (c % 16) * 8;
      *reinterpret_cast<f32x4 *>(&sQ[rr * SQ + cc]) = qn[u];
    }
    if (i0 + 64 < np_) fetch_q(i0 + 64);
    __syncthreads();
#pragma unroll
    for (int ms = 0; ms < 2; ++ms) {
      const bf16 *arow = &sQ[(32 * ms + col) * SQ + 8 * h];
      f32x16 lsum = Mfma<bf16>::mma(*reinterpret_cast<const bf16x8 *>(arow), bfr[0], zero16());
#pragma unroll
      for (int ks = 1; ks < 8; ++ks) {
        const f32x16 part = Mfma<bf16>::mma(*reinterpret_cast<const bf16x8 *>(arow + ks * 16), bfr[ks], zero16());
#pragma unroll
        for (int v = 0; v < 16; ++v) lsum[v] += part[v];
      }
      float e[16];
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = i0 + 32 * ms + acc_row(v, lane);
        const float ev = i < n ? __builtin_amdgcn_exp2f(fmaf(lsum[v], c2, -zs2)) : 0.0f;
        ss = fma((double)ev, (double)ev, ss);
        e[v] = ev;
      }
      if (rvalid) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
          *reinterpret_cast<f32x4 *>(urow + i0 + 32 * ms + 8 * g + 4 * h) =
              f32x4{e[4 * g], e[4 * g + 1], e[4 * g + 2], e[4 * g + 3]};
      }
    }
  }
  ss += __shfl_xor(ss, 32, 64);
  if (rvalid && h == 0) anorm[(size_t)b * tp + r] = sqrt(ss);
}

// fp32 inputs: the same profiles with float64 logits and exponentials (one
// workgroup per anchor, one thread per query).
__global__ void __launch_bounds__(256) k_prof_anchor_f32(const float *__restrict__ Q, const float *__restrict__ K,
                                                         const int32_t *__restrict__ anchors,
                                                         const float *__restrict__ zmerge, int n, int T, int t,
                                                         int64_t tp, int64_t np_, double scale,
                                                         float *__restrict__ Ua, double *__restrict__ anorm) {
  __shared__ double kr[kHeadDim];
  __shared__ double red[4];
  const int b = blockIdx.y, r = blockIdx.x, tid = threadIdx.x;
  if (tid < kHeadDim) kr[tid] = (double)K[((size_t)b * T + anchors[(size_t)b * t + r]) * kHeadDim + tid];
  __syncthreads();
  const double zm = (double)zmerge[b];
  float *urow = Ua + ((size_t)b * tp + r) * np_;
  double ss = 0.0;
  for (int64_t i = tid; i < np_; i += 256) {
    double ev = 0.0;
    if (i < n) {
      const float *q = Q + ((size_t)b * n + i) * kHeadDim;
      double l = 0.0;
      for (int k = 0; k < kHeadDim; ++k) l = fma((double)q[k], kr[k], l);
      ev = exp(scale * l - zm);
    }
    ss = fma(ev, ev, ss);
    urow[i] = (float)ev;
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) red[tid >> 6] = ss;
  __syncthreads();
  if (tid == 0) anorm[(size_t)b * tp + r] = sqrt(red[0] + red[1] + red[2] + red[3]);
}

// The contraction's anchor operand U [P][tp][np]: Ua / anorm, stored in fp16
// scaled by 2^15 for bf16 inputs (one rounding of the fp32 product) or in
// fp32; rows r >= t and columns i >= n are zero.  One wave per row, four
// consecutive columns per lane (np_ is a multiple of 256).
template <typename T>
__global__ void __launch_bounds__(256) k_anchor_u(const float *__restrict__ Ua, const double *__restrict__ anorm,
                                                  int n, int t, int64_t tp, int64_t np_, float uscale,
                                                  T *__restrict__ U) {
  typedef __attribute__((__vector_size__(4 * sizeof(T)))) T T4;
  const int b = blockIdx.y, lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= tp) return;
  T *urow = U + ((size_t)b * tp + r) * np_;
  const float *arow = Ua + ((size_t)b * tp + r) * np_;
  const double nr = r < t ? anorm[(size_t)b * tp + r] : 0.0;
  const float inv = nr > 0.0 ? (float)((double)uscale / nr) : 0.0f;
  for (int64_t i = 4 * lane; i < np_; i += 256) {
    f32x4 a = {0.0f, 0.0f, 0.0f, 0.0f};
    if (r < t && i < n) a = *reinterpret_cast<const f32x4 *>(arow + i);
    T4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = (T)(i + e < n ? a[e] * inv : 0.0f);
    *reinterpret_cast<T4 *>(urow + i) = o;
  }
}

// ---------------------------------------------------------------- pass A bounds
// Relative (eta) and absolute (alpha, in the units of the stored similarity)
// error bound of one pass-A similarity of key j, whose key has norm kn and mass
// weight phi.  Every term of S(j, r) = sum_i E_ij U_ir is >= 0, so a relative
// bound on each term bounds the sum.
//  bf16 inputs, fp16 operands scaled by 2^15 (S_A = 2^30 S):
//   E'  logit on MFMA, fp32 accumulation over d: gamma_128 s ||q|| ||k_j||;
//       exponent argument formed in fp32 and v_exp_f32 (1 ulp); fp16 rounding.
//   U'  the precise profile (gamma_23 s ||q|| ||k_r|| + exp32_err, fp32),
//       divided by its float64 norm (same bound), a fp32 product and one fp16
//       rounding.
//   fp16 x fp16 products are exact in fp32; the fp32 accumulation of n >= 0
//   terms adds gamma_n; the epilogue truncates the stored value by < 2^-18.  Operands below the fp16 normal range (E' or U' < 2^-14)
//   carry an absolute error <= 2^-25 instead: alpha = 2^-25 (||U'_r||_1 + ||E'_j||_1)
//   <= 2^-10 (sqrt(n) + n phi_j), with ||U_r||_2 = 1.
//  fp32 inputs: fp32 products are rounded (u each, d + 2 terms in the logit and
//   one in every product of the contraction); the anchor operand is the float64
//   profile rounded to fp32 and normalised in fp32.
struct BoundA {
  double eta, alpha;
};

__device__ inline BoundA bound_a(bool bf16in, int n, double s, double zm, const AssignPair &pn, double kn,
                                 double phi) {
  const double A = s * pn.qmax * kn * 1.4426950408889634 * 1.001;   // |logit| log2(e) bound of the key
  BoundA o;
  if (bf16in) {
    const double Z = fabs(zm) * 1.4426950408889634 + (double)kProfLog2Scale;
    const double e_key = gamma_m(kHeadDim) * s * pn.qmax * kn + 0.6931471805599453 * kU32 * (3.0 * A + 4.0 * Z) +
                         2.0 * kU32;
    const double e_anc = gamma_m(kSliceTerms) * s * pn.qmax * pn.amax +
                         exp32_err(s * pn.qmax * pn.amax * 1.4426950408889634 * 1.001, fabs(zm) * 1.4426950408889634);
    const double eE = (1.0 + e_key) * (1.0 + kU16) - 1.0;
    const double eU = (1.0 + e_anc + kU32) / (1.0 - e_anc) * (1.0 + 2.0 * kU32) * (1.0 + kU16) - 1.0;
    // the contraction's epilogue stores similarities with the low 5 bits
    // cleared (relative truncation < 2^-18)
    o.eta = (1.0 + eE) * (1.0 + eU) * (1.0 + gamma_m(n)) * (1.0 + 3.814697265625e-06) - 1.0;
    o.alpha = 9.765625e-04 * 1.01 * (sqrt((double)n) + (double)n * phi * 1.001) + (double)n * 1e-18;
  } else {
    const double Z = fabs(zm) * 1.4426950408889634;
    const double e_key = gamma_m(kHeadDim + 2) * s * pn.qmax * kn +
                         0.6931471805599453 * kU32 * (3.0 * A + 4.0 * Z) + 2.0 * kU32;
    const double eU = 3.0 * kU32 + 1e-14;
    o.eta = (1.0 + e_key) * (1.0 + eU) * (1.0 + kU32) * (1.0 + gamma_m(n)) - 1.0;
    o.alpha = (double)n * 1e-36;
  }
  return o;
}

__device__ inline float threshold_a(float s1, const BoundA &bd) {
  const double th = ((double)s1 - bd.alpha) * (1.0 - bd.eta) / (1.0 + bd.eta) - bd.alpha;
  // round down so that a similarity equal to the exact threshold is kept
  return (float)th - fabsf((float)th) * 1.2e-7f - 1e-37f;
}

template <typename E>
__device__ inline double row_norm(const E *x) {
  double ss = 0.0;
  for (int k = 0; k < kHeadDim; ++k) {
    const double v = (double)(float)x[k];
    ss = fma(v, v, ss);
  }
  return sqrt(ss) * (1.0 + 1e-12);
}

// Candidate anchors of one key after pass A.  For each anchor tile the best
// two above the threshold are candidates; a tile whose third value reaches the
// threshold may hold more, and contributes all its anchors ("overflow").
struct CandA {
  int singles, overflow;
  float th;
  uint64_t g1;
};

__device__ inline CandA cand_a(const uint64_t *p1, const uint64_t *p2, const uint32_t *p3, int64_t stride, int MT,
                               int t, float th_or_nan, uint64_t g1) {
  CandA c;
  c.g1 = g1;
  c.th = th_or_nan;
  c.singles = 0;
  c.overflow = 0;
  for (int mt = 0; mt < MT; ++mt) {
    const uint64_t a = p1[(size_t)mt * stride], b2 = p2[(size_t)mt * stride];
    const float v3 = __uint_as_float(p3[(size_t)mt * stride]);
    if (v3 >= c.th) {
      ++c.overflow;
      continue;
    }
    if (a != 0ull && packed_r(a) < (uint32_t)t && packed_sim(a) >= c.th) ++c.singles;
    if (b2 != 0ull && packed_r(b2) < (uint32_t)t && packed_sim(b2) >= c.th) ++c.singles;
  }
  return c;
}

// Queue key j for the float64 pass with its k surviving candidates, which sit
// at pool offset off (off = -1, k = t: every anchor).
// Queue key j for the float64 pass with k candidates starting at pool offset
// off (off < 0: all t anchors).  More than kPassDSplit pool candidates are
// split over consecutive entries; the capacity dcap covers the largest split
// the pool allows.
__device__ inline void push_d(const AssignLists &L, int b, int j, int off, int k) {
  const bool split = off >= 0 && k > kPassDSplit;
  const int ne = split ? (k + kPassDSplit - 1) / kPassDSplit : 1;
  const int slot = atomicAdd(&L.dcnt[b], ne);
  for (int e = 0; e < ne; ++e) {
    const size_t q = (size_t)b * L.dcap + slot + e;
    L.dkey[q] = j;
    L.doff[q] = split ? off + e * kPassDSplit : off;
    L.dn[q] = split ? min(kPassDSplit, k - e * kPassDSplit) : k;
    L.dgrp[q] = split ? slot : -1;
    L.dgn[q] = ne;
  }
  atomicAdd(&L.stats[b * kAssignStats + 1], 1);
}

// Pass A decision, one thread per position j: anchors map to themselves
// (eq. anchor_assignment); a key with one candidate takes it; the others take
// the pass-A best for now, and their candidates go to the pair's pool for
// pass C.  Anchor tiles have TR rows.
template <typename E>
__global__ void __launch_bounds__(256) k_assign_finalize(
    const uint64_t *__restrict__ part1, const uint64_t *__restrict__ part2, const uint32_t *__restrict__ part3,
    int MT, int64_t Np, const int32_t *__restrict__ anchors, const E *__restrict__ K, const float *__restrict__ phi,
    const float *__restrict__ zmerge, const AssignPair *__restrict__ pn, int T, int t, int n, int TR, double s,
    int32_t *__restrict__ kappa, AssignLists L) {
  const int b = blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= T) return;
  const int32_t *S = anchors + (size_t)b * t;
  int lo = 0, hi = t;   // lo = #{anchors < j}
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (S[mid] < j) lo = mid + 1;
    else hi = mid;
  }
  if (lo < t && S[lo] == j) {
    kappa[(size_t)b * T + j] = lo;
    return;
  }
  const size_t c = (size_t)b * MT * Np + (size_t)(j - lo);
  const uint64_t *p1 = part1 + c, *p2 = part2 + c;
  const uint32_t *p3 = part3 + c;
  uint64_t g1 = 0;
  for (int mt = 0; mt < MT; ++mt) g1 = max(g1, p1[(size_t)mt * Np]);
  const uint32_t r1 = packed_r(g1);
  const double kn = row_norm(K + ((size_t)b * T + j) * kHeadDim);
  const BoundA bd = bound_a(sizeof(E) == 2, n, s, (double)zmerge[b], pn[b], kn, (double)phi[(size_t)b * T + j]);
  const float th = threshold_a(packed_sim(g1), bd);
  const CandA ca = cand_a(p1, p2, p3, Np, MT, t, th, g1);
  kappa[(size_t)b * T + j] = (int32_t)(r1 < (uint32_t)t ? r1 : 0u);
  if (ca.overflow == 0 && ca.singles == 1) return;
  int32_t *st = L.stats + (size_t)b * kAssignStats;
  atomicAdd(&st[0], 1);
  if (ca.overflow) atomicAdd(&st[7], 1);
  // the key's candidates: the best two above the threshold of each tile, or
  // every anchor of a tile whose third value reaches it
  int nc = 0;
  for (int mt = 0; mt < MT; ++mt) {
    if (__uint_as_float(p3[(size_t)mt * Np]) >= th) {
      nc += min(t, (mt + 1) * TR) - mt * TR;
      continue;
    }
    const uint64_t a = p1[(size_t)mt * Np], a2 = p2[(size_t)mt * Np];
    nc += (a != 0ull && packed_r(a) < (uint32_t)t && packed_sim(a) >= th);
    nc += (a2 != 0ull && packed_r(a2) < (uint32_t)t && packed_sim(a2) >= th);
  }
  atomicAdd(&st[2], nc);
  if (nc == 0) {   // no finite similarity reaches the threshold (non-finite input): the pass-A best stands
    atomicAdd(&st[3], 1);
    atomicAdd(&st[4], 1);
    return;
  }
  const int off = atomicAdd(&L.pcnt[b], nc);
  if ((int64_t)off + nc > L.pcap) {   // pool full (near-equal profiles): decided in float64 over all t anchors
    push_d(L, b, j, -1, t);
    return;
  }
  int32_t *pl = L.pool + (size_t)b * L.pcap + off;
  int k = 0;
  for (int mt = 0; mt < MT; ++mt) {
    if (__uint_as_float(p3[(size_t)mt * Np]) >= th) {
      for (int r = mt * TR; r < min(t, (mt + 1) * TR); ++r) pl[k++] = r;
      continue;
    }
    const uint64_t a = p1[(size_t)mt * Np], a2 = p2[(size_t)mt * Np];
    if (a != 0ull && packed_r(a) < (uint32_t)t && packed_sim(a) >= th) pl[k++] = (int32_t)packed_r(a);
    if (a2 != 0ull && packed_r(a2) < (uint32_t)t && packed_sim(a2) >= th) pl[k++] = (int32_t)packed_r(a2);
  }
  const int slot = atomicAdd(&L.fcnt[b], 1);
  L.fkey[(size_t)b * L.cap + slot] = j;
  L.foff[(size_t)b * L.cap + slot] = off;
  L.fn[(size_t)b * L.cap + slot] = nc;
  atomicAdd(&st[6], 1);
}

// Workgroup barrier that waits for this wave's LDS operations only: global
// loads issued before it stay in flight across it.
__device__ __forceinline__ void lds_only_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt and expcnt unconstrained
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------- pass C
// Refine the keys queued by pass A.  The queued keys of a pair form groups of
// 64 (in queue order) and a group's candidates in the pool form chunks of CAP;
// each (group, chunk) is one work item.  The keys' profiles are formed in
// fp32 and each candidate pair accumulates sum_i e_ij e_ir (fp32 products
// summed four at a time, then in float64) against the anchor's stored
// profile; the similarity e_j . e_r / ||e_r|| goes back to the pool, and
// k_assign_decide takes the decisions once every item is done.
//  bf16 inputs: logits from eight MFMA slices as in k_prof_anchor_bf16
//   (kSliceTerms), exponentials within exp32_err.  Bound of one similarity:
//   (1 + eps_k)(1 + eps_a)/(1 - eps_a)(1 + gamma_4) - 1 with eps_k = gamma_23 s
//   ||q|| ||k_j|| + exp32_err and eps_a the same with max ||k_r|| (profile and norm).
//  fp32 inputs: float64 logits and exponentials; the bound is the fp32
//   rounding of the two profiles and of the partial products.
// A key whose best similarity exceeds every other candidate's by more than the
// bound on both is decided; the survivors of the others go to pass D.
// Work distribution: k_refine_plan lays out each pair's items (goff); a fixed
// grid of kRefineBlocks workgroups per pair takes items it = blockIdx.x,
// blockIdx.x + kRefineBlocks, ..., so the chunks of one group with many
// candidates (keys whose candidates include whole anchor tiles) spread over
// workgroups instead of running in sequence on one.  The queries are swept in
// tiles of 128.  Per tile the eight waves form the 64 keys' profiles (one
// 32 x 32 MFMA tile each: a key half by a quarter of the queries) into a
// shared LDS tile; each wave takes 32 candidates, two per load instruction: a
// half-wave covers one candidate's 128 queries, four per lane, so every load
// reads two contiguous 512-byte runs of anchor profile rows.  The candidates'
// partial sums stay in registers (float64) across the tiles and are reduced
// over the half-waves once per item.
constexpr int kRefineBlocks = 128;
constexpr int kRefineCpw = 32;   // candidates per wave

template <typename E>
__global__ void __launch_bounds__(512, 2) k_assign_refine(const E *__restrict__ Q, const E *__restrict__ K,
                                                       const float *__restrict__ zmerge,
                                                       const float *__restrict__ Ua, const double *__restrict__ anorm,
                                                       int T, int n, int64_t tp, int64_t np_, double s,
                                                       AssignLists L) {
  constexpr bool BF = sizeof(E) == 2;
  constexpr int NK = 64, NW = 8, CPW = kRefineCpw, CAP = NW * CPW, QT = 128, SE = QT + 4;
  constexpr int SKB = BF ? kHeadDim + 8 : kHeadDim + 4;   // key-row stride (elements)
  __shared__ int32_t kpos[NK], koff[NK], kbase[NK + 1], khalf, item_g, item_c0;
  __shared__ int32_t cr[CAP];
  __shared__ int32_t ck[CAP];
  __shared__ __attribute__((aligned(16))) E sK[NK * SKB];
  __shared__ __attribute__((aligned(16))) float eS[NK * SE];   // the keys' profiles on one query tile
  // pair-major over the whole grid (no XCD remap): the anchor profiles do not
  // fit an L2 anyway, and a pair with many candidates spreads over every XCD
  const int bx = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int F = L.fcnt[b];
  const double zm = (double)zmerge[b];
  const float c2 = (float)(s * 1.4426950408889634), zs2 = zmerge[b] * 1.4426950408889634f;
  const E *Qb = Q + (size_t)b * n * kHeadDim;
  const float *Uab = Ua + (size_t)b * tp * np_;
  int32_t *pool = L.pool + (size_t)b * L.pcap;
  double *psim = L.psim + (size_t)b * L.pcap;
  const int kt = wave >> 2, qsub = wave & 3;   // this wave's key half and query quarter in the profile phase
  const int G = (F + NK - 1) / NK;
  const int32_t *goff = L.goff + (size_t)b * L.gcap;
  const int items = F > 0 ? goff[G] : 0;
  int cur = -1;   // the group whose keys are in the shared arrays
  for (int it = bx; it < items; it += kRefineBlocks) {   // uniform over the workgroup
    __syncthreads();   // the previous item is done with the shared arrays
    if (tid == 0) {   // the group g with goff[g] <= it < goff[g + 1]
      int lo = 0, hi = G;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (goff[mid] <= it) lo = mid;
        else hi = mid;
      }
      item_g = lo;
      item_c0 = (it - goff[lo]) * CAP;
    }
    __syncthreads();
    const int g = item_g, c0 = item_c0;
    if (g != cur) {   // load the group's keys (uniform)
      cur = g;
      const int f0 = g * NK, nk = min(NK, F - f0);
      if (tid < NK) {
        kpos[tid] = -1;
        koff[tid] = 0;
        if (tid < nk) {
          const size_t q = (size_t)b * L.cap + f0 + tid;
          kpos[tid] = L.fkey[q];
          koff[tid] = L.foff[q];
        }
      }
      __syncthreads();
      if (tid == 0) {
        int acc = 0;
        for (int k = 0; k < NK; ++k) {
          kbase[k] = acc;
          acc += k < nk ? L.fn[(size_t)b * L.cap + f0 + k] : 0;
        }
        kbase[NK] = acc;
      }
      for (int x = tid; x < NK * kHeadDim; x += NW * 64) {   // the keys' rows (zero for empty slots)
        const int k = x / kHeadDim, c = x % kHeadDim;
        sK[k * SKB + c] = kpos[k] >= 0 ? K[((size_t)b * T + kpos[k]) * kHeadDim + c] : (E)0.0f;
      }
      __syncthreads();
    }
    const int total = kbase[NK];
    {
      const int cn = min(CAP, total - c0);
      __syncthreads();   // the previous chunk is done with cr / ck / khalf
      if (tid == 0) khalf = 0;
      __syncthreads();
      for (int c = tid; c < CAP; c += NW * 64) {
        int lo = -1, r = 0;
        if (c < cn) {
          const int gi = c0 + c;
          int lo2 = 0, hi = NK;   // the key k with kbase[k] <= gi < kbase[k + 1]
          while (hi - lo2 > 1) {
            const int mid = (lo2 + hi) >> 1;
            if (kbase[mid] <= gi) lo2 = mid;
            else hi = mid;
          }
          lo = lo2;
          r = pool[koff[lo] + gi - kbase[lo]];
          atomicOr(&khalf, 1 << (lo >> 5));   // which 32-key halves this chunk's candidates belong to
        }
        ck[c] = lo;
        cr[c] = r;
      }
      __syncthreads();
      const int need = khalf;
      double acc[CPW / 2];
#pragma unroll
      for (int u = 0; u < CPW / 2; ++u) acc[u] = 0.0;
      const int cw0 = wave * CPW;   // this wave's candidates cw0 + 2u + h
      const int qo = 4 * col;        // half-wave lane col covers queries i0 + 4 col .. + 3
      const bool prof = (need >> kt) & 1;   // this wave forms profiles in this chunk
      // Loads are unconditional so that the compiler can count them exactly
      // across the tile loop (a load under a branch may not have been issued,
      // which forces a full drain at the next use): an empty candidate slot
      // holds anchor 0 and is skipped when used; query rows past n are
      // clamped, and their profiles are zeroed below.
      auto load_w = [&](int i0, int u) -> f32x4 {
        const int c = cw0 + 2 * u + h;
        return *reinterpret_cast<const f32x4 *>(Uab + (size_t)cr[c] * np_ + i0 + qo);
      };
      // bf16 inputs: the loads run one query tile ahead.  The query fragments
      // of tile i0 + 128 are issued as soon as the MFMAs of tile i0 have read
      // theirs, and each anchor-profile value of tile i0 + 128 as soon as its
      // tile-i0 value is used; the tile barriers wait for LDS only.  Vector
      // loads complete in issue order, so the profile phase waits for its
      // query fragments alone while the anchor values stay in flight.
      // fp32 inputs: one tile at a time.
      bf16x8 qa[BF ? 8 : 1];
      auto load_q = [&](int i0) {
        if constexpr (BF) {
          const int iq = i0 + 32 * qsub + col;   // this lane's query row of the MFMA A operand
          const bf16 *qrow = reinterpret_cast<const bf16 *>(Qb) + (size_t)(iq < n ? iq : n - 1) * kHeadDim + 8 * h;
#pragma unroll
          for (int ks = 0; ks < 8; ++ks) qa[ks] = *reinterpret_cast<const bf16x8 *>(qrow + ks * 16);
        }
      };
      auto tile_barrier = [&]() {
        if constexpr (BF) lds_only_barrier();
        else __syncthreads();
      };
      f32x4 w[CPW / 2];
      if constexpr (BF) {
        load_q(0);
        // the same issue order as at the end of each tile (query fragments,
        // then anchor values), so that the counts agree at the loop head
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < CPW / 2; ++u) w[u] = load_w(0, u);
      }
      for (int i0 = 0; i0 < n; i0 += QT) {
        const int nxt = i0 + QT < n ? i0 + QT : i0;   // the last tile reloads itself
        if constexpr (!BF) {
#pragma unroll
          for (int u = 0; u < CPW / 2; ++u) w[u] = load_w(i0, u);
        }
        // ---- the 64 keys' profiles on queries [i0, i0 + 128) (bf16: always, so
        // that no load or MFMA of the tile loop sits under a branch)
        if (BF || prof) {
          double l[BF ? 1 : 16];
          f32x16 lsum;
          if constexpr (BF) {
            const bf16 *krow = reinterpret_cast<const bf16 *>(sK) + (kt * 32 + col) * SKB + 8 * h;
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
              const bf16x8 bk = *reinterpret_cast<const bf16x8 *>(krow + ks * 16);
              const f32x16 part = Mfma<bf16>::mma(qa[ks], bk, zero16());
              if (ks == 0) lsum = part;
              else {
#pragma unroll
                for (int v = 0; v < 16; ++v) lsum[v] += part[v];
              }
            }
          } else {
#pragma unroll
            for (int v = 0; v < 16; ++v) l[v] = 0.0;
            const float *krow = reinterpret_cast<const float *>(sK) + (kt * 32 + col) * SKB;
            for (int k = 0; k < kHeadDim; k += 4) {
              const f32x4 kv = *reinterpret_cast<const f32x4 *>(krow + k);
#pragma unroll
              for (int v = 0; v < 16; ++v) {
                const int qi = i0 + 32 * qsub + acc_row(v, lane);
                if (qi < n) {
                  const f32x4 qv = *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(Qb) +
                                                                   (size_t)qi * kHeadDim + k);
#pragma unroll
                  for (int e = 0; e < 4; ++e) l[v] = fma((double)qv[e], (double)kv[e], l[v]);
                }
              }
            }
          }
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int qi = 32 * qsub + acc_row(v, lane);
            float ev = 0.0f;
            if (i0 + qi < n) {
              if constexpr (BF) ev = __builtin_amdgcn_exp2f(fmaf(lsum[v], c2, -zs2));
              else ev = (float)exp(s * l[v] - zm);
            }
            eS[(kt * 32 + col) * SE + qi] = ev;
          }
        }
        if constexpr (BF) load_q(nxt);   // the MFMAs above have read qa
        tile_barrier();   // the tile's profiles are complete
        // ---- CPW candidates per wave: half-wave h takes candidate cw0 + 2u + h
        // Branch-free: an empty slot reads key 0's profile and adds an exact zero.
#pragma unroll
        for (int u = 0; u < CPW / 2; ++u) {
          const int k = ck[cw0 + 2 * u + h];
          const f32x4 e4 = *reinterpret_cast<const f32x4 *>(&eS[(k >= 0 ? k : 0) * SE + qo]);
          float p4 = e4[0] * w[u][0];   // four non-negative products in fp32 (within gamma_4), then float64
#pragma unroll
          for (int e = 1; e < 4; ++e) p4 = fmaf(e4[e], w[u][e], p4);
          acc[u] += k >= 0 ? (double)p4 : 0.0;
          if constexpr (BF) w[u] = load_w(nxt, u);
        }
        tile_barrier();   // reads of the tile done before the next one overwrites it
      }
      // ---- reduce each candidate's partial sums over its half-wave
#pragma unroll
      for (int u = 0; u < CPW / 2; ++u) {
        double d = acc[u];
#pragma unroll
        for (int m = 16; m >= 1; m >>= 1) d += __shfl_xor(d, m, 64);
        const int c = cw0 + 2 * u + h;
        if (col == 0 && c < cn) {
          const int k = ck[c];
          psim[koff[k] + c0 + c - kbase[k]] = d / anorm[(size_t)b * tp + cr[c]];
        }
      }
    }
  }
}

// Pass C work items: each group of 64 queued keys (in queue order) has
// ceil(candidates / cap_c) chunks; goff[g] is the first item of group g (an
// exclusive prefix) and goff[G] the pair's item count.  One workgroup per
// pair, 256 groups per scan step.
__global__ void __launch_bounds__(256) k_refine_plan(AssignLists L, int cap_c) {
  __shared__ int32_t sc[256];
  __shared__ int32_t carry;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int F = L.fcnt[b], G = (F + 63) / 64;
  int32_t *goff = L.goff + (size_t)b * L.gcap;
  const int32_t *fn = L.fn + (size_t)b * L.cap;
  if (tid == 0) carry = 0;
  for (int g0 = 0; g0 < G; g0 += 256) {   // uniform over the workgroup
    const int g = g0 + tid;
    int nit = 0;
    if (g < G) {
      int tot = 0;
      for (int k = g * 64; k < min(F, g * 64 + 64); ++k) tot += fn[k];
      nit = (tot + cap_c - 1) / cap_c;
    }
    __syncthreads();   // carry holds the previous steps' total
    sc[tid] = nit;
    __syncthreads();
    for (int d = 1; d < 256; d <<= 1) {   // inclusive scan
      const int v = tid >= d ? sc[tid - d] : 0;
      __syncthreads();
      sc[tid] += v;
      __syncthreads();
    }
    if (g < G) goff[g] = carry + sc[tid] - nit;
    __syncthreads();
    if (tid == 0) carry += sc[255];
  }
  __syncthreads();
  if (tid == 0) goff[G] = carry;
}

// Pass C decision, one thread per queued key, once every chunk of its
// candidates has its similarity: the best one (equal ones to the lower r)
// becomes the key's anchor for now, the candidates within the bound of it
// survive, compacted in place at the front of the key's pool segment, and a
// key with more than one survivor goes to pass D.
template <typename E>
__global__ void __launch_bounds__(256) k_assign_decide(const E *__restrict__ K, const float *__restrict__ zmerge,
                                                       const AssignPair *__restrict__ pn, int T, double s,
                                                       int32_t *__restrict__ kappa, AssignLists L) {
  constexpr bool BF = sizeof(E) == 2;
  const int b = blockIdx.y;
  const int F = L.fcnt[b];
  const AssignPair pp = pn[b];
  const double zm = (double)zmerge[b];
  int32_t *pool = L.pool + (size_t)b * L.pcap;
  const double *psim = L.psim + (size_t)b * L.pcap;
  for (int f = blockIdx.x * 256 + threadIdx.x; f < F; f += gridDim.x * 256) {
    const size_t q = (size_t)b * L.cap + f;
    const int j = L.fkey[q], o = L.foff[q], m = L.fn[q];
    if (m <= 0) continue;
    int best = 0;
    for (int c = 1; c < m; ++c)
      if (psim[o + c] > psim[o + best] || (psim[o + c] == psim[o + best] && pool[o + c] < pool[o + best]))
        best = c;
    double eta;
    if constexpr (BF) {
      const double kn = row_norm(K + ((size_t)b * T + j) * kHeadDim);
      const double g = gamma_m(kSliceTerms) * s * pp.qmax, Z = fabs(zm) * 1.4426950408889634;
      const double ek = g * kn + exp32_err(s * pp.qmax * kn * 1.4426950408889634 * 1.001, Z);
      const double ea = g * pp.amax + exp32_err(s * pp.qmax * pp.amax * 1.4426950408889634 * 1.001, Z);
      eta = (1.0 + ek) * (1.0 + ea) / (1.0 - ea) * (1.0 + gamma_m(4)) * (1.0 + 1e-12) - 1.0;
    } else {
      eta = 3.0 * kU32 + gamma_m(4) + 1e-12;
    }
    const double bs = psim[o + best];
    const double thc = bs * (1.0 - eta) / (1.0 + eta) - 1e-300;
    kappa[(size_t)b * T + j] = pool[o + best];
    // writes trail reads: this thread alone owns the key's pool segment
    int ns = 0;
    for (int c = 0; c < m; ++c)
      if (psim[o + c] >= thc) pool[o + ns++] = pool[o + c];
    if (ns > 1) push_d(L, b, j, o, ns);
  }
}

// ---------------------------------------------------------------- pass D
// Float64 decision for the remaining keys: logits as float64 sums of exact
// products, exp in float64, norms and dot products in float64; the largest
// similarity wins and equal ones go to the lower r.  A key's entries are the
// anchors that survived pass C.  k_exact_plan packs consecutive queued
// entries into items of up to 32 vectors (an entry is its key and its
// candidates); a fixed grid of kExactBlocks workgroups per pair takes items
// it = blockIdx.x, blockIdx.x + kExactBlocks, ...  An item's keys and
// candidate anchors share one sweep over the queries in tiles of 64, and an
// entry with more candidates than fit (all t anchors) continues in the next
// sweep.  An entry of a split key leaves its best (similarity, anchor) for
// k_exact_merge instead of deciding the key.
constexpr int kExactBlocks = 128;

// Pass D work items: greedy packing of consecutive entries into items of at
// most 32 vectors (an entry needs 1 + its candidates; a larger one forms an
// item of its own).  ditem = {count, first entry of each item, dcnt}.  One
// workgroup per pair; entry sizes staged in LDS, packed by one thread.
__global__ void __launch_bounds__(256) k_exact_plan(AssignLists L) {
  constexpr int W = 2048;
  __shared__ int32_t sdn[W];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int D = L.dcnt[b];
  const int32_t *dn = L.dn + (size_t)b * L.dcap;
  int32_t *items = L.ditem + (size_t)b * (L.dcap + 2);
  int nit = 0, nv = 0;   // thread 0 only
  for (int w0 = 0; w0 < D; w0 += W) {   // uniform over the workgroup
    const int nw = min(W, D - w0);
    __syncthreads();   // thread 0 is done with the previous window
    for (int x = tid; x < nw; x += 256) sdn[x] = dn[w0 + x];
    __syncthreads();
    if (tid == 0) {
      for (int x = 0; x < nw; ++x) {
        const int need = 1 + sdn[x];
        if (w0 + x == 0 || nv + need > 32) {
          items[1 + nit++] = w0 + x;
          nv = 0;
        }
        nv += need;
      }
    }
  }
  if (tid == 0) {
    items[0] = nit;
    items[1 + nit] = D;
  }
}

// A split key's decision from its entries' bests: the largest similarity,
// equal ones to the lower r (the same order as within an entry).  One thread
// per first entry of a split key.
__global__ void __launch_bounds__(256) k_exact_merge(int T, int32_t *__restrict__ kappa, AssignLists L) {
  const int b = blockIdx.y;
  const int D = L.dcnt[b];
  for (int di = blockIdx.x * 256 + threadIdx.x; di < D; di += gridDim.x * 256) {
    const size_t q = (size_t)b * L.dcap + di;
    if (L.dgrp[q] != di) continue;
    const int ne = L.dgn[q];
    double bs = L.dsim[q];
    int br = L.dr[q];
    for (int e = 1; e < ne; ++e) {
      const double sim = L.dsim[q + e];
      const int r = L.dr[q + e];
      if (sim > bs || (sim == bs && r < br)) {
        bs = sim;
        br = r;
      }
    }
    kappa[(size_t)b * T + L.dkey[q]] = br;
  }
}

template <typename E>
__global__ void __launch_bounds__(256) k_assign_exact(const E *__restrict__ Q, const E *__restrict__ K,
                                                      const int32_t *__restrict__ anchors,
                                                      const float *__restrict__ zmerge, int T, int t, int n, double s,
                                                      int32_t *__restrict__ kappa, AssignLists L) {
  constexpr int NV = 32, NQ = 64, SK = kHeadDim + 4;
  __shared__ __attribute__((aligned(16))) float sK[NV * SK];
  __shared__ __attribute__((aligned(16))) float sQ[NQ * SK];
  __shared__ double sE[NV * (NQ + 1)];
  __shared__ int32_t vpos[NV], vown[NV], vr[NV];
  __shared__ double vdot[NV], vnn[NV];
  // batch segments: first and one-past-last vector, continues, final
  __shared__ int32_t sg_v0[NV], sg_v1[NV], sg_cont[NV], sg_final[NV], sg_di[NV];
  __shared__ int32_t nv_s, nseg_s, di_s, ci_s, done_s;
  __shared__ double run_sim;
  __shared__ int32_t run_r;
  int bx, b;
  pair_block(kExactBlocks, gridDim.y, bx, b);
  const int tid = threadIdx.x;
  const int D = L.dcnt[b];
  const int32_t *S = anchors + (size_t)b * t;
  const double zm = (double)zmerge[b];
  const E *Qb = Q + (size_t)b * n * kHeadDim;
  auto n_cand = [&](int di) { return L.dn[(size_t)b * L.dcap + di]; };
  auto cand_at = [&](int di, int ci) {   // doff < 0: every anchor is a candidate
    const int off = L.doff[(size_t)b * L.dcap + di];
    return off < 0 ? ci : L.pool[(size_t)b * L.pcap + off + ci];
  };
  // register tile of the logit pass: vectors tv, tv + 16 and queries tq + 16 m, m = 0..3
  const int tv = tid >> 4, tq = tid & 15;
  // rows of 128 elements of E as 4 floats per thread-step (bf16: 4 values = 8 bytes)
  auto load4 = [](const E *p) -> f32x4 {
    if constexpr (sizeof(E) == 2) {
      const bf16x4 v = *reinterpret_cast<const bf16x4 *>(p);
      return f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
    } else {
      return *reinterpret_cast<const f32x4 *>(p);
    }
  };
  const int32_t *items = L.ditem + (size_t)b * (L.dcap + 2);
  const int nitems = D > 0 ? items[0] : 0;
  for (int it = bx; it < nitems; it += kExactBlocks) {   // uniform over the workgroup
    const int g0 = items[1 + it], g1 = items[2 + it];
    __syncthreads();   // every thread has left the previous item's loop
    if (tid == 0) {
      di_s = g0;
      ci_s = 0;
      done_s = 0;
    }
    __syncthreads();
    while (!done_s) {
      if (tid == 0) {   // build the next batch from keys di_s .. g1 - 1
        int nv = 0, ns = 0, di = di_s, ci = ci_s;
        while (di < g1 && nv + 2 <= NV) {
          const int nck = n_cand(di);
          sg_cont[ns] = ci > 0;
          sg_di[ns] = di;
          sg_v0[ns] = nv;
          vpos[nv] = L.dkey[(size_t)b * L.dcap + di];
          vown[nv] = -1;
          vr[nv] = -1;
          const int kv = nv++;
          while (nv < NV && ci < nck) {
            const int r = cand_at(di, ci++);
            vpos[nv] = S[r];
            vown[nv] = kv;
            vr[nv] = r;
            ++nv;
          }
          sg_v1[ns] = nv;
          sg_final[ns] = ci >= nck;
          ++ns;
          if (ci >= nck) {
            ++di;
            ci = 0;
          }
        }
        nv_s = nv;
        nseg_s = ns;
        di_s = di;
        ci_s = ci;
      }
      __syncthreads();
      const int nv = nv_s;
      for (int x = tid; x < NV * kHeadDim / 4; x += 256) {
        const int v = x / (kHeadDim / 4), k = 4 * (x % (kHeadDim / 4));
        const f32x4 w = v < nv ? load4(K + ((size_t)b * T + vpos[v]) * kHeadDim + k) : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<f32x4 *>(&sK[v * SK + k]) = w;
      }
      __syncthreads();   // sK and the batch's vectors are published
      // Running sums of vector rv: eight lanes per vector (queries 8 rq .. 8 rq + 7
      // of each tile), combined in a fixed tree and kept by the first lane.
      const int rv = tid >> 3, rq = tid & 7;
      const int vo = rv < nv ? vown[rv] : -1;
      double acc_d = 0.0, acc_n = 0.0;
      const int lane = tid & 63, wave = tid >> 6, lr = lane & 15, lk = lane >> 4;
      // the next query tile is loaded into registers while this one's products run
      constexpr int QCH = NQ * kHeadDim / 4 / 256;   // groups of 4 values per thread
      using Raw = std::conditional_t<sizeof(E) == 2, bf16x4, f32x4>;
      Raw qn[QCH];
      auto fetch_q = [&](int j0) {
#pragma unroll
        for (int c = 0; c < QCH; ++c) {
          const int x = tid + 256 * c, q = x / (kHeadDim / 4), k = 4 * (x % (kHeadDim / 4));
          qn[c] = j0 + q < n ? *reinterpret_cast<const Raw *>(Qb + (size_t)(j0 + q) * kHeadDim + k) : Raw{};
        }
      };
      fetch_q(0);
      for (int i0 = 0; i0 < n; i0 += NQ) {
        __syncthreads();   // every wave is done with the previous tile
#pragma unroll
        for (int c = 0; c < QCH; ++c) {
          const int x = tid + 256 * c, q = x / (kHeadDim / 4), k = 4 * (x % (kHeadDim / 4));
          f32x4 w;
#pragma unroll
          for (int u = 0; u < 4; ++u) w[u] = (float)qn[c][u];
          *reinterpret_cast<f32x4 *>(&sQ[q * SK + k]) = w;
        }
        if (i0 + NQ < n) fetch_q(i0 + NQ);
        __syncthreads();
        // logits on fp64 MFMA (16 x 16 x 4): wave w owns queries 16 w .. 16 w + 15
        // of the tile and both 16-vector halves; each lane supplies k = 16 g + 4 lk + u
        // to the four products of group g (bf16 / fp32 values are exact in fp64)
        f64x4 c0 = {0.0, 0.0, 0.0, 0.0}, c1 = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 2
        for (int g = 0; g < kHeadDim / 16; ++g) {
          const f32x4 a0 = *reinterpret_cast<const f32x4 *>(&sK[lr * SK + 16 * g + 4 * lk]);
          const f32x4 a1 = *reinterpret_cast<const f32x4 *>(&sK[(16 + lr) * SK + 16 * g + 4 * lk]);
          const f32x4 bq = *reinterpret_cast<const f32x4 *>(&sQ[(16 * wave + lr) * SK + 16 * g + 4 * lk]);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            c0 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a0[u], (double)bq[u], c0, 0, 0, 0);
            c1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)a1[u], (double)bq[u], c1, 0, 0, 0);
          }
        }
        // lane holds vectors 4 r + lk (and + 16) for query 16 w + lr
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int v = 4 * r + lk, q = 16 * wave + lr;
          const bool qv = i0 + q < n;
          sE[v * (NQ + 1) + q] = v < nv && qv ? exp(s * c0[r] - zm) : 0.0;
          sE[(v + 16) * (NQ + 1) + q] = v + 16 < nv && qv ? exp(s * c1[r] - zm) : 0.0;
        }
        __syncthreads();
        double d = 0.0, nn = 0.0;
        if (vo >= 0) {
#pragma unroll
          for (int x = 0; x < 8; ++x) {
            const int q = 8 * rq + x;
            const double ev = sE[rv * (NQ + 1) + q];
            d = fma(sE[vo * (NQ + 1) + q], ev, d);
            nn = fma(ev, ev, nn);
          }
        }
        d += __shfl_xor(d, 1, 64);
        nn += __shfl_xor(nn, 1, 64);
        d += __shfl_xor(d, 2, 64);
        nn += __shfl_xor(nn, 2, 64);
        d += __shfl_xor(d, 4, 64);
        nn += __shfl_xor(nn, 4, 64);
        acc_d += d;
        acc_n += nn;
      }
      if (rq == 0) {
        vdot[rv] = acc_d;
        vnn[rv] = acc_n;
      }
      __syncthreads();
      if (tid == 0) {
        for (int g = 0; g < nseg_s; ++g) {
          double bs = sg_cont[g] ? run_sim : -1.0;
          int br = sg_cont[g] ? run_r : 0x7FFFFFFF;
          for (int v = sg_v0[g] + 1; v < sg_v1[g]; ++v) {
            const double sim = vnn[v] > 0.0 ? vdot[v] / sqrt(vnn[v]) : 0.0;
            if (sim > bs || (sim == bs && vr[v] < br)) {
              bs = sim;
              br = vr[v];
            }
          }
          if (sg_final[g]) {
            const size_t q = (size_t)b * L.dcap + sg_di[g];
            if (L.dgrp[q] >= 0) {   // part of a split key: k_exact_merge decides
              L.dsim[q] = bs;
              L.dr[q] = br;
            } else if (br != 0x7FFFFFFF) {
              kappa[(size_t)b * T + vpos[sg_v0[g]]] = br;
            }
          } else {
            run_sim = bs;
            run_r = br;
          }
        }
        done_s = di_s >= g1;
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------- launchers
hipError_t launch_pair_norms(int dtype, const void *Q, const void *K, const int32_t *anchors, int P, int n, int T,
                             int t, void *pn, hipStream_t s) {
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_pair_norms<bf16>, dim3(P), dim3(256), 0, s, (const bf16 *)Q, (const bf16 *)K, anchors, n,
                       T, t, (AssignPair *)pn);
  else
    hipLaunchKernelGGL(k_pair_norms<float>, dim3(P), dim3(256), 0, s, (const float *)Q, (const float *)K, anchors,
                       n, T, t, (AssignPair *)pn);
  return hipGetLastError();
}

hipError_t launch_anchor_profiles(int dtype, const void *Q, const void *K, const int32_t *anchors,
                                  const float *zmerge, int P, int n, int T, int t, int64_t tp, int64_t np_,
                                  float scale, float *Ua, double *anorm, void *U, hipStream_t s) {
  if (dtype == ARCKV_BF16) {
    hipLaunchKernelGGL(k_prof_anchor_bf16, dim3((unsigned)((t + 127) / 128), P), dim3(256), 0, s, (const bf16 *)Q,
                       (const bf16 *)K, anchors, zmerge, n, T, t, tp, np_, (double)scale, Ua, anorm);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    hipLaunchKernelGGL(k_anchor_u<f16>, dim3((unsigned)(tp / 4), P), dim3(256), 0, s, (const float *)Ua,
                       (const double *)anorm, n, t, tp, np_, kProfScale, (f16 *)U);
  } else {
    hipLaunchKernelGGL(k_prof_anchor_f32, dim3((unsigned)t, P), dim3(256), 0, s, (const float *)Q, (const float *)K,
                       anchors, zmerge, n, T, t, tp, np_, (double)scale, Ua, anorm);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    hipLaunchKernelGGL(k_anchor_u<float>, dim3((unsigned)(tp / 4), P), dim3(256), 0, s, (const float *)Ua,
                       (const double *)anorm, n, t, tp, np_, 1.0f, (float *)U);
  }
  return hipGetLastError();
}

__global__ void k_fill_i32(int32_t *p, int64_t count, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < count) p[i] = v;
}

hipError_t launch_fill_i32(int32_t *p, int64_t count, int32_t v, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, p, count, v);
  return hipGetLastError();
}

// Pass A decision (clears the counters first).  MT anchor tiles of TR rows;
// Np = the partials' row stride (compacted key columns).
hipError_t launch_assign_finalize(int dtype, const void *K, const uint64_t *part1, const uint64_t *part2,
                                  const uint32_t *part3, int MT, int TR, int64_t Np, const int32_t *anchors,
                                  const float *phi, const float *zmerge, const void *pn, int P, int T, int t, int n,
                                  float scale, int32_t *kappa, const AssignLists &L, hipStream_t s) {
  hipError_t e = launch_fill_i32(L.fcnt, P, 0, s);
  if (e == hipSuccess) e = launch_fill_i32(L.dcnt, P, 0, s);
  if (e == hipSuccess) e = launch_fill_i32(L.pcnt, P, 0, s);
  if (e == hipSuccess) e = launch_fill_i32(L.stats, (int64_t)P * kAssignStats, 0, s);
  if (e != hipSuccess) return e;
  const dim3 gf((unsigned)((T + 255) / 256), P);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_assign_finalize<bf16>, gf, dim3(256), 0, s, part1, part2, part3, MT, Np, anchors,
                       (const bf16 *)K, phi, zmerge, (const AssignPair *)pn, T, t, n, TR, (double)scale, kappa, L);
  else
    hipLaunchKernelGGL(k_assign_finalize<float>, gf, dim3(256), 0, s, part1, part2, part3, MT, Np, anchors,
                       (const float *)K, phi, zmerge, (const AssignPair *)pn, T, t, n, TR, (double)scale, kappa, L);
  return hipGetLastError();
}

// Pass C (a grid of early exits where nothing is queued).
hipError_t launch_assign_refine(int dtype, const void *Q, const void *K, const float *zmerge, const void *pn,
                                const float *Ua, const double *anorm, int P, int T, int t, int n, int64_t tp,
                                int64_t np_, float scale, int32_t *kappa, const AssignLists &L, hipStream_t s) {
  if (T - t <= 0) return hipSuccess;
  const bool bf = dtype == ARCKV_BF16;
  hipLaunchKernelGGL(k_refine_plan, dim3(P), dim3(256), 0, s, L, 8 * kRefineCpw);
  const dim3 g(kRefineBlocks, P), gd(8, P);
  if (bf) {
    hipLaunchKernelGGL(k_assign_refine<bf16>, g, dim3(512), 0, s, (const bf16 *)Q, (const bf16 *)K, zmerge, Ua,
                       anorm, T, n, tp, np_, (double)scale, L);
    hipLaunchKernelGGL(k_assign_decide<bf16>, gd, dim3(256), 0, s, (const bf16 *)K, zmerge, (const AssignPair *)pn,
                       T, (double)scale, kappa, L);
  } else {
    hipLaunchKernelGGL(k_assign_refine<float>, g, dim3(512), 0, s, (const float *)Q, (const float *)K, zmerge, Ua,
                       anorm, T, n, tp, np_, (double)scale, L);
    hipLaunchKernelGGL(k_assign_decide<float>, gd, dim3(256), 0, s, (const float *)K, zmerge,
                       (const AssignPair *)pn, T, (double)scale, kappa, L);
  }
  return hipGetLastError();
}

// Pass D.
hipError_t launch_assign_exact(int dtype, const void *Q, const void *K, const int32_t *anchors, const float *zmerge,
                               int P, int T, int t, int n, float scale, int32_t *kappa, const AssignLists &L,
                               hipStream_t s) {
  hipLaunchKernelGGL(k_exact_plan, dim3(P), dim3(256), 0, s, L);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_assign_exact<bf16>, dim3(kExactBlocks, P), dim3(256), 0, s, (const bf16 *)Q,
                       (const bf16 *)K, anchors, zmerge, T, t, n, (double)scale, kappa, L);
  else
    hipLaunchKernelGGL(k_assign_exact<float>, dim3(kExactBlocks, P), dim3(256), 0, s, (const float *)Q,
                       (const float *)K, anchors, zmerge, T, t, n, (double)scale, kappa, L);
  hipLaunchKernelGGL(k_exact_merge, dim3(8, P), dim3(256), 0, s, T, kappa, L);
  return hipGetLastError();
}

}  // namespace arckv
