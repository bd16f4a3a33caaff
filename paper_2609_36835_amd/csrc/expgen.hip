// Exponentiated score matrices, written transposed (query index contiguous)
// so that the later contractions over queries read both operands K-contiguous.
//
// MODE_PROFILE (Section 3.4, eq. response_profile / mass_centroid):
//   E^T[j][i] = exp(s q_i.k_j - z_merge) for every cached key j that is not an
//   anchor, phi_j = (1/n) sum_i E[i][j] for every key.  Non-anchor key j writes
//   row j - #{anchors < j} of the compacted E^T, so the assignment contraction
//   runs over the T - t non-anchor keys only.  For bf16 inputs E^T is stored in
//   fp16 scaled by 2^15 (kProfScale; a power of two, so the scaling is exact and
//   the fp16 normal range covers E >= 2^-29); for fp32 inputs in fp32.  The
//   anchors' own profiles come from the precise anchor-profile pass.
// MODE_PHIC (Appendix A.9):
//   L^T[r][i]   = s q_i.c_r            (logits of the compact keys, fp32)
//   Phi^T[r][i] = exp(L - z_i)         (z_i: full-cache row maxima)
//
// A workgroup owns 128 output rows (keys or compact keys) whose fragments stay
// in registers, and sweeps all query tiles through LDS.  Padding rows/columns
// of the workspace are written as zeros.
#include <type_traits>

#include "common.hpp"

namespace arckv {
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;

enum { MODE_PROFILE = 0, MODE_PHIC = 1 };

template <typename T, int MODE>
__global__ void __launch_bounds__(256) k_expgen(const T *__restrict__ Q, const void *__restrict__ Bsrc,
                                                int64_t b_pair_stride, int64_t b_plane_stride, int b_rows,
                                                const float *__restrict__ shift, void *__restrict__ out,
                                                int64_t out_pair_stride, int64_t out_plane_stride,
                                                float *__restrict__ aux, int64_t aux_pair_stride, int n,
                                                int n_pad, float scale, const int32_t *__restrict__ anchors, int t,
                                                void *__restrict__ uout, float *__restrict__ ssq, int64_t tp,
                                                const float *__restrict__ mvec, double *__restrict__ hout) {
  using M = Mfma<T>;
  constexpr int KPL = M::KPL, KSTEP = M::KSTEP, NKS = kHeadDim / KSTEP;
  constexpr bool SPLIT_B = (MODE == MODE_PHIC) && sizeof(T) == 2;   // compact keys kept as bf16 hi + lo
  constexpr int NB = SPLIT_B ? 2 : 1;
  constexpr int EPC = 16 / sizeof(T);
  constexpr int SQ = kHeadDim + EPC;
  __shared__ __attribute__((aligned(16))) T sQ[64 * SQ];

  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int row = blockIdx.x * 128 + wave * 32 + col;   // key j or compact-key r
  const bool rvalid = row < b_rows;
  const T *Bp = reinterpret_cast<const T *>(Bsrc) + (size_t)b * b_pair_stride;
  typename M::frag bf[NB][NKS];
  #pragma unroll
  for (int p = 0; p < NB; ++p)
    #pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      bf[p][ks] = rvalid ? M::load(Bp + p * b_plane_stride + (size_t)row * kHeadDim + ks * KSTEP + KPL * h)
                         : M::zero();
  const T *Qb = Q + (size_t)b * n * kHeadDim;
  const float c2 = scale * 1.4426950408889634f;
  const float zshift = (MODE == MODE_PROFILE) ? shift[b] : 0.0f;
  float rowsum = 0.0f;
  double hsum = 0.0;   // PHIC: h_r = sum_i Phi[i][r] m_i (when hout is given)
  // PROFILE destination of this lane's key: >= 0 compacted E^T row, <= -2
  // anchor -(r + 2), -1 none (padding key)
  int dest = -1;
  if (MODE == MODE_PROFILE && rvalid) {
    const int32_t *S = anchors + (size_t)b * t;
    int lo = 0, hi = t;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (S[mid] < row) lo = mid + 1;
      else hi = mid;
    }
    dest = (lo < t && S[lo] == row) ? -(lo + 2) : row - lo;
  }
  // base pointer of staged row rr of this wave (MODE_PROFILE), or null
  auto row_dst = [&](int rr, int i0) -> T * {
    const int d = __shfl(dest, rr, 64);
    if (d < 0) return nullptr;   // padding key or anchor: nothing stored
    return reinterpret_cast<T *>(out) + (size_t)b * out_pair_stride + (size_t)d * n_pad + i0;
  };

  // Output tiles (this wave's 32 rows x 64 queries) are staged in LDS so that
  // global stores are whole 128/256-byte row segments.
  constexpr int SO = 64 + 4;                               // staging row (4-byte words)
  __shared__ float sOut[4][32 * SO];
  float *so = sOut[wave];
  // dst_base: row 0 of this wave at column i0; routed: rows go to row_dst()
  auto flush_f32 = [&](const float (&v)[2][16], float *dst_base, bool routed, int i0) {
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) so[col * SO + 32 * ms + acc_row(vv, lane)] = v[ms][vv];
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 8; ++pass) {             // 32 rows x 16 chunks of 16 B
      const int chunk = pass * 64 + lane, r = chunk / 16, c4 = (chunk % 16) * 4;
      const f32x4 w = {so[r * SO + c4], so[r * SO + c4 + 1], so[r * SO + c4 + 2], so[r * SO + c4 + 3]};
      float *dst = routed ? reinterpret_cast<float *>(row_dst(r, i0)) : dst_base + (size_t)r * n_pad;
      if (dst) *reinterpret_cast<f32x4 *>(dst + c4) = w;
    }
    __syncthreads();
  };
  auto flush_bf16 = [&](const float (&v)[2][16], int part, bf16 *dst_base, bool routed, int i0) {   // part: 0 value, 1 hi, 2 lo
    bf16 *sb = reinterpret_cast<bf16 *>(so);
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        bf16 hi, lo;
        split_bf16(v[ms][vv], hi, lo);
        sb[col * (2 * SO) + 32 * ms + acc_row(vv, lane)] = part == 2 ? lo : hi;
      }
    __syncthreads();
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {             // 32 rows x 8 chunks of 16 B
      const int chunk = pass * 64 + lane, r = chunk / 8, c8 = (chunk % 8) * 8;
      bf16 *dst = routed ? reinterpret_cast<bf16 *>(row_dst(r, i0)) : dst_base + (size_t)r * n_pad;
      if (dst) *reinterpret_cast<bf16x8 *>(dst + c8) = *reinterpret_cast<const bf16x8 *>(&sb[r * (2 * SO) + c8]);
    }
    __syncthreads();
  };
  const int row0 = blockIdx.x * 128 + wave * 32;          // first output row of this wave

  for (int i0 = 0; i0 < n_pad; i0 += 64) {
    for (int c = tid; c < 64 * (kHeadDim / EPC); c += 256) {
      int r = c / (kHeadDim / EPC), cc = (c % (kHeadDim / EPC)) * EPC;
      f32x4 v = {0.f, 0.f, 0.f, 0.f};
      if (i0 + r < n) v = *reinterpret_cast<const f32x4 *>(Qb + (size_t)(i0 + r) * kHeadDim + cc);
      *reinterpret_cast<f32x4 *>(&sQ[r * SQ + cc]) = v;
    }
    __syncthreads();
    float val[2][16], lg[2][16];
#pragma unroll
    for (int ms = 0; ms < 2; ++ms) {
      f32x16 acc = zero16();
      const T *arow = &sQ[(32 * ms + col) * SQ + KPL * h];
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        typename M::frag a = M::load(arow + ks * KSTEP);
#pragma unroll
        for (int p = 0; p < NB; ++p) acc = M::mma(a, bf[p][ks], acc);
      }
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        const int i = i0 + 32 * ms + acc_row(vv, lane);
        const bool ok = rvalid && i < n;
        if (MODE == MODE_PROFILE) {
          val[ms][vv] = ok ? exp2f(acc[vv] * c2 - zshift * 1.4426950408889634f) : 0.0f;
          rowsum += val[ms][vv];
          lg[ms][vv] = 0.0f;
        } else {
          lg[ms][vv] = ok ? acc[vv] * scale : 0.0f;
          val[ms][vv] = ok ? expf(lg[ms][vv] - (shift ? shift[(size_t)b * n + i] : 0.0f)) : 0.0f;
          if (hout && ok) hsum += (double)val[ms][vv] * (double)mvec[(size_t)b * n + i];
        }
      }
    }
    __syncthreads();   // sQ is refilled at the next i0; sOut is free
    char *ob = reinterpret_cast<char *>(out);
    constexpr bool routed = MODE == MODE_PROFILE;
    if constexpr (sizeof(T) == 4) {
      flush_f32(val, reinterpret_cast<float *>(ob) + (size_t)b * out_pair_stride + (size_t)row0 * n_pad + i0, routed,
                i0);
    } else if constexpr (MODE == MODE_PROFILE) {
      flush_bf16(val, 0, nullptr, true, i0);
    } else {
      bf16 *o = reinterpret_cast<bf16 *>(ob) + (size_t)b * out_pair_stride + (size_t)row0 * n_pad + i0;
      flush_bf16(val, 1, o, false, i0);
      flush_bf16(val, 2, o + out_plane_stride, false, i0);
    }
    if (MODE == MODE_PHIC) flush_f32(lg, aux + (size_t)b * aux_pair_stride + (size_t)row0 * n_pad + i0, false, i0);
  }
  if (MODE == MODE_PROFILE) {
    rowsum += __shfl_xor(rowsum, 32, 64);
    if (h == 0 && rvalid) aux[(size_t)b * aux_pair_stride + row] = rowsum / (float)n;
  }
  if (MODE == MODE_PHIC && hout) {
    hsum += __shfl_xor(hsum, 32, 64);
    if (h == 0) hout[(size_t)b * tp + row] = hsum;
  }
}

// ---------------------------------------------------------------- bf16 path
// Same products as k_expgen, for bf16 inputs, with the query tiles double-
// buffered: tile i+1 (64 queries x 256 B) goes global -> LDS with the
// direct-to-LDS loads while tile i's products are formed (rows stored unpadded,
// 16-byte chunks XOR-swizzled by (row & 15) so the fragment reads of 16
// consecutive rows hit distinct banks).  One barrier per query tile hands the
// next Q stage over, after the products and before the stores.  Each wave
// stages its 32 x 64 output block in a private LDS area, so no workgroup
// barrier guards the staging.
typedef __attribute__((address_space(3))) void eg_lds_t;

// LDS of k_expgen_bf16: two Q stages of 64 rows (16 KB each), four wave-private
// staging areas of 32 rows (bf16 rows of 64 + 8 in profile mode, fp32 rows of
// 64 + 4 in phic mode), and in phic mode z_i and m_i of both Q stages.
template <int MODE>
constexpr int eg_stage_bytes() {
  return MODE == MODE_PHIC ? 32 * (64 + 4) * 4 : 32 * (64 + 8) * 2;
}
template <int MODE>
constexpr size_t eg_lds_bytes() {
  return 2 * 64 * kHeadDim * 2 + 4 * eg_stage_bytes<MODE>() + (MODE == MODE_PHIC ? 2 * 2 * 64 * 4 : 0);
}

template <int MODE>
__global__ void __launch_bounds__(256, 2) k_expgen_bf16(const bf16 *__restrict__ Q, const bf16 *__restrict__ Bsrc,
                                                     int64_t b_pair_stride, int64_t b_plane_stride, int b_rows,
                                                     const float *__restrict__ shift, bf16 *__restrict__ out,
                                                     int64_t out_pair_stride, int64_t out_plane_stride,
                                                     float *__restrict__ aux, int64_t aux_pair_stride, int n,
                                                     int n_pad, float scale, const int32_t *__restrict__ anchors,
                                                     int t, bf16 *__restrict__ uout, float *__restrict__ ssq,
                                                     int64_t tp, const float *__restrict__ mvec,
                                                     double *__restrict__ hout) {
  constexpr int NB = MODE == MODE_PHIC ? 2 : 1;           // compact keys kept as bf16 hi + lo
  constexpr int NKS = kHeadDim / 16;
  constexpr int QB = 64 * kHeadDim * 2;                   // one Q stage (16 KB)
  // staging: bf16 rows of 64 + 8 (profile) or fp32 rows of 64 + 4 (phic)
  constexpr int SO_F = 64 + 4, SO_H = 64 + 8;
  constexpr int STG = eg_stage_bytes<MODE>();
  // Dynamic LDS (eg_lds_bytes<MODE>): two Q stages, four wave-private output
  // staging areas, and in phic mode z_i and m_i of both Q stages.  A dynamic
  // array also keeps the compiler from waiting for every direct-to-LDS load
  // in flight before each LDS read, which would serialise the prefetch.
  extern __shared__ __attribute__((aligned(1024))) char eg_smem[];
  char *sQ = eg_smem, *sOut = eg_smem + 2 * QB;
  float *sZ = reinterpret_cast<float *>(sOut + 4 * STG), *sM = sZ + 128;   // [stage][64]

  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, col = lane & 31;
  const int row = blockIdx.x * 128 + wave * 32 + col;   // key j or compact-key r
  const bool rvalid = row < b_rows;
  const bf16 *Bp = Bsrc + (size_t)b * b_pair_stride;
  bf16x8 bf[NB][NKS];
#pragma unroll
  for (int p = 0; p < NB; ++p)
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks)
      bf[p][ks] = rvalid ? *reinterpret_cast<const bf16x8 *>(Bp + p * b_plane_stride + (size_t)row * kHeadDim +
                                                              ks * 16 + 8 * h)
                         : Mfma<bf16>::zero();
  const bf16 *Qb = Q + (size_t)b * n * kHeadDim;
  const float c2 = scale * 1.4426950408889634f;
  // profile: E' = 2^15 E, folded into the exponent (exact)
  const float zs2 = MODE == MODE_PROFILE ? shift[b] * 1.4426950408889634f - (float)kProfLog2Scale : 0.0f;
  float rowsum = 0.0f;
  double hsum = 0.0;   // PHIC: h_r = sum_i Phi[i][r] m_i (when hout is given)
  // profile: the compacted E^T row of a non-anchor key.  Padding keys j >= T
  // write their (zero) rows to row j - t, in [T - t, Tp - t), and anchor r to
  // row Tp - t + r, in [Tp - t, Tp): past the rows of the real keys, so those
  // rows only feed assignment columns that are never read, and every lane
  // stores unconditionally with a fixed per-tile store count.
  int dest = row - t;
  if (MODE == MODE_PROFILE && rvalid) {
    const int32_t *S = anchors + (size_t)b * t;
    int lo = 0, hi = t;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (S[mid] < row) lo = mid + 1;
      else hi = mid;
    }
    dest = (lo < t && S[lo] == row) ? (int)(out_pair_stride / n_pad) - t + lo : row - lo;
  }
  // Q stage loads: run 4 wave + u covers tile rows 4 (4 wave + u) .. + 3; lane l
  // fills physical chunk l % 16 of its row with logical chunk (l % 16) ^ row.
  // Rows past n read row n - 1 (their outputs are masked).
  auto issue_q = [&](int i0, int st) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int r = 4 * (4 * wave + u) + lane / 16;
      const int qrow = min(i0 + r, n - 1);
      const bf16 *src = Qb + (size_t)qrow * kHeadDim + 8 * ((lane % 16) ^ (r & 15));
      __builtin_amdgcn_global_load_lds((const void *)src, (eg_lds_t *)(sQ + st * QB + (4 * wave + u) * 1024), 16,
                                       0, 0);
    }
    // phic: the stage's z_i (and m_i) ride along, so the loop body issues no
    // vector-memory loads of its own
    if (MODE == MODE_PHIC && wave == 0) {
      const size_t iq = (size_t)b * n + min(i0 + lane, n - 1);
      if (shift) __builtin_amdgcn_global_load_lds((const void *)(shift + iq), (eg_lds_t *)(sZ + 64 * st), 4, 0, 0);
      if (hout) __builtin_amdgcn_global_load_lds((const void *)(mvec + iq), (eg_lds_t *)(sM + 64 * st), 4, 0, 0);
    }
  };
  char *so = sOut + wave * STG;
  auto wave_fence = [] { asm volatile("" ::: "memory"); };
  const int row0 = blockIdx.x * 128 + wave * 32;
  auto row_dst = [&](int rr, int i0) -> bf16 * {
    const int d = __shfl(dest, rr, 64);
    return out + (size_t)b * out_pair_stride + (size_t)d * n_pad + i0;
  };
  // stage v (rows = this wave's 32 outputs, 64 query columns) and copy out
  auto flush_bf16 = [&](const float (&v)[2][16], int part, bf16 *dst_base, bool routed, int i0) {
    bf16 *sb = reinterpret_cast<bf16 *>(so);
    wave_fence();
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        bf16 hi, lo;
        split_bf16(v[ms][vv], hi, lo);
        sb[col * SO_H + 32 * ms + acc_row(vv, lane)] = part == 2 ? lo : hi;
      }
    wave_fence();
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {             // 32 rows x 8 chunks of 16 B
      const int chunk = pass * 64 + lane, r = chunk / 8, c8 = (chunk % 8) * 8;
      bf16 *dst = routed ? row_dst(r, i0) : dst_base + (size_t)r * n_pad;
      *reinterpret_cast<bf16x8 *>(dst + c8) = *reinterpret_cast<const bf16x8 *>(&sb[r * SO_H + c8]);
    }
    wave_fence();
  };
  auto flush_f32 = [&](const float (&v)[2][16], float *dst_base) {
    float *sf = reinterpret_cast<float *>(so);
    wave_fence();
#pragma unroll
    for (int ms = 0; ms < 2; ++ms)
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) sf[col * SO_F + 32 * ms + acc_row(vv, lane)] = v[ms][vv];
    wave_fence();
#pragma unroll
    for (int pass = 0; pass < 8; ++pass) {             // 32 rows x 16 chunks of 16 B
      const int chunk = pass * 64 + lane, r = chunk / 16, c4 = (chunk % 16) * 4;
      const f32x4 w = {sf[r * SO_F + c4], sf[r * SO_F + c4 + 1], sf[r * SO_F + c4 + 2], sf[r * SO_F + c4 + 3]};
      *reinterpret_cast<f32x4 *>(dst_base + (size_t)r * n_pad + c4) = w;
    }
    wave_fence();
  };

  const int ntile = n_pad / 64;
  // without z (logits only) the shift is zero; the stages stay zero-filled
  if (MODE == MODE_PHIC && !shift && tid < 128) sZ[tid] = 0.0f;
  // profile: destination row of each of this lane's four store passes (row
  // 8 pass + lane / 8 of the wave), fixed over the query sweep
  bf16 *prow[4];
  if constexpr (MODE == MODE_PROFILE) {
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) prow[pass] = row_dst(8 * pass + lane / 8, 0);
  }
  // wave-uniform: this wave's 32 rows are all real keys
  const bool rows_full = row0 + 32 <= b_rows;
  issue_q(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  for (int it = 0; it < ntile; ++it) {
    const int i0 = it * 64, st = it & 1;
    if (it + 1 < ntile) issue_q(i0 + 64, st ^ 1);
    const char *sq = sQ + st * QB;
    if constexpr (MODE == MODE_PROFILE) {
      // E' = 2^(acc c2 - zs2) by the hardware exponential (results below
      // 2^-126 flush to zero); masks only on ragged tiles; each pair of rows
      // rounded to fp16 (nearest even) once
      uint32_t pk[2][8];
      auto products = [&](auto full_c) {
        constexpr bool FULL = decltype(full_c)::value;
#pragma unroll
        for (int ms = 0; ms < 2; ++ms) {
          f32x16 acc = zero16();
          const int r = 32 * ms + col;
#pragma unroll
          for (int ks = 0; ks < NKS; ++ks) {
            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(sq + r * 256 + 16 * ((2 * ks + h) ^ (r & 15)));
            acc = Mfma<bf16>::mma(a, bf[0][ks], acc);
          }
#pragma unroll
          for (int u = 0; u < 8; ++u) {
            float e0 = __builtin_amdgcn_exp2f(fmaf(acc[2 * u], c2, -zs2));
            float e1 = __builtin_amdgcn_exp2f(fmaf(acc[2 * u + 1], c2, -zs2));
            if constexpr (!FULL) {
              const int i = i0 + 32 * ms + acc_row(2 * u, lane);   // rows i and i + 1
              e0 = rvalid && i < n ? e0 : 0.0f;
              e1 = rvalid && i + 1 < n ? e1 : 0.0f;
            }
            rowsum += e0;
            rowsum += e1;
            const f16x2 h2 = {(f16)e0, (f16)e1};
            pk[ms][u] = __builtin_bit_cast(uint32_t, h2);
          }
        }
      };
      // wave-uniform: a whole tile of real keys and queries needs no masks
      if (__builtin_amdgcn_readfirstlane((int)(rows_full && i0 + 64 <= n)))
        products(std::true_type{});
      else
        products(std::false_type{});
      bf16 *sb = reinterpret_cast<bf16 *>(so);
      wave_fence();
#pragma unroll
      for (int ms = 0; ms < 2; ++ms)
#pragma unroll
        for (int u = 0; u < 8; ++u)
          *reinterpret_cast<uint32_t *>(&sb[col * SO_H + 32 * ms + acc_row(2 * u, lane)]) = pk[ms][u];
      wave_fence();
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {             // 32 rows x 8 chunks of 16 B
        const int chunk = pass * 64 + lane, r = chunk / 8, c8 = (chunk % 8) * 8;
        // E^T is written once and read back much later: streaming stores
        __builtin_nontemporal_store(*reinterpret_cast<const u32x4 *>(&sb[r * SO_H + c8]),
                                    reinterpret_cast<u32x4 *>(prow[pass] + i0 + c8));
      }
      wave_fence();
    } else {
    float val[2][16], lg[2][16];
#pragma unroll
    for (int ms = 0; ms < 2; ++ms) {
      f32x16 acc = zero16();
      const int r = 32 * ms + col;
#pragma unroll
      for (int ks = 0; ks < NKS; ++ks) {
        const bf16x8 a = *reinterpret_cast<const bf16x8 *>(sq + r * 256 + 16 * ((2 * ks + h) ^ (r & 15)));
#pragma unroll
        for (int p = 0; p < NB; ++p) acc = Mfma<bf16>::mma(a, bf[p][ks], acc);
      }
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        const int i = i0 + 32 * ms + acc_row(vv, lane);
        const bool ok = rvalid && i < n;
        // evaluated on every lane (masked lanes see finite inputs), then
        // selected, so the exponential stays free of branches
        lg[ms][vv] = ok ? acc[vv] * scale : 0.0f;
        const float e = expf(lg[ms][vv] - sZ[64 * st + 32 * ms + acc_row(vv, lane)]);
        val[ms][vv] = ok ? e : 0.0f;
      }
    }
    if (hout) {   // masked entries of val are zero
#pragma unroll
      for (int ms = 0; ms < 2; ++ms)
#pragma unroll
        for (int vv = 0; vv < 16; ++vv)
          hsum += (double)val[ms][vv] * (double)sM[64 * st + 32 * ms + acc_row(vv, lane)];
    }
    bf16 *o = out + (size_t)b * out_pair_stride + (size_t)row0 * n_pad + i0;
    flush_bf16(val, 1, o, false, i0);
    flush_bf16(val, 2, o + out_plane_stride, false, i0);
    flush_f32(lg, aux + (size_t)b * aux_pair_stride + (size_t)row0 * n_pad + i0);
    }
    // The next Q stage has landed: it was issued before this tile's stores (4
    // per lane in profile mode, 4 + 4 + 8 in phic mode, all unconditional) and
    // the vector-memory counter retires in issue order, so waiting until only
    // the stores may be outstanding suffices.  After the barrier every wave's
    // share has landed and every wave is done reading stage st.
    if constexpr (MODE == MODE_PROFILE) __builtin_amdgcn_s_waitcnt(4 | (7 << 4) | (15 << 8));        // vmcnt(4)
    else __builtin_amdgcn_s_waitcnt(0 | (1 << 14) | (7 << 4) | (15 << 8));                            // vmcnt(16)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  }
  if (MODE == MODE_PROFILE) {
    rowsum += __shfl_xor(rowsum, 32, 64);
    if (h == 0 && rvalid) aux[(size_t)b * aux_pair_stride + row] = rowsum * (kProfInvScale / (float)n);
  }
  if (MODE == MODE_PHIC && hout) {
    hsum += __shfl_xor(hsum, 32, 64);
    if (h == 0) hout[(size_t)b * tp + row] = hsum;
  }
}

template <int MODE>
static hipError_t eg_set_lds() {
  return hipFuncSetAttribute((const void *)k_expgen_bf16<MODE>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)eg_lds_bytes<MODE>());
}

// Compacted E^T [B][Tp][np] of the non-anchor keys (fp16 scaled by 2^15 for
// bf16 inputs, fp32 for fp32 inputs) and phi [B][T] of every key.
hipError_t launch_profiles(int dtype, const void *Q, const void *K, const float *zmerge, const int32_t *anchors,
                           int t, void *Et, float *phi, int B, int T, int n, int64_t Tp, int64_t np_, float scale,
                           hipStream_t s) {
  dim3 grid(Tp / 128, B);
  if (dtype == ARCKV_BF16) {
    hipError_t e = eg_set_lds<MODE_PROFILE>();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_expgen_bf16<MODE_PROFILE>), grid, dim3(256), eg_lds_bytes<MODE_PROFILE>(), s, (const bf16 *)Q, (const bf16 *)K,
                       (int64_t)T * kHeadDim, (int64_t)0, T, zmerge, (bf16 *)Et, Tp * np_, (int64_t)0, phi,
                       (int64_t)T, n, (int)np_, scale, anchors, t, (bf16 *)nullptr, (float *)nullptr, (int64_t)0,
                       (const float *)nullptr, (double *)nullptr);
  } else
    hipLaunchKernelGGL((k_expgen<float, MODE_PROFILE>), grid, dim3(256), 0, s, (const float *)Q, K,
                       (int64_t)T * kHeadDim, (int64_t)0, T, zmerge, Et, Tp * np_, (int64_t)0, phi, (int64_t)T,
                       n, (int)np_, scale, anchors, t, (void *)nullptr, (float *)nullptr, (int64_t)0,
                       (const float *)nullptr, (double *)nullptr);
  return hipGetLastError();
}

// Ckp: padded compact keys [B][planes][tp][128]; Phi^T [B][planes][tp][np]; L^T [B][tp][np].
// With m and h given, also h_r = sum_i Phi[i][r] m_i (float64) [B][tp].
hipError_t launch_phic(int dtype, const void *Q, const void *Ckp, const float *z, void *PhiT, float *LT,
                       const float *m, double *h, int B, int t, int n, int64_t tp, int64_t np_, float scale,
                       hipStream_t s) {
  if (h && !m) return hipErrorInvalidValue;   // h = Phi_C^T m needs m
  dim3 grid(tp / 128, B);
  if (dtype == ARCKV_BF16) {
    hipError_t e = eg_set_lds<MODE_PHIC>();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_expgen_bf16<MODE_PHIC>), grid, dim3(256), eg_lds_bytes<MODE_PHIC>(), s, (const bf16 *)Q, (const bf16 *)Ckp,
                       2 * tp * kHeadDim, tp * kHeadDim, t, z, (bf16 *)PhiT, 2 * tp * np_, tp * np_, LT, tp * np_,
                       n, (int)np_, scale, (const int32_t *)nullptr, 0, (bf16 *)nullptr, (float *)nullptr, tp, m, h);
  } else
    hipLaunchKernelGGL((k_expgen<float, MODE_PHIC>), grid, dim3(256), 0, s, (const float *)Q, Ckp,
                       tp * kHeadDim, (int64_t)0, t, z, PhiT, tp * np_, (int64_t)0, LT, tp * np_, n, (int)np_,
                       scale, (const int32_t *)nullptr, 0, (void *)nullptr, (float *)nullptr, tp, m, h);
  return hipGetLastError();
}

}  // namespace arckv
