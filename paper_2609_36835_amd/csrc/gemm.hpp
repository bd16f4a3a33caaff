// Batched "TN" contraction D[p][m][n] = sum_k A[p][m][k] * B[p][n][k] on MFMA,
// both operands K-contiguous (row-major [rows][K]).  Every contraction of the
// compaction path over the reference-query axis has this shape:
//   anchor assignment  U_S E^T      (bf16, or fp32 for fp32 inputs)
//   mass Gram          Phi_C^T Phi_C  (split bf16: hi*hi + hi*lo + lo*hi)
//   value Gram / rhs   P^T P, P^T Y   (split bf16)
//   refinement residuals          (fp32)
// Operands may carry two bf16 planes (hi, lo); the product then adds the
// three leading terms, giving ~16 significant bits per operand.
//
// Tiles: 128 x 128 per workgroup, 4 waves of 64 x 64 (2 x 2 MFMA 32x32 tiles),
// K staged through LDS in slabs of 32 with register prefetch of the next slab.
// Dimensions M, N, K must be multiples of the tile (callers pad workspace).
// Workgroups are remapped so each XCD receives a contiguous, M-grouped range
// of tiles (operand reuse in that XCD's L2).
#pragma once
#include "common.hpp"

namespace arckv {

struct GemmShape {
  int batch, M, N, K;                 // per-batch dims (multiples of 128 / 32)
  int64_t a_pair, a_plane, lda;       // element strides
  int64_t b_pair, b_plane, ldb;
  bool syrk;                          // only tiles with m-tile >= n-tile (lower triangle)
  int group_m;                        // M-tiles per group in the tile order
};

constexpr int kGBM = 128, kGBN = 128, kGBK = 32;

// Decode a logical tile id into (batch, mt, nt).
__device__ inline void gemm_tile(const GemmShape &g, int64_t tile, int &p, int &mt, int &nt) {
  const int MT = g.M / kGBM, NT = g.N / kGBN;
  if (g.syrk) {
    const int64_t per = (int64_t)MT * (MT + 1) / 2;
    p = (int)(tile / per);
    int64_t r = tile % per;
    // row-major lower triangle: idx = mt*(mt+1)/2 + nt
    int m = (int)((sqrt(8.0 * (double)r + 1.0) - 1.0) * 0.5);
    while ((int64_t)m * (m + 1) / 2 > r) --m;
    while ((int64_t)(m + 1) * (m + 2) / 2 <= r) ++m;
    mt = m;
    nt = (int)(r - (int64_t)m * (m + 1) / 2);
    return;
  }
  const int64_t per = (int64_t)MT * NT;
  p = (int)(tile / per);
  int64_t r = tile % per;
  const int gm = g.group_m;
  const int64_t per_group = (int64_t)gm * NT;
  const int grp = (int)(r / per_group);
  const int first_m = grp * gm;
  const int gsize = min(MT - first_m, gm);
  const int64_t rr = r % per_group;
  mt = first_m + (int)(rr % gsize);
  nt = (int)(rr / gsize);
}

__host__ inline int64_t gemm_tiles(const GemmShape &g) {
  const int64_t MT = g.M / kGBM, NT = g.N / kGBN;
  return (int64_t)g.batch * (g.syrk ? MT * (MT + 1) / 2 : MT * NT);
}

template <typename T, int NA, int NB, class Epi>
__global__ void __launch_bounds__(256) k_gemm_tn(GemmShape g, const T *__restrict__ A, const T *__restrict__ B,
                                                 Epi epi) {
  using Mf = Mfma<T>;
  constexpr int KPL = Mf::KPL, KSTEP = Mf::KSTEP;
  constexpr int EPC = 16 / sizeof(T);             // elements per 16-byte chunk
  constexpr int SL = kGBK + EPC;                  // padded LDS row stride (elements)
  constexpr int CPR = kGBK / EPC;                 // chunks per row
  constexpr int CH = kGBM * CPR / 256;            // chunks per thread per plane
  __shared__ __attribute__((aligned(16))) T sA[NA][kGBM * SL];
  __shared__ __attribute__((aligned(16))) T sB[NB][kGBN * SL];

  const int64_t nblocks = gridDim.x;
  const int64_t tile = xcd_remap(blockIdx.x, nblocks);
  int p, mt, nt;
  gemm_tile(g, tile, p, mt, nt);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int h = lane >> 5, col = lane & 31;
  const T *Ab = A + (size_t)p * g.a_pair + (size_t)mt * kGBM * g.lda;
  const T *Bb = B + (size_t)p * g.b_pair + (size_t)nt * kGBN * g.ldb;

  f32x4 ra[NA][CH], rb[NB][CH];
  auto prefetch = [&](int k0) {
    #pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = tid + 256 * c, r = idx / CPR, cc = (idx % CPR) * EPC;
      #pragma unroll
      for (int q = 0; q < NA; ++q)
        ra[q][c] = *reinterpret_cast<const f32x4 *>(Ab + q * g.a_plane + (size_t)r * g.lda + k0 + cc);
      #pragma unroll
      for (int q = 0; q < NB; ++q)
        rb[q][c] = *reinterpret_cast<const f32x4 *>(Bb + q * g.b_plane + (size_t)r * g.ldb + k0 + cc);
    }
  };
  f32x16 acc[2][2];
  #pragma unroll
  for (int i = 0; i < 2; ++i)
    #pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = zero16();

  prefetch(0);
  for (int k0 = 0; k0 < g.K; k0 += kGBK) {
    __syncthreads();
    #pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = tid + 256 * c, r = idx / CPR, cc = (idx % CPR) * EPC;
      #pragma unroll
      for (int q = 0; q < NA; ++q) *reinterpret_cast<f32x4 *>(&sA[q][r * SL + cc]) = ra[q][c];
      #pragma unroll
      for (int q = 0; q < NB; ++q) *reinterpret_cast<f32x4 *>(&sB[q][r * SL + cc]) = rb[q][c];
    }
    __syncthreads();
    if (k0 + kGBK < g.K) prefetch(k0 + kGBK);
    #pragma unroll
    for (int ks = 0; ks < kGBK / KSTEP; ++ks) {
      typename Mf::frag fa[NA][2], fb[NB][2];
      #pragma unroll
      for (int i = 0; i < 2; ++i) {
        #pragma unroll
        for (int q = 0; q < NA; ++q) fa[q][i] = Mf::load(&sA[q][(wm * 64 + 32 * i + col) * SL + ks * KSTEP + KPL * h]);
        #pragma unroll
        for (int q = 0; q < NB; ++q) fb[q][i] = Mf::load(&sB[q][(wn * 64 + 32 * i + col) * SL + ks * KSTEP + KPL * h]);
      }
      #pragma unroll
      for (int i = 0; i < 2; ++i)
        #pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = Mf::mma(fa[0][i], fb[0][j], acc[i][j]);
          if constexpr (NB > 1) acc[i][j] = Mf::mma(fa[0][i], fb[1][j], acc[i][j]);
          if constexpr (NA > 1) acc[i][j] = Mf::mma(fa[1][i], fb[0][j], acc[i][j]);
        }
    }
  }
  epi(acc, p, mt * kGBM + wm * 64, nt * kGBN + wn * 64, mt, nt, lane, wm);
}

// ------------------------------------------------------------------ epilogues
// Rows are anchors r, columns keys j.  For each key, keep the best two
// (similarity, lowest r) as packed 64-bit keys and the third similarity
// (Top3), one partial per (M-tile, key).  Similarities are >= 0, so their float
// bits order like uints.
struct EpiArgmax {
  uint64_t *part1, *part2;  // [P][MT][Np]
  uint32_t *part3;          // [P][MT][Np]
  int64_t pair_stride;      // MT * Np
  int Np, t;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[2][2], int p, int row0, int col0, int mt, int nt, int lane,
                             int wm) const {
    __shared__ uint64_t red1[128], red2[128];
    __shared__ uint32_t red3[128];
    const int h = lane >> 5, col = lane & 31;
    uint64_t k1[2], k2[2];
    uint32_t k3[2];
    #pragma unroll
    for (int j = 0; j < 2; ++j) {
      Top3 tp;
      tp.init();
      #pragma unroll
      for (int i = 0; i < 2; ++i)
        #pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = row0 + 32 * i + acc_row(v, lane);
          tp.add(acc[i][j][v], (uint32_t)r, r < t);
        }
      k1[j] = pack_sim(tp.v1, tp.r1);
      k2[j] = pack_sim(tp.v2, tp.r2);
      k3[j] = tp.v3 < 0.0f ? 0u : __float_as_uint(tp.v3);
      merge_top3(k1[j], k2[j], k3[j], __shfl_xor(k1[j], 32, 64), __shfl_xor(k2[j], 32, 64),
                 __shfl_xor(k3[j], 32, 64));
    }
    const int cl = col0 - nt * kGBN;   // 0 or 64 within the block
    if (wm == 1 && h == 0)
      #pragma unroll
      for (int j = 0; j < 2; ++j) {
        red1[cl + 32 * j + col] = k1[j];
        red2[cl + 32 * j + col] = k2[j];
        red3[cl + 32 * j + col] = k3[j];
      }
    __syncthreads();
    if (wm == 0 && h == 0)
      #pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = cl + 32 * j + col;
        merge_top3(k1[j], k2[j], k3[j], red1[c], red2[c], red3[c]);
        const size_t o = (size_t)p * pair_stride + (size_t)mt * Np + col0 + 32 * j + col;
        part1[o] = k1[j];
        part2[o] = k2[j];
        part3[o] = k3[j];
      }
  }
};

// Symmetric Gram: write the tile to G and Gc, and its transpose for tiles
// below the diagonal.
struct EpiSym {
  float *G, *Gc;
  int64_t pair_stride;  // ld * ld
  int ld;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[2][2], int p, int row0, int col0, int mt, int nt, int lane,
                             int) const {
    const int h = lane >> 5, col = lane & 31;
    float *Gp = G + (size_t)p * pair_stride, *Gcp = Gc + (size_t)p * pair_stride;
    #pragma unroll
    for (int i = 0; i < 2; ++i)
      #pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = col0 + 32 * j + col;
        #pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r0 = row0 + 32 * i + 8 * g + 4 * h;
          #pragma unroll
          for (int e = 0; e < 4; ++e) {
            Gp[(size_t)(r0 + e) * ld + c] = acc[i][j][4 * g + e];
            Gcp[(size_t)(r0 + e) * ld + c] = acc[i][j][4 * g + e];
          }
          if (mt != nt) {
            f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
            *reinterpret_cast<f32x4 *>(Gp + (size_t)c * ld + r0) = v;
            *reinterpret_cast<f32x4 *>(Gcp + (size_t)c * ld + r0) = v;
          }
        }
      }
  }
};

// out[r][c] = acc, or acc - lam[p] * X[r][c] when X is given (the value-fit
// residual P^T U - lam X).
struct EpiStore {
  float *out;
  int64_t pair_stride;
  int ld;
  const float *X;        // nullptr: plain store
  const float *lam;      // [P]
  __device__ __forceinline__ void operator()(f32x16 (&acc)[2][2], int p, int row0, int col0, int, int, int lane, int) const {
    const size_t base = (size_t)p * pair_stride;
    const int col = lane & 31;
    #pragma unroll
    for (int i = 0; i < 2; ++i)
      #pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int c = col0 + 32 * j + col;
        #pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = row0 + 32 * i + acc_row(v, lane);
          const size_t o = base + (size_t)r * ld + c;
          float val = acc[i][j][v];
          if (X) val -= lam[p] * X[o];
          out[o] = val;
        }
      }
  }
};

// U^T[c][i] = Y[i][c] - acc[c][i] (rows c < 128, columns queries i; zero for
// i >= n), stored as bf16 hi/lo planes or fp32 [P][planes][128][ld].
template <bool SPLIT>
struct EpiValueResid {
  void *out;
  int64_t pair_stride, plane_stride;   // elements
  int ld, n;
  const float *Y;                      // [P][n][128]
  __device__ __forceinline__ void operator()(f32x16 (&acc)[2][2], int p, int row0, int col0, int, int, int lane, int) const {
    const int h = lane >> 5, col = lane & 31;
    #pragma unroll
    for (int i = 0; i < 2; ++i)
      #pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int q = col0 + 32 * j + col;   // query index
        #pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c0 = row0 + 32 * i + 8 * g + 4 * h;
          f32x4 y = {0.f, 0.f, 0.f, 0.f};
          if (q < n) y = *reinterpret_cast<const f32x4 *>(Y + ((size_t)p * n + q) * kHeadDim + c0);
          #pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float u = q < n ? y[e] - acc[i][j][4 * g + e] : 0.0f;
            const size_t o = (size_t)p * pair_stride + (size_t)(c0 + e) * ld + q;
            if constexpr (SPLIT) {
              bf16 hi, lo;
              split_bf16(u, hi, lo);
              reinterpret_cast<bf16 *>(out)[o] = hi;
              reinterpret_cast<bf16 *>(out)[o + plane_stride] = lo;
            } else {
              reinterpret_cast<float *>(out)[o] = u;
            }
          }
        }
      }
  }
};

template <typename T, int NA, int NB, class Epi>
hipError_t launch_gemm(const GemmShape &g, const T *A, const T *B, const Epi &epi, hipStream_t s) {
  const int64_t tiles = gemm_tiles(g);
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_tn<T, NA, NB, Epi>), dim3((unsigned)tiles), dim3(256), 0, s, g, A, B, epi);
  return hipGetLastError();
}

}  // namespace arckv
