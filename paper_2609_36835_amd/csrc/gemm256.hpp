// Large-tile variant of the batched TN contraction for the big bf16 / split-
// bf16 contractions (anchor assignment, Gram matrices).
//
// Workgroup tile 256 x 256, 4 waves of 128 x 128 (4 x 4 MFMA 32x32x16 tiles,
// 256 fp32 accumulators per lane).  K advances in slabs of BK (64 for one
// bf16 plane, 32 for hi/lo planes) through two LDS buffers: the next slab is
// fetched into registers while the current one feeds the MFMAs, then written
// to the other buffer, so each K step needs a single barrier.  At 256 x 256
// the operand traffic from L2 is ~16 B/clk per CU at the MFMA peak (a 128 x
// 128 tile needs ~64 B/clk, the L2 limit).
#pragma once
#include "gemm.hpp"

namespace arckv {

constexpr int kLBM = 256, kLBN = 256;

struct GemmShape256 {
  int batch, M, N, K;               // multiples of 256 / BK
  int64_t a_pair, a_plane, lda;
  int64_t b_pair, b_plane, ldb;
  bool syrk;
  int group_m;
};

__device__ inline void gemm256_tile(const GemmShape256 &g, int64_t tile, int &p, int &mt, int &nt) {
  const int MT = g.M / kLBM, NT = g.N / kLBN;
  if (g.syrk) {
    const int64_t per = (int64_t)MT * (MT + 1) / 2;
    p = (int)(tile / per);
    const int64_t r = tile % per;
    int m = (int)((sqrt(8.0 * (double)r + 1.0) - 1.0) * 0.5);
    while ((int64_t)m * (m + 1) / 2 > r) --m;
    while ((int64_t)(m + 1) * (m + 2) / 2 <= r) ++m;
    mt = m;
    nt = (int)(r - (int64_t)m * (m + 1) / 2);
    return;
  }
  const int64_t per = (int64_t)MT * NT;
  p = (int)(tile / per);
  const int64_t r = tile % per;
  const int gm = g.group_m;
  const int64_t per_group = (int64_t)gm * NT;
  const int grp = (int)(r / per_group);
  const int first_m = grp * gm;
  const int gsize = min(MT - first_m, gm);
  const int64_t rr = r % per_group;
  mt = first_m + (int)(rr % gsize);
  nt = (int)(rr / gsize);
}

__host__ inline int64_t gemm256_tiles(const GemmShape256 &g) {
  const int64_t MT = g.M / kLBM, NT = g.N / kLBN;
  return (int64_t)g.batch * (g.syrk ? MT * (MT + 1) / 2 : MT * NT);
}

template <int NA, int NB, class Epi>
__global__ void __launch_bounds__(256, 1) k_gemm256(GemmShape256 g, const bf16 *__restrict__ A,
                                                    const bf16 *__restrict__ B, Epi epi) {
  constexpr int BK = (NA + NB > 2) ? 32 : 64;
  constexpr int SL = BK + 8;                         // padded LDS row (elements): 16 B pad
  constexpr int CPR = BK / 8;                        // 16-byte chunks per row
  constexpr int CH = kLBM * CPR / 256;               // chunks per thread per plane
  constexpr int KS = BK / 16;                        // MFMA k-steps per slab
  constexpr int STAGE = (NA + NB) * kLBM * SL;        // elements per LDS buffer
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];

  const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
  int p, mt, nt;
  gemm256_tile(g, tile, p, mt, nt);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int h = lane >> 5, col = lane & 31;
  const bf16 *Ab = A + (size_t)p * g.a_pair + (size_t)mt * kLBM * g.lda;
  const bf16 *Bb = B + (size_t)p * g.b_pair + (size_t)nt * kLBN * g.ldb;

  f32x4 ra[NA][CH], rb[NB][CH];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = tid + 256 * c, r = idx / CPR, cc = (idx % CPR) * 8;
#pragma unroll
      for (int q = 0; q < NA; ++q)
        ra[q][c] = *reinterpret_cast<const f32x4 *>(Ab + q * g.a_plane + (size_t)r * g.lda + k0 + cc);
#pragma unroll
      for (int q = 0; q < NB; ++q)
        rb[q][c] = *reinterpret_cast<const f32x4 *>(Bb + q * g.b_plane + (size_t)r * g.ldb + k0 + cc);
    }
  };
  auto stash = [&](bf16 *s) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const int idx = tid + 256 * c, r = idx / CPR, cc = (idx % CPR) * 8;
#pragma unroll
      for (int q = 0; q < NA; ++q) *reinterpret_cast<f32x4 *>(&s[(q * kLBM + r) * SL + cc]) = ra[q][c];
#pragma unroll
      for (int q = 0; q < NB; ++q) *reinterpret_cast<f32x4 *>(&s[((NA + q) * kLBM + r) * SL + cc]) = rb[q][c];
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = zero16();

  fetch(0);
  stash(smem);
  __syncthreads();
  int buf = 0;
  for (int k0 = 0; k0 < g.K; k0 += BK) {
    const bool more = k0 + BK < g.K;
    if (more) fetch(k0 + BK);
    const bf16 *s = smem + buf * STAGE;
#pragma unroll 1
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 fa[NA][4], fb[NB][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int q = 0; q < NA; ++q)
          fa[q][i] = *reinterpret_cast<const bf16x8 *>(&s[(q * kLBM + wm * 128 + 32 * i + col) * SL + ks * 16 + 8 * h]);
#pragma unroll
        for (int q = 0; q < NB; ++q)
          fb[q][i] = *reinterpret_cast<const bf16x8 *>(
              &s[((NA + q) * kLBM + wn * 128 + 32 * i + col) * SL + ks * 16 + 8 * h]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = Mfma<bf16>::mma(fa[0][i], fb[0][j], acc[i][j]);
          if constexpr (NB > 1) acc[i][j] = Mfma<bf16>::mma(fa[0][i], fb[1][j], acc[i][j]);
          if constexpr (NA > 1) acc[i][j] = Mfma<bf16>::mma(fa[1][i], fb[0][j], acc[i][j]);
        }
    }
    if (more) stash(smem + (buf ^ 1) * STAGE);
    __syncthreads();
    buf ^= 1;
  }
  epi(acc, p, mt * kLBM + wm * 128, nt * kLBN + wn * 128, mt, nt, lane, wm);
}

// ------------------------------------------------------------------ epilogues
// Anchor assignment: rows anchors r, columns keys j; packed (similarity, lowest
// r) maxima per (256-row M-tile, key).
struct EpiArgmax256 {
  uint64_t *part;       // [P][MT][Np]
  int64_t pair_stride;  // MT * Np
  int Np, t;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int p, int row0, int col0, int mt, int nt,
                                             int lane, int wm) const {
    __shared__ uint64_t red[256];
    const int h = lane >> 5, col = lane & 31;
    uint64_t best[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      best[j] = 0ull;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = row0 + 32 * i + acc_row(v, lane);
          const uint64_t key =
              ((uint64_t)__float_as_uint(acc[i][j][v]) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)r);
          best[j] = (r < t && key > best[j]) ? key : best[j];
        }
      const uint64_t o = __shfl_xor(best[j], 32, 64);
      best[j] = o > best[j] ? o : best[j];
    }
    const int cl = col0 - nt * kLBN;   // 0 or 128
    if (wm == 1 && h == 0)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[cl + 32 * j + col] = best[j];
    __syncthreads();
    if (wm == 0 && h == 0)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint64_t o = red[cl + 32 * j + col];
        part[(size_t)p * pair_stride + (size_t)mt * Np + col0 + 32 * j + col] = o > best[j] ? o : best[j];
      }
  }
};

// Symmetric Gram: write the tile to G and Gc, and its transpose below the diagonal.
struct EpiSym256 {
  float *G, *Gc;
  int64_t pair_stride;
  int ld;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[4][4], int p, int row0, int col0, int mt, int nt,
                                             int lane, int) const {
    const int h = lane >> 5, col = lane & 31;
    float *Gp = G + (size_t)p * pair_stride, *Gcp = Gc + (size_t)p * pair_stride;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
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
            const f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
            *reinterpret_cast<f32x4 *>(Gp + (size_t)c * ld + r0) = v;
            *reinterpret_cast<f32x4 *>(Gcp + (size_t)c * ld + r0) = v;
          }
        }
      }
  }
};

template <int NA, int NB, class Epi>
hipError_t launch_gemm256(const GemmShape256 &g, const bf16 *A, const bf16 *B, const Epi &epi, hipStream_t s) {
  const int64_t tiles = gemm256_tiles(g);
  if (tiles == 0) return hipSuccess;
  constexpr int BK = (NA + NB > 2) ? 32 : 64;
  const size_t lds = 2 * (size_t)(NA + NB) * kLBM * (BK + 8) * sizeof(bf16);
  auto kern = k_gemm256<NA, NB, Epi>;
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)tiles), dim3(256), lds, s, g, A, B, epi);
  return hipGetLastError();
}

}  // namespace arckv
