// Large-tile batched TN contraction on bf16 or fp16 MFMA (32x32x16) for the
// big contractions of the path: the anchor assignment (one fp16 plane), the
// split-bf16 Gram matrices (hi/lo planes, three products) and the Cholesky
// trailing updates (row-scaled fp16 hi/lo planes of an fp32 panel, three
// products as one contraction over three K segments, about 2^-22 relative).
//
// C[M][N] = sum_k A[m][k] B[n][k], both operands K-contiguous.  A workgroup of
// WM x WN waves owns a (32 WM TM) x (32 WN TN) tile; each wave a 32TM x 32TN
// block of accumulators.  Operand slabs of BK elements go global -> LDS with
// the CDNA4 direct-to-LDS loads (global_load_lds_dwordx4: lane l of a wave
// writes bytes [16 l, 16 l + 16) of a 1 KB LDS run), so no VGPRs are spent on
// staging.  Rows are stored unpadded and each row's 16-byte chunks are XOR-
// swizzled with the row index, which makes the MFMA fragment reads (32 rows x
// one chunk per half-wave) free of bank conflicts.  NS LDS stages: slabs
// i+1 .. i+NS-1 are in flight while slab i feeds the MFMAs (a counted vmcnt
// wait lets the younger slabs stay outstanding); fragments for k-step ks+1 are
// read while the MFMAs of ks run, and a slab's last k-step of MFMAs runs after
// the next slab's barrier.  One workgroup barrier per slab, without the full
// memory fence of __syncthreads(), so the prefetch stays in flight.
// Dimensions must be multiples of the tile; workgroups are remapped so that
// each XCD owns a contiguous, M-grouped (or lower-triangular) range of tiles.
#pragma once
#include <type_traits>
#include <utility>

#include "gemm.hpp"

namespace arckv {

typedef __attribute__((address_space(3))) void lds_void_t;

struct BigShape {
  int batch, M, N, K;
  int64_t a_pair, a_plane, lda;   // elements
  int64_t b_pair, b_plane, ldb;
  bool syrk;                      // lower-triangular tiles only (nt <= mt)
  int group_m;
  // Segmented K (single-plane configurations): K = segments x kseg, and
  // segment s reads plane (sega >> 2s) & 3 of A and (segb >> 2s) & 3 of B at
  // columns 0 .. kseg - 1.  One accumulation then sums several plane products
  // (kseg = 0: plain K).
  int kseg = 0;
  uint32_t sega = 0, segb = 0;
};

template <int WM, int WN, int TM, int TN, int BK, int NA, int NB, int NS = 2>
struct BigCfg {
  static constexpr int NW = WM * WN, THREADS = 64 * NW;
  static constexpr int BM = 32 * WM * TM, BN = 32 * WN * TN;
  static constexpr int RB = BK * 2;                 // LDS row bytes
  static constexpr int CPR = BK / 8;                // 16-byte chunks per row
  static constexpr int RPI = 1024 / RB;             // rows per 1 KB load run
  static constexpr int A_BYTES = BM * RB, B_BYTES = BN * RB;
  static constexpr int STAGE = NA * A_BYTES + NB * B_BYTES;
  static constexpr int LDS = NS * STAGE;
  static constexpr int A_INST = A_BYTES / 1024 / NW, B_INST = B_BYTES / 1024 / NW;
  static constexpr int SLAB_INST = NA * A_INST + NB * B_INST;   // load instructions per slab per wave
  static constexpr int KS = BK / 16;
  static_assert(A_INST * NW * 1024 == A_BYTES && B_INST * NW * 1024 == B_BYTES, "load split");
  static_assert(CPR == 4 || CPR == 8, "BK must be 32 or 64");
  static_assert(NA == NB || NA == 1 || NB == 1, "plane counts");
  static_assert(LDS <= 160 * 1024 - 16 * 1024, "LDS budget");
  static_assert(NS >= 2 && (NS - 2) * SLAB_INST < 64, "stages");
  // chunk swizzle: 16 consecutive rows at one logical chunk cover all 64 banks
  __device__ static __forceinline__ int swz(int row) { return (row * RB / 256) & (CPR - 1); }
};

template <int BM, int BN>
__device__ inline void big_tile(const BigShape &g, int64_t tile, int &p, int &mt, int &nt) {
  const int MT = g.M / BM, NT = g.N / BN;
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

inline int64_t big_tiles(const BigShape &g, int BM, int BN) {
  const int64_t MT = g.M / BM, NT = g.N / BN;
  return (int64_t)g.batch * (g.syrk ? MT * (MT + 1) / 2 : MT * NT);
}

// s_waitcnt until at most N vector-memory instructions of this wave are
// outstanding (expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// s_waitcnt lgkmcnt(0) (vmcnt and expcnt left unconstrained).
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4)); }

// Workgroup barrier without a memory fence; the empty asm statements keep the
// compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// An epilogue may expose skip(p): the whole tile is skipped for pair p (a
// factorisation that failed or no longer needs updating).
template <typename E, typename = void>
struct epi_has_skip : std::false_type {};
template <typename E>
struct epi_has_skip<E, std::void_t<decltype(std::declval<const E &>().skip(0))>> : std::true_type {};

template <int WM, int WN, int TM, int TN, int BK, int NA, int NB, int NS, typename E, class Epi>
__global__ void __launch_bounds__(64 * WM * WN, 1) k_gemm_big(BigShape g, const bf16 *__restrict__ A,
                                                              const bf16 *__restrict__ B, Epi epi) {
  using C = BigCfg<WM, WN, TM, TN, BK, NA, NB, NS>;
  extern __shared__ __attribute__((aligned(1024))) char big_smem[];

  const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
  int p, mt, nt;
  big_tile<C::BM, C::BN>(g, tile, p, mt, nt);
  if constexpr (epi_has_skip<Epi>::value) {
    if (epi.skip(p)) return;   // uniform over the workgroup: no barrier has run yet
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int h = lane >> 5, col = lane & 31;
  const bf16 *Ab = A + (size_t)p * g.a_pair + (size_t)mt * C::BM * g.lda;
  const bf16 *Bb = B + (size_t)p * g.b_pair + (size_t)nt * C::BN * g.ldb;

  // Per-lane source offsets of this wave's load runs: run gi covers rows
  // [gi RPI, gi RPI + RPI); lane l fills physical chunk l % CPR of row
  // gi RPI + l / CPR, i.e. logical chunk (l % CPR) ^ swz(row).
  int64_t offA[C::A_INST], offB[C::B_INST];
#pragma unroll
  for (int i = 0; i < C::A_INST; ++i) {
    const int row = (wave * C::A_INST + i) * C::RPI + lane / C::CPR;
    offA[i] = (int64_t)row * g.lda + 8 * ((lane % C::CPR) ^ C::swz(row));
  }
#pragma unroll
  for (int i = 0; i < C::B_INST; ++i) {
    const int row = (wave * C::B_INST + i) * C::RPI + lane / C::CPR;
    offB[i] = (int64_t)row * g.ldb + 8 * ((lane % C::CPR) ^ C::swz(row));
  }
  auto issue = [&](int slab, int st) {
    const int k0 = slab * BK;
    int64_t ka = k0, kb = k0;
    if (g.kseg) {   // wave-uniform: a slab never straddles two segments
      const int sg = k0 / g.kseg, kk = k0 - sg * g.kseg;
      ka = (int64_t)((g.sega >> (2 * sg)) & 3u) * g.a_plane + kk;
      kb = (int64_t)((g.segb >> (2 * sg)) & 3u) * g.b_plane + kk;
    }
    char *s = big_smem + st * C::STAGE;
#pragma unroll
    for (int q = 0; q < NA; ++q)
#pragma unroll
      for (int i = 0; i < C::A_INST; ++i)
        __builtin_amdgcn_global_load_lds((const void *)(Ab + q * g.a_plane + offA[i] + ka),
                                         (lds_void_t *)(s + q * C::A_BYTES + (wave * C::A_INST + i) * 1024), 16, 0,
                                         0);
#pragma unroll
    for (int q = 0; q < NB; ++q)
#pragma unroll
      for (int i = 0; i < C::B_INST; ++i)
        __builtin_amdgcn_global_load_lds(
            (const void *)(Bb + q * g.b_plane + offB[i] + kb),
            (lds_void_t *)(s + NA * C::A_BYTES + q * C::B_BYTES + (wave * C::B_INST + i) * 1024), 16, 0, 0);
  };

  int rowA[TM], rowB[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) rowA[i] = wm * 32 * TM + 32 * i + col;
#pragma unroll
  for (int j = 0; j < TN; ++j) rowB[j] = wn * 32 * TN + 32 * j + col;
  auto rd = [&](const char *s, int ks, bf16x8 (&fa)[NA][TM], bf16x8 (&fb)[NB][TN]) {
    const int c = 2 * ks + h;
#pragma unroll
    for (int q = 0; q < NA; ++q)
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[q][i] = *reinterpret_cast<const bf16x8 *>(s + q * C::A_BYTES + rowA[i] * C::RB +
                                                     16 * (c ^ C::swz(rowA[i])));
#pragma unroll
    for (int q = 0; q < NB; ++q)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[q][j] = *reinterpret_cast<const bf16x8 *>(s + NA * C::A_BYTES + q * C::B_BYTES + rowB[j] * C::RB +
                                                     16 * (c ^ C::swz(rowB[j])));
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = zero16();

  // one k-step of products from fragments in registers
  auto step = [&](bf16x8 (&fa)[NA][TM], bf16x8 (&fb)[NB][TN]) {
#pragma unroll
    for (int ii = 0; ii < TM; ++ii)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        acc[ii][j] = mma16<E>(fa[0][ii], fb[0][j], acc[ii][j]);
        if constexpr (NB > 1) acc[ii][j] = mma16<E>(fa[0][ii], fb[1][j], acc[ii][j]);
        if constexpr (NA > 1) acc[ii][j] = mma16<E>(fa[1][ii], fb[0][j], acc[ii][j]);
        if constexpr (NA > 2 && NB > 2) {
          acc[ii][j] = mma16<E>(fa[0][ii], fb[2][j], acc[ii][j]);
          acc[ii][j] = mma16<E>(fa[2][ii], fb[0][j], acc[ii][j]);
          acc[ii][j] = mma16<E>(fa[1][ii], fb[1][j], acc[ii][j]);
        }
      }
  };

  // Fragments of k-step ks go to buffer ks & 1.  The products of a slab's last
  // k-step (buffer 1) run after the next slab's barrier, under the LDS reads
  // of that slab's first k-step, so the matrix cores are not idle while every
  // wave fetches its first fragments; the sums keep their order.
  static_assert(C::KS % 2 == 0, "the last k-step of a slab sits in buffer 1");
  const int nk = g.K / BK;
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) issue(st, st);
  bf16x8 fa[2][NA][TM], fb[2][NB][TN];
  for (int i = 0; i < nk; ++i) {
    // this wave's runs of slab i have landed (the younger slabs i+1 ..
    // i+NS-2 may still be in flight); after the barrier every wave's have, and
    // every wave is done reading slab i-1, whose stage is refilled next
    if (i + NS - 2 < nk) wait_vmcnt<(NS - 2) * C::SLAB_INST>();
    else if constexpr (NS > 2) {   // last slabs: wait conservatively
      if (i + 1 < nk) wait_vmcnt<C::SLAB_INST>();
      else wait_vmcnt<0>();
    }
    wait_lgkmcnt0();   // the deferred fragments are in registers
    lds_barrier();
    const char *s = big_smem + (i % NS) * C::STAGE;
    rd(s, 0, fa[0], fb[0]);
    __builtin_amdgcn_sched_barrier(0);
    if (i > 0) step(fa[1], fb[1]);
    // the next slab's loads go out once the deferred MFMAs are issued (before
    // them they hold up the first fragment reads, later they land late)
    __builtin_amdgcn_sched_barrier(0);
    if (i + NS - 1 < nk) issue(i + NS - 1, (i + NS - 1) % NS);
#pragma unroll
    for (int ks = 0; ks + 1 < C::KS; ++ks) {
      rd(s, ks + 1, fa[(ks + 1) & 1], fb[(ks + 1) & 1]);
      step(fa[ks & 1], fb[ks & 1]);
    }
    asm volatile("" ::: "memory");
  }
  if (nk > 0) step(fa[1], fb[1]);
  __syncthreads();
  epi(acc, p, mt * C::BM + wm * 32 * TM, nt * C::BN + wn * 32 * TN, mt, nt, lane, wm, wn);
}

// ------------------------------------------------------------------ epilogues
// Anchor assignment: rows anchors r, columns keys j.  For every (M-tile,
// key) the best two similarities as packed keys and the third as float bits
// (Top3), so a later pass can tell which anchors of the tile may be the
// argmax once the rounding of the operands is accounted for.
template <int WM, int WN, int TM, int TN>
struct EpiArgmaxBig {
  uint64_t *part1, *part2;  // [P][MT][Np]
  uint32_t *part3;          // [P][MT][Np]
  int64_t pair_stride;      // MT * Np
  int Np, t;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int mt, int nt,
                                             int lane, int wm, int wn) const {
    constexpr int BN = 32 * WN * TN;
    // the operand stages are free once the contraction has finished (the
    // caller synchronised the workgroup before the epilogue)
    extern __shared__ __attribute__((aligned(1024))) char big_smem[];
    uint64_t *red1 = reinterpret_cast<uint64_t *>(big_smem);    // [WM][BN]
    uint64_t *red2 = red1 + WM * BN;                             // [WM][BN]
    uint32_t *red3 = reinterpret_cast<uint32_t *>(red2 + WM * BN);
    const int h = lane >> 5, col = lane & 31;
    // Per lane and column, the top three of its 32 values as uint32 keys: the
    // similarity's bits with the low 5 cleared (a relative truncation below
    // 2^-18, which the decision bound includes) and 31 - position in the low 5,
    // so max / med3 keep the larger value and, among equal keys, the lower r.
    const bool all_valid = row0 + 32 * TM <= t;   // wave-uniform
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      uint32_t q1 = 0u, q2 = 0u, q3 = 0u;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          uint32_t key = (__float_as_uint(acc[i][j][v]) & ~31u) | (uint32_t)(31 - (16 * i + v));
          if (!all_valid) key = row0 + 32 * i + acc_row(v, lane) < t ? key : 0u;
          const uint32_t n2 = med3u(q1, q2, key);
          q3 = med3u(q2, q3, key);
          q2 = n2;
          q1 = max(q1, key);
        }
      auto unpack = [&](uint32_t q) -> uint64_t {
        if (q == 0u) return 0ull;
        const int pos = 31 - (int)(q & 31u);
        const int r = row0 + 32 * (pos >> 4) + acc_row(pos & 15, lane);
        return ((uint64_t)(q & ~31u) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)r);
      };
      uint64_t k1 = unpack(q1), k2 = unpack(q2);
      uint32_t k3 = q3 & ~31u;
      merge_top3(k1, k2, k3, __shfl_xor(k1, 32, 64), __shfl_xor(k2, 32, 64), __shfl_xor(k3, 32, 64));
      if (h == 0) {
        const int c = wm * BN + wn * 32 * TN + 32 * j + col;
        red1[c] = k1;
        red2[c] = k2;
        red3[c] = k3;
      }
    }
    __syncthreads();
    for (int c = threadIdx.x; c < BN; c += 64 * WM * WN) {
      uint64_t k1 = red1[c], k2 = red2[c];
      uint32_t k3 = red3[c];
#pragma unroll
      for (int w = 1; w < WM; ++w) merge_top3(k1, k2, k3, red1[w * BN + c], red2[w * BN + c], red3[w * BN + c]);
      const size_t o = (size_t)p * pair_stride + (size_t)mt * Np + (size_t)nt * BN + c;
      part1[o] = k1;
      part2[o] = k2;
      part3[o] = k3;
    }
  }
};

// Symmetric Gram: write the lower tile to G and Gc.  The strict upper triangle
// outside the diagonal tiles is left unwritten: the factorisation, the solves
// and the free-set gathers read the lower triangle only.
template <int TM, int TN>
struct EpiSymBig {
  float *G, *Gc;
  int64_t pair_stride;
  int ld;
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int, int,
                                             int lane, int, int) const {
    const int h = lane >> 5, col = lane & 31;
    float *Gp = G + (size_t)p * pair_stride, *Gcp = Gc + (size_t)p * pair_stride;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int c = col0 + 32 * j + col;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int r0 = row0 + 32 * i + 8 * g + 4 * h;
          const f32x4 v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            Gp[(size_t)(r0 + e) * ld + c] = v[e];
            Gcp[(size_t)(r0 + e) * ld + c] = v[e];
          }
        }
      }
  }
};

// out[r][c] = acc (minus lam[p] X[r][c] when X is given), fp32 [P][rows][ld].
template <int TM, int TN>
struct EpiStoreBig {
  float *out;
  int64_t pair_stride;
  int ld;
  const float *X;      // nullptr: plain store
  const float *lam;    // [P]
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int, int, int lane,
                                             int, int) const {
    const size_t base = (size_t)p * pair_stride;
    const int col = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
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

// U^T[c][q] = Y[q][c] - acc[c][q] (rows c < 128, columns queries q; zero for
// q >= n), stored as bf16 hi/lo planes [P][2][128][ld].
template <int TM, int TN>
struct EpiValueResidBig {
  bf16 *out;
  int64_t pair_stride, plane_stride;   // elements
  int ld, n;
  const float *Y;                      // [P][n][128]
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int, int, int lane,
                                             int, int) const {
    const int h = lane >> 5, col = lane & 31;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int q = col0 + 32 * j + col;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int c0 = row0 + 32 * i + 8 * g + 4 * h;
          f32x4 y = {0.f, 0.f, 0.f, 0.f};
          if (q < n) y = *reinterpret_cast<const f32x4 *>(Y + ((size_t)p * n + q) * kHeadDim + c0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float u = q < n ? y[e] - acc[i][j][4 * g + e] : 0.0f;
            const size_t o = (size_t)p * pair_stride + (size_t)(c0 + e) * ld + q;
            bf16 hi, lo;
            split_bf16(u, hi, lo);
            out[o] = hi;
            out[o + plane_stride] = lo;
          }
        }
      }
  }
};

template <int WM, int WN, int TM, int TN, int BK, int NA, int NB, int NS, typename E = bf16, class Epi>
hipError_t launch_gemm_big(const BigShape &g, const bf16 *A, const bf16 *B, const Epi &epi, hipStream_t s) {
  using C = BigCfg<WM, WN, TM, TN, BK, NA, NB, NS>;
  if (g.M % C::BM || g.N % C::BN || g.K % BK) return hipErrorInvalidValue;
  if (g.kseg && (NA != 1 || NB != 1 || g.kseg % BK || g.K % g.kseg || g.K / g.kseg > 16))
    return hipErrorInvalidValue;
  const int64_t tiles = big_tiles(g, C::BM, C::BN);
  if (tiles == 0) return hipSuccess;
  auto kern = k_gemm_big<WM, WN, TM, TN, BK, NA, NB, NS, E, Epi>;
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)tiles), dim3(C::THREADS), C::LDS, s, g, A, B, epi);
  return hipGetLastError();
}

}  // namespace arckv
