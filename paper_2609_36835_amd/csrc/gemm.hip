// Instantiations of the batched TN contraction for the compaction stages.
#include "gemm.hpp"
#include "gemm_big.hpp"

namespace arckv {

// Anchor assignment (eq. anchor_assignment): S[r][j] = sum_i U_S[r][i] E^T[j][i];
// per-(M-tile, key) top-3 partials (EpiArgmax*) [P][MT][N].  U [P][tp][np],
// Et [P][Et_rows][np] with the first N rows used (the compacted non-anchor
// keys).  Operands are fp16 for bf16 inputs (large-tile kernel, M-tiles of 256
// rows, 8 waves of 64 x 128) and fp32 for fp32 inputs (M-tiles of 128).
hipError_t launch_assign_gemm(int dtype, const void *U, const void *Et, uint64_t *part1, uint64_t *part2,
                              uint32_t *part3, int P, int t, int64_t tp, int64_t N, int64_t Et_rows, int64_t np_,
                              hipStream_t s) {
  if (N == 0) return hipSuccess;
  if (dtype == ARCKV_BF16) {
    // tile order: all anchor tiles of a pair walk the key tiles together (about 13 x 2.5 tiles per XCD
    // at a time): half the L2 misses of groups of 7, 2-3% faster
    BigShape g2{P, (int)tp, (int)N, (int)np_, tp * np_, 0, np_, Et_rows * np_, 0, np_, false, 13};
    EpiArgmaxBig<4, 2, 2, 4> e2{part1, part2, part3, (tp / 256) * N, (int)N, t};
    return launch_gemm_big<4, 2, 2, 4, 64, 1, 1, 2, f16>(g2, (const bf16 *)U, (const bf16 *)Et, e2, s);
  }
  GemmShape g;
  g.batch = P;
  g.M = (int)tp;
  g.N = (int)N;
  g.K = (int)np_;
  g.a_pair = tp * np_;
  g.a_plane = 0;
  g.lda = np_;
  g.b_pair = Et_rows * np_;
  g.b_plane = 0;
  g.ldb = np_;
  g.syrk = false;
  g.group_m = 8;
  EpiArgmax e{part1, part2, part3, (tp / kGBM) * N, (int)N, t};
  return launch_gemm<float, 1, 1>(g, (const float *)U, (const float *)Et, e, s);
}

// Gram matrix X^T X of a [P][planes][tp][np] operand (rows = columns of the
// design matrix), written to both G and Gc ([P][tp][tp]).
hipError_t launch_gram(int dtype, const void *X, float *G, float *Gc, int P, int64_t tp, int64_t np_,
                       hipStream_t s) {
  GemmShape g;
  g.batch = P;
  g.M = g.N = (int)tp;
  g.K = (int)np_;
  g.syrk = true;
  g.group_m = 8;
  g.lda = g.ldb = np_;
  EpiSym e{G, Gc, tp * tp, (int)tp};
  if (dtype == ARCKV_BF16) {
    BigShape g2{P, (int)tp, (int)tp, (int)np_, 2 * tp * np_, tp * np_, np_, 2 * tp * np_, tp * np_, np_, true, 4};
    EpiSymBig<2, 4> e2{G, Gc, tp * tp, (int)tp};
    return launch_gemm_big<4, 2, 2, 4, 32, 2, 2, 2>(g2, (const bf16 *)X, (const bf16 *)X, e2, s);
  }
  g.a_pair = g.b_pair = tp * np_;
  g.a_plane = g.b_plane = 0;
  return launch_gemm<float, 1, 1>(g, (const float *)X, (const float *)X, e, s);
}

// Right-hand side P^T Y: PT [P][planes][tp][np], YT [P][planes][128][np] -> Bm [P][tp][128].
hipError_t launch_rhs_gemm(int dtype, const void *PT, const void *YT, float *Bm, int P, int64_t tp, int64_t np_,
                           hipStream_t s) {
  GemmShape g;
  g.batch = P;
  g.M = (int)tp;
  g.N = kHeadDim;
  g.K = (int)np_;
  g.syrk = false;
  g.group_m = 8;
  g.lda = g.ldb = np_;
  EpiStore e{Bm, tp * kHeadDim, kHeadDim, nullptr, nullptr};
  if (dtype == ARCKV_BF16) {
    BigShape g2{P, (int)tp, kHeadDim, (int)np_, 2 * tp * np_, tp * np_, np_, 2 * (int64_t)kHeadDim * np_,
                (int64_t)kHeadDim * np_, np_, false, (int)(tp / 256)};
    EpiStoreBig<2, 2> e2{Bm, tp * kHeadDim, kHeadDim, nullptr, nullptr};
    return launch_gemm_big<4, 2, 2, 2, 32, 2, 2, 2>(g2, (const bf16 *)PT, (const bf16 *)YT, e2, s);
  }
  g.a_pair = tp * np_;
  g.a_plane = 0;
  g.b_pair = (int64_t)kHeadDim * np_;
  g.b_plane = 0;
  return launch_gemm<float, 1, 1>(g, (const float *)PT, (const float *)YT, e, s);
}

// Value-fit refinement residual from the data, in two contractions over the
// split (or fp32) operands:
//   U^T = Y^T - X^T P^T      A = X^T [P][pl][128][tp], B = P [P][pl][np][tp], K = tp
//   R   = P^T U - lam X       A = P^T [P][pl][tp][np],  B = U^T [P][pl][128][np], K = np
hipError_t launch_value_residual(int dtype, const void *XT, const void *Pm, const void *PT, const float *Y, void *UT,
                                 const float *X, const float *lam, float *R, int P, int n, int64_t tp, int64_t np_,
                                 hipStream_t s) {
  const bool split = dtype == ARCKV_BF16;
  const int64_t pl = split ? 2 : 1;
  GemmShape g1;
  g1.batch = P;
  g1.M = kHeadDim;
  g1.N = (int)np_;
  g1.K = (int)tp;
  g1.syrk = false;
  g1.group_m = 8;
  g1.a_pair = pl * kHeadDim * tp;
  g1.a_plane = split ? kHeadDim * tp : 0;
  g1.lda = tp;
  g1.b_pair = pl * np_ * tp;
  g1.b_plane = split ? np_ * tp : 0;
  g1.ldb = tp;
  hipError_t e;
  if (split) {
    BigShape gb{P, kHeadDim, (int)np_, (int)tp, pl * kHeadDim * tp, kHeadDim * tp, tp, pl * np_ * tp, np_ * tp, tp,
                false, 1};
    EpiValueResidBig<2, 2> ep{(bf16 *)UT, pl * kHeadDim * np_, kHeadDim * np_, (int)np_, n, Y};
    e = launch_gemm_big<2, 4, 2, 2, 32, 2, 2, 2>(gb, (const bf16 *)XT, (const bf16 *)Pm, ep, s);
  } else {
    EpiValueResid<false> ep{UT, kHeadDim * np_, 0, (int)np_, n, Y};
    e = launch_gemm<float, 1, 1>(g1, (const float *)XT, (const float *)Pm, ep, s);
  }
  if (e != hipSuccess) return e;
  GemmShape g2;
  g2.batch = P;
  g2.M = (int)tp;
  g2.N = kHeadDim;
  g2.K = (int)np_;
  g2.syrk = false;
  g2.group_m = 8;
  g2.a_pair = pl * tp * np_;
  g2.a_plane = split ? tp * np_ : 0;
  g2.lda = np_;
  g2.b_pair = pl * kHeadDim * np_;
  g2.b_plane = split ? kHeadDim * np_ : 0;
  g2.ldb = np_;
  EpiStore e2{R, tp * kHeadDim, kHeadDim, X, lam};
  if (split) {
    BigShape gb{P, (int)tp, kHeadDim, (int)np_, pl * tp * np_, tp * np_, np_, pl * kHeadDim * np_, kHeadDim * np_, np_,
                false, (int)(tp / 256)};
    EpiStoreBig<2, 2> eb{R, tp * kHeadDim, kHeadDim, X, lam};
    return launch_gemm_big<4, 2, 2, 2, 32, 2, 2, 2>(gb, (const bf16 *)PT, (const bf16 *)UT, eb, s);
  }
  return launch_gemm<float, 1, 1>(g2, (const float *)PT, (const float *)UT, e2, s);
}

}  // namespace arckv
