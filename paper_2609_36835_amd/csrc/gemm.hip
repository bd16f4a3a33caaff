// Instantiations of the batched TN contraction for the compaction stages.
#include "gemm.hpp"

namespace arckv {

// Anchor assignment (eq. anchor_assignment): S[r][j] = sum_i U_S[r][i] E^T[j][i];
// per-(M-tile, key) packed argmax partials.  U [P][tp][np], Et [P][Tp][np].
hipError_t launch_assign_gemm(int dtype, const void *U, const void *Et, uint64_t *part, int P, int t, int64_t tp,
                              int64_t Tp, int64_t np_, hipStream_t s) {
  GemmShape g;
  g.batch = P;
  g.M = (int)tp;
  g.N = (int)Tp;
  g.K = (int)np_;
  g.a_pair = tp * np_;
  g.a_plane = 0;
  g.lda = np_;
  g.b_pair = Tp * np_;
  g.b_plane = 0;
  g.ldb = np_;
  g.syrk = false;
  g.group_m = 8;
  EpiArgmax e{part, (tp / kGBM) * Tp, (int)Tp, t};
  if (dtype == ARCKV_BF16) return launch_gemm<bf16, 1, 1>(g, (const bf16 *)U, (const bf16 *)Et, e, s);
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
    g.a_pair = g.b_pair = 2 * tp * np_;
    g.a_plane = g.b_plane = tp * np_;
    return launch_gemm<bf16, 2, 2>(g, (const bf16 *)X, (const bf16 *)X, e, s);
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
  EpiStore e{Bm, tp * kHeadDim, kHeadDim, nullptr, nullptr, nullptr};
  if (dtype == ARCKV_BF16) {
    g.a_pair = 2 * tp * np_;
    g.a_plane = tp * np_;
    g.b_pair = 2 * (int64_t)kHeadDim * np_;
    g.b_plane = (int64_t)kHeadDim * np_;
    return launch_gemm<bf16, 2, 2>(g, (const bf16 *)PT, (const bf16 *)YT, e, s);
  }
  g.a_pair = tp * np_;
  g.a_plane = 0;
  g.b_pair = (int64_t)kHeadDim * np_;
  g.b_plane = 0;
  return launch_gemm<float, 1, 1>(g, (const float *)PT, (const float *)YT, e, s);
}

// Refinement residual R = Bm - Gc X - lam X for 128 right-hand sides, fp32 MFMA.
// Gc [P][tp][tp], XT [P][128][tp] (X transposed), X / Bm / R [P][tp][128].
hipError_t launch_value_residual(const float *Gc, const float *XT, const float *Bm, const float *X,
                                 const float *lam, float *R, int P, int64_t tp, hipStream_t s) {
  GemmShape g;
  g.batch = P;
  g.M = (int)tp;
  g.N = kHeadDim;
  g.K = (int)tp;
  g.syrk = false;
  g.group_m = 8;
  g.a_pair = tp * tp;
  g.a_plane = 0;
  g.lda = tp;
  g.b_pair = (int64_t)kHeadDim * tp;
  g.b_plane = 0;
  g.ldb = tp;
  EpiStore e{R, tp * kHeadDim, kHeadDim, Bm, X, lam};
  return launch_gemm<float, 1, 1>(g, Gc, XT, e, s);
}

}  // namespace arckv
