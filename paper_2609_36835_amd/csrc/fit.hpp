// Per-pair state of the two ridge fits (fit.hip), shared by the kernels and
// the host-side stage sequencing.  All pointers are device arrays for one
// chunk of P pairs.
#pragma once
#include <stdint.h>

namespace arckv {

struct FitState {
  double *trace;   // [P] tr(M) of the unregularised Gram
  float *lam;      // [P] ridge lam = delta tr(M) / t
  float *delta;    // [P] relative ridge in use
  int32_t *nesc;   // [P] escalations taken (pivot failures and cut-off refinements)
  int32_t *info;   // [P] status (0 ok, > 0 failed pivot + 1, < 0 see arckv.h and fit.hip)
};

// Work arrays of the exact non-negative fit ([P][tp] unless noted).
struct NnlsWork {
  int32_t *F, *idx, *bidx, *pos;   // free flags, free and bound lists, slot of each key
  int32_t *nf, *nb;                // [P] free- and bound-set sizes
  int32_t *state;                  // [P][4]
  int32_t *red;                    // [2] max free-set size, unsettled pairs
  double *y, *rf, *xf;             // dual, compressed right-hand side and solution
};

// Buffers of the mass-fit solve with guarded refinement ([P][tp] doubles
// unless noted).
struct MassSolve {
  const float *LT;   // [P][tp][np] logits s Q C_k^T, transposed (zero beyond n)
  const float *z;    // [P][n] row maxima
  const float *m;    // [P][n] row masses
  const double *h;   // right-hand side Phi_C^T m
  double *w;         // solution
  double *x;         // last refinement correction
  double *y, *sw;    // triangular-solve work
  double *u;         // [P][np] data residual m - Phi_C w
  double *res;       // normal-equation residual
  double *rprev;     // [P] norm of the previous refinement correction
  int32_t *div;      // [P] pair to be refactored with a larger ridge
};

}  // namespace arckv
