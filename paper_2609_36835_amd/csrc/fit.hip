// Mass-bias and compact-value fits (Appendix A.9, eq. mass_fit, eq. value_lstsq).
//
// Both fits solve ridge-regularised normal equations (M + lam I) x = rhs with
// M a float32 Gram matrix of size tp (padded; the padding is an identity
// block with zero right-hand side, so padded unknowns solve to 0):
//   k_ridge_init     lam = delta * tr(M)/t, write M + lam I into the work copy
//   Cholesky         float32, left-looking over 256-wide outer panels:
//                      k_chol_scales  per-row power-of-two shifts s_r from the
//                                     diagonal (sqrt(A_rr) s_r in [2^13, 2^14))
//                      (contraction)  before a panel is factored, the big
//                                     contraction on fp16 MFMA applies every
//                                     earlier panel to it (hi / lo planes of
//                                     L s_r, three products, about 2^-22
//                                     relative)
//                      k_chol_diag    factor a 64 x 64 diagonal block and
//                                     invert it (1024 threads, four entries
//                                     of a row each, one barrier per column)
//                      k_chol_panel   L_ik = A_ik L_kk^-T inside the panel's
//                                     256 x 256 diagonal block (fp32 MFMA
//                                     with the inverse)
//                      k_chol_upd     A -= L L^T inside that block (fp32 MFMA)
//                      k_chol_strip16 the rows below it: the same panel steps
//                                     and updates on a 128 x 256 strip held in
//                                     LDS as hi / lo planes (fp16 MFMA), then
//                                     L and its planes written back
//                    a failed pivot records info = column + 1 for that pair
//   escalation       pairs that failed are refactored by the same kernels with
//                    delta raised tenfold (from 1e-7 when zero), at most
//                    max_escalations times (launch_cholesky)
//   solves           TRSV (one rhs, float64 accumulation) / TRSM (128 rhs; the
//                    forward one in 256-row blocks on the planes of L)
//   residuals        rhs - (M + lam I) x, float64 (mass fit) or float32 MFMA
//                    (value fit), for iterative refinement
#include "common.hpp"
#include "gemm.hpp"
#include "gemm_big.hpp"
#include "fit.hpp"

namespace arckv {

constexpr int kNB = 64;          // Cholesky block
constexpr int kSD = kNB + 1;     // LDS stride of a 64x64 fp32 tile

// --------------------------------------------------------------- ridge
// info starts at -1 for pairs flagged with non-finite inputs (bad, may be
// null), which every later kernel then skips, and 0 otherwise.
__global__ void __launch_bounds__(256) k_ridge_init(float *__restrict__ Gw, const float *__restrict__ Gc, int t,
                                                    int64_t ld, float delta0, FitState st,
                                                    const int32_t *__restrict__ bad) {
  __shared__ double red[4];
  const int b = blockIdx.x, tid = threadIdx.x;
  const size_t base = (size_t)b * ld * ld;
  double tr = 0.0;
  for (int r = tid; r < t; r += 256) tr += (double)Gc[base + (size_t)r * ld + r];
  tr = wave_sum(tr);
  if ((tid & 63) == 0) red[tid >> 6] = tr;
  __syncthreads();
  tr = red[0] + red[1] + red[2] + red[3];
  const float lam = (float)((double)delta0 * tr / (double)t);
  for (int64_t r = tid; r < ld; r += 256) Gw[base + (size_t)r * ld + r] = r < t ? Gc[base + (size_t)r * ld + r] + lam : 1.0f;
  if (tid == 0) {
    st.trace[b] = tr;
    st.lam[b] = lam;
    st.delta[b] = delta0;
    st.nesc[b] = 0;
    st.info[b] = bad && bad[b] ? -1 : 0;
  }
}

// ---------------------------------------------------------------- ridge escalation
// A pair whose factorisation failed (info > 0) is refactored with the ridge
// raised tenfold, from kDeltaFloor when it was zero, by the same batched
// blocked factorisation, while it has escalations left (nesc < max_esc); pairs
// that are settled carry kEscSkip meanwhile (every factorisation kernel skips
// info != 0), non-finite ones keep -1.
constexpr int32_t kEscSkip = -0x30000000;
constexpr float kDeltaFloor = 1e-7f;

__global__ void k_esc_state(int B, int t, FitState st, int max_esc) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const int32_t f = st.info[b];
  if (f > 0 && st.nesc[b] < max_esc) {
    const float delta = fmaxf(10.0f * st.delta[b], kDeltaFloor);
    st.delta[b] = delta;
    st.lam[b] = (float)((double)delta * st.trace[b] / (double)t);
    st.nesc[b] += 1;
    st.info[b] = 0;
  } else if (f == 0) {
    st.info[b] = kEscSkip;
  }
}

// Gw = Gc + lam I (lower triangle and diagonal; padding diagonal 1) for the
// pairs being refactored (info == 0).  One row per thread-block row.
__global__ void __launch_bounds__(256) k_esc_copy(float *__restrict__ Gw, const float *__restrict__ Gc, int t,
                                                  int64_t ld, FitState st) {
  const int b = blockIdx.y;
  const int64_t r = blockIdx.x;
  if (st.info[b] != 0) return;
  const float lam = st.lam[b];
  const size_t base = (size_t)b * ld * ld + (size_t)r * ld;
  for (int64_t c = threadIdx.x; c <= r; c += 256)
    Gw[base + c] = c == r ? (r < t ? Gc[base + c] + lam : 1.0f) : Gc[base + c];
}

__global__ void k_esc_restore(int B, int32_t *__restrict__ info) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < B && info[b] == kEscSkip) info[b] = 0;
}

// cnt[0] = number of pairs whose factorisation failed (info > 0) and that
// have escalations left.
__global__ void __launch_bounds__(256) k_count_failed(int B, const FitState st, int max_esc, int32_t *cnt) {
  __shared__ int red[4];
  int c = 0;
  for (int b = threadIdx.x; b < B; b += 256) c += st.info[b] > 0 && st.nesc[b] < max_esc;
  for (int m = 32; m >= 1; m >>= 1) c += __shfl_xor(c, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) cnt[0] = red[0] + red[1] + red[2] + red[3];
}

// ---------------------------------------------------------------- refinement guard
// Each refinement step recomputes the residual from the data, so it converges
// at a rate set by how far the float32 factor is from those normal equations.
// Where the ridge is small next to the Gram's float32 rounding (a
// rank-deficient Gram, t > n, with a ridge near 1e-6 of its mean diagonal) the
// steps instead grow the solution along the Gram's near-null directions.  After
// every step but the first the correction is compared with the previous one:
// a correction above 1e-10 |w| that is not at most half the previous one is
// undone and ends the pair's refinement (kRefStop); while it has escalations
// left the pair is then refactored with the ridge raised tenfold and solved
// again (div).  Pairs not being refactored meanwhile carry kDoneSkip.
constexpr int32_t kRefStop = -0x20000000;
constexpr int32_t kDoneSkip = -0x10000000;

// One workgroup per pair, after step it (w already holds w + x); it = 0 records
// the first correction's norm.
__global__ void __launch_bounds__(256) k_refine_watch(double *__restrict__ w, const double *__restrict__ x,
                                                      int64_t tp, int it, double *__restrict__ xprev,
                                                      int32_t *__restrict__ div, FitState st, int max_esc) {
  __shared__ double red[2][4];
  const int b = blockIdx.x, tid = threadIdx.x;
  if (st.info[b] != 0) return;
  const double xp = xprev[b];   // read by every thread before thread 0 rewrites it
  const size_t o = (size_t)b * tp;
  double x2 = 0.0, w2 = 0.0;
  for (int64_t r = tid; r < tp; r += 256) {
    const double a = x[o + r], c = w[o + r];
    x2 = fma(a, a, x2);
    w2 = fma(c, c, w2);
  }
  x2 = wave_sum(x2);
  w2 = wave_sum(w2);
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = x2;
    red[1][tid >> 6] = w2;
  }
  __syncthreads();
  const double xn = sqrt(red[0][0] + red[0][1] + red[0][2] + red[0][3]);
  const double wn = sqrt(red[1][0] + red[1][1] + red[1][2] + red[1][3]);
  if (it == 0 || !(xn > 0.5 * xp && xn > 1e-10 * wn)) {
    if (tid == 0) xprev[b] = xn;
    return;
  }
  for (int64_t r = tid; r < tp; r += 256) w[o + r] -= x[o + r];
  if (tid == 0) {
    st.info[b] = kRefStop;
    div[b] = st.nesc[b] < max_esc;
  }
}

// cnt[0] = number of nonzero flags.
__global__ void __launch_bounds__(256) k_count_flags(int B, const int32_t *__restrict__ flag, int32_t *cnt) {
  __shared__ int red[4];
  int c = 0;
  for (int b = threadIdx.x; b < B; b += 256) c += flag[b] != 0;
  for (int m = 32; m >= 1; m >>= 1) c += __shfl_xor(c, m, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) cnt[0] = red[0] + red[1] + red[2] + red[3];
}

// Pairs to refactor get info = 1 (picked up by k_esc_state); the settled rest kDoneSkip.
__global__ void k_div_mark(int B, int32_t *__restrict__ div, int32_t *__restrict__ info) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const int32_t f = info[b];
  if (div[b]) {
    info[b] = 1;
    div[b] = 0;
  } else if (f == 0 || f == kRefStop) {
    info[b] = kDoneSkip;
  }
}

__global__ void k_refine_restore(int B, int32_t *__restrict__ info) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < B && (info[b] == kRefStop || info[b] == kDoneSkip)) info[b] = 0;
}

// ---------------------------------------------------------------- non-finite inputs
// bad[b] |= 1 when any of the `per` values of pair b in a is not finite (a
// grid-stride pass over [B][per]; bad is cleared by the caller).
__global__ void __launch_bounds__(256) k_nonfinite(const float *__restrict__ a, int64_t per, int32_t *__restrict__ bad) {
  const int b = blockIdx.y;
  bool any = false;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < per; i += (int64_t)gridDim.x * 256)
    any |= !isfinite(a[(size_t)b * per + i]);
  if (__any(any) && (threadIdx.x & 63) == 0) atomicOr(&bad[b], 1);
}

// Factor the 64 x 64 diagonal block k in place and write L_kk^-1 to
// dinv[b][k] (one workgroup of 256 threads per pair).  Thread (r, cls) with
// r = tid / 4, cls = tid % 4 keeps A[r][4j + cls] (j < 16) in registers.
// Threads of k_chol_diag: 64 rows x kDiagCls column classes, each thread
// holding kDiagPer entries of its row (four waves per SIMD hide each other's
// latency along the per-column dependence chain).
constexpr int kDiagCls = 16, kDiagPer = kNB / kDiagCls, kDiagThreads = kNB * kDiagCls;

// Right-looking over the 64 columns c with one barrier per column: column c,
// updated through column c - 1 but not yet scaled, sits in LDS (its owners
// publish it right after their own update of step c - 1), so every thread
// reads the pivot, takes d = sqrt and 1 / d itself, scales the entries it
// needs, L[x][c] = A'[x][c] / d, and subtracts L[r][c] L[q][c] from its
// entries.  The inverse X = L^-1 is an elimination on the identity in the
// same loop: row c of X is row c of the updated identity times 1 / d,
// published at step c, and rows below subtract L[r][c] X[c][q] one step
// later, when that row is visible.  Both recurrences accumulate in column
// order with the same products and fused multiply-adds as a plain
// column-by-column factorisation and row-by-row substitution.  A failed pivot
// records info = column + 1 and leaves the block and dinv unwritten.
__global__ void __launch_bounds__(kDiagThreads) k_chol_diag(float *__restrict__ Gw, int64_t ld, int k,
                                                   int32_t *__restrict__ info, float *__restrict__ dinv) {
  __shared__ float sA[kNB * kSD];   // column c: A updated through column c - 1, unscaled
  __shared__ float sX[kNB * kSD];   // L^-1, one row per column step
  __shared__ float sd[kNB], sdg[kNB];   // 1 / L[c][c] and L[c][c]
  const int b = blockIdx.x, tid = threadIdx.x;
  if (info[b] != 0) return;   // uniform over the workgroup
  const int r = tid / kDiagCls, cls = tid % kDiagCls;
  float *D = Gw + (size_t)b * ld * ld + (size_t)k * kNB * ld + (size_t)k * kNB;
  for (int e = tid; e < kNB * kNB / 4; e += kDiagThreads) {
    const int rr = e >> 4, c4 = (e & 15) * 4;
    const f32x4 v = *reinterpret_cast<const f32x4 *>(D + (size_t)rr * ld + c4);
#pragma unroll
    for (int q = 0; q < 4; ++q) sA[rr * kSD + c4 + q] = v[q];
  }
  __syncthreads();
  // Each thread reads only its own entries, and column 0 needs no update.
  float a[kDiagPer], y[kDiagPer];
#pragma unroll
  for (int j = 0; j < kDiagPer; ++j) {
    const int q = kDiagCls * j + cls;
    a[j] = sA[r * kSD + q];
    y[j] = q == r ? 1.0f : 0.0f;
  }
  int fail = 0;
  float plrc = 0.0f;   // L[r][c - 1]
#pragma unroll 1
  for (int c = 0; c < kNB; ++c) {
    const float piv = sA[c * kSD + c];
    const float arc = sA[r * kSD + c];
    float col[kDiagPer], xp[kDiagPer];
#pragma unroll
    for (int j = 0; j < kDiagPer; ++j) col[j] = sA[(kDiagCls * j + cls) * kSD + c];
    if (c > 0) {
#pragma unroll
      for (int j = 0; j < kDiagPer; ++j) xp[j] = sX[(c - 1) * kSD + kDiagCls * j + cls];
    }
    if (!(piv > 0.0f) || !isfinite(piv)) {   // uniform: every thread read the same pivot
      fail = c + 1;
      break;
    }
    const float d = sqrtf(piv), inv = 1.0f / d;
    if (c > 0 && r >= c) {
#pragma unroll
      for (int j = 0; j < kDiagPer; ++j) y[j] = fmaf(-plrc, xp[j], y[j]);
    }
    if (r == c) {
#pragma unroll
      for (int j = 0; j < kDiagPer; ++j) sX[c * kSD + kDiagCls * j + cls] = y[j] * inv;
    }
    const float lrc = arc * inv;
    if (r > c) {
#pragma unroll
      for (int j = 0; j < kDiagPer; ++j) a[j] = fmaf(-lrc, col[j] * inv, a[j]);
    }
    plrc = lrc;
    if (c + 1 < kNB && cls == (c + 1) % kDiagCls) {
      const int jn = (c + 1) / kDiagCls;
      float v = a[0];
#pragma unroll
      for (int j = 1; j < kDiagPer; ++j) v = j == jn ? a[j] : v;
      sA[r * kSD + c + 1] = v;
    }
    if (tid == 0) {
      sd[c] = inv;
      sdg[c] = d;
    }
    __syncthreads();
  }
  if (fail) {
    if (tid == 0) info[b] = k * kNB + fail;
    return;
  }
  float *Xi = dinv + ((size_t)b * (ld / kNB) + k) * kNB * kNB;
  for (int e = tid; e < kNB * kNB; e += kDiagThreads) {
    const int rr = e >> 6, q = e & 63;
    if (q < rr) D[(size_t)rr * ld + q] = sA[rr * kSD + q] * sd[q];
    else if (q == rr) D[(size_t)rr * ld + q] = sdg[q];
    Xi[e] = sX[rr * kSD + q];
  }
}

// Panel: L_ik = A_ik L_kk^-T for the rows below diagonal block k up to row
// r_end, as an fp32 MFMA product with the inverse from k_chol_diag.  A
// workgroup takes 128 rows (4 waves x 32 rows x 64 columns).
__global__ void __launch_bounds__(256) k_chol_panel(float *__restrict__ Gw, int64_t ld, int k, int64_t r_end,
                                                    const float *__restrict__ dinv,
                                                    const int32_t *__restrict__ info) {
  __shared__ float sLi[kNB * kSD], sA[128 * kSD];
  const int b = blockIdx.y;
  if (info[b] != 0) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, h = lane >> 5, col = lane & 31;
  const int64_t rb = (int64_t)(k + 1) * kNB + 128 * (int64_t)blockIdx.x;
  float *G = Gw + (size_t)b * ld * ld;
  const float *Li = dinv + ((size_t)b * (ld / kNB) + k) * kNB * kNB;
  for (int e = tid; e < kNB * kNB / 4; e += 256) {
    const int r = e / 16, c4 = (e % 16) * 4;
    const f32x4 v = *reinterpret_cast<const f32x4 *>(Li + r * kNB + c4);
#pragma unroll
    for (int q = 0; q < 4; ++q) sLi[r * kSD + c4 + q] = v[q];
  }
  for (int e = tid; e < 128 * kNB / 4; e += 256) {
    const int r = e / 16, c4 = (e % 16) * 4;
    f32x4 v = {0.f, 0.f, 0.f, 0.f};
    if (rb + r < r_end) v = *reinterpret_cast<const f32x4 *>(G + (size_t)(rb + r) * ld + (size_t)k * kNB + c4);
#pragma unroll
    for (int q = 0; q < 4; ++q) sA[r * kSD + c4 + q] = v[q];
  }
  __syncthreads();
  f32x16 acc0 = zero16(), acc1 = zero16();
#pragma unroll
  for (int ks = 0; ks < kNB / 2; ++ks) {
    const float fa = sA[(32 * wave + col) * kSD + 2 * ks + h];
    acc0 = Mfma<float>::mma(fa, sLi[col * kSD + 2 * ks + h], acc0);
    acc1 = Mfma<float>::mma(fa, sLi[(32 + col) * kSD + 2 * ks + h], acc1);
  }
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int64_t r = rb + 32 * wave + acc_row(v, lane);
    if (r < r_end) {
      G[(size_t)r * ld + (size_t)k * kNB + col] = acc0[v];
      G[(size_t)r * ld + (size_t)k * kNB + 32 + col] = acc1[v];
    }
  }
}

// Trailing update of the blocked factorisation on fp32 MFMA:
//   G[r][c] -= sum_{q in [q0, q0+kw)} L[r][q] L[c][q]
// for r in [r_lo, r_hi), c in [r_lo, c_hi), c <= r (up to the 64-wide diagonal
// block), with 128 x 128 output tiles (4 waves of 64 x 64).  Only tiles on or
// below the diagonal are launched: row tile ti holds column tiles
// tj < min(ti + 1, n_ct); workgroups are remapped so each XCD owns a
// contiguous range of (pair, tile).  The L operands are the finished panel
// columns [q0, q0+kw), streamed through LDS in slabs of 32.
__device__ inline void chol_upd_tile(int64_t idx, int n_ct, int &ti, int &tj) {
  const int64_t tri = (int64_t)n_ct * (n_ct + 1) / 2;
  if (idx < tri) {
    int m = (int)((sqrt(8.0 * (double)idx + 1.0) - 1.0) * 0.5);
    while ((int64_t)m * (m + 1) / 2 > idx) --m;
    while ((int64_t)(m + 1) * (m + 2) / 2 <= idx) ++m;
    ti = m;
    tj = (int)(idx - (int64_t)m * (m + 1) / 2);
  } else {
    const int64_t r = idx - tri;
    ti = n_ct + (int)(r / n_ct);
    tj = (int)(r % n_ct);
  }
}

__host__ __device__ inline int64_t chol_upd_tiles(int n_rt, int n_ct) {
  return (int64_t)n_ct * (n_ct + 1) / 2 + (int64_t)(n_rt - n_ct) * n_ct;
}

__global__ void __launch_bounds__(256) k_chol_upd(float *__restrict__ Gw, int64_t ld, int r_lo, int r_hi, int c_hi,
                                                  int q0, int kw, int n_rt, int n_ct,
                                                  const int32_t *__restrict__ info) {
  // LDS rows of 33 floats: the 4-byte fragment reads of 32 consecutive rows
  // then fall in 32 distinct banks.  Two buffers; the next slab is fetched into
  // registers while the current one is consumed.
  constexpr int TB = 128, BKc = 32, SLc = BKc + 1, CHc = TB * BKc / 4 / 256;
  __shared__ float sA[2][TB * SLc], sB[2][TB * SLc];
  const int64_t per = chol_upd_tiles(n_rt, n_ct);
  const int64_t tile = xcd_remap(blockIdx.x, gridDim.x);
  const int b = (int)(tile / per);
  if (info[b] != 0) return;
  int ti, tj;
  chol_upd_tile(tile % per, n_ct, ti, tj);
  const int rb = r_lo + TB * ti, cb = r_lo + TB * tj;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, col = lane & 31;
  float *G = Gw + (size_t)b * ld * ld;
  f32x4 ra[CHc], rbv[CHc];
  auto fetch = [&](int kq) {
#pragma unroll
    for (int c = 0; c < CHc; ++c) {
      const int e = tid + 256 * c, r = e / (BKc / 4), c4 = (e % (BKc / 4)) * 4;
      const int row_a = rb + r, row_b = cb + r;
      ra[c] = f32x4{0.f, 0.f, 0.f, 0.f};
      rbv[c] = ra[c];
      if (row_a < r_hi) ra[c] = *reinterpret_cast<const f32x4 *>(G + (size_t)row_a * ld + q0 + kq + c4);
      if (row_b < c_hi) rbv[c] = *reinterpret_cast<const f32x4 *>(G + (size_t)row_b * ld + q0 + kq + c4);
    }
  };
  auto stash = [&](int bf) {
#pragma unroll
    for (int c = 0; c < CHc; ++c) {
      const int e = tid + 256 * c, r = e / (BKc / 4), c4 = (e % (BKc / 4)) * 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        sA[bf][r * SLc + c4 + q] = ra[c][q];
        sB[bf][r * SLc + c4 + q] = rbv[c][q];
      }
    }
  };
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = zero16();
  fetch(0);
  stash(0);
  __syncthreads();
  int bf = 0;
  for (int kq = 0; kq < kw; kq += BKc) {
    const bool more = kq + BKc < kw;
    if (more) fetch(kq + BKc);
#pragma unroll
    for (int ks = 0; ks < BKc / 2; ++ks) {
      float fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fa[i] = sA[bf][(wm * 64 + 32 * i + col) * SLc + 2 * ks + h];
        fb[i] = sB[bf][(wn * 64 + 32 * i + col) * SLc + 2 * ks + h];
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = Mfma<float>::mma(fa[i], fb[j], acc[i][j]);
    }
    if (more) stash(bf ^ 1);
    __syncthreads();
    bf ^= 1;
  }
  // Read-modify-write of the tile: every old value is loaded (unconditionally,
  // from a clamped in-range address) before any store, so the loads pipeline
  // instead of paying one memory round trip each.
  const int64_t lm = ld - 1;
  float old[2][2][16];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t c = cb + wn * 64 + 32 * j + col, cc = c < lm ? c : lm;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t r = rb + wm * 64 + 32 * i + acc_row(v, lane), rr = r < lm ? r : lm;
        old[i][j][v] = __builtin_nontemporal_load(&G[rr * ld + cc]);
      }
    }
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = cb + wn * 64 + 32 * j + col;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = rb + wm * 64 + 32 * i + acc_row(v, lane);
        if (r < r_hi && c < c_hi && c <= r + 63) G[(size_t)r * ld + c] = old[i][j][v] - acc[i][j][v];
      }
    }
}

// Left-looking update of the column panel K0 .. K0 + 255:
// G[K0 + r][K0 + c] -= acc s_r s_c for the tile's entries with c <= r + 63
// (the lower triangle, up to whole diagonal 64-blocks), s the rows' inverse
// scales 2^-shift (k_chol_scales; 256 x 256 tiles, 512 threads); per row
// block of the wave, every old value is loaded before any store so the loads
// pipeline.
template <int TM, int TN>
struct EpiCholUpd {
  float *G;
  int64_t ld;
  int K0;
  const int32_t *info;
  const float *rs;        // inverse scales of pair 0, rows from K0
  int64_t rs_pair;        // floats between pairs
  __device__ __forceinline__ bool skip(int p) const { return info[p] != 0; }
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int mt, int nt,
                                             int lane, int, int) const {
    if (info[p] != 0) return;   // uniform over the workgroup
    // the tile's 256 row and 256 column scales, staged in LDS (the operand
    // stages are free: the caller synchronised the workgroup before the epilogue)
    extern __shared__ __attribute__((aligned(1024))) char big_smem[];
    float *ssc = reinterpret_cast<float *>(big_smem);
    const float *sp = rs + (size_t)p * rs_pair;
    for (int x = threadIdx.x; x < 512; x += blockDim.x) ssc[x] = sp[(x < 256 ? mt : nt) * 256 + (x & 255)];
    __syncthreads();
    float *Gp = G + (size_t)p * ld * ld + (size_t)K0 * ld + K0;
    const int col = lane & 31, rl = row0 - mt * 256, cl = col0 - nt * 256;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      float old[TN][16];
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = row0 + 32 * i + acc_row(v, lane), c = col0 + 32 * j + col;
          old[j][v] = __builtin_nontemporal_load(&Gp[(size_t)r * ld + c]);
        }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const float scj = ssc[256 + cl + 32 * j + col];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int r = row0 + 32 * i + acc_row(v, lane), c = col0 + 32 * j + col;
          const float sr = ssc[rl + 32 * i + acc_row(v, lane)];
          if (c <= r + 63) Gp[(size_t)r * ld + c] = old[j][v] - acc[i][j][v] * (sr * scj);
        }
      }
    }
  }
};

// Rows K1 .. ld of the outer panel (columns K0 .. K1 = K0 + 256), once its
// 256 x 256 diagonal block is factored: for each 64-column block k in order,
// the panel step L_rk = A_rk L_kk^-T (with the stored inverse), then the
// update of the panel's later blocks j, A_rj -= L_rk L_jk^T; then the rows' L
// is written back with the fp16 hi / lo planes of the left-looking updates'
// operand.  A workgroup of 8 waves keeps 128 rows x 256 columns in LDS, so
// the strip is read and written once instead of once per step; each
// 128 x 64 product is 4 x 2 waves of 32 x 32.
constexpr int kStripRows = 128;

// k_chol_strip16: the strip on fp16 MFMA (32x32x16), every product as hi.hi + hi.lo +
// lo.hi of fp16 planes (about 2^-22 relative, as in the trailing
// contraction).  With s_x = 2^shift[x] (sqrt(A_xx) s_x in [2^13, 2^14)):
//  - an entry of a block not yet factored, |A'_rc| <= sqrt(A_rr A_cc), is held
//    as A'_rc s_r s_c 2^-14, a factored one, |L_rc| <= sqrt(A_rr), as L_rc s_r,
//    both below 2^14, as hi / lo planes in LDS;
//  - the B operand rows (D_k with its columns m scaled by 2^14 / s_m, or L_jk)
//    are split after scaling each row by the power of two that brings its
//    largest magnitude into [2^13, 2^14);
//  - an update recombines hi + lo in fp32, subtracts and splits again.
// The planes left in LDS are the split the left-looking contractions read,
// and G gets (hi + lo) / s_r.  LDS rows are unpadded with their 16-byte chunks XOR-swizzled by
// row, so each quarter-wave's fragment reads touch 16 distinct bank groups.
constexpr size_t kStrip16Lds = ((size_t)2 * kStripRows * 256 + (size_t)2 * kNB * kNB) * sizeof(f16) +
                               (size_t)(kNB + kStripRows + 256) * sizeof(int32_t);

__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_chol_strip16(float *__restrict__ Gw, int64_t ld, int K0, const float *__restrict__ dinv, f16 *__restrict__ Lp,
               const int32_t *__restrict__ shift, const int32_t *__restrict__ info) {
  extern __shared__ __attribute__((aligned(16))) char strip16_smem[];
  f16 *sTh = reinterpret_cast<f16 *>(strip16_smem);        // [128][256] hi
  f16 *sTl = sTh + kStripRows * 256;                         // [128][256] lo
  f16 *sBh = sTl + kStripRows * 256;                         // [64][64] hi
  f16 *sBl = sBh + kNB * kNB;                                // [64][64] lo
  int32_t *sBe = reinterpret_cast<int32_t *>(sBl + kNB * kNB);   // [64] row exponents of B
  int32_t *sSh = sBe + kNB;                                  // [128] row shifts of the strip
  int32_t *sShC = sSh + kStripRows;                          // [256] shifts of the panel's columns
  const int b = blockIdx.y;
  if (info[b] != 0) return;   // uniform over the workgroup
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, col = lane & 31;
  const int K1 = K0 + 256;
  const int64_t R = K1 + (int64_t)blockIdx.x * kStripRows;
  float *G = Gw + (size_t)b * ld * ld;
  const int nb = (int)(ld / kNB);
  // element (r, c) of a plane: T rows of 32 chunks, B rows of 8 chunks
  auto tix = [](int r, int c) { return r * 256 + 8 * ((c >> 3) ^ (r & 15)) + (c & 7); };
  auto bix = [](int i, int m) { return i * kNB + 8 * ((m >> 3) ^ ((i >> 1) & 7)) + (m & 7); };
  auto split4 = [](f32x4 x, f16x4 &hi, f16x4 &lo) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      hi[q] = (f16)x[q];
      lo[q] = (f16)(x[q] - (float)hi[q]);
    }
  };
  if (tid < kStripRows) sSh[tid] = shift[(size_t)b * ld + R + tid];
  if (tid < 256) sShC[tid] = shift[(size_t)b * ld + K0 + tid];
  constexpr int kSteps = 10;
  constexpr int8_t step_k[kSteps] = {0, 0, 0, 0, 1, 1, 1, 2, 2, 3};
  constexpr int8_t step_j[kSteps] = {0, 1, 2, 3, 1, 2, 3, 2, 3, 3};
  f32x4 pre[2];
  auto load_b = [&](int st) {
    const int k = step_k[st], j = step_j[st];
    const float *src = j == k ? dinv + ((size_t)b * nb + K0 / kNB + k) * kNB * kNB
                              : G + (size_t)(K0 + kNB * j) * ld + K0 + kNB * k;
    const int64_t lds = j == k ? kNB : ld;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int e = tid + 512 * c, i = e >> 4, c4 = (e & 15) * 4;
      pre[c] = *reinterpret_cast<const f32x4 *>(src + (size_t)i * lds + c4);
    }
  };
  // B rows scaled by their own power of two (16 consecutive lanes hold a row);
  // for D_k its columns first take 2^14 / s_m
  auto stash_b = [&](int k, bool panel) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int e = tid + 512 * c, i = e >> 4, c4 = (e & 15) * 4;
      if (panel) {
#pragma unroll
        for (int q = 0; q < 4; ++q) pre[c][q] = ldexpf(pre[c][q], 14 - sShC[64 * k + c4 + q]);
      }
      float m = fmaxf(fmaxf(fabsf(pre[c][0]), fabsf(pre[c][1])), fmaxf(fabsf(pre[c][2]), fabsf(pre[c][3])));
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
      int ex = 0;
      if (m > 0.0f) frexpf(m, &ex);
      const int sc = max(min(14 - ex, 126), -126);
      f32x4 x;
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = ldexpf(pre[c][q], sc);
      f16x4 hi, lo;
      split4(x, hi, lo);
      *reinterpret_cast<f16x4 *>(&sBh[bix(i, c4)]) = hi;
      *reinterpret_cast<f16x4 *>(&sBl[bix(i, c4)]) = lo;
      if ((e & 15) == 0) sBe[i] = sc;
    }
  };
  // this wave's 32 x 32 block of T[:, 64 ka ..] x B^T, in the scaled units
  const int arow = 32 * wm + col, brow = 32 * wn + col;
  auto product = [&](int ka) {
    f32x16 acc = zero16();
#pragma unroll
    for (int ks = 0; ks < kNB / 16; ++ks) {
      const int ca = 64 * ka + 16 * ks + 8 * h, cb = 16 * ks + 8 * h;
      const bf16x8 ah = *reinterpret_cast<const bf16x8 *>(&sTh[tix(arow, ca)]);
      const bf16x8 al = *reinterpret_cast<const bf16x8 *>(&sTl[tix(arow, ca)]);
      const bf16x8 bh = *reinterpret_cast<const bf16x8 *>(&sBh[bix(brow, cb)]);
      const bf16x8 bl = *reinterpret_cast<const bf16x8 *>(&sBl[bix(brow, cb)]);
      acc = mma16<f16>(ah, bh, acc);
      acc = mma16<f16>(ah, bl, acc);
      acc = mma16<f16>(al, bh, acc);
    }
    return acc;
  };
  {  // the strip, 128 rows x 64 groups of 4, scaled by s_r s_c 2^-14 and split
    f32x4 v[kStripRows * 64 / 512];
#pragma unroll
    for (int i = 0; i < kStripRows * 64 / 512; ++i) {
      const int e = tid + 512 * i, r = e >> 6, c4 = (e & 63) * 4;
      v[i] = *reinterpret_cast<const f32x4 *>(G + (size_t)(R + r) * ld + K0 + c4);
    }
    load_b(0);
    __syncthreads();   // sSh, sShC
#pragma unroll
    for (int i = 0; i < kStripRows * 64 / 512; ++i) {
      const int e = tid + 512 * i, r = e >> 6, c4 = (e & 63) * 4;
      const int sh = sSh[r] - 14;
      f32x4 x;
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = ldexpf(v[i][q], sh + sShC[c4 + q]);
      f16x4 hi, lo;
      split4(x, hi, lo);
      *reinterpret_cast<f16x4 *>(&sTh[tix(r, c4)]) = hi;
      *reinterpret_cast<f16x4 *>(&sTl[tix(r, c4)]) = lo;
    }
  }
  // block kb (final after its panel step): planes and L = (hi + lo) / s_r of
  // all 128 rows, four columns per thread-group, issued while later steps run
  f16 *hib = Lp + (size_t)b * 2 * ld * ld, *lob = hib + (size_t)ld * ld;
  auto write_block = [&](int kb) {
#pragma unroll
    for (int q = 0; q < kStripRows * 16 / 512; ++q) {
      const int g = tid + 512 * q, rr = g >> 4, c = 64 * kb + (g & 15) * 4;
      const int64_t r = R + rr;
      const f16x4 hi = *reinterpret_cast<const f16x4 *>(&sTh[tix(rr, c)]);
      const f16x4 lo = *reinterpret_cast<const f16x4 *>(&sTl[tix(rr, c)]);
      const float us = ldexpf(1.0f, -sSh[rr]);
      f32x4 x;
#pragma unroll
      for (int u = 0; u < 4; ++u) x[u] = ((float)hi[u] + (float)lo[u]) * us;
      *reinterpret_cast<f32x4 *>(G + (size_t)r * ld + K0 + c) = x;
      *reinterpret_cast<f16x4 *>(hib + (size_t)r * ld + K0 + c) = hi;
      *reinterpret_cast<f16x4 *>(lob + (size_t)r * ld + K0 + c) = lo;
    }
  };
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
    const int k = step_k[st], j = step_j[st];
    __syncthreads();   // the strip is up to date and every wave is done with sB
    if (st > 0 && step_j[st - 1] == step_k[st - 1]) write_block(step_k[st - 1]);
    stash_b(k, j == k);
    if (st + 1 < kSteps) load_b(st + 1);
    __syncthreads();
    const f32x16 acc = product(k);
    if (j == k) {      // panel step: L_k s_r replaces block k
      const float inv_b = ldexpf(1.0f, -sBe[brow]);
      __syncthreads();
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 32 * wm + acc_row(v, lane), c = 64 * k + 32 * wn + col;
        const float x = acc[v] * inv_b;
        const f16 hi = (f16)x;
        sTh[tix(r, c)] = hi;
        sTl[tix(r, c)] = (f16)(x - (float)hi);
      }
    } else {           // update of block j (this wave's own entries), in its units s_r s_c 2^-14
      const float inv_b = ldexpf(1.0f, sShC[64 * j + brow] - 14 - sBe[brow]);
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int r = 32 * wm + acc_row(v, lane), c = 64 * j + 32 * wn + col;
        const float x = ((float)sTh[tix(r, c)] + (float)sTl[tix(r, c)]) - acc[v] * inv_b;
        const f16 hi = (f16)x;
        sTh[tix(r, c)] = hi;
        sTl[tix(r, c)] = (f16)(x - (float)hi);
      }
    }
  }
  __syncthreads();
  write_block(step_k[kSteps - 1]);   // the last panel step's block
}

// Per-row shifts of the left-looking updates' operand.  |L_rk| <= sqrt(A_rr)
// for every k (row r of L L^T = A), so 2^sh with sqrt(A_rr) 2^sh in
// [2^13, 2^14) keeps every scaled entry of the row below 2^14, inside fp16's
// range with the lo part carrying the next 11 bits; one shift per row for the
// whole factorisation lets a contraction run over all earlier panels at once.
// shift[r] = sh, inv[r] = 2^-sh (rows of a non-positive diagonal get 0: their
// factorisation fails at that pivot).
__global__ void __launch_bounds__(256) k_chol_scales(const float *__restrict__ Gw, int64_t ld,
                                                     int32_t *__restrict__ shift, float *__restrict__ inv,
                                                     const int32_t *__restrict__ info) {
  const int b = blockIdx.y;
  if (info[b] != 0) return;
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= ld) return;
  const float d = Gw[(size_t)b * ld * ld + (size_t)r * ld + r];
  int sh = 0;
  if (d > 0.0f && isfinite(d)) {
    int ex = 0;
    frexpf(sqrtf(d), &ex);   // sqrt(d) = f 2^ex, f in [0.5, 1)
    sh = max(min(14 - ex, 126), -126);
  }
  shift[(size_t)b * ld + r] = sh;
  inv[(size_t)b * ld + r] = ldexpf(1.0f, -sh);
}

// --------------------------------------------------------------- one right-hand side
// One-rhs triangular solves, float64 vectors, right-looking over 64-row
// blocks with one launch per block j, so that every block row below (forward)
// or above (backward) is updated by its own workgroup:
//   forward  L y = rhs:   y_j = D_j s_j,   s_i -= L_ij y_j      (i > j)
//   backward L^T x = y:   x_j = D_j^T y_j, y_i -= L_ji^T x_j    (i < j)
// D_j is the inverse of diagonal block j from the factorisation.  Each
// workgroup recomputes the block solution (a 64 x 64 product) and updates its
// target block; workgroup 0 also writes the solution (and adds it to `acc` on
// the backward pass when given).  Forward step 0 reads the rhs, later steps the
// work vector s; the backward pass updates y in place.
template <bool FWD>
__global__ void __launch_bounds__(256) k_trsv_step(const float *__restrict__ Gw, const float *__restrict__ dinv,
                                                   int64_t ld, int j, const double *__restrict__ rhs,
                                                   double *__restrict__ work, double *__restrict__ out,
                                                   double *__restrict__ acc, const int32_t *__restrict__ info) {
  __shared__ double sv[kNB], sol[kNB], red[4][kNB];
  const int b = blockIdx.y, g = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (info[b] != 0) return;
  const int nb = (int)(ld / kNB);
  const int i = FWD ? j + 1 + g : g;                       // target block
  const bool has_target = FWD ? i < nb : i < j;
  const float *L = Gw + (size_t)b * ld * ld;
  const float *D = dinv + ((size_t)b * nb + j) * kNB * kNB;
  const double *src = (FWD && j == 0) ? rhs + (size_t)b * ld : work + (size_t)b * ld;
  if (tid < kNB) sv[tid] = src[(size_t)j * kNB + tid];
  __syncthreads();
  if constexpr (FWD) {
    // row-major tiles: four lanes per row, each over 16 contiguous columns
    // (16-byte loads); a lane's partial is the sum the column-quarter took in
    // the transposed form, and the quarters meet in the same order
    const int rr = tid >> 2, qs = tid & 3;
    auto rowdot = [&](const float *row, const double *vec) {
      double pr = 0.0;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const f32x4 v = *reinterpret_cast<const f32x4 *>(row + 16 * qs + 4 * c);
#pragma unroll
        for (int q = 0; q < 4; ++q) pr += (double)v[q] * vec[16 * qs + 4 * c + q];
      }
      const double p1 = __shfl_down(pr, 1, 4), p2 = __shfl_down(pr, 2, 4), p3 = __shfl_down(pr, 3, 4);
      return ((pr + p1) + p2) + p3;   // valid in the row's first lane
    };
    const double sr = rowdot(D + rr * kNB, sv);
    if (qs == 0) sol[rr] = sr;
    __syncthreads();
    if (g == 0 && tid < kNB) out[(size_t)b * ld + (size_t)j * kNB + tid] = sol[tid];
    if (!has_target) return;
    const double ur = rowdot(L + ((size_t)i * kNB + rr) * ld + (size_t)j * kNB, sol);
    if (qs == 0) {
      const size_t e = (size_t)b * ld + (size_t)i * kNB + rr;
      const double base = j == 0 ? rhs[e] : work[e];
      work[e] = base - ur;
    }
    return;
  }
  double part = 0.0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int q = 16 * wave + e;
    part += (double)D[q * kNB + lane] * sv[q];
  }
  red[wave][lane] = part;
  __syncthreads();
  if (tid < kNB) sol[tid] = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
  __syncthreads();
  if (g == 0 && tid < kNB) {
    out[(size_t)b * ld + (size_t)j * kNB + tid] = sol[tid];
    if (!FWD && acc) acc[(size_t)b * ld + (size_t)j * kNB + tid] += sol[tid];
  }
  if (!has_target) return;
  part = 0.0;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int q = 16 * wave + e;
    part += (double)L[((size_t)j * kNB + q) * ld + (size_t)i * kNB + lane] * sol[q];
  }
  red[wave][lane] = part;     // red is free: every thread read it before the last barrier
  __syncthreads();
  if (tid < kNB) {
    const size_t e = (size_t)b * ld + (size_t)i * kNB + tid;
    work[e] = work[e] - (red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid]);
  }
}

// Refinement residual of the mass fit computed from the data, not from the
// float32 Gram: res = Phi_C^T (m - Phi_C w) - lam w with Phi_C = exp(L^T - z)
// re-evaluated in fp32 and every sum in float64.
// Optional key lists restrict either stage to a subset of the compact keys
// (list [P][tp], count [P]): the exact non-negative fit sums only over its free
// keys (w = 0 elsewhere) and needs each residual only on one side of its
// partition.  Without a list every key r < t takes part.
// Stage 1: u_i = m_i - sum_{r<t} Phi[i][r] w_r.  256 queries per workgroup,
// four per lane (16-byte loads of the L^T rows); wave s sums the compact keys
// r = s (mod 4) with two accumulator sets, and the four partial sums meet in LDS.
__global__ void __launch_bounds__(256) k_mass_resid_rows(const float *__restrict__ LT, const float *__restrict__ z,
                                                         const float *__restrict__ m, const double *__restrict__ w,
                                                         int n, int t, int64_t tp, int64_t np_,
                                                         double *__restrict__ u, const int32_t *__restrict__ info,
                                                         const int32_t *__restrict__ list,
                                                         const int32_t *__restrict__ count) {
  __shared__ double red[4][256];
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (info[b] != 0) return;
  const int i0 = blockIdx.x * 256 + 4 * lane;
  double a0[4] = {0.0, 0.0, 0.0, 0.0}, a1[4] = {0.0, 0.0, 0.0, 0.0};
  if (i0 < n) {
    const float *L = LT + (size_t)b * tp * np_ + i0;   // L^T rows are zero beyond n
    const double *wb = w + (size_t)b * tp;
    float zi[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) zi[k] = i0 + k < n ? z[(size_t)b * n + i0 + k] : 0.0f;
    auto term = [&](int r, double (&a)[4]) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(L + (size_t)r * np_);
      const double wr = wb[r];
#pragma unroll
      for (int k = 0; k < 4; ++k) a[k] += (double)expf(v[k] - zi[k]) * wr;
    };
    if (list) {
      const int32_t *lb = list + (size_t)b * tp;
      const int c = count[b];
      int k = wave;
      for (; k + 4 < c; k += 8) {
        term(lb[k], a0);
        term(lb[k + 4], a1);
      }
      if (k < c) term(lb[k], a0);
    } else {
      int r = wave;
      for (; r + 4 < t; r += 8) {
        term(r, a0);
        term(r + 4, a1);
      }
      if (r < t) term(r, a0);
    }
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) red[wave][4 * lane + k] = a0[k] + a1[k];
  __syncthreads();
  const int i = blockIdx.x * 256 + tid;
  if (i < np_) {
    const double acc = red[0][tid] + red[1][tid] + red[2][tid] + red[3][tid];
    u[(size_t)b * np_ + i] = i < n ? (double)m[(size_t)b * n + i] - acc : 0.0;
  }
}

// Stage 2: res_r = sum_i Phi[i][r] u_i - lam w_r.  Each wave takes four
// compact keys (16 per workgroup) so that the z and u loads are shared by
// them; four queries per lane per step (16-byte loads of the L^T rows and of
// u).  With a list, slot k handles key list[k] (k < count) and writes only there.
constexpr int kResKeys = 4;   // compact keys per wave
__global__ void __launch_bounds__(256) k_mass_resid_cols(const float *__restrict__ LT, const float *__restrict__ z,
                                                         const double *__restrict__ u, const double *__restrict__ w,
                                                         const float *__restrict__ lam, int n, int t, int64_t tp,
                                                         int64_t np_, double *__restrict__ res,
                                                         const int32_t *__restrict__ info,
                                                         const int32_t *__restrict__ list,
                                                         const int32_t *__restrict__ count) {
  typedef __attribute__((__vector_size__(2 * sizeof(double)))) double f64x2;
  const int b = blockIdx.y, lane = threadIdx.x & 63;
  const int k0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * kResKeys;   // first slot of this wave
  if (k0 >= tp || info[b] != 0) return;
  const int lim = list ? count[b] : t;   // slots k < lim are live keys
  if (k0 >= lim) {
    if (!list && lane < kResKeys) res[(size_t)b * tp + k0 + lane] = 0.0;   // padding keys r >= t
    return;
  }
  int r[kResKeys];
  const float *row[kResKeys];
#pragma unroll
  for (int q = 0; q < kResKeys; ++q) {
    const int k = k0 + q < lim ? k0 + q : lim - 1;   // dead slots repeat a live key, unstored
    r[q] = list ? list[(size_t)b * tp + k] : k;
    row[q] = LT + ((size_t)b * tp + r[q]) * np_;
  }
  const float *zb = z + (size_t)b * n;
  const double *ub = u + (size_t)b * np_;   // zero beyond n
  double acc[kResKeys] = {0.0, 0.0, 0.0, 0.0};
  for (int i0 = 4 * lane; i0 < n; i0 += 256) {
    const f64x2 u01 = *reinterpret_cast<const f64x2 *>(ub + i0);
    const f64x2 u23 = *reinterpret_cast<const f64x2 *>(ub + i0 + 2);
    const double uu[4] = {u01[0], u01[1], u23[0], u23[1]};
    float zz[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) zz[e] = zb[i0 + e < n ? i0 + e : n - 1];
#pragma unroll
    for (int q = 0; q < kResKeys; ++q) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(row[q] + i0);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const double term = (double)expf(v[e] - zz[e]) * uu[e];
        acc[q] += i0 + e < n ? term : 0.0;
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kResKeys; ++q) {
    const double sum = wave_sum(acc[q]);
    if (lane == 0 && k0 + q < lim)
      res[(size_t)b * tp + r[q]] = sum - (double)lam[b] * w[(size_t)b * tp + r[q]];
  }
  if (!list && lane >= kResKeys && lane < 2 * kResKeys) {   // padding keys r >= t within this wave's slots
    const int k = k0 + lane - kResKeys;
    if (k >= lim && k < tp) res[(size_t)b * tp + k] = 0.0;
  }
}

// beta = clip(log(max(max(w, 0), eps)), bmin, bmax); NaN for failed pairs.
__global__ void __launch_bounds__(256) k_bias_finalize(const double *__restrict__ w, int64_t ld, int t, float eps,
                                                       float bmin, float bmax, const int32_t *__restrict__ info,
                                                       float *__restrict__ beta, float *__restrict__ beta_ws) {
  const int b = blockIdx.y;
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= ld) return;
  float v = 0.0f;
  if (r < t) {
    if (info[b] != 0) {
      v = NAN;
    } else {
      const double wv = w[(size_t)b * ld + r];
      const double ws = wv > 0.0 ? wv : 0.0;
      v = (float)log(ws > (double)eps ? ws : (double)eps);
      v = fminf(fmaxf(v, bmin), bmax);
    }
    beta[(size_t)b * t + r] = v;
  }
  if (beta_ws) beta_ws[(size_t)b * ld + r] = v;
}

// --------------------------------------------------------------- value-fit operands
// P^T[r][i] = softmax_r(L^T[r][i] + beta_r) for r < t, i < n (own column max),
// split into bf16 hi/lo planes (or fp32), written in both layouts the value fit
// contracts over: PT [planes][tp][np] and, if Pm is given, Pm [planes][np][tp].
// A workgroup takes 64 queries: each wave first runs an online max/sum over the
// compact keys r = wave (mod 4) and the four partial (max, sum) pairs are
// merged in LDS; then the 64 x 64 (r, i) tiles are formed, stored row-wise into
// PT and, through an LDS transpose, into Pm.
template <typename T>
__global__ void __launch_bounds__(256) k_phat(const float *__restrict__ LT, const float *__restrict__ beta, int n,
                                              int t, int64_t tp, int64_t np_, void *__restrict__ out,
                                              void *__restrict__ outm) {
  constexpr int PL = sizeof(T) == 2 ? 2 : 1;
  __shared__ float smx[4][64], ssum[4][64];
  __shared__ __attribute__((aligned(16))) T sp[PL][64][64 + 8];
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i0 = blockIdx.x * 64, i = i0 + lane;
  const float *L = LT + (size_t)b * tp * np_ + i;
  const float *bb = beta + (size_t)b * tp;
  // exp(d) for d = x - max <= 0 as the hardware 2^(d log2(e)); the online max
  // advances eight keys at a time and rescales the running sum only when the
  // lane's maximum grew.
  constexpr float kLog2e = 1.4426950408889634f;
  float mx = -INFINITY, sum = 0.0f;
  if (i < n) {
    int r = wave;
    for (; r + 28 < t; r += 32) {
      float x[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) x[u] = L[(size_t)(r + 4 * u) * np_] + bb[r + 4 * u];
      float cm = x[0];
#pragma unroll
      for (int u = 1; u < 8; ++u) cm = fmaxf(cm, x[u]);
      if (cm > mx) {
        sum *= __builtin_amdgcn_exp2f((mx - cm) * kLog2e);
        mx = cm;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) sum += __builtin_amdgcn_exp2f((x[u] - mx) * kLog2e);
    }
    for (; r < t; r += 4) {
      const float x = L[(size_t)r * np_] + bb[r];
      if (x > mx) {
        sum *= __builtin_amdgcn_exp2f((mx - x) * kLog2e);
        mx = x;
      }
      sum += __builtin_amdgcn_exp2f((x - mx) * kLog2e);
    }
  }
  smx[wave][lane] = mx;
  ssum[wave][lane] = sum;
  __syncthreads();
  const float M = fmaxf(fmaxf(smx[0][lane], smx[1][lane]), fmaxf(smx[2][lane], smx[3][lane]));
  float S = 0.0f;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    S += smx[q][lane] == -INFINITY ? 0.0f : ssum[q][lane] * __builtin_amdgcn_exp2f((smx[q][lane] - M) * kLog2e);
  const float inv = (i < n && S > 0.0f) ? 1.0f / S : 0.0f;
  T *PT = reinterpret_cast<T *>(out) + (size_t)b * PL * tp * np_;
  T *Pm = reinterpret_cast<T *>(outm) + (size_t)b * PL * tp * np_;
  constexpr int EPV = 16 / sizeof(T);                     // elements per 16-byte store
  typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
  // this wave's 16 keys of the next tile: logits and biases loaded while the
  // current tile is stored
  float ln[16], bn[16];
  auto fetch_l = [&](int64_t q0) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t r = q0 + 16 * wave + e;
      const bool ok = i < n && r < t;
      ln[e] = ok ? L[(size_t)r * np_] : 0.0f;
      bn[e] = ok ? bb[r] : 0.0f;
    }
  };
  fetch_l(0);
  for (int64_t r0 = 0; r0 < tp; r0 += 64) {
    __syncthreads();   // the previous tile's stores have read sp
    float lc[16], bc[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      lc[e] = ln[e];
      bc[e] = bn[e];
    }
    if (r0 + 64 < tp) fetch_l(r0 + 64);
#pragma unroll
    for (int e4 = 0; e4 < 16; e4 += 4) {   // four consecutive keys per LDS write
      float pv[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t r = r0 + 16 * wave + e4 + e;
        pv[e] = (i < n && r < t) ? __builtin_amdgcn_exp2f((lc[e4 + e] + bc[e4 + e] - M) * kLog2e) * inv : 0.0f;
      }
      const int rr = 16 * wave + e4;
      if constexpr (PL == 2) {
        bf16x4 hi, lo;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hi[e] = (bf16)pv[e];
          lo[e] = (bf16)(pv[e] - (float)hi[e]);
        }
        *reinterpret_cast<bf16x4 *>(&sp[0][lane][rr]) = hi;
        *reinterpret_cast<bf16x4 *>(&sp[1][lane][rr]) = lo;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) sp[0][lane][rr + e] = pv[e];
      }
    }
    __syncthreads();
    // P^T rows r0 + rr, columns i0 .. i0 + 63 (gathered down the tile)
    for (int e = tid; e < PL * 64 * (64 / EPV); e += 256) {
      const int q = e / (64 * (64 / EPV)), rr = (e / (64 / EPV)) % 64, c = (e % (64 / EPV)) * EPV;
      T v[EPV];
#pragma unroll
      for (int k = 0; k < EPV; ++k) v[k] = sp[q][c + k][rr];
      *reinterpret_cast<u32x4 *>(&PT[(size_t)q * tp * np_ + (size_t)(r0 + rr) * np_ + i0 + c]) =
          *reinterpret_cast<const u32x4 *>(v);
    }
    if (outm)   // P rows i0 + row, columns r0 .. r0 + 63
      for (int e = tid; e < PL * 64 * (64 / EPV); e += 256) {
        const int q = e / (64 * (64 / EPV)), row = (e / (64 / EPV)) % 64, c = (e % (64 / EPV)) * EPV;
        *reinterpret_cast<u32x4 *>(&Pm[(size_t)q * np_ * tp + (size_t)(i0 + row) * tp + r0 + c]) =
            *reinterpret_cast<const u32x4 *>(&sp[q][row][c]);
      }
  }
}

// out[c][i] = in[i][c] for a [rows][128] fp32 matrix, zero-padded to rows_pad
// columns; bf16 hi/lo planes or fp32.
template <typename T>
__global__ void __launch_bounds__(256) k_transpose128(const float *__restrict__ in, int rows, int64_t in_pair,
                                                      int64_t rows_pad, void *__restrict__ out, int64_t out_pair) {
  __shared__ float s[64][kHeadDim + 1];
  const int b = blockIdx.y, tid = threadIdx.x;
  const int i0 = blockIdx.x * 64;
  for (int e = tid; e < 64 * kHeadDim; e += 256) {
    const int r = e / kHeadDim, c = e % kHeadDim;
    s[r][c] = (i0 + r < rows) ? in[(size_t)b * in_pair + (size_t)(i0 + r) * kHeadDim + c] : 0.0f;
  }
  __syncthreads();
  for (int e = tid; e < 64 * kHeadDim; e += 256) {
    const int c = e / 64, r = e % 64;
    const float v = s[r][c];
    const size_t o = (size_t)b * out_pair + (size_t)c * rows_pad + i0 + r;
    if constexpr (sizeof(T) == 2) {
      bf16 *ob = reinterpret_cast<bf16 *>(out);
      split_bf16(v, ob[o], ob[o + (size_t)kHeadDim * rows_pad]);
    } else {
      reinterpret_cast<float *>(out)[o] = v;
    }
  }
}

// --------------------------------------------------------------- 128 right-hand sides
// 128-rhs triangular solve on fp32 MFMA: L X = R (forward) or L^T X = R
// (backward), one workgroup per pair (8 waves = 2 row tiles x 4 column tiles
// of 32), 64-row blocks, so L is read once per solve.  For block kb the
// update  acc = sum_p L_kb,p X_p  (forward) or  sum_p L_p,kb^T X_p  (backward)
// is an MFMA product with the L tile and the X tile staged in LDS; the block
// is then X_kb = D (R_kb - acc) with D = L_kb,kb^-1 (forward) or its
// transpose (backward), the diagonal-block inverses written by the
// factorisation.
constexpr int kTrsmRB = 64, kTrsmSLD = kTrsmRB + 1, kTrsmSXD = kHeadDim + 1;
constexpr size_t kTrsmLds = (size_t)2 * (kTrsmRB * kTrsmSLD + kTrsmRB * kTrsmSXD) * sizeof(float);

template <bool FWD>
__global__ void __launch_bounds__(512) k_trsm_mfma(const float *__restrict__ Gw, int64_t ld,
                                                   const float *__restrict__ dinv, const float *__restrict__ R,
                                                   float *__restrict__ X, const int32_t *__restrict__ info) {
  constexpr int RB = kTrsmRB, SLD = kTrsmSLD, SXD = kTrsmSXD;
  extern __shared__ float trsm_smem[];
  auto sL = [&](int bf) { return trsm_smem + bf * RB * SLD; };
  auto sX = [&](int bf) { return trsm_smem + 2 * RB * SLD + bf * RB * SXD; };
  const int b = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (info[b] != 0) return;
  const int wr = wave >> 2, wc = wave & 3, h = lane >> 5, col = lane & 31;
  const float *L = Gw + (size_t)b * ld * ld;
  const float *Rb = R + (size_t)b * ld * kHeadDim;
  float *Xb = X + (size_t)b * ld * kHeadDim;
  const int nb = (int)(ld / RB);
  const float *Db = dinv + (size_t)b * nb * RB * RB;
  f32x4 rl[2], rx[4];
  // tile (i, k) of the operand: forward L[r0+i][p0+k], backward L[p0+k][r0+i]
  auto fetch = [&](int r0, int p0) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int e = tid + 512 * c, i = e / 16, k4 = (e % 16) * 4;
      rl[c] = FWD ? *reinterpret_cast<const f32x4 *>(L + (size_t)(r0 + i) * ld + p0 + k4)
                  : *reinterpret_cast<const f32x4 *>(L + (size_t)(p0 + i) * ld + r0 + k4);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int e = tid + 512 * c, i = e / 32, k4 = (e % 32) * 4;
      rx[c] = *reinterpret_cast<const f32x4 *>(Xb + (size_t)(p0 + i) * kHeadDim + k4);
    }
  };
  auto stash = [&](int bf) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int e = tid + 512 * c, i = e / 16, k4 = (e % 16) * 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (FWD) sL(bf)[i * SLD + k4 + q] = rl[c][q];
        else sL(bf)[(k4 + q) * SLD + i] = rl[c][q];
      }
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int e = tid + 512 * c, i = e / 32, k4 = (e % 32) * 4;
#pragma unroll
      for (int q = 0; q < 4; ++q) sX(bf)[i * SXD + k4 + q] = rx[c][q];
    }
  };
  for (int step = 0; step < nb; ++step) {
    const int kb = FWD ? step : nb - 1 - step;
    const int r0 = kb * RB;
    f32x16 acc = zero16();
    const int pb0 = FWD ? 0 : kb + 1, pb1 = FWD ? kb : nb;
    int bf = 0;
    if (pb0 < pb1) {
      __syncthreads();
      fetch(r0, pb0 * RB);
      stash(0);
      __syncthreads();
    }
    for (int pb = pb0; pb < pb1; ++pb) {
      const bool more = pb + 1 < pb1;
      if (more) fetch(r0, (pb + 1) * RB);
#pragma unroll 8
      for (int ks = 0; ks < RB / 2; ++ks)
        acc = Mfma<float>::mma(sL(bf)[(32 * wr + col) * SLD + 2 * ks + h],
                               sX(bf)[(2 * ks + h) * SXD + 32 * wc + col], acc);
      if (more) stash(bf ^ 1);
      __syncthreads();
      bf ^= 1;
    }
    __syncthreads();
    // right-hand side minus update into sX(0); D into sL(0) (row r = output row)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = 32 * wr + acc_row(v, lane), c = 32 * wc + col;
      sX(0)[r * SXD + c] = Rb[(size_t)(r0 + r) * kHeadDim + c] - acc[v];
    }
    const float *Dk = Db + (size_t)kb * RB * RB;
    for (int e = tid; e < RB * RB / 4; e += 512) {
      const int i = e / 16, k4 = (e % 16) * 4;
      const f32x4 v = *reinterpret_cast<const f32x4 *>(Dk + i * RB + k4);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (FWD) sL(0)[i * SLD + k4 + q] = v[q];
        else sL(0)[(k4 + q) * SLD + i] = v[q];
      }
    }
    __syncthreads();
    f32x16 out = zero16();
#pragma unroll 8
    for (int ks = 0; ks < RB / 2; ++ks)
      out = Mfma<float>::mma(sL(0)[(32 * wr + col) * SLD + 2 * ks + h], sX(0)[(2 * ks + h) * SXD + 32 * wc + col],
                             out);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int r = 32 * wr + acc_row(v, lane), c = 32 * wc + col;
      Xb[(size_t)(r0 + r) * kHeadDim + c] = out[v];
    }
    __threadfence_block();
  }
}

// ---------------------------------------------------------------- blocked forward solve
// L Y = R for 128 right-hand sides in 256-row blocks kb: the contribution of the
// earlier blocks, L[kb, 0:kb] Y[0:kb], is one contraction on fp16 MFMA over the
// factorisation's hi / lo planes of L (row r scaled by 2^shift[r]) and hi / lo
// planes of Y^T (column c scaled by 2^e_c), the three products hi.hi, hi.lo,
// lo.hi as in the left-looking update (about 2^-22 relative); the 256 x 256
// diagonal block is then solved by one workgroup per pair with the stored
// 64 x 64 inverses on fp32 MFMA.  Pairs flagged here are solved again by the
// fp32 kernel (k_trsm_mfma).

// e_c with 2 ||R_c|| / sqrt(lam) 2^e_c < 2^10: |Y_rc| <= ||R_c|| / sigma_min(L)
// and sigma_min(L)^2 is about the smallest eigenvalue of the ridged Gram, at
// least lam, so the scaled values keep 2^6 of headroom under fp16's largest.
// A pair without a ridge, or with a non-finite right-hand side, is flagged.
__global__ void __launch_bounds__(1024) k_trsm_colexp(const float *__restrict__ R, int64_t ld,
                                                      const float *__restrict__ lam, const int32_t *__restrict__ info,
                                                      int32_t *__restrict__ ex, int32_t *__restrict__ flag) {
  __shared__ double part[8][kHeadDim];
  const int b = blockIdx.x, tid = threadIdx.x, c = tid & (kHeadDim - 1), g = tid >> 7;
  if (info[b] != 0) return;
  // eight row groups per column, eight loads in flight per thread
  const float *Rb = R + (size_t)b * ld * kHeadDim + c;
  double ss = 0.0;
#pragma unroll 8
  for (int64_t r = g; r < ld; r += 8) {
    const double v = Rb[r * kHeadDim];
    ss = fma(v, v, ss);
  }
  part[g][c] = ss;
  if (tid == 0) flag[b] = 0;
  __syncthreads();
  if (g != 0) return;
  ss = 0.0;
#pragma unroll
  for (int q = 0; q < 8; ++q) ss += part[q][c];
  const float lb = lam[b];
  const double bound = lb > 0.0f ? 2.0 * sqrt(ss) / sqrt((double)lb) : INFINITY;
  int e = 0;
  const bool ok = isfinite(bound);
  if (ok && bound > 0.0) {
    int x = 0;
    frexp(bound, &x);   // bound < 2^x
    e = max(min(10 - x, 126), -126);
  }
  ex[(size_t)b * kHeadDim + c] = e;
  if (!ok) flag[b] = 1;
}

// Y[r0 + m][c] = R[r0 + m][c] - acc 2^-shift[r0 + m] 2^-e_c for one 256-row block
// (tile rows m, columns c < 128).
template <int TM, int TN>
struct EpiTrsmFwd {
  const float *R;
  float *Y;
  int64_t ld;
  int r0;
  const float *sinv;     // L's inverse row scales [P][ld]
  const int32_t *ex;     // [P][128]
  const int32_t *info, *flag;
  __device__ __forceinline__ bool skip(int p) const { return info[p] != 0 || flag[p] != 0; }
  __device__ __forceinline__ void operator()(f32x16 (&acc)[TM][TN], int p, int row0, int col0, int, int, int lane,
                                             int, int) const {
    const int col = lane & 31;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int c = col0 + 32 * j + col;
      const float sc = ldexpf(1.0f, -ex[(size_t)p * kHeadDim + c]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int64_t r = r0 + row0 + 32 * i + acc_row(v, lane);
          const size_t o = ((size_t)p * ld + r) * kHeadDim + c;
          Y[o] = R[o] - acc[i][j][v] * (sinv[(size_t)p * ld + r] * sc);
        }
    }
  }
};

// One 256-row block per pair: right-hand sides rows r0 .. r0 + 255 (src), four
// 64-row steps y_s = D_s r_s with r_s' -= L_s's y_s for the later steps s'
// (right-looking inside the block, the right-hand sides held in registers:
// wave (wm, wn) owns rows 32 wm and columns 32 wn of every 64-row step).  Writes
// Y (fp32) and the planes of Y^T for the later blocks' contractions; a scaled
// value at or above 2^15 flags the pair.
__global__ void __launch_bounds__(512) k_trsm_fwd_blk(const float *__restrict__ Gw, const float *__restrict__ dinv,
                                                      int64_t ld, int kb, const float *__restrict__ src,
                                                      float *__restrict__ Y, f16 *__restrict__ Yt,
                                                      const int32_t *__restrict__ ex,
                                                      const int32_t *__restrict__ info, int32_t *__restrict__ flag) {
  constexpr int SY = 160;             // row stride of the [64][128] operand: the two half-waves on opposite banks
  __shared__ float sD[kNB * kSD];      // D_s, then L_s's
  __shared__ float sY[kNB * SY];       // r_s, then y_s, [k][c]
  const int b = blockIdx.x;
  if (info[b] != 0 || flag[b] != 0) return;   // uniform over the workgroup
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3, h = lane >> 5, col = lane & 31;
  const int nb = (int)(ld / kNB);
  const int64_t r0 = (int64_t)kb * 256;
  const float *L = Gw + (size_t)b * ld * ld;
  const int c = 32 * wn + col;
  const int e = ex[(size_t)b * kHeadDim + c];
  f32x16 rt[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      rt[s][v] = src[((size_t)b * ld + r0 + 64 * s + 32 * wm + acc_row(v, lane)) * kHeadDim + c];
  auto stage = [&](const float *A, int64_t lda) {   // a 64 x 64 operand into sD, row-major
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int g = tid + 512 * q, i = g >> 4, c4 = (g & 15) * 4;
      const f32x4 v = *reinterpret_cast<const f32x4 *>(A + (size_t)i * lda + c4);
#pragma unroll
      for (int u = 0; u < 4; ++u) sD[i * kSD + c4 + u] = v[u];
    }
  };
  auto product = [&]() {   // this wave's 32 x 32 block of sD x sY
    f32x16 acc = zero16();
#pragma unroll 8
    for (int ks = 0; ks < kNB / 2; ++ks)
      acc = Mfma<float>::mma(sD[(32 * wm + col) * kSD + 2 * ks + h], sY[(2 * ks + h) * SY + c], acc);
    return acc;
  };
  bool over = false;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 16; ++v) sY[(32 * wm + acc_row(v, lane)) * SY + c] = rt[s][v];
    stage(dinv + ((size_t)b * nb + 4 * kb + s) * kNB * kNB, kNB);
    __syncthreads();
    const f32x16 y = product();
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t r = r0 + 64 * s + 32 * wm + acc_row(v, lane);
      sY[(32 * wm + acc_row(v, lane)) * SY + c] = y[v];
      Y[((size_t)b * ld + r) * kHeadDim + c] = y[v];
    }
    // planes of Y^T: rows 8 g + 4 h .. + 3 of this lane are four consecutive r
    f16 *hi = Yt + ((size_t)b * 2 * kHeadDim + c) * ld + r0 + 64 * s + 32 * wm + 4 * h;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      f16x4 xh, xl;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float x = ldexpf(y[4 * g + u], e);
        over |= !(fabsf(x) < 32768.0f);
        xh[u] = (f16)x;
        xl[u] = (f16)(x - (float)xh[u]);
      }
      *reinterpret_cast<f16x4 *>(hi + 8 * g) = xh;
      *reinterpret_cast<f16x4 *>(hi + (size_t)kHeadDim * ld + 8 * g) = xl;
    }
#pragma unroll
    for (int s2 = s + 1; s2 < 4; ++s2) {
      __syncthreads();   // every wave is done with sD; sY holds y_s
      stage(L + (size_t)(r0 + 64 * s2) * ld + r0 + 64 * s, ld);
      __syncthreads();
      const f32x16 u = product();
#pragma unroll
      for (int v = 0; v < 16; ++v) rt[s2][v] -= u[v];
    }
  }
  if (over) flag[b] = 1;
}

// After the blocked solve: a column whose largest scaled value |Y_rc| 2^e_c is
// below 2^-6 (a bound far above the solution) kept fewer than about 18
// significant bits in its planes; its pair is flagged for the fp32 solve.
__global__ void __launch_bounds__(1024) k_trsm_colcheck(const float *__restrict__ Y, int64_t ld,
                                                        const int32_t *__restrict__ ex,
                                                        const int32_t *__restrict__ info, int32_t *__restrict__ flag) {
  __shared__ float part[8][kHeadDim];
  const int b = blockIdx.x, tid = threadIdx.x, c = tid & (kHeadDim - 1), g = tid >> 7;
  if (info[b] != 0 || flag[b] != 0) return;   // uniform over the workgroup
  const float *Yb = Y + (size_t)b * ld * kHeadDim + c;
  float m = 0.0f;
#pragma unroll 8
  for (int64_t r = g; r < ld; r += 8) m = fmaxf(m, fabsf(Yb[r * kHeadDim]));
  part[g][c] = m;
  __syncthreads();
  if (g != 0) return;
#pragma unroll
  for (int q = 1; q < 8; ++q) m = fmaxf(m, part[q][c]);
  if (m > 0.0f && ldexpf(m, ex[(size_t)b * kHeadDim + c]) < 0.015625f) flag[b] = 1;
}

// out[b] = 1 where the fp32 solve must skip pair b (failed, or solved above)
__global__ void k_trsm_fallback_mask(const int32_t *__restrict__ info, const int32_t *__restrict__ flag, int B,
                                     int32_t *__restrict__ out) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b < B) out[b] = (info[b] != 0 || flag[b] == 0) ? 1 : 0;
}

__global__ void __launch_bounds__(256) k_add_copy(float *__restrict__ x, const float *__restrict__ dx, int64_t n_per,
                                                  const int32_t *__restrict__ info) {
  const int b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= n_per || info[b] != 0) return;
  x[(size_t)b * n_per + e] += dx[(size_t)b * n_per + e];
}

// Copy the first t rows of the padded [tp][128] solution to the output, NaN
// for pairs whose factorisation failed.
__global__ void __launch_bounds__(256) k_values_out(const float *__restrict__ Xp, int64_t tp, int t,
                                                    const int32_t *__restrict__ info, float *__restrict__ Cv) {
  const int b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)t * kHeadDim) return;
  Cv[(size_t)b * t * kHeadDim + e] = info[b] != 0 ? NAN : Xp[(size_t)b * tp * kHeadDim + e];
}

// --------------------------------------------------------------- exact NNLS (bias_mode 1)
// Block principal pivoting (Judice & Pires 1994, in the single-right-hand-side
// form of Kim & Park 2011) for min ||Phi_C w - m||^2 + lam ||w||^2, w >= 0, the
// ridged system of the projected fit.  Per pair: F (passive set, 1 = free), x,
// y = (G + lam I) x - h from the data residual, and the state
// {best infeasible count N, backup budget p, done, spare}.  The iteration starts
// from the unconstrained solution (F = every key), which the projected fit has
// already computed; each later iteration solves the free-set system compressed
// to its |F| x |F| block.
constexpr int32_t kNnlsSkip = -0x40000000;   // info marker of a pair that has converged

__global__ void __launch_bounds__(256) k_nnls_init(int t, int64_t tp, const int32_t *__restrict__ info,
                                                   int32_t *__restrict__ F, double *__restrict__ y,
                                                   int32_t *__restrict__ state) {
  const int b = blockIdx.y;
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r < tp) {
    F[(size_t)b * tp + r] = r < t;
    y[(size_t)b * tp + r] = 0.0;
  }
  if (r == 0) {
    state[4 * b] = t + 1;
    state[4 * b + 1] = 3;
    state[4 * b + 2] = info[b] != 0;   // a failed projected fit is not iterated
    state[4 * b + 3] = 0;
  }
}

// One workgroup per pair: the infeasible set V = {free x < -tol} u {bound y < -tol},
// then the exchange rule: all of V while |V| improves on the best count (or the
// backup budget lasts), otherwise only its largest index.  Marks the pair done
// (and skipped by the factor and solve kernels) when V is empty.
__global__ void __launch_bounds__(256) k_nnls_update(const double *__restrict__ x, const double *__restrict__ y,
                                                     const double *__restrict__ h, int t, int64_t tp,
                                                     int32_t *__restrict__ F, int32_t *__restrict__ state,
                                                     int32_t *__restrict__ info) {
  __shared__ double sx[4], sh[4];
  __shared__ int32_t scnt[4], smax[4];
  __shared__ int32_t s_mode;   // 0 none, 1 all of V, 2 the largest index only
  __shared__ int32_t s_j;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (state[4 * b + 2] || info[b] != 0) return;   // settled, or a factorisation failed
  const double *xb = x + (size_t)b * tp, *yb = y + (size_t)b * tp, *hb = h + (size_t)b * tp;
  int32_t *Fb = F + (size_t)b * tp;
  double mx = 0.0, mh = 0.0;
  for (int r = tid; r < t; r += 256) {
    mx = fmax(mx, fabs(xb[r]));
    mh = fmax(mh, fabs(hb[r]));
  }
  for (int o = 32; o >= 1; o >>= 1) {
    mx = fmax(mx, __shfl_xor(mx, o, 64));
    mh = fmax(mh, __shfl_xor(mh, o, 64));
  }
  if (lane == 0) {
    sx[wave] = mx;
    sh[wave] = mh;
  }
  __syncthreads();
  // tolerances: float32-level relative to the solution and right-hand side scales
  const double tx = 1e-6 * fmax(fmax(sx[0], sx[1]), fmax(sx[2], sx[3]));
  const double ty = 1e-6 * fmax(fmax(sh[0], sh[1]), fmax(sh[2], sh[3]));
  auto infeasible = [&](int r) { return Fb[r] ? xb[r] < -tx : yb[r] < -ty; };
  int32_t cnt = 0, jmax = -1;
  for (int r = tid; r < t; r += 256)
    if (infeasible(r)) {
      ++cnt;
      jmax = r;
    }
  for (int o = 32; o >= 1; o >>= 1) {
    cnt += __shfl_xor(cnt, o, 64);
    jmax = max(jmax, __shfl_xor(jmax, o, 64));
  }
  if (lane == 0) {
    scnt[wave] = cnt;
    smax[wave] = jmax;
  }
  __syncthreads();
  if (tid == 0) {
    const int32_t V = scnt[0] + scnt[1] + scnt[2] + scnt[3];
    s_j = max(max(smax[0], smax[1]), max(smax[2], smax[3]));
    int32_t mode = 0;
    if (V == 0) {
      state[4 * b + 2] = 1;
      info[b] = kNnlsSkip;
    } else if (V < state[4 * b]) {
      state[4 * b] = V;
      state[4 * b + 1] = 3;
      mode = 1;
    } else if (state[4 * b + 1] >= 1) {
      state[4 * b + 1] -= 1;
      mode = 1;
    } else {
      mode = 2;
    }
    state[4 * b + 3] += mode != 0;   // iterations taken
    s_mode = mode;
  }
  __syncthreads();
  if (s_mode == 1) {
    // infeasible(r) reads only F[r], which this thread alone owns
    for (int r = tid; r < t; r += 256)
      if (infeasible(r)) Fb[r] ^= 1;
  } else if (s_mode == 2 && tid == 0) {
    Fb[s_j] ^= 1;
  }
}

__global__ void k_nnls_zero(int32_t *__restrict__ red) {
  if (threadIdx.x < 2) red[threadIdx.x] = 0;
}

// Free list of every unsettled pair: idx[k] = the k-th free key (ascending),
// pos[r] = its slot or -1, nf = |F|; red = {max nf, unsettled pairs}.
// Free and bound lists of every unsettled pair: idx[k] = the k-th free key,
// bidx[k] = the k-th bound key (both ascending), pos[r] = the free slot of r or
// -1; nf = |F|, nb = t - |F|; red = {max nf, unsettled pairs}.
__global__ void __launch_bounds__(256) k_nnls_index(const int32_t *__restrict__ F, int t, int64_t tp,
                                                    const int32_t *__restrict__ info, int32_t *__restrict__ idx,
                                                    int32_t *__restrict__ bidx, int32_t *__restrict__ pos,
                                                    int32_t *__restrict__ nf, int32_t *__restrict__ nb,
                                                    int32_t *__restrict__ red) {
  __shared__ int32_t wsum[4];
  __shared__ int32_t base;
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (info[b] != 0) return;   // settled or failed
  if (tid == 0) base = 0;
  __syncthreads();
  const int32_t *Fb = F + (size_t)b * tp;
  int32_t *ib = idx + (size_t)b * tp, *bb = bidx + (size_t)b * tp, *pb = pos + (size_t)b * tp;
  for (int64_t r0 = 0; r0 < tp; r0 += 256) {
    const int64_t r = r0 + tid;
    const bool f = r < t && Fb[r] != 0;
    const uint64_t m = __ballot(f);
    if (lane == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    int32_t before = base + __popcll(m & ((1ull << lane) - 1ull));   // free keys below r
    for (int w = 0; w < wave; ++w) before += wsum[w];
    if (f) ib[before] = (int32_t)r;
    else if (r < t) bb[r - before] = (int32_t)r;
    if (r < tp) pb[r] = f ? before : -1;
    __syncthreads();
    if (tid == 0) base += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
  }
  if (tid == 0) {
    nf[b] = base;
    nb[b] = t - base;
    atomicMax(&red[0], base);
    atomicAdd(&red[1], 1);
  }
}

// Compressed free-set system [ldf][ldf]: G_{idx_i idx_j} + lam [i = j] for
// i, j < nf, identity beyond.
__global__ void __launch_bounds__(256) k_nnls_gather_gram(const float *__restrict__ Gc, int64_t tp,
                                                          const int32_t *__restrict__ idx,
                                                          const int32_t *__restrict__ nf, const FitState st,
                                                          int64_t ldf, float *__restrict__ Gw) {
  const int b = blockIdx.y;
  if (st.info[b] != 0) return;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= ldf * ldf) return;
  const int64_t i = e / ldf, j = e % ldf;
  // the factorisation reads the lower triangle only
  if (j > i) return;
  const int32_t n = nf[b];
  float v = i == j ? 1.0f : 0.0f;
  if (i < n) {   // then j <= i < n; the free list ascends, so (idx_i, idx_j) is in the stored lower triangle
    const int32_t *ib = idx + (size_t)b * tp;
    v = Gc[(size_t)b * tp * tp + (size_t)ib[i] * tp + ib[j]] + (i == j ? st.lam[b] : 0.0f);
  }
  Gw[(size_t)b * ldf * ldf + e] = v;
}

// out[k] = in[idx_k] for k < nf, 0 beyond (a compressed right-hand side).
__global__ void __launch_bounds__(256) k_nnls_gather_vec(const double *__restrict__ in, int64_t tp,
                                                         const int32_t *__restrict__ idx,
                                                         const int32_t *__restrict__ nf,
                                                         const int32_t *__restrict__ info, int64_t ldf,
                                                         double *__restrict__ out) {
  const int b = blockIdx.y;
  const int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (k >= ldf || info[b] != 0) return;
  out[(size_t)b * ldf + k] = k < nf[b] ? in[(size_t)b * tp + idx[(size_t)b * tp + k]] : 0.0;
}

// x[r] = xf[pos_r] on free keys and 0 on bound ones (acc: x[r] += ...).
__global__ void __launch_bounds__(256) k_nnls_scatter(const double *__restrict__ xf, int64_t ldf,
                                                      const int32_t *__restrict__ pos, int64_t tp,
                                                      const int32_t *__restrict__ info, int acc,
                                                      double *__restrict__ x) {
  const int b = blockIdx.y;
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= tp || info[b] != 0) return;
  const int32_t p = pos[(size_t)b * tp + r];
  const double v = p >= 0 ? xf[(size_t)b * ldf + p] : 0.0;
  double *o = x + (size_t)b * tp + r;
  *o = acc ? *o + v : v;
}

// y = -(data residual) on bound keys, 0 on free ones.
__global__ void __launch_bounds__(256) k_nnls_dual(const double *__restrict__ res, const int32_t *__restrict__ F,
                                                   int64_t tp, const int32_t *__restrict__ info,
                                                   double *__restrict__ y) {
  const int b = blockIdx.y;
  const int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (r >= tp || info[b] != 0) return;
  const size_t o = (size_t)b * tp + r;
  y[o] = F[o] ? 0.0 : -res[o];
}

// After the iterations: converged pairs are ok again; pairs still iterating get -2.
__global__ void k_nnls_finish(const int32_t *__restrict__ state, int B, int32_t *__restrict__ info) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  if (info[b] == kNnlsSkip) info[b] = 0;
  else if (info[b] == 0 && !state[4 * b + 2]) info[b] = -2;
}

// ------------------------------------------------------------------ launchers
hipError_t launch_fill_i32(int32_t *p, int64_t count, int32_t v, hipStream_t s);
hipError_t launch_trsv(const float *Gw, const float *dinv, int B, int64_t ld, const double *rhs, double *sw,
                       double *y, double *x, double *acc, const int32_t *info, hipStream_t s);
hipError_t launch_cholesky_factor(float *Gw, const float *Gc, int B, int t, int64_t ld, float delta0, int max_esc,
                                  FitState st, float *dinv, void *lsplit, hipStream_t s);

// Escalation rounds over the pairs whose factorisation failed and that have
// escalations left.  Before each round the number of such pairs is read back
// to the host (cnt: one device int32), so rounds run only when a pair needs
// one; with max_esc = 0 nothing is read back.
static hipError_t launch_esc_rounds(float *Gw, const float *Gc, int B, int t, int64_t ld, int max_esc, FitState st,
                                    float *dinv, void *lsplit, int32_t *cnt, hipStream_t s) {
  hipError_t e = hipSuccess;
  for (int round = 0; round < max_esc; ++round) {
    hipLaunchKernelGGL(k_count_failed, dim3(1), dim3(256), 0, s, B, st, max_esc, cnt);
    int32_t failed = 0;
    if ((e = hipMemcpyAsync(&failed, cnt, sizeof(failed), hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
    if (failed == 0) break;
    hipLaunchKernelGGL(k_esc_state, dim3((B + 255) / 256), dim3(256), 0, s, B, t, st, max_esc);
    hipLaunchKernelGGL(k_esc_copy, dim3((unsigned)ld, B), dim3(256), 0, s, Gw, Gc, t, ld, st);
    if ((e = launch_cholesky_factor(Gw, Gc, B, t, ld, 0.0f, 0, st, dinv, lsplit, s)) != hipSuccess) return e;
    hipLaunchKernelGGL(k_esc_restore, dim3((B + 255) / 256), dim3(256), 0, s, B, st.info);
  }
  return hipGetLastError();
}

// Ridge + factorisation of the work copy Gw of Gc, then the escalation rounds.
hipError_t launch_cholesky(float *Gw, const float *Gc, int B, int t, int64_t ld, float delta0, int max_esc,
                           FitState st, float *dinv, void *lsplit, const int32_t *bad, int32_t *cnt,
                           hipStream_t s) {
  hipLaunchKernelGGL(k_ridge_init, dim3(B), dim3(256), 0, s, Gw, Gc, t, ld, delta0, st, bad);
  hipError_t e = launch_cholesky_factor(Gw, Gc, B, t, ld, delta0, 0, st, dinv, lsplit, s);
  if (e != hipSuccess) return e;
  return launch_esc_rounds(Gw, Gc, B, t, ld, max_esc, st, dinv, lsplit, cnt, s);
}

hipError_t launch_nonfinite(const float *a, int B, int64_t per, int32_t *bad, hipStream_t s) {
  if (per <= 0) return hipSuccess;
  const int64_t blocks = (per + 255) / 256;
  hipLaunchKernelGGL(k_nonfinite, dim3((unsigned)(blocks < 64 ? blocks : 64), B), dim3(256), 0, s, a, per, bad);
  return hipGetLastError();
}

// Factor the prepared work copy Gw in place (no ridge set-up, no escalation).
hipError_t launch_cholesky_factor(float *Gw, const float *Gc, int B, int t, int64_t ld, float delta0, int max_esc,
                                  FitState st, float *dinv, void *lsplit, hipStream_t s) {
  // 256-wide outer panels, left-looking: before a panel is factored, one
  // contraction applies every earlier panel to it (rows K0 .. ld, K = 3 K0 over
  // the fp16 hi / lo planes of L), so each trailing entry is read and written
  // once per factorisation instead of once per outer panel.  Inside the panel,
  // 64-wide diagonal factor + panel-solve steps on its 256 x 256 diagonal block,
  // then the fused strip kernel on the rows below, which also writes their
  // planes for the later panels' contractions.
  // lsplit layout (B (4 ld^2 + 8 ld) bytes): planes [B][2][ld][ld] fp16 (hi,
  // lo), then shifts [B][ld] int32, then inverse scales [B][ld] fp32.
  constexpr int kOuter = 256;
  f16 *Lp = reinterpret_cast<f16 *>(lsplit);
  int32_t *shift = reinterpret_cast<int32_t *>(Lp + (size_t)B * 2 * ld * ld);
  float *sinv = reinterpret_cast<float *>(shift + (size_t)B * ld);
  hipLaunchKernelGGL(k_chol_scales, dim3((unsigned)((ld + 255) / 256), B), dim3(256), 0, s, Gw, ld, shift, sinv,
                     st.info);
  const hipError_t ea = hipFuncSetAttribute((const void *)k_chol_strip16, hipFuncAttributeMaxDynamicSharedMemorySize,
                                            (int)kStrip16Lds);
  if (ea != hipSuccess) return ea;
  for (int K0 = 0; K0 < ld; K0 += kOuter) {
    const int K1 = (int)(K0 + kOuter < ld ? K0 + kOuter : ld);
    if (K0 > 0) {
      // A[K0.., K0..K1) -= L[K0.., 0..K0) L[K0..K1, 0..K0)^T: the three products
      // hi.hi, hi.lo, lo.hi per k-step from both planes of each operand (each
      // plane is read once), 256 x 256 tiles down the panel
      const f16 *Ar = Lp + (size_t)K0 * ld;
      BigShape g{B, (int)(ld - K0), kOuter, K0, 2 * ld * ld, ld * ld, ld, 2 * ld * ld, ld * ld, ld, false, 4};
      EpiCholUpd<2, 4> e{Gw, ld, K0, st.info, sinv + K0, ld};
      const hipError_t err = launch_gemm_big<4, 2, 2, 4, 32, 2, 2, 2, f16>(
          g, reinterpret_cast<const bf16 *>(Ar), reinterpret_cast<const bf16 *>(Ar), e, s);
      if (err != hipSuccess) return err;
    }
    // the 256 x 256 diagonal block: 64-wide steps restricted to its rows
    for (int c = K0; c < K1; c += kNB) {
      const int k = c / kNB;
      hipLaunchKernelGGL(k_chol_diag, dim3(B), dim3(kDiagThreads), 0, s, Gw, ld, k, st.info, dinv);
      const int rem = (K1 - c) / kNB - 1;   // row blocks of the diagonal block below block k
      if (rem > 0)
        hipLaunchKernelGGL(k_chol_panel, dim3((rem + 1) / 2, B), dim3(256), 0, s, Gw, ld, k, (int64_t)K1, dinv,
                           st.info);
      if (c + kNB < K1) {
        const int r_lo = c + kNB, n_rt = (K1 - r_lo + 127) / 128, n_ct = (K1 - r_lo + 127) / 128;
        hipLaunchKernelGGL(k_chol_upd, dim3((unsigned)(chol_upd_tiles(n_rt, n_ct) * B)), dim3(256), 0, s, Gw, ld,
                           r_lo, K1, K1, c, kNB, n_rt, n_ct, st.info);
      }
    }
    // the rows below: all four steps, written back once, with their planes
    if (K1 < ld)
      hipLaunchKernelGGL(k_chol_strip16, dim3((unsigned)((ld - K1) / kStripRows), B), dim3(512), kStrip16Lds, s, Gw,
                         ld, K0, dinv, Lp, shift, st.info);
  }
  (void)Gc;
  (void)delta0;
  (void)max_esc;
  return hipGetLastError();
}

// Forward L y = rhs then backward L^T x = y; sw and y are work vectors
// [B][ld]; x receives the solution, acc (optional) accumulates it.
hipError_t launch_trsv(const float *Gw, const float *dinv, int B, int64_t ld, const double *rhs, double *sw,
                       double *y, double *x, double *acc, const int32_t *info, hipStream_t s) {
  const int nb = (int)(ld / kNB);
  for (int j = 0; j < nb; ++j) {
    const int ng = nb - 1 - j > 0 ? nb - 1 - j : 1;
    hipLaunchKernelGGL(k_trsv_step<true>, dim3(ng, B), dim3(256), 0, s, Gw, dinv, ld, j, rhs, sw, y,
                       (double *)nullptr, info);
  }
  for (int j = nb - 1; j >= 0; --j) {
    const int ng = j > 0 ? j : 1;
    hipLaunchKernelGGL(k_trsv_step<false>, dim3(ng, B), dim3(256), 0, s, Gw, dinv, ld, j, (const double *)nullptr,
                       y, x, acc, info);
  }
  return hipGetLastError();
}

hipError_t launch_mass_residual(const float *LT, const float *z, const float *m, const double *w, const float *lam,
                                int B, int n, int t, int64_t tp, int64_t np_, double *u, double *res,
                                const int32_t *info, hipStream_t s, const int32_t *row_list,
                                const int32_t *row_count, const int32_t *col_list, const int32_t *col_count) {
  hipLaunchKernelGGL(k_mass_resid_rows, dim3((unsigned)(np_ / 256), B), dim3(256), 0, s, LT, z, m, w, n, t, tp, np_,
                     u, info, row_list, row_count);
  hipLaunchKernelGGL(k_mass_resid_cols, dim3((unsigned)(tp / (4 * kResKeys)), B), dim3(256), 0, s, LT, z, u, w, lam,
                     n, t, tp, np_, res, info, col_list, col_count);
  return hipGetLastError();
}

// Mass-fit solve for the factored pairs (info == 0): w = (G + lam I)^-1 h by
// the float32 factor, then refine_steps refinement steps against the data
// under the refinement guard above (which needs two steps to compare); pairs the guard cuts off are refactored
// with the ridge raised tenfold and solved again, while escalations remain.
// Each such round reads back one integer (the number of pairs to refactor).
hipError_t launch_mass_solve(float *Gw, const float *Gc, float *dinv, void *lsplit, const MassSolve &ms, int B, int n,
                             int t, int64_t tp, int64_t np_, int refine_steps, int max_esc, FitState st, int32_t *cnt,
                             hipStream_t s) {
  hipError_t e;
  const dim3 gb((B + 255) / 256);
  if ((e = launch_fill_i32(ms.div, B, 0, s)) != hipSuccess) return e;
  for (int round = 0;; ++round) {
    if ((e = launch_trsv(Gw, dinv, B, tp, ms.h, ms.sw, ms.y, ms.w, nullptr, st.info, s)) != hipSuccess) return e;
    for (int it = 0; it < refine_steps; ++it) {
      if ((e = launch_mass_residual(ms.LT, ms.z, ms.m, ms.w, st.lam, B, n, t, tp, np_, ms.u, ms.res, st.info, s,
                                      nullptr, nullptr, nullptr, nullptr)) != hipSuccess)
        return e;
      if ((e = launch_trsv(Gw, dinv, B, tp, ms.res, ms.sw, ms.y, ms.x, ms.w, st.info, s)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_refine_watch, dim3(B), dim3(256), 0, s, ms.w, ms.x, tp, it, ms.rprev, ms.div, st,
                         max_esc);
    }
    if (refine_steps < 2 || round == max_esc) break;
    hipLaunchKernelGGL(k_count_flags, dim3(1), dim3(256), 0, s, B, (const int32_t *)ms.div, cnt);
    int32_t flagged = 0;
    if ((e = hipMemcpyAsync(&flagged, cnt, sizeof(flagged), hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
    if (flagged == 0) break;
    hipLaunchKernelGGL(k_div_mark, gb, dim3(256), 0, s, B, ms.div, st.info);
    if ((e = launch_esc_rounds(Gw, Gc, B, t, tp, max_esc, st, dinv, lsplit, cnt, s)) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_refine_restore, gb, dim3(256), 0, s, B, st.info);
  return hipGetLastError();
}

// Pivoting iterations on the projected fit's refined solution x (in place).
// Each iteration reads back {largest free set, unsettled pairs} to size the
// compressed system and to stop once every pair has settled, so this
// synchronises the stream once per iteration.
hipError_t launch_nnls(const float *Gc, float *Gw, const double *h, const float *LT, const float *z, const float *m,
                       int B, int n, int t, int64_t tp, int64_t np_, int max_iter, int refine_steps, FitState st,
                       float *dinv, void *lsplit, NnlsWork nw, double *x, double *sw, double *yw, double *u,
                       double *res, hipStream_t s) {
  const dim3 gv((unsigned)((tp + 255) / 256), (unsigned)B);
  hipLaunchKernelGGL(k_nnls_init, gv, dim3(256), 0, s, t, tp, st.info, nw.F, nw.y, nw.state);
  hipError_t e;
  for (int it = 0;; ++it) {
    // the update after the last solve only checks feasibility (and marks done)
    hipLaunchKernelGGL(k_nnls_update, dim3(B), dim3(256), 0, s, x, nw.y, h, t, tp, nw.F, nw.state, st.info);
    if (it == max_iter) break;
    hipLaunchKernelGGL(k_nnls_zero, dim3(1), dim3(64), 0, s, nw.red);
    hipLaunchKernelGGL(k_nnls_index, dim3(B), dim3(256), 0, s, nw.F, t, tp, st.info, nw.idx, nw.bidx, nw.pos,
                       nw.nf, nw.nb, nw.red);
    int32_t red[2] = {0, 0};
    if ((e = hipMemcpyAsync(red, nw.red, sizeof(red), hipMemcpyDeviceToHost, s)) != hipSuccess) return e;
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
    if (red[1] == 0) break;   // every pair has settled (or failed)
    const int64_t ldf = red[0] > 256 ? (red[0] + 255) / 256 * 256 : 256;
    const dim3 gf((unsigned)((ldf + 255) / 256), (unsigned)B);
    hipLaunchKernelGGL(k_nnls_gather_gram, dim3((unsigned)((ldf * ldf + 255) / 256), (unsigned)B), dim3(256), 0, s,
                       Gc, tp, nw.idx, nw.nf, st, ldf, Gw);
    if ((e = launch_cholesky_factor(Gw, Gc, B, t, ldf, 0.0f, 0, st, dinv, lsplit, s)) != hipSuccess) return e;
    for (int rs = 0; rs <= refine_steps; ++rs) {
      // rs = 0 solves for x from h; later steps solve for a correction from the
      // residual of the full ridged system against the data, h - (G + lam I) x
      hipLaunchKernelGGL(k_nnls_gather_vec, gf, dim3(256), 0, s, rs == 0 ? h : res, tp, nw.idx, nw.nf, st.info, ldf,
                         nw.rf);
      if ((e = launch_trsv(Gw, dinv, B, ldf, nw.rf, sw, yw, nw.xf, nullptr, st.info, s)) != hipSuccess) return e;
      hipLaunchKernelGGL(k_nnls_scatter, gv, dim3(256), 0, s, nw.xf, ldf, nw.pos, tp, st.info, rs > 0 ? 1 : 0, x);
      // x vanishes off F, so Phi_C x sums over the free keys; the residual is
      // needed on the free keys for a correction, on the bound keys (the dual)
      // after the last one
      const bool last = rs == refine_steps;
      if ((e = launch_mass_residual(LT, z, m, x, st.lam, B, n, t, tp, np_, u, res, st.info, s, nw.idx, nw.nf,
                                    last ? nw.bidx : nw.idx, last ? nw.nb : nw.nf)) != hipSuccess)
        return e;
    }
    hipLaunchKernelGGL(k_nnls_dual, gv, dim3(256), 0, s, res, nw.F, tp, st.info, nw.y);
  }
  hipLaunchKernelGGL(k_nnls_finish, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, nw.state, B, st.info);
  return hipGetLastError();
}

hipError_t launch_bias_finalize(const double *w, int B, int64_t ld, int t, float eps, float bmin, float bmax,
                                const int32_t *info, float *beta, float *beta_ws, hipStream_t s) {
  hipLaunchKernelGGL(k_bias_finalize, dim3((unsigned)((ld + 255) / 256), B), dim3(256), 0, s, w, ld, t, eps, bmin,
                     bmax, info, beta, beta_ws);
  return hipGetLastError();
}

hipError_t launch_phat(int dtype, const float *LT, const float *beta_ws, int B, int n, int t, int64_t tp,
                       int64_t np_, void *out, void *outm, hipStream_t s) {
  dim3 grid((unsigned)(np_ / 64), B);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_phat<bf16>, grid, dim3(256), 0, s, LT, beta_ws, n, t, tp, np_, out, outm);
  else
    hipLaunchKernelGGL(k_phat<float>, grid, dim3(256), 0, s, LT, beta_ws, n, t, tp, np_, out, outm);
  return hipGetLastError();
}

hipError_t launch_transpose128(int dtype, const float *in, int B, int rows, int64_t in_pair, int64_t rows_pad,
                               void *out, int64_t out_pair, hipStream_t s) {
  dim3 grid((unsigned)(rows_pad / 64), B);
  if (dtype == ARCKV_BF16)
    hipLaunchKernelGGL(k_transpose128<bf16>, grid, dim3(256), 0, s, in, rows, in_pair, rows_pad, out, out_pair);
  else
    hipLaunchKernelGGL(k_transpose128<float>, grid, dim3(256), 0, s, in, rows, in_pair, rows_pad, out, out_pair);
  return hipGetLastError();
}

hipError_t launch_trsm(bool fwd, const float *Gw, const float *dinv, int B, int64_t ld, const float *R, float *X,
                       const int32_t *info, hipStream_t s) {
  const void *kern = fwd ? (const void *)k_trsm_mfma<true> : (const void *)k_trsm_mfma<false>;
  const hipError_t e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kTrsmLds);
  if (e != hipSuccess) return e;
  dim3 grid(1, B);
  if (fwd)
    hipLaunchKernelGGL(k_trsm_mfma<true>, grid, dim3(512), kTrsmLds, s, Gw, ld, dinv, R, X, info);
  else
    hipLaunchKernelGGL(k_trsm_mfma<false>, grid, dim3(512), kTrsmLds, s, Gw, ld, dinv, R, X, info);
  return hipGetLastError();
}

// Blocked forward solve L Y = R (see k_trsm_fwd_blk) with the fp32 solve for the
// pairs it flags.  lsplit holds the factorisation's planes, shifts and inverse
// scales (launch_cholesky_factor); tw: Y^T planes [B][2][128][ld] fp16, then
// e [B][128], flags [B] and the fallback mask [B] (int32).
hipError_t launch_trsm_fwd_blocked(const float *Gw, const float *dinv, const void *lsplit, int B, int64_t ld,
                                   const float *R, float *Y, const float *lam, const int32_t *info, void *tw,
                                   hipStream_t s) {
  const f16 *Lp = reinterpret_cast<const f16 *>(lsplit);
  const float *sinv = reinterpret_cast<const float *>(reinterpret_cast<const int32_t *>(Lp + (size_t)B * 2 * ld * ld) +
                                                      (size_t)B * ld);
  f16 *Yt = reinterpret_cast<f16 *>(tw);
  int32_t *ex = reinterpret_cast<int32_t *>(Yt + (size_t)B * 2 * kHeadDim * ld);
  int32_t *flag = ex + (size_t)B * kHeadDim;
  int32_t *mask = flag + B;
  hipLaunchKernelGGL(k_trsm_colexp, dim3(B), dim3(1024), 0, s, R, ld, lam, info, ex, flag);
  const int nblk = (int)(ld / 256);
  for (int kb = 0; kb < nblk; ++kb) {
    if (kb > 0) {
      const int K0 = 256 * kb;
      BigShape g{B, 256, kHeadDim, K0, 2 * ld * ld, ld * ld, ld, 2 * kHeadDim * ld, kHeadDim * ld, ld, false, 1};
      EpiTrsmFwd<2, 2> e{R, Y, ld, K0, sinv, ex, info, flag};
      const hipError_t err = launch_gemm_big<4, 2, 2, 2, 32, 2, 2, 3, f16>(
          g, reinterpret_cast<const bf16 *>(Lp + (size_t)K0 * ld), reinterpret_cast<const bf16 *>(Yt), e, s);
      if (err != hipSuccess) return err;
    }
    hipLaunchKernelGGL(k_trsm_fwd_blk, dim3(B), dim3(512), 0, s, Gw, dinv, ld, kb, kb == 0 ? R : Y, Y, Yt, ex, info,
                       flag);
  }
  hipLaunchKernelGGL(k_trsm_colcheck, dim3(B), dim3(1024), 0, s, Y, ld, ex, info, flag);
  hipLaunchKernelGGL(k_trsm_fallback_mask, dim3((B + 255) / 256), dim3(256), 0, s, info, flag, B, mask);
  return launch_trsm(true, Gw, dinv, B, ld, R, Y, mask, s);
}

hipError_t launch_add(float *x, const float *dx, int B, int64_t n_per, const int32_t *info, hipStream_t s) {
  hipLaunchKernelGGL(k_add_copy, dim3((unsigned)((n_per + 255) / 256), B), dim3(256), 0, s, x, dx, n_per, info);
  return hipGetLastError();
}

hipError_t launch_values_out(const float *Xp, int B, int64_t tp, int t, const int32_t *info, float *Cv,
                             hipStream_t s) {
  hipLaunchKernelGGL(k_values_out, dim3((unsigned)(((int64_t)t * kHeadDim + 255) / 256), B), dim3(256), 0, s, Xp, tp,
                     t, info, Cv);
  return hipGetLastError();
}

}  // namespace arckv
