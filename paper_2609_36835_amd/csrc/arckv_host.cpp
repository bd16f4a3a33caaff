// Host side of the ARC-KV library: argument validation (before any HIP call),
// workspace planning, and stage sequencing on the caller's stream.
#include <math.h>
#include <mutex>
#include <stdint.h>
#include <string.h>
#include <vector>

#include <hip/hip_runtime.h>

#include "arckv.h"
#include "assign.hpp"
#include "fit.hpp"

namespace arckv {
typedef uint16_t bf16_t_;   // bfloat16 storage, opaque on the host
constexpr int kHeadDimH = 128;
constexpr int64_t kPadH = 256;
inline int64_t rup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

hipError_t launch_score(int dtype, const void *K, const void *V, const void *W1, const float *b1, const float *w2,
                        const float *b2, float *scores, int B, int T, hipStream_t s);
hipError_t launch_select(const float *scores, int B, int T, int t, int32_t *anchors, hipStream_t s);
hipError_t launch_select_ex(const float *scores, int B, int T, int t, const int32_t *t_pair, int chunk_len,
                            int t_stride, int32_t *anchors, hipStream_t s);
constexpr int kChunkThresholdH = 10000;   // chunked selection applies when T > 10,000

// Realised anchor count of chunked selection (Appendix A.3), in double exactly as
// the select kernel computes each chunk's share.
static int64_t chunked_count(int64_t T, int64_t t, int64_t chunk_len) {
  if (chunk_len <= 0 || T <= kChunkThresholdH) return t;
  int64_t total = 0;
  for (int64_t start = 0; start < T; start += chunk_len) {
    const int64_t Tc = T - start < chunk_len ? T - start : chunk_len;
    int64_t v = (int64_t)floor((double)t * (double)Tc / (double)T + 0.5);
    v = v < 1 ? 1 : (v > Tc ? Tc : v);
    total += v;
  }
  return total;
}
hipError_t launch_rowstats(int dtype, const void *K, const void *V, const void *Q, float *z, float *m, float *Y,
                           int B, int T, int n, float scale, hipStream_t s);
hipError_t launch_profiles(int dtype, const void *Q, const void *K, const float *zmerge, const int32_t *anchors,
                           int t, void *Et, float *phi, int B, int T, int n, int64_t Tp, int64_t np_, float scale,
                           hipStream_t s);
hipError_t launch_phic(int dtype, const void *Q, const void *Ckp, const float *z, void *PhiT, float *LT,
                       const float *m, double *h, int B, int t, int n, int64_t tp, int64_t np_, float scale,
                       hipStream_t s);
hipError_t launch_zmax(const float *z, int B, int n, float *zmax, hipStream_t s);
hipError_t launch_pair_norms(int dtype, const void *Q, const void *K, const int32_t *anchors, int P, int n, int T,
                             int t, void *pn, hipStream_t s);
hipError_t launch_anchor_profiles(int dtype, const void *Q, const void *K, const int32_t *anchors,
                                  const float *zmerge, int P, int n, int T, int t, int64_t tp, int64_t np_,
                                  float scale, float *Ua, double *anorm, void *U, hipStream_t s);
hipError_t launch_assign_finalize(int dtype, const void *K, const uint64_t *part1, const uint64_t *part2,
                                  const uint32_t *part3, int MT, int TR, int64_t Np, const int32_t *anchors,
                                  const float *phi, const float *zmerge, const void *pn, int P, int T, int t, int n,
                                  float scale, int32_t *kappa, const AssignLists &L, hipStream_t s);
hipError_t launch_assign_refine(int dtype, const void *Q, const void *K, const float *zmerge, const void *pn,
                                const float *Ua, const double *anorm, int P, int T, int t, int n, int64_t tp,
                                int64_t np_, float scale, int32_t *kappa, const AssignLists &L, hipStream_t s);
hipError_t launch_assign_exact(int dtype, const void *Q, const void *K, const int32_t *anchors, const float *zmerge,
                               int P, int T, int t, int n, float scale, int32_t *kappa, const AssignLists &L,
                               hipStream_t s);
hipError_t launch_fill_i32(int32_t *p, int64_t count, int32_t v, hipStream_t s);
hipError_t launch_group_merge(int dtype, const void *K, const float *phi, const int32_t *kappa,
                              const int32_t *anchors, int B, int T, int t, int64_t tp, float lambda,
                              int32_t *offsets, int32_t *cursor, int32_t *perm, float *Ck, void *Ckp, hipStream_t s);
hipError_t launch_assign_gemm(int dtype, const void *U, const void *Et, uint64_t *part1, uint64_t *part2,
                              uint32_t *part3, int P, int t, int64_t tp, int64_t N, int64_t Et_rows, int64_t np_,
                              hipStream_t s);
hipError_t launch_gram(int dtype, const void *X, float *G, float *Gc, int P, int64_t tp, int64_t np_, hipStream_t s);
hipError_t launch_rhs_gemm(int dtype, const void *PT, const void *YT, float *Bm, int P, int64_t tp, int64_t np_,
                           hipStream_t s);
hipError_t launch_value_residual(int dtype, const void *XT, const void *Pm, const void *PT, const float *Y, void *UT,
                                 const float *X, const float *lam, float *R, int P, int n, int64_t tp, int64_t np_,
                                 hipStream_t s);
hipError_t launch_mass_residual(const float *LT, const float *z, const float *m, const double *w, const float *lam,
                                int B, int n, int t, int64_t tp, int64_t np_, double *u, double *res,
                                const int32_t *info, hipStream_t s, const int32_t *row_list = nullptr,
                                const int32_t *row_count = nullptr, const int32_t *col_list = nullptr,
                                const int32_t *col_count = nullptr);
hipError_t launch_mass_solve(float *Gw, const float *Gc, float *dinv, void *lsplit, const MassSolve &ms, int B, int n,
                             int t, int64_t tp, int64_t np_, int refine_steps, int max_esc, FitState st, int32_t *cnt,
                             hipStream_t s);
hipError_t launch_cholesky(float *Gw, const float *Gc, int B, int t, int64_t ld, float delta0, int max_esc,
                           FitState st, float *dinv, void *lsplit, const int32_t *bad, int32_t *cnt,
                           hipStream_t s);
hipError_t launch_nonfinite(const float *a, int B, int64_t per, int32_t *bad, hipStream_t s);
hipError_t launch_trsv(const float *Gw, const float *dinv, int B, int64_t ld, const double *rhs, double *sw,
                       double *y, double *x, double *acc, const int32_t *info, hipStream_t s);
hipError_t launch_cholesky_factor(float *Gw, const float *Gc, int B, int t, int64_t ld, float delta0, int max_esc,
                                  FitState st, float *dinv, void *lsplit, hipStream_t s);
hipError_t launch_nnls(const float *Gc, float *Gw, const double *h, const float *LT, const float *z, const float *m,
                       int B, int n, int t, int64_t tp, int64_t np_, int max_iter, int refine_steps, FitState st,
                       float *dinv, void *lsplit, NnlsWork nw, double *x, double *sw, double *yw, double *u,
                       double *res, hipStream_t s);
hipError_t launch_bias_finalize(const double *w, int B, int64_t ld, int t, float eps, float bmin, float bmax,
                                const int32_t *info, float *beta, float *beta_ws, hipStream_t s);
hipError_t launch_phat(int dtype, const float *LT, const float *beta_ws, int B, int n, int t, int64_t tp,
                       int64_t np_, void *out, void *outm, hipStream_t s);
hipError_t launch_transpose128(int dtype, const float *in, int B, int rows, int64_t in_pair, int64_t rows_pad,
                               void *out, int64_t out_pair, hipStream_t s);
hipError_t launch_trsm(bool fwd, const float *Gw, const float *dinv, int B, int64_t ld, const float *R, float *X,
                       const int32_t *info, hipStream_t s);
hipError_t launch_trsm_fwd_blocked(const float *Gw, const float *dinv, const void *lsplit, int B, int64_t ld,
                                   const float *R, float *Y, const float *lam, const int32_t *info, void *tw,
                                   hipStream_t s);
hipError_t launch_add(float *x, const float *dx, int B, int64_t n_per, const int32_t *info, hipStream_t s);
hipError_t launch_values_out(const float *Xp, int B, int64_t tp, int t, const int32_t *info, float *Cv,
                             hipStream_t s);
hipError_t launch_copy_info(const int32_t *a, const int32_t *b, int B, int32_t *info, hipStream_t s);
hipError_t launch_copy_f32(const float *src, float *dst, int B, hipStream_t s);
int attend_chunks(int t, int F);
size_t attend_scratch_bytes();
hipError_t attend_scratch(void **ptr);
hipError_t launch_dsa_proj(const void *X1, const void *X2, bool x2_f32, const void *W1, const void *W2, int B,
                           int nrows, int n_blocks, bool norm, void *out, hipStream_t s);
hipError_t launch_dsa_w(const void *X, const void *Lx, const float *bx, int B, int n_pos, int dx, int x_group,
                        int p_off, float *w, hipStream_t s);
hipError_t launch_dsa_index(int pass, const void *qbar, const void *kbar, const float *w, int B, int n, int n_pos,
                            int T, float *z, float *m, float *part, hipStream_t s);
hipError_t launch_dsa_pool(const float *part, int B, int n, int T, float *scores, hipStream_t s);
int dsa_query_blocks(int n);
hipError_t launch_attend(int P, int G, int t, int F, float scale, const void *Q, const void *Ck, const float *beta,
                         const void *Cv, const void *Kf, const void *Vf, float *part_o, float *part_ml, float *out,
                         hipStream_t s);

// ------------------------------------------------------------------ timing
enum Stage {
  ST_SCORE, ST_SELECT, ST_ROWSTATS, ST_ZMAX, ST_PROFILES, ST_ANCHOR_PROF, ST_ASSIGN, ST_FINALIZE, ST_MERGE,
  ST_PHIC, ST_GRAM_G, ST_CHOL_G, ST_SOLVE_W, ST_PHAT, ST_GRAM_A, ST_RHS, ST_CHOL_A, ST_SOLVE_V, ST_ATTEND,
  ST_DSA_PROJ, ST_DSA_VALUE, ST_DSA_INDEX, ST_ASSIGN_REFINE, ST_ASSIGN_EXACT, ST_COUNT
};
static const char *kStageNames[ST_COUNT] = {
    "score", "select", "rowstats", "zmax", "profiles", "anchor_profiles", "assign_gemm", "assign_finalize",
    "merge", "phic", "gram_G", "chol_G", "solve_beta", "phat", "gram_A", "rhs_B", "chol_A", "solve_values",
    "attend", "dsa_proj", "dsa_value_head", "dsa_index", "assign_refine", "assign_exact"};

struct TimingState {
  std::mutex mu;
  bool enabled = false;
  struct Rec { int stage; hipEvent_t a, b; };
  std::vector<Rec> pending;
  std::vector<hipEvent_t> pool;
  double ms[ST_COUNT] = {0};
  int32_t cnt[ST_COUNT] = {0};
};
static TimingState g_timing;

static hipEvent_t take_event() {
  if (!g_timing.pool.empty()) {
    hipEvent_t e = g_timing.pool.back();
    g_timing.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct StageScope {
  int stage;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  StageScope(int st, hipStream_t str) : stage(st), s(str) {
    if (!g_timing.enabled) return;
    std::lock_guard<std::mutex> lk(g_timing.mu);
    a = take_event();
    b = take_event();
    if (a) (void)hipEventRecord(a, s);
  }
  ~StageScope() {
    if (!a || !b) return;
    (void)hipEventRecord(b, s);
    std::lock_guard<std::mutex> lk(g_timing.mu);
    g_timing.pending.push_back({stage, a, b});
  }
};
#define STAGE(id, expr)                              \
  do {                                               \
    StageScope _sc(id, stream);                      \
    if ((expr) != hipSuccess) return ARCKV_ERR_HIP;  \
  } while (0)

// ------------------------------------------------------------------ workspace plan
struct Dims {
  int B, T, n, t, dtype;
  int64_t Tp, np_, tp, MT;
  int64_t esz;   // bytes per element of E^T / U_S
};

static Dims make_dims(const arckv_problem *p, int t) {
  Dims d;
  d.B = p->B;
  d.T = p->T;
  d.n = p->n;
  d.t = t;
  d.dtype = p->dtype;
  d.Tp = rup(p->T, kPadH);
  d.np_ = rup(p->n, kPadH);
  d.tp = rup(t, kPadH);
  d.MT = d.tp / 128;
  d.esz = p->dtype == ARCKV_BF16 ? 2 : 4;
  return d;
}

// Capacity of the assignment's candidate pool, per cached key of a pair (about 1
// candidate per key at the 32K workload; a key whose list does not fit keeps its
// first-pass decision and is counted as undecided).
constexpr int64_t kPoolPerKey = 8;

struct Bump {
  int64_t off = 0;
  int64_t take(int64_t bytes) {
    int64_t o = off;
    off += rup(bytes, 256);
    return o;
  }
};

// Persistent per-pair arrays ([B]-sized) followed by a chunk region for P pairs.
struct Plan {
  // persistent
  int64_t scores, z, m, Y, zmax, kappa, phi, beta_ws, info_g, info_a, st_g, st_a, astats, bad, cnt;
  int64_t persistent_bytes;
  // chunk region (offsets relative to chunk base)
  int64_t Ckp;
  int64_t Et, U, Ua, anorm, pn, part1, part2, part3, fcnt, fkey, foff, fn, pcnt, pool, psim, dcnt, dkey, dn,
      doff, goff, dgrp, dgn, dsim, dr, ditem;   // merge phase
  int64_t offsets, cursor, perm;
  int64_t PhiT, LT, Gw, Gc, dinv, lsplit, tw, h, w, y, x, res, sw, rprev, div, u, YT, Bm, X, R, Y2, XT, Pm, UT;  // fit phase
  int64_t nF, nidx, nbidx, npos, nnf, nnb, nstate, nred, ny, nrhs, ndx;   // exact NNLS (bias_mode 1)
  int64_t chunk_bytes;
};

static Plan make_plan(const Dims &d, int64_t P) {
  Plan pl;
  Bump a;
  const int64_t B = d.B;
  pl.scores = a.take(B * d.T * 4);
  pl.z = a.take(B * d.n * 4);
  pl.m = a.take(B * d.n * 4);
  pl.Y = a.take(B * d.n * kHeadDimH * 4);
  pl.zmax = a.take(B * 4);
  pl.kappa = a.take(B * d.T * 4);
  pl.phi = a.take(B * d.T * 4);
  pl.beta_ws = a.take(B * d.tp * 4);
  pl.info_g = a.take(B * 4);
  pl.info_a = a.take(B * 4);
  pl.st_g = a.take(B * 24);    // trace (8) + lam (4) + delta (4) + nesc (4) + pad (4)
  pl.st_a = a.take(B * 24);
  pl.astats = a.take(B * kAssignStats * 4);  // assignment statistics [B][kAssignStats]
  pl.bad = a.take(B * 4);                     // non-finite inputs of the current fit [B]
  pl.cnt = a.take(16);                        // failed-factorisation count read back by the host
  pl.persistent_bytes = a.off;

  Bump c;
  pl.Ckp = c.take(P * d.tp * kHeadDimH * 4);
  const int64_t phase0 = c.off;
  Bump m = c;
  pl.Et = m.take(P * d.Tp * d.np_ * d.esz);
  pl.U = m.take(P * d.tp * d.np_ * d.esz);
  pl.Ua = m.take(P * d.tp * d.np_ * 4);       // precise anchor profiles (fp32)
  pl.anorm = m.take(P * d.tp * 8);
  pl.pn = m.take(P * 16);
  pl.part1 = m.take(P * d.MT * d.Tp * 8);     // top-3 partials per (anchor tile, key)
  pl.part2 = m.take(P * d.MT * d.Tp * 8);
  pl.part3 = m.take(P * d.MT * d.Tp * 4);
  pl.fcnt = m.take(P * 4);
  pl.fkey = m.take(P * d.Tp * 4);
  pl.foff = m.take(P * d.Tp * 4);
  pl.fn = m.take(P * d.Tp * 4);
  pl.pcnt = m.take(P * 4);
  pl.pool = m.take(P * kPoolPerKey * d.Tp * 4);   // candidate pool: kPoolPerKey entries per key on average
  pl.psim = m.take(P * kPoolPerKey * d.Tp * 8);
  pl.dcnt = m.take(P * 4);
  const int64_t dcap = pass_d_capacity(d.Tp, kPoolPerKey);
  pl.dkey = m.take(P * dcap * 4);
  pl.dn = m.take(P * dcap * 4);
  pl.doff = m.take(P * dcap * 4);
  pl.goff = m.take(P * (d.Tp / 64 + 2) * 4);   // pass C work items per group of 64 queued keys
  pl.dgrp = m.take(P * dcap * 4);
  pl.dgn = m.take(P * dcap * 4);
  pl.dsim = m.take(P * dcap * 8);
  pl.dr = m.take(P * dcap * 4);
  pl.ditem = m.take(P * (dcap + 2) * 4);
  pl.offsets = m.take(P * (int64_t)(d.t + 1) * 4);
  pl.cursor = m.take(P * (int64_t)d.t * 4);
  pl.perm = m.take(P * (int64_t)d.T * 4);
  Bump f = c;
  pl.PhiT = f.take(P * d.tp * d.np_ * 4);   // two bf16 planes or one fp32 plane
  pl.LT = f.take(P * d.tp * d.np_ * 4);
  pl.Gw = f.take(P * d.tp * d.tp * 4);
  pl.Gc = f.take(P * d.tp * d.tp * 4);
  pl.dinv = f.take(P * d.tp * 64 * 4);   // one 64 x 64 inverse per diagonal block
  pl.lsplit = f.take(P * (4 * d.tp * d.tp + 8 * d.tp));   // L's fp16 hi / lo planes, row shifts and scales
  pl.tw = f.take(P * (4 * kHeadDimH * d.tp + 4 * kHeadDimH + 8));   // forward solve: Y^T planes, column scales, flags
  pl.h = f.take(P * d.tp * 8);
  pl.w = f.take(P * d.tp * 8);
  pl.y = f.take(P * d.tp * 8);
  pl.x = f.take(P * d.tp * 8);
  pl.res = f.take(P * d.tp * 8);
  pl.sw = f.take(P * d.tp * 8);
  pl.rprev = f.take(P * 8);
  pl.div = f.take(P * 4);
  pl.u = f.take(P * d.np_ * 8);
  pl.YT = f.take(P * kHeadDimH * d.np_ * 4);
  pl.Bm = f.take(P * d.tp * kHeadDimH * 4);
  pl.X = f.take(P * d.tp * kHeadDimH * 4);
  pl.R = f.take(P * d.tp * kHeadDimH * 4);
  pl.Y2 = f.take(P * d.tp * kHeadDimH * 4);
  pl.XT = f.take(P * d.tp * kHeadDimH * 4);
  pl.Pm = f.take(P * d.tp * d.np_ * 4);
  pl.UT = f.take(P * kHeadDimH * d.np_ * 4);
  pl.nF = f.take(P * d.tp * 4);
  pl.nidx = f.take(P * d.tp * 4);
  pl.nbidx = f.take(P * d.tp * 4);
  pl.npos = f.take(P * d.tp * 4);
  pl.nnf = f.take(P * 4);
  pl.nnb = f.take(P * 4);
  pl.nstate = f.take(P * 16);
  pl.nred = f.take(16);
  pl.ny = f.take(P * d.tp * 8);
  pl.nrhs = f.take(P * d.tp * 8);
  pl.ndx = f.take(P * d.tp * 8);
  (void)phase0;
  pl.chunk_bytes = m.off > f.off ? m.off : f.off;
  return pl;
}

static size_t plan_total(const Dims &d, int64_t P) {
  Plan pl = make_plan(d, P);
  return (size_t)(pl.persistent_bytes + pl.chunk_bytes);
}

// Largest chunk of pairs that fits the workspace (0 if not even one).
static int64_t chunk_for(const Dims &d, size_t ws_bytes, int64_t want) {
  const size_t one = plan_total(d, 1);
  if (ws_bytes < one) return 0;
  const size_t per = plan_total(d, 2) - one;
  int64_t P = 1 + (int64_t)((ws_bytes - one) / (per ? per : 1));
  const int64_t cap = (want > 0 && want < d.B) ? want : d.B;
  if (P > cap) P = cap;
  while (P > 1 && plan_total(d, P) > ws_bytes) --P;
  while (P < cap && plan_total(d, P + 1) <= ws_bytes) ++P;
  return P;
}

// ------------------------------------------------------------------ validation
static bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

static arckv_status check_problem(const arckv_problem *p) {
  if (!p) return ARCKV_ERR_INVALID_ARG;
  if (p->B < 1 || p->T < 1 || p->n < 1) return ARCKV_ERR_INVALID_ARG;
  if (p->d != kHeadDimH) return ARCKV_ERR_UNSUPPORTED;
  if (p->dtype != ARCKV_F32 && p->dtype != ARCKV_BF16) return ARCKV_ERR_UNSUPPORTED;
  if (!isfinite(p->scale)) return ARCKV_ERR_INVALID_ARG;
  if ((int64_t)p->T > (1ll << 30) || (int64_t)p->n > (1ll << 30)) return ARCKV_ERR_UNSUPPORTED;
  return ARCKV_OK;
}

static arckv_status check_params(const arckv_fit_params *p) {
  if (!p) return ARCKV_ERR_INVALID_ARG;
  if (!(p->lambda_m >= 0.0f && p->lambda_m <= 1.0f)) return ARCKV_ERR_INVALID_ARG;
  if (!(p->delta_beta >= 0.0f) || !isfinite(p->delta_beta)) return ARCKV_ERR_INVALID_ARG;
  if (!(p->delta_v >= 0.0f) || !isfinite(p->delta_v)) return ARCKV_ERR_INVALID_ARG;
  if (!(p->eps_w > 0.0f) || !isfinite(p->eps_w)) return ARCKV_ERR_INVALID_ARG;
  if (!(p->b_min <= p->b_max) || !isfinite(p->b_min) || !isfinite(p->b_max)) return ARCKV_ERR_INVALID_ARG;
  if (p->bias_mode != 0 && p->bias_mode != 1) return ARCKV_ERR_UNSUPPORTED;
  if (p->nnls_max_iter < 1 || p->nnls_max_iter > 256) return ARCKV_ERR_INVALID_ARG;
  if (p->max_escalations < 0 || p->max_escalations > 6) return ARCKV_ERR_INVALID_ARG;
  if (p->refine_steps < 0 || p->refine_steps > 4) return ARCKV_ERR_INVALID_ARG;
  if (p->value_refine_steps < 0 || p->value_refine_steps > 4) return ARCKV_ERR_INVALID_ARG;
  if (p->pair_chunk < 0) return ARCKV_ERR_INVALID_ARG;
  if (p->select_chunk < 0) return ARCKV_ERR_INVALID_ARG;
  return ARCKV_OK;
}

static float eff_scale(const arckv_problem *p) {
  return p->scale > 0.0f ? p->scale : 1.0f / sqrtf((float)p->d);
}

static arckv_status check_ws(const Dims &d, void *ws, size_t ws_bytes, int64_t want, int64_t *P) {
  if (!ws || !aligned(ws, 256)) return ARCKV_ERR_WORKSPACE;
  *P = chunk_for(d, ws_bytes, want);
  return *P >= 1 ? ARCKV_OK : ARCKV_ERR_WORKSPACE;
}

#define CHECK(x)                              \
  do {                                        \
    arckv_status _s = (x);                    \
    if (_s != ARCKV_OK) return _s;            \
  } while (0)

// ------------------------------------------------------------------ stage bodies
struct Ctx {
  Dims d;
  Plan pl;
  char *ws;
  float scale;
  hipStream_t stream;
  template <typename T> T *pers(int64_t off) const { return reinterpret_cast<T *>(ws + off); }
  template <typename T> T *chunk(int64_t off) const { return reinterpret_cast<T *>(ws + pl.persistent_bytes + off); }
  int64_t in_esz() const { return d.dtype == ARCKV_BF16 ? 2 : 4; }
};

// Merge stage for pairs [b0, b0+P): needs zmax for those pairs.
static arckv_status run_merge_chunk(const Ctx &c, int b0, int P, const void *K, const void *Q,
                                    const int32_t *anchors, float lambda_m, float *Ck, int32_t *kappa, float *phi,
                                    const float *zmax) {
  const Dims &d = c.d;
  hipStream_t stream = c.stream;
  const char *Kc = (const char *)K + (size_t)b0 * d.T * kHeadDimH * c.in_esz();
  const char *Qc = (const char *)Q + (size_t)b0 * d.n * kHeadDimH * c.in_esz();
  const int32_t *anc = anchors + (size_t)b0 * d.t;
  void *Et = c.chunk<char>(c.pl.Et);
  void *U = c.chunk<char>(c.pl.U);
  float *Ua = c.chunk<float>(c.pl.Ua);
  double *anorm = c.chunk<double>(c.pl.anorm);
  void *pn = c.chunk<char>(c.pl.pn);
  uint64_t *part1 = c.chunk<uint64_t>(c.pl.part1), *part2 = c.chunk<uint64_t>(c.pl.part2);
  uint32_t *part3 = c.chunk<uint32_t>(c.pl.part3);
  AssignLists L{c.chunk<int32_t>(c.pl.fcnt), c.chunk<int32_t>(c.pl.fkey),  c.chunk<int32_t>(c.pl.foff),
                c.chunk<int32_t>(c.pl.fn),   c.chunk<int32_t>(c.pl.pcnt),  c.chunk<int32_t>(c.pl.pool),
                c.chunk<double>(c.pl.psim),  kPoolPerKey * d.Tp,           c.chunk<int32_t>(c.pl.dcnt),
                c.chunk<int32_t>(c.pl.dkey), c.chunk<int32_t>(c.pl.dn),    c.chunk<int32_t>(c.pl.doff),
                c.pers<int32_t>(c.pl.astats) + (size_t)b0 * kAssignStats, d.Tp,
                c.chunk<int32_t>(c.pl.goff), d.Tp / 64 + 2,
                c.chunk<int32_t>(c.pl.dgrp), c.chunk<int32_t>(c.pl.dgn), c.chunk<double>(c.pl.dsim),
                c.chunk<int32_t>(c.pl.dr),   c.chunk<int32_t>(c.pl.ditem), pass_d_capacity(d.Tp, kPoolPerKey)};
  const float *zm = zmax + b0;
  int32_t *kap = kappa + (size_t)b0 * d.T;
  const float *phib = phi + (size_t)b0 * d.T;
  // the assignment contraction runs over the T - t non-anchor keys (compacted E^T rows)
  const int64_t Tc = rup(d.T - d.t, kPadH);
  const int TR = d.dtype == ARCKV_BF16 ? 256 : 128;               // anchor rows per contraction tile
  const int mt_used = (int)(d.tp / TR);
  STAGE(ST_PROFILES, launch_profiles(d.dtype, Qc, Kc, zm, anc, d.t, Et, phi + (size_t)b0 * d.T, P, d.T, d.n, d.Tp,
                                     d.np_, c.scale, stream));
  STAGE(ST_ANCHOR_PROF, launch_pair_norms(d.dtype, Qc, Kc, anc, P, d.n, d.T, d.t, pn, stream));
  STAGE(ST_ANCHOR_PROF, launch_anchor_profiles(d.dtype, Qc, Kc, anc, zm, P, d.n, d.T, d.t, d.tp, d.np_, c.scale, Ua,
                                               anorm, U, stream));
  STAGE(ST_ASSIGN, launch_assign_gemm(d.dtype, U, Et, part1, part2, part3, P, d.t, d.tp, Tc, d.Tp, d.np_, stream));
  STAGE(ST_FINALIZE, launch_assign_finalize(d.dtype, Kc, part1, part2, part3, mt_used, TR, Tc, anc, phib, zm, pn, P,
                                            d.T, d.t, d.n, c.scale, kap, L, stream));
  STAGE(ST_ASSIGN_REFINE, launch_assign_refine(d.dtype, Qc, Kc, zm, pn, Ua, anorm, P, d.T, d.t, d.n, d.tp, d.np_,
                                               c.scale, kap, L, stream));
  STAGE(ST_ASSIGN_EXACT, launch_assign_exact(d.dtype, Qc, Kc, anc, zm, P, d.T, d.t, d.n, c.scale, kap, L, stream));
  STAGE(ST_MERGE, launch_group_merge(d.dtype, Kc, phi + (size_t)b0 * d.T, kappa + (size_t)b0 * d.T, anc, P, d.T,
                                     d.t, d.tp, lambda_m, c.chunk<int32_t>(c.pl.offsets),
                                     c.chunk<int32_t>(c.pl.cursor), c.chunk<int32_t>(c.pl.perm),
                                     Ck + (size_t)b0 * d.t * kHeadDimH, c.chunk<char>(c.pl.Ckp), stream));
  return ARCKV_OK;
}

// Padded compact-key operand copy for pairs [b0, b0+P) from a user C_k.
hipError_t launch_pad_ck(int dtype, const float *Ck, int P, int t, int64_t tp, void *Ckp, hipStream_t s);

static FitState fit_state(const Ctx &c, int64_t st_off, int64_t info_off, int b0) {
  FitState st;
  char *base = c.pers<char>(st_off);
  const int B = c.d.B;
  st.trace = reinterpret_cast<double *>(base) + b0;
  st.lam = reinterpret_cast<float *>(base + (size_t)B * 8) + b0;
  st.delta = reinterpret_cast<float *>(base + (size_t)B * 12) + b0;
  st.nesc = reinterpret_cast<int32_t *>(base + (size_t)B * 16) + b0;
  st.info = c.pers<int32_t>(info_off) + b0;
  return st;
}

// Mass fit for pairs [b0, b0+P): needs Ckp (chunk), z, m.
// Y (may be null) is only checked for non-finite values, so that arckv_compact
// reports a non-finite V (which reaches Y alone) in both fits.
static arckv_status run_fit_bias_chunk(const Ctx &c, int b0, int P, const void *Q, const float *z, const float *m,
                                       const float *Ck, const arckv_fit_params &fp, float *beta, FitState st,
                                       const float *Y = nullptr) {
  const Dims &d = c.d;
  hipStream_t stream = c.stream;
  const char *Qc = (const char *)Q + (size_t)b0 * d.n * kHeadDimH * c.in_esz();
  const float *zc = z + (size_t)b0 * d.n, *mc = m + (size_t)b0 * d.n;
  void *PhiT = c.chunk<char>(c.pl.PhiT);
  float *LT = c.chunk<float>(c.pl.LT), *Gw = c.chunk<float>(c.pl.Gw), *Gc = c.chunk<float>(c.pl.Gc);
  double *h = c.chunk<double>(c.pl.h), *w = c.chunk<double>(c.pl.w), *y = c.chunk<double>(c.pl.y);
  double *x = c.chunk<double>(c.pl.x), *res = c.chunk<double>(c.pl.res), *sw = c.chunk<double>(c.pl.sw);
  float *dinv = c.chunk<float>(c.pl.dinv);
  // pairs whose inputs (z, m, C_k, and Y when given) hold a non-finite value report info = -1
  int32_t *bad = c.pers<int32_t>(c.pl.bad) + b0;
  if (launch_fill_i32(bad, P, 0, stream) != hipSuccess || launch_nonfinite(zc, P, d.n, bad, stream) != hipSuccess ||
      (Y && launch_nonfinite(Y + (size_t)b0 * d.n * kHeadDimH, P, (int64_t)d.n * kHeadDimH, bad, stream) !=
                hipSuccess) ||
      launch_nonfinite(mc, P, d.n, bad, stream) != hipSuccess ||
      launch_nonfinite(Ck + (size_t)b0 * d.t * kHeadDimH, P, (int64_t)d.t * kHeadDimH, bad, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  // Phi_C^T (split planes), the logits L^T, and h = Phi_C^T m in one pass
  STAGE(ST_PHIC, launch_phic(d.dtype, Qc, c.chunk<char>(c.pl.Ckp), zc, PhiT, LT, mc, h, P, d.t, d.n, d.tp, d.np_,
                             c.scale, stream));
  STAGE(ST_GRAM_G, launch_gram(d.dtype, PhiT, Gw, Gc, P, d.tp, d.np_, stream));
  STAGE(ST_CHOL_G, launch_cholesky(Gw, Gc, P, d.t, d.tp, fp.delta_beta, fp.max_escalations, st, dinv,
                                   c.chunk<char>(c.pl.lsplit), bad, c.pers<int32_t>(c.pl.cnt), stream));
  {
    StageScope _sc(ST_SOLVE_W, stream);
    double *u = c.chunk<double>(c.pl.u);
    const MassSolve ms{LT, zc, mc, h, w, x, y, sw, u, res, c.chunk<double>(c.pl.rprev), c.chunk<int32_t>(c.pl.div)};
    if (launch_mass_solve(Gw, Gc, dinv, c.chunk<char>(c.pl.lsplit), ms, P, d.n, d.t, d.tp, d.np_, fp.refine_steps,
                          fp.max_escalations, st, c.pers<int32_t>(c.pl.cnt), stream) != hipSuccess)
      return ARCKV_ERR_HIP;
    if (fp.bias_mode == 1) {
      // exact NNLS on the ridged system whose ridge the factorisation above
      // settled, pivoting from the unconstrained solution w
      NnlsWork nw{c.chunk<int32_t>(c.pl.nF),  c.chunk<int32_t>(c.pl.nidx),   c.chunk<int32_t>(c.pl.nbidx),
                  c.chunk<int32_t>(c.pl.npos), c.chunk<int32_t>(c.pl.nnf),    c.chunk<int32_t>(c.pl.nnb),
                  c.chunk<int32_t>(c.pl.nstate), c.chunk<int32_t>(c.pl.nred), c.chunk<double>(c.pl.ny),
                  c.chunk<double>(c.pl.nrhs),  c.chunk<double>(c.pl.ndx)};
      if (launch_nnls(Gc, Gw, h, LT, zc, mc, P, d.n, d.t, d.tp, d.np_, fp.nnls_max_iter, fp.refine_steps, st, dinv,
                      c.chunk<char>(c.pl.lsplit), nw, w, sw, y, u, res, stream) != hipSuccess)
        return ARCKV_ERR_HIP;
    }
    if (launch_bias_finalize(w, P, d.tp, d.t, fp.eps_w, fp.b_min, fp.b_max, st.info, beta + (size_t)b0 * d.t,
                             c.pers<float>(c.pl.beta_ws) + (size_t)b0 * d.tp, stream) != hipSuccess)
      return ARCKV_ERR_HIP;
  }
  return ARCKV_OK;
}

hipError_t launch_pad_beta(const float *beta, int P, int t, int64_t tp, float *beta_ws, hipStream_t s);

// Value fit for pairs [b0, b0+P): needs LT (from the mass fit, or recomputed),
// beta_ws, Y.
static arckv_status run_fit_values_chunk(const Ctx &c, int b0, int P, const float *Y, const float *Ck,
                                         const float *beta, const arckv_fit_params &fp, float *Cv, FitState st) {
  const Dims &d = c.d;
  hipStream_t stream = c.stream;
  void *PT = c.chunk<char>(c.pl.PhiT);
  float *LT = c.chunk<float>(c.pl.LT), *Gw = c.chunk<float>(c.pl.Gw), *Gc = c.chunk<float>(c.pl.Gc);
  void *YT = c.chunk<char>(c.pl.YT);
  float *Bm = c.chunk<float>(c.pl.Bm), *X = c.chunk<float>(c.pl.X), *R = c.chunk<float>(c.pl.R);
  float *Y2 = c.chunk<float>(c.pl.Y2), *dinv = c.chunk<float>(c.pl.dinv);
  void *XT = c.chunk<char>(c.pl.XT), *Pm = c.chunk<char>(c.pl.Pm), *UT = c.chunk<char>(c.pl.UT);
  const float *Yc = Y + (size_t)b0 * d.n * kHeadDimH;
  const int64_t pl = d.dtype == ARCKV_BF16 ? 2 : 1;
  const int64_t yt_pair = (d.dtype == ARCKV_BF16 ? 2 : 1) * (int64_t)kHeadDimH * d.np_;
  // pairs whose inputs (Y, C_k, beta) hold a non-finite value report info = -1
  // (a failed mass fit leaves beta NaN)
  int32_t *bad = c.pers<int32_t>(c.pl.bad) + b0;
  if (launch_fill_i32(bad, P, 0, stream) != hipSuccess ||
      launch_nonfinite(Yc, P, (int64_t)d.n * kHeadDimH, bad, stream) != hipSuccess ||
      launch_nonfinite(Ck + (size_t)b0 * d.t * kHeadDimH, P, (int64_t)d.t * kHeadDimH, bad, stream) != hipSuccess ||
      launch_nonfinite(beta + (size_t)b0 * d.t, P, d.t, bad, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  // P^T for the Gram and right-hand side, and P (query-major) for the refinement residuals
  STAGE(ST_PHAT, launch_phat(d.dtype, LT, c.pers<float>(c.pl.beta_ws) + (size_t)b0 * d.tp, P, d.n, d.t, d.tp,
                             d.np_, PT, fp.value_refine_steps > 0 ? Pm : nullptr, stream));
  STAGE(ST_GRAM_A, launch_gram(d.dtype, PT, Gw, Gc, P, d.tp, d.np_, stream));
  {
    StageScope _sc(ST_RHS, stream);
    if (launch_transpose128(d.dtype, Y + (size_t)b0 * d.n * kHeadDimH, P, d.n, (int64_t)d.n * kHeadDimH, d.np_, YT,
                            yt_pair, stream) != hipSuccess)
      return ARCKV_ERR_HIP;
    if (launch_rhs_gemm(d.dtype, PT, YT, Bm, P, d.tp, d.np_, stream) != hipSuccess) return ARCKV_ERR_HIP;
  }
  STAGE(ST_CHOL_A, launch_cholesky(Gw, Gc, P, d.t, d.tp, fp.delta_v, fp.max_escalations, st, dinv,
                                   c.chunk<char>(c.pl.lsplit), bad, c.pers<int32_t>(c.pl.cnt), stream));
  {
    StageScope _sc(ST_SOLVE_V, stream);
    void *lsp = c.chunk<char>(c.pl.lsplit), *tw = c.chunk<char>(c.pl.tw);
    if (launch_trsm_fwd_blocked(Gw, dinv, lsp, P, d.tp, Bm, Y2, st.lam, st.info, tw, stream) != hipSuccess)
      return ARCKV_ERR_HIP;
    if (launch_trsm(false, Gw, dinv, P, d.tp, Y2, X, st.info, stream) != hipSuccess) return ARCKV_ERR_HIP;
    // refinement against the data: R = P^T (Y - P X) - lam X
    for (int it = 0; it < fp.value_refine_steps; ++it) {
      if (launch_transpose128(d.dtype, X, P, (int)d.tp, d.tp * kHeadDimH, d.tp, XT, pl * d.tp * kHeadDimH, stream) !=
          hipSuccess)
        return ARCKV_ERR_HIP;
      if (launch_value_residual(d.dtype, XT, Pm, PT, Yc, UT, X, st.lam, R, P, d.n, d.tp, d.np_, stream) != hipSuccess)
        return ARCKV_ERR_HIP;
      if (launch_trsm_fwd_blocked(Gw, dinv, lsp, P, d.tp, R, Y2, st.lam, st.info, tw, stream) != hipSuccess)
        return ARCKV_ERR_HIP;
      if (launch_trsm(false, Gw, dinv, P, d.tp, Y2, R, st.info, stream) != hipSuccess) return ARCKV_ERR_HIP;
      if (launch_add(X, R, P, d.tp * kHeadDimH, st.info, stream) != hipSuccess) return ARCKV_ERR_HIP;
    }
    if (launch_values_out(X, P, d.tp, d.t, st.info, Cv + (size_t)b0 * d.t * kHeadDimH, stream) != hipSuccess)
      return ARCKV_ERR_HIP;
  }
  return ARCKV_OK;
}

}  // namespace arckv

using namespace arckv;

// ====================================================================== C ABI
extern "C" {

arckv_status arckv_default_params(arckv_fit_params *p) {
  if (!p) return ARCKV_ERR_INVALID_ARG;
  p->lambda_m = 0.25f;
  p->delta_beta = 1e-6f;
  p->delta_v = 1e-3f;
  p->eps_w = 1e-12f;
  p->b_min = -30.0f;
  p->b_max = 30.0f;
  p->bias_mode = 0;
  p->max_escalations = 6;
  p->refine_steps = 2;
  p->value_refine_steps = 1;
  p->pair_chunk = 0;
  p->select_chunk = 0;
  p->nnls_max_iter = 32;
  return ARCKV_OK;
}

arckv_status arckv_budget(int64_t T, double rho, int32_t *t) {
  if (!t || T < 1 || !isfinite(rho) || rho < 0.0) return ARCKV_ERR_INVALID_ARG;
  if (T > (1ll << 30)) return ARCKV_ERR_UNSUPPORTED;
  double v = floor(rho * (double)T + 0.5);
  if (v < 1.0) v = 1.0;
  if (v > (double)T) v = (double)T;
  *t = (int32_t)v;
  return ARCKV_OK;
}

arckv_status arckv_workspace_size(const arckv_problem *prob, int32_t t, const arckv_fit_params *p, size_t *bytes) {
  CHECK(check_problem(prob));
  if (!bytes || t < 1 || t > prob->T) return ARCKV_ERR_INVALID_ARG;
  arckv_fit_params def;
  arckv_default_params(&def);
  if (!p) p = &def;
  CHECK(check_params(p));
  // with chunked selection t is the nominal budget: size for the realised count
  const int64_t tr = chunked_count(prob->T, t, p->select_chunk);
  Dims d = make_dims(prob, (int32_t)(tr > t ? tr : t));
  int64_t P = p->pair_chunk > 0 && p->pair_chunk < d.B ? p->pair_chunk : d.B;
  *bytes = plan_total(d, P);
  return ARCKV_OK;
}

arckv_status arckv_budgets(int32_t P, const double *a, int32_t t, int64_t T, int32_t *t_out) {
  if (P < 1 || !a || !t_out || t < 1 || T < 1) return ARCKV_ERR_INVALID_ARG;
  if (T > (1ll << 30)) return ARCKV_ERR_UNSUPPORTED;
  double sum = 0.0;
  for (int32_t i = 0; i < P; ++i) {
    if (!isfinite(a[i]) || a[i] < 0.0) return ARCKV_ERR_INVALID_ARG;
    sum += a[i];
  }
  if (!(sum > 0.0) || !isfinite(sum)) return ARCKV_ERR_INVALID_ARG;
  for (int32_t i = 0; i < P; ++i) {
    double v = floor(a[i] / sum * (double)P * (double)t);
    v = v < 1.0 ? 1.0 : (v > (double)T ? (double)T : v);
    t_out[i] = (int32_t)v;
  }
  return ARCKV_OK;
}

arckv_status arckv_select_count(int64_t T, int32_t t, int32_t chunk_len, int32_t *t_real) {
  if (!t_real || T < 1 || t < 1 || t > T || chunk_len < 0) return ARCKV_ERR_INVALID_ARG;
  if (T > (1ll << 30)) return ARCKV_ERR_UNSUPPORTED;
  *t_real = (int32_t)chunked_count(T, t, chunk_len);
  return ARCKV_OK;
}

arckv_status arckv_score(const arckv_problem *prob, const void *K, const void *V, const arckv_indexer *ix,
                         float *scores, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!K || !V || !ix || !scores || !ix->W1 || !ix->b1 || !ix->w2 || !ix->b2) return ARCKV_ERR_INVALID_ARG;
  if (ix->hidden != 64) return ARCKV_ERR_UNSUPPORTED;
  if (ix->w1_dtype != prob->dtype) return ARCKV_ERR_UNSUPPORTED;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(ix->W1, 16)) return ARCKV_ERR_INVALID_ARG;
  STAGE(ST_SCORE, launch_score(prob->dtype, K, V, ix->W1, ix->b1, ix->w2, ix->b2, scores, prob->B, prob->T, stream));
  return ARCKV_OK;
}

arckv_status arckv_select(const arckv_problem *prob, const float *scores, int32_t t, int32_t *anchors, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!scores || !anchors || t < 1 || t > prob->T) return ARCKV_ERR_INVALID_ARG;
  (void)ws;
  (void)ws_bytes;
  STAGE(ST_SELECT, launch_select(scores, prob->B, prob->T, t, anchors, stream));
  return ARCKV_OK;
}

arckv_status arckv_select_ex(const arckv_problem *prob, const float *scores, int32_t t, const int32_t *t_pair,
                             int32_t chunk_len, int32_t t_stride, int32_t *anchors, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!scores || !anchors || t < 1 || t > prob->T || chunk_len < 0 || t_stride < 1) return ARCKV_ERR_INVALID_ARG;
  if (!t_pair && t_stride < chunked_count(prob->T, t, chunk_len)) return ARCKV_ERR_INVALID_ARG;
  STAGE(ST_SELECT, launch_select_ex(scores, prob->B, prob->T, t, t_pair, chunk_len, t_stride, anchors, stream));
  return ARCKV_OK;
}

arckv_status arckv_rowstats(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref, float *z,
                            float *m, float *Y, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!K || !V || !Q_ref || !z || !m || !Y) return ARCKV_ERR_INVALID_ARG;
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(Q_ref, 16) || !aligned(Y, 16)) return ARCKV_ERR_INVALID_ARG;
  STAGE(ST_ROWSTATS, launch_rowstats(prob->dtype, K, V, Q_ref, z, m, Y, prob->B, prob->T, prob->n,
                                     eff_scale(prob), stream));
  return ARCKV_OK;
}

arckv_status arckv_merge(const arckv_problem *prob, const void *K, const void *Q_ref, const float *z,
                         const int32_t *anchors, int32_t t, float lambda_m, float *C_k, int32_t *assign, float *phi,
                         void *ws, size_t ws_bytes, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!K || !Q_ref || !z || !anchors || !C_k || t < 1 || t > prob->T) return ARCKV_ERR_INVALID_ARG;
  if (!(lambda_m >= 0.0f && lambda_m <= 1.0f)) return ARCKV_ERR_INVALID_ARG;
  if (!aligned(K, 16) || !aligned(Q_ref, 16) || !aligned(C_k, 16)) return ARCKV_ERR_INVALID_ARG;
  Ctx c;
  c.d = make_dims(prob, t);
  int64_t P = 0;
  CHECK(check_ws(c.d, ws, ws_bytes, 0, &P));
  c.pl = make_plan(c.d, P);
  c.ws = (char *)ws;
  c.scale = eff_scale(prob);
  c.stream = stream;
  float *zmax = c.pers<float>(c.pl.zmax);
  int32_t *kappa = assign ? assign : c.pers<int32_t>(c.pl.kappa);
  float *phiw = phi ? phi : c.pers<float>(c.pl.phi);
  STAGE(ST_ZMAX, launch_zmax(z, c.d.B, c.d.n, zmax, stream));
  for (int b0 = 0; b0 < c.d.B; b0 += (int)P) {
    const int Pc = (int)(c.d.B - b0 < P ? c.d.B - b0 : P);
    CHECK(run_merge_chunk(c, b0, Pc, K, Q_ref, anchors, lambda_m, C_k, kappa, phiw, zmax));
  }
  return ARCKV_OK;
}

static arckv_status fit_common(const arckv_problem *prob, const float *C_k, int32_t t, const arckv_fit_params *p,
                               void *ws, size_t ws_bytes, hipStream_t stream, Ctx &c, int64_t &P) {
  CHECK(check_problem(prob));
  if (!C_k || t < 1 || t > prob->T) return ARCKV_ERR_INVALID_ARG;
  CHECK(check_params(p));
  c.d = make_dims(prob, t);
  CHECK(check_ws(c.d, ws, ws_bytes, p->pair_chunk, &P));
  c.pl = make_plan(c.d, P);
  c.ws = (char *)ws;
  c.scale = eff_scale(prob);
  c.stream = stream;
  return ARCKV_OK;
}

// z, m (mass fit) or Y (value fit) given, or recomputed into the workspace
// from K, V by the row-statistics kernel.
static arckv_status fit_rowstats(const Ctx &c, const void *K, const void *V, const void *Q_ref, const float **z,
                                 const float **m, const float **Y) {
  if ((z && *z && m && *m) || (Y && *Y)) return ARCKV_OK;
  if (!K || !V || !aligned(K, 16) || !aligned(V, 16)) return ARCKV_ERR_INVALID_ARG;
  float *zw = c.pers<float>(c.pl.z), *mw = c.pers<float>(c.pl.m), *Yw = c.pers<float>(c.pl.Y);
  hipStream_t stream = c.stream;
  STAGE(ST_ROWSTATS, launch_rowstats(c.d.dtype, K, V, Q_ref, zw, mw, Yw, c.d.B, c.d.T, c.d.n, c.scale, stream));
  if (z) *z = zw;
  if (m) *m = mw;
  if (Y) *Y = Yw;
  return ARCKV_OK;
}

arckv_status arckv_fit_bias(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                            const float *C_k, int32_t t, const float *z, const float *m, const arckv_fit_params *p,
                            float *beta, int32_t *info, float *delta_used, void *ws, size_t ws_bytes,
                            hipStream_t stream) {
  arckv_fit_params def;
  arckv_default_params(&def);
  if (!p) p = &def;
  if (!Q_ref || !beta || !info) return ARCKV_ERR_INVALID_ARG;
  if (!aligned(Q_ref, 16) || !aligned(C_k, 16)) return ARCKV_ERR_INVALID_ARG;
  if ((!z || !m) && (!K || !V)) return ARCKV_ERR_INVALID_ARG;   // z and m are recomputed from K, V
  Ctx c;
  int64_t P = 0;
  CHECK(fit_common(prob, C_k, t, p, ws, ws_bytes, stream, c, P));
  if (!z || !m) {
    z = m = nullptr;
    CHECK(fit_rowstats(c, K, V, Q_ref, &z, &m, nullptr));
  }
  for (int b0 = 0; b0 < c.d.B; b0 += (int)P) {
    const int Pc = (int)(c.d.B - b0 < P ? c.d.B - b0 : P);
    if (launch_pad_ck(c.d.dtype, C_k + (size_t)b0 * t * kHeadDimH, Pc, t, c.d.tp, c.chunk<char>(c.pl.Ckp), stream) !=
        hipSuccess)
      return ARCKV_ERR_HIP;
    FitState st = fit_state(c, c.pl.st_g, c.pl.info_g, b0);
    CHECK(run_fit_bias_chunk(c, b0, Pc, Q_ref, z, m, C_k, *p, beta, st));
  }
  if (launch_copy_info(c.pers<int32_t>(c.pl.info_g), nullptr, c.d.B, info, stream) != hipSuccess) return ARCKV_ERR_HIP;
  if (delta_used && launch_copy_f32(reinterpret_cast<float *>(c.pers<char>(c.pl.st_g) + (size_t)c.d.B * 12),
                                    delta_used, c.d.B, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  return ARCKV_OK;
}

arckv_status arckv_fit_values(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                              const float *C_k, const float *beta, int32_t t, const float *Y,
                              const arckv_fit_params *p, float *C_v, int32_t *info, float *delta_used, void *ws,
                              size_t ws_bytes, hipStream_t stream) {
  arckv_fit_params def;
  arckv_default_params(&def);
  if (!p) p = &def;
  if (!Q_ref || !beta || !C_v || !info) return ARCKV_ERR_INVALID_ARG;
  if (!aligned(Q_ref, 16) || !aligned(C_k, 16) || (Y && !aligned(Y, 16))) return ARCKV_ERR_INVALID_ARG;
  if (!Y && (!K || !V)) return ARCKV_ERR_INVALID_ARG;   // Y is recomputed from K, V
  Ctx c;
  int64_t P = 0;
  CHECK(fit_common(prob, C_k, t, p, ws, ws_bytes, stream, c, P));
  if (!Y) CHECK(fit_rowstats(c, K, V, Q_ref, nullptr, nullptr, &Y));
  const Dims &d = c.d;
  for (int b0 = 0; b0 < d.B; b0 += (int)P) {
    const int Pc = (int)(d.B - b0 < P ? d.B - b0 : P);
    if (launch_pad_ck(d.dtype, C_k + (size_t)b0 * t * kHeadDimH, Pc, t, d.tp, c.chunk<char>(c.pl.Ckp), stream) !=
        hipSuccess)
      return ARCKV_ERR_HIP;
    if (launch_pad_beta(beta + (size_t)b0 * t, Pc, t, d.tp, c.pers<float>(c.pl.beta_ws) + (size_t)b0 * d.tp,
                        stream) != hipSuccess)
      return ARCKV_ERR_HIP;
    // logits of the compact keys (the exp-part is unused here; z only shifts it)
    const char *Qc = (const char *)Q_ref + (size_t)b0 * d.n * kHeadDimH * c.in_esz();
    STAGE(ST_PHIC, launch_phic(d.dtype, Qc, c.chunk<char>(c.pl.Ckp), nullptr, c.chunk<char>(c.pl.PhiT),
                               c.chunk<float>(c.pl.LT), nullptr, nullptr, Pc, d.t, d.n, d.tp, d.np_, c.scale, stream));
    FitState st = fit_state(c, c.pl.st_a, c.pl.info_a, b0);
    CHECK(run_fit_values_chunk(c, b0, Pc, Y, C_k, beta, *p, C_v, st));
  }
  if (launch_copy_info(c.pers<int32_t>(c.pl.info_a), nullptr, d.B, info, stream) != hipSuccess) return ARCKV_ERR_HIP;
  if (delta_used && launch_copy_f32(reinterpret_cast<float *>(c.pers<char>(c.pl.st_a) + (size_t)d.B * 12),
                                    delta_used, d.B, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  return ARCKV_OK;
}

// arckv_compact (ix given) and arckv_compact_scored (scores_in given).
static arckv_status compact_impl(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                                 const arckv_indexer *ix, const float *scores_in, double rho,
                                 const arckv_fit_params *p, int32_t *t_out, int32_t *anchors, float *C_k,
                                 float *beta, float *C_v, int32_t *info, void *ws, size_t ws_bytes,
                                 hipStream_t stream) {
  arckv_fit_params def;
  arckv_default_params(&def);
  if (!p) p = &def;
  CHECK(check_problem(prob));
  CHECK(check_params(p));
  if (!K || !V || !Q_ref || !t_out || !anchors || !C_k || !beta || !C_v || !info) return ARCKV_ERR_INVALID_ARG;
  if (!ix && !scores_in) return ARCKV_ERR_INVALID_ARG;
  if (ix) {
    if (!ix->W1 || !ix->b1 || !ix->w2 || !ix->b2) return ARCKV_ERR_INVALID_ARG;
    if (ix->hidden != 64 || ix->w1_dtype != prob->dtype) return ARCKV_ERR_UNSUPPORTED;
    if (!aligned(ix->W1, 16)) return ARCKV_ERR_INVALID_ARG;
  }
  if (!aligned(K, 16) || !aligned(V, 16) || !aligned(Q_ref, 16) || !aligned(C_k, 16)) return ARCKV_ERR_INVALID_ARG;
  int32_t t = 0;
  CHECK(arckv_budget(prob->T, rho, &t));
  const int32_t t_nominal = t;
  t = (int32_t)chunked_count(prob->T, t, p->select_chunk);   // realised count under chunked selection
  Ctx c;
  c.d = make_dims(prob, t);
  int64_t P = 0;
  CHECK(check_ws(c.d, ws, ws_bytes, p->pair_chunk, &P));
  *t_out = t;
  c.pl = make_plan(c.d, P);
  c.ws = (char *)ws;
  c.scale = eff_scale(prob);
  c.stream = stream;
  const Dims &d = c.d;
  const float *scores = scores_in ? scores_in : c.pers<float>(c.pl.scores);
  float *z = c.pers<float>(c.pl.z), *m = c.pers<float>(c.pl.m), *Y = c.pers<float>(c.pl.Y);
  float *zmax = c.pers<float>(c.pl.zmax), *phi = c.pers<float>(c.pl.phi);
  int32_t *kappa = c.pers<int32_t>(c.pl.kappa);
  if (ix)
    STAGE(ST_SCORE, launch_score(d.dtype, K, V, ix->W1, ix->b1, ix->w2, ix->b2, c.pers<float>(c.pl.scores), d.B, d.T,
                                 stream));
  STAGE(ST_SELECT, launch_select_ex(scores, d.B, d.T, t_nominal, nullptr, p->select_chunk, t, anchors, stream));
  STAGE(ST_ROWSTATS, launch_rowstats(d.dtype, K, V, Q_ref, z, m, Y, d.B, d.T, d.n, c.scale, stream));
  STAGE(ST_ZMAX, launch_zmax(z, d.B, d.n, zmax, stream));
  for (int b0 = 0; b0 < d.B; b0 += (int)P) {
    const int Pc = (int)(d.B - b0 < P ? d.B - b0 : P);
    CHECK(run_merge_chunk(c, b0, Pc, K, Q_ref, anchors, p->lambda_m, C_k, kappa, phi, zmax));
    CHECK(run_fit_bias_chunk(c, b0, Pc, Q_ref, z, m, C_k, *p, beta, fit_state(c, c.pl.st_g, c.pl.info_g, b0), Y));
    CHECK(run_fit_values_chunk(c, b0, Pc, Y, C_k, beta, *p, C_v, fit_state(c, c.pl.st_a, c.pl.info_a, b0)));
  }
  if (launch_copy_info(c.pers<int32_t>(c.pl.info_g), c.pers<int32_t>(c.pl.info_a), d.B, info, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  return ARCKV_OK;
}

static arckv_status check_attend(int32_t P, int32_t G, int32_t t, int32_t F) {
  if (P < 1 || t < 0 || F < 0 || (int64_t)t + F < 1) return ARCKV_ERR_INVALID_ARG;
  if ((int64_t)t + F > (1ll << 30)) return ARCKV_ERR_UNSUPPORTED;
  if (G != 1 && G != 2 && G != 4 && G != 8) return ARCKV_ERR_UNSUPPORTED;
  return ARCKV_OK;
}

static size_t attend_ws_bytes(int32_t P, int32_t G, int32_t t, int32_t F) {
  const size_t nch = (size_t)attend_chunks(t, F);
  return rup((int64_t)((size_t)P * nch * G * kHeadDimH * 4), 256) + rup((int64_t)((size_t)P * nch * G * 2 * 4), 256);
}

arckv_status arckv_attend_workspace_size(int32_t P, int32_t G, int32_t t, int32_t F, size_t *bytes) {
  CHECK(check_attend(P, G, t, F));
  if (!bytes) return ARCKV_ERR_INVALID_ARG;
  *bytes = attend_ws_bytes(P, G, t, F);
  return ARCKV_OK;
}

static arckv_status check_attend_args(int32_t P, int32_t G, int32_t t, int32_t F, float scale, const void *Q,
                                      const void *C_k, const void *C_v, const void *K_f, const void *V_f,
                                      const float *out) {
  CHECK(check_attend(P, G, t, F));
  if (!Q || !out) return ARCKV_ERR_INVALID_ARG;
  if (t > 0 && (!C_k || !C_v)) return ARCKV_ERR_INVALID_ARG;
  if (F > 0 && (!K_f || !V_f)) return ARCKV_ERR_INVALID_ARG;
  if (!isfinite(scale)) return ARCKV_ERR_INVALID_ARG;
  if (!aligned(Q, 16) || (C_k && !aligned(C_k, 16)) || (C_v && !aligned(C_v, 16)) || (K_f && !aligned(K_f, 16)) ||
      (V_f && !aligned(V_f, 16)))
    return ARCKV_ERR_INVALID_ARG;
  return ARCKV_OK;
}

arckv_status arckv_attend(int32_t P, int32_t G, int32_t t, int32_t F, float scale, const void *Q, const void *C_k,
                          const float *beta, const void *C_v, const void *K_f, const void *V_f, float *out, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
  CHECK(check_attend_args(P, G, t, F, scale, Q, C_k, C_v, K_f, V_f, out));
  if (!ws || !aligned(ws, 256) || ws_bytes < attend_ws_bytes(P, G, t, F)) return ARCKV_ERR_WORKSPACE;
  const float s = scale > 0.0f ? scale : 1.0f / sqrtf((float)kHeadDimH);
  const size_t nch = (size_t)attend_chunks(t, F);
  float *part_o = reinterpret_cast<float *>(ws);
  float *part_ml = reinterpret_cast<float *>((char *)ws + rup((int64_t)((size_t)P * nch * G * kHeadDimH * 4), 256));
  STAGE(ST_ATTEND, launch_attend(P, G, t, F, s, Q, t > 0 ? C_k : nullptr, t > 0 ? beta : nullptr,
                                 t > 0 ? C_v : nullptr, F > 0 ? K_f : nullptr, F > 0 ? V_f : nullptr, part_o, part_ml,
                                 out, stream));
  return ARCKV_OK;
}

arckv_status arckv_attend_noalloc(int32_t P, int32_t G, int32_t t, int32_t F, float scale, const void *Q,
                                  const void *C_k, const float *beta, const void *C_v, const void *K_f,
                                  const void *V_f, float *out, hipStream_t stream) {
  CHECK(check_attend_args(P, G, t, F, scale, Q, C_k, C_v, K_f, V_f, out));
  if (attend_ws_bytes(P, G, t, F) > attend_scratch_bytes()) return ARCKV_ERR_WORKSPACE;
  void *base = nullptr;
  if (attend_scratch(&base) != hipSuccess) return ARCKV_ERR_HIP;
  const float s = scale > 0.0f ? scale : 1.0f / sqrtf((float)kHeadDimH);
  const size_t nch = (size_t)attend_chunks(t, F);
  // every partial is written before the combine reads it: nothing to clear
  float *part_o = reinterpret_cast<float *>(base);
  float *part_ml = reinterpret_cast<float *>((char *)base + rup((int64_t)((size_t)P * nch * G * kHeadDimH * 4), 256));
  if (launch_attend(P, G, t, F, s, Q, t > 0 ? C_k : nullptr, t > 0 ? beta : nullptr, t > 0 ? C_v : nullptr,
                    F > 0 ? K_f : nullptr, F > 0 ? V_f : nullptr, part_o, part_ml, out, stream) != hipSuccess)
    return ARCKV_ERR_HIP;
  return ARCKV_OK;
}

arckv_status arckv_compact(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                           const arckv_indexer *ix, double rho, const arckv_fit_params *p, int32_t *t_out,
                           int32_t *anchors, float *C_k, float *beta, float *C_v, int32_t *info, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!ix) return ARCKV_ERR_INVALID_ARG;
  return compact_impl(prob, K, V, Q_ref, ix, nullptr, rho, p, t_out, anchors, C_k, beta, C_v, info, ws, ws_bytes,
                      stream);
}

arckv_status arckv_compact_scored(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                                  const float *scores, double rho, const arckv_fit_params *p, int32_t *t_out,
                                  int32_t *anchors, float *C_k, float *beta, float *C_v, int32_t *info, void *ws,
                                  size_t ws_bytes, hipStream_t stream) {
  if (!scores) return ARCKV_ERR_INVALID_ARG;
  return compact_impl(prob, K, V, Q_ref, nullptr, scores, rho, p, t_out, anchors, C_k, beta, C_v, info, ws,
                      ws_bytes, stream);
}

// ---------------------------------------------------------------- value-aware indexer
struct DsaPlan {
  int64_t ka, va, qa, c, za, ma, qbar, kbar, w, z, m, part, bytes;
};

static DsaPlan dsa_plan(int64_t P, int64_t T, int64_t n, int64_t n_pos) {
  DsaPlan d;
  Bump b;
  d.ka = b.take(P * T * 128 * 2);
  d.va = b.take(P * T * 128 * 2);
  d.qa = b.take(P * n * 128 * 2);
  d.c = b.take(P * n * 128 * 4);
  d.za = b.take(P * n * 4);
  d.ma = b.take(P * n * 4);
  d.qbar = b.take(P * n * 1024 * 2);
  d.kbar = b.take(P * T * 1024 * 2);
  d.w = b.take(P * n_pos * 8 * 4);
  d.z = b.take(P * n * 4);
  d.m = b.take(P * n * 4);
  d.part = b.take(P * (int64_t)dsa_query_blocks((int)n) * T * 4);
  d.bytes = b.off;
  return d;
}

arckv_status arckv_dsa_workspace_size(const arckv_problem *prob, int32_t pair_chunk, size_t *bytes) {
  CHECK(check_problem(prob));
  if (!bytes || pair_chunk < 0) return ARCKV_ERR_INVALID_ARG;
  const int64_t P = pair_chunk > 0 && pair_chunk < prob->B ? pair_chunk : prob->B;
  *bytes = (size_t)dsa_plan(P, prob->T, prob->n, prob->n).bytes;   // sized for n_pos = n, the largest allowed
  return ARCKV_OK;
}

arckv_status arckv_score_dsa(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                             const arckv_dsa_indexer *ix, float *scores, void *ws, size_t ws_bytes,
                             hipStream_t stream) {
  CHECK(check_problem(prob));
  if (prob->dtype != ARCKV_BF16) return ARCKV_ERR_UNSUPPORTED;
  if (!K || !V || !Q_ref || !ix || !scores) return ARCKV_ERR_INVALID_ARG;
  if (!ix->X_ref || !ix->L_q || !ix->L_k || !ix->L_x || !ix->b_x || !ix->U_q || !ix->U_k || !ix->U_v || !ix->L_c ||
      !ix->L_v)
    return ARCKV_ERR_INVALID_ARG;
  if (ix->n_pos < 1 || prob->n % ix->n_pos != 0 || ix->d_x < 1 || ix->x_group < 1 || !isfinite(ix->scale_a))
    return ARCKV_ERR_INVALID_ARG;
  const void *al[] = {K, V, Q_ref, ix->L_q, ix->L_k, ix->U_q, ix->U_k, ix->U_v, ix->L_c, ix->L_v};
  for (const void *q : al)
    if (!aligned(q, 16)) return ARCKV_ERR_INVALID_ARG;
  if (!ws || !aligned(ws, 256)) return ARCKV_ERR_WORKSPACE;
  const int64_t B = prob->B, T = prob->T, n = prob->n;
  // largest chunk of pairs whose plan fits
  int64_t P = B;
  while (P > 1 && (size_t)dsa_plan(P, T, n, ix->n_pos).bytes > ws_bytes) P = (P + 1) / 2;
  if ((size_t)dsa_plan(P, T, n, ix->n_pos).bytes > ws_bytes) return ARCKV_ERR_WORKSPACE;
  const DsaPlan pl = dsa_plan(P, T, n, ix->n_pos);
  char *w0 = (char *)ws;
  const float sa = ix->scale_a > 0.0f ? ix->scale_a : 1.0f / sqrtf(128.0f);
  for (int64_t b0 = 0; b0 < B; b0 += P) {
    const int Pc = (int)(B - b0 < P ? B - b0 : P);
    const bf16_t_ *Kc = (const bf16_t_ *)K + b0 * T * 128, *Vc = (const bf16_t_ *)V + b0 * T * 128;
    const bf16_t_ *Qc = (const bf16_t_ *)Q_ref + b0 * n * 128;
    auto mat = [&](const void *base, int64_t per) { return (const bf16_t_ *)base + b0 * per; };
    {
      StageScope _sc(ST_DSA_PROJ, stream);
      if (launch_dsa_proj(Kc, nullptr, false, mat(ix->U_k, 128 * 128), nullptr, Pc, (int)T, 1, false, w0 + pl.ka,
                          stream) != hipSuccess ||
          launch_dsa_proj(Vc, nullptr, false, mat(ix->U_v, 128 * 128), nullptr, Pc, (int)T, 1, false, w0 + pl.va,
                          stream) != hipSuccess ||
          launch_dsa_proj(Qc, nullptr, false, mat(ix->U_q, 128 * 128), nullptr, Pc, (int)n, 1, false, w0 + pl.qa,
                          stream) != hipSuccess)
        return ARCKV_ERR_HIP;
    }
    STAGE(ST_DSA_VALUE, launch_rowstats(ARCKV_BF16, w0 + pl.ka, w0 + pl.va, w0 + pl.qa, (float *)(w0 + pl.za),
                                        (float *)(w0 + pl.ma), (float *)(w0 + pl.c), Pc, (int)T, (int)n, sa, stream));
    {
      StageScope _sc(ST_DSA_PROJ, stream);
      if (launch_dsa_proj(Kc, Vc, false, mat(ix->L_k, 1024 * 128), mat(ix->L_v, 1024 * 128), Pc, (int)T, 8, true,
                          w0 + pl.kbar, stream) != hipSuccess ||
          launch_dsa_proj(Qc, w0 + pl.c, true, mat(ix->L_q, 1024 * 128), mat(ix->L_c, 1024 * 128), Pc, (int)n, 8,
                          true, w0 + pl.qbar, stream) != hipSuccess ||
          launch_dsa_w(ix->X_ref, mat(ix->L_x, 8 * (int64_t)ix->d_x), ix->b_x + b0 * 8, Pc, ix->n_pos, ix->d_x,
                       ix->x_group, (int)b0, (float *)(w0 + pl.w), stream) != hipSuccess)
        return ARCKV_ERR_HIP;
    }
    {
      StageScope _sc(ST_DSA_INDEX, stream);
      float *z = (float *)(w0 + pl.z), *m = (float *)(w0 + pl.m), *part = (float *)(w0 + pl.part);
      if (launch_dsa_index(1, w0 + pl.qbar, w0 + pl.kbar, (float *)(w0 + pl.w), Pc, (int)n, ix->n_pos, (int)T, z, m,
                           part, stream) != hipSuccess ||
          launch_dsa_index(2, w0 + pl.qbar, w0 + pl.kbar, (float *)(w0 + pl.w), Pc, (int)n, ix->n_pos, (int)T, z, m,
                           part, stream) != hipSuccess ||
          launch_dsa_pool(part, Pc, (int)n, (int)T, scores + b0 * T, stream) != hipSuccess)
        return ARCKV_ERR_HIP;
    }
  }
  return ARCKV_OK;
}

const char *arckv_status_string(arckv_status s) {
  switch (s) {
    case ARCKV_OK: return "ok";
    case ARCKV_ERR_INVALID_ARG: return "invalid argument";
    case ARCKV_ERR_UNSUPPORTED: return "unsupported configuration";
    case ARCKV_ERR_WORKSPACE: return "workspace too small or misaligned";
    case ARCKV_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

arckv_status arckv_assign_stats(const arckv_problem *prob, int32_t t, const void *ws, size_t ws_bytes,
                                int32_t *stats, hipStream_t stream) {
  CHECK(check_problem(prob));
  if (!ws || !stats || t < 1 || t > prob->T) return ARCKV_ERR_INVALID_ARG;
  const Dims d = make_dims(prob, t);
  if (!aligned(ws, 256) || ws_bytes < plan_total(d, 1)) return ARCKV_ERR_WORKSPACE;
  const Plan pl = make_plan(d, 1);   // the persistent region does not depend on the chunk size
  if (hipMemcpyAsync(stats, (const char *)ws + pl.astats, (size_t)prob->B * kAssignStats * 4, hipMemcpyDeviceToDevice, stream) !=
      hipSuccess)
    return ARCKV_ERR_HIP;
  return ARCKV_OK;
}

arckv_status arckv_set_timing(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  g_timing.enabled = enable != 0;
  return ARCKV_OK;
}

arckv_status arckv_reset_timing(void) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto &r : g_timing.pending) {
    g_timing.pool.push_back(r.a);
    g_timing.pool.push_back(r.b);
  }
  g_timing.pending.clear();
  for (int i = 0; i < ST_COUNT; ++i) {
    g_timing.ms[i] = 0.0;
    g_timing.cnt[i] = 0;
  }
  return ARCKV_OK;
}

arckv_status arckv_stage_times(int32_t max_stages, const char **names, double *ms, int32_t *counts,
                               int32_t *n_stages) {
  if (!n_stages || max_stages < 0 || (max_stages > 0 && !ms)) return ARCKV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  for (auto &r : g_timing.pending) {
    if (hipEventSynchronize(r.b) != hipSuccess) return ARCKV_ERR_HIP;
    float t = 0.0f;
    if (hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) return ARCKV_ERR_HIP;
    g_timing.ms[r.stage] += t;
    g_timing.cnt[r.stage] += 1;
    g_timing.pool.push_back(r.a);
    g_timing.pool.push_back(r.b);
  }
  g_timing.pending.clear();
  *n_stages = ST_COUNT;
  for (int i = 0; i < ST_COUNT && i < max_stages; ++i) {
    if (names) names[i] = kStageNames[i];
    ms[i] = g_timing.ms[i];
    if (counts) counts[i] = g_timing.cnt[i];
  }
  return ARCKV_OK;
}

}  // extern "C"
