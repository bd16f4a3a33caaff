/*
 * arckv.h -- C ABI of the MI355X (gfx950) ARC-KV per-context compaction library.
 *
 * ARC-KV (arXiv 2609.36835) replaces a long key/value cache block (K, V, T rows
 * of head dimension d) of one layer-KV-head pair by t << T compact entries
 * (C_k, beta, C_v) so that softmax(q C_k^T + beta) C_v approximates full
 * attention softmax(q K^T) V and the block's attention mass (Section 3.1,
 * eq. compact_attention and eq. block_attention_mass).  Per context, four
 * stages run (Section 3.2):
 *   1. score every cached token and take the top-t tokens as anchors (Section 3.3);
 *   2. assign every key to the anchor with the most similar normalised
 *      attention-response profile and merge each group into one compact key
 *      inside the group's convex hull (Section 3.4);
 *   3. fit the mass bias beta by projected least squares (Appendix A.9, eq. mass_fit;
 *      optionally by exact non-negative least squares);
 *   4. fit the compact values C_v by ridge least squares (Appendix A.9, eq. value_lstsq).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - A call processes B independent pairs (flattened [layer][kv_head]).
 *  - All array arguments are DEVICE pointers owned by the caller, row-major and
 *    contiguous: K, V [B][T][d]; Q_ref [B][n][d] (each pair's n rows ordered
 *    [query head][position]); per-pair vectors [B][len].  Inputs are read-only.
 *    K, V, Q_ref, Y, W1 and C_k move in 16-byte vectors and must be 16-byte
 *    aligned (ARCKV_ERR_INVALID_ARG otherwise).
 *  - K, V and Q_ref share one element type (arckv_problem.dtype): float32 or
 *    bfloat16.  Only d = 128 is supported.  Outputs are float32 (indices int32).
 *  - The library never allocates device memory.  Entry points that need scratch
 *    take a caller-owned device workspace (ws, ws_bytes) of at least
 *    arckv_workspace_size() bytes, 256-byte aligned.  Its contents are
 *    undefined on entry and exit (apart from the counters arckv_assign_stats
 *    reads); it must not be shared by calls that may overlap in time.
 *  - All device work is enqueued on the caller's stream.  The host is
 *    synchronised only where the next launches depend on a device result: the
 *    fits read back the number of pairs to refactor (a failed Cholesky pivot;
 *    in the mass fit also a cut-off refinement) before each possible
 *    ridge-escalation round (not with max_escalations = 0), and the
 *    exact non-negative mass fit (bias_mode = 1) reads two integers back once
 *    per pivoting iteration, to size the next iteration's system and to stop
 *    when every pair has settled.  Results are valid once the stream reaches
 *    them.
 *  - Argument errors are returned synchronously BEFORE any HIP call, so they can
 *    be checked on a machine without a GPU.  A failed kernel launch returns
 *    ARCKV_ERR_HIP.  Numerical failures are reported asynchronously in the
 *    per-pair `info` arrays.  No C++ exception crosses this interface.
 *  - The logit scale s multiplies q.k everywhere (the paper omits 1/sqrt(d) by
 *    convention, Section 3.1); scale <= 0 selects 1/sqrt(d).
 */
#ifndef ARCKV_H
#define ARCKV_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ARCKV_OK = 0,
  ARCKV_ERR_INVALID_ARG = 1,   /* null pointer, bad size, t outside [1, T], ... */
  ARCKV_ERR_UNSUPPORTED = 2,   /* d != 128, unknown dtype, bias_mode outside {0, 1}, ... */
  ARCKV_ERR_WORKSPACE = 3,     /* ws too small or misaligned */
  ARCKV_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} arckv_status;

typedef enum { ARCKV_F32 = 0, ARCKV_BF16 = 1 } arckv_dtype;

typedef struct {
  int32_t B;       /* pairs in the call, >= 1 */
  int32_t T;       /* cached tokens per pair, >= 1 */
  int32_t n;       /* reference queries per pair, >= 1 */
  int32_t d;       /* head dimension; must be 128 */
  int32_t dtype;   /* arckv_dtype of K, V, Q_ref */
  float scale;     /* logit scale s; <= 0 selects 1/sqrt(d) */
} arckv_problem;

/* The token scorer: a 2-layer MLP on concat(k_j, v_j),
 * I_j = w2 . GELU(W1 [k_j; v_j] + b1) + b2, GELU(x) = x Phi(x) (erf form).
 * The bfloat16 path evaluates erfc with the rational approximation of
 * Abramowitz & Stegun 7.1.26 (absolute error <= 1.5e-7), so each GELU is
 * within about 3.3e-7 of the exact one for |x| <= 4 (about 1e-7 relative
 * beyond); the float32 path calls erff.
 * It is query-independent, so the root-mean-square pooling of eq.
 * indexer_pooling reduces to softmax(I), and ranking by I ranks by the pooled
 * score (Section 3.3). */
typedef struct {
  int32_t hidden;     /* hidden width; must be 64 */
  int32_t w1_dtype;   /* arckv_dtype of W1 */
  const void *W1;     /* [B][hidden][2d], input order [k ; v] */
  const float *b1;    /* [B][hidden] */
  const float *w2;    /* [B][hidden] */
  const float *b2;    /* [B] */
} arckv_indexer;

/* Fit parameters (Section 3.4 and Appendix A.9).  The paper gives lambda_m;
 * the remaining values are this library's readings. */
typedef struct {
  float lambda_m;        /* key-merge coefficient in [0, 1]; default 0.25 */
  float delta_beta;      /* relative ridge of the mass fit: G + delta_beta*tr(G)/t*I; default 1e-6 */
  float delta_v;         /* relative ridge of the value fit: lambda_v = delta_v*tr(A)/t; default 1e-3 */
  float eps_w;           /* epsilon_w of eq. mass_fit; default 1e-12 */
  float b_min, b_max;    /* clip range of beta; default [-30, 30] */
  int32_t bias_mode;     /* 0 = projected least squares (eq. mass_fit, the paper's: w* = max(w~, 0));
                          * 1 = exact non-negative least squares on the same ridged system, by block
                          * principal pivoting; other values unsupported */
  int32_t max_escalations; /* ridge x10 retries (from 1e-7 when the ridge is 0) after a failed
                            * Cholesky pivot or a cut-off mass-fit refinement, 0..6; default 6 */
  int32_t refine_steps;  /* iterative-refinement steps after each mass-fit Cholesky solve, 0..4;
                          * default 2.  Each step recomputes the residual from the data
                          * (Phi_C; P_hat for the value fit), not from the float32 Gram, so
                          * the solves converge to the least-squares solutions of the exact
                          * normal equations.  With refine_steps >= 2 a correction (above 1e-10 |w|) that
                          * is not at most half the previous one is undone and ends the
                          * refinement; the pair is then refactored with the ridge raised
                          * tenfold, as after a failed pivot (a ridge small next to the
                          * float32 rounding of a rank-deficient Gram, t > n, makes the
                          * steps diverge). */
  int32_t pair_chunk;    /* pairs processed together by arckv_compact (0 = all B); sizes the workspace */
  int32_t select_chunk;  /* 0 = global top-t (default).  L > 0: when T > 10,000, anchors are the union of
                          * each L-position chunk's local top-t_c (Appendix A.3), so arckv_compact keeps
                          * arckv_select_count(T, t, L) anchors; merge and fits stay global. */
  int32_t nnls_max_iter; /* bias_mode 1: pivoting iterations (one masked Cholesky solve each), 1..256;
                          * default 32.  A pair not settled by then reports info = -2. */
  int32_t value_refine_steps; /* refinement steps after the value-fit solve, 0..4; default 1 (its ridge
                               * keeps the system well conditioned: one step reaches the float32
                               * floor of its residual) */
} arckv_fit_params;

/* Fill *p with the defaults listed above.  Returns ARCKV_ERR_INVALID_ARG on NULL. */
arckv_status arckv_default_params(arckv_fit_params *p);

/* Budget t = clip_[1,T](floor(rho*T + 1/2)), computed in double (the paper
 * rounds the budget by ceil in training, floor per head and round per chunk,
 * Section 3.5 and Appendix A.2-A.3; round-half-up is this library's reading).
 * Errors: T < 1, rho not finite or rho < 0, t == NULL. */
arckv_status arckv_budget(int64_t T, double rho, int32_t *t);

/* Bytes of workspace needed by every entry point below for this problem and
 * budget (the maximum over stages; arckv_compact with p->pair_chunk pairs in
 * flight).  p may be NULL (defaults). */
arckv_status arckv_workspace_size(const arckv_problem *prob, int32_t t,
                                  const arckv_fit_params *p, size_t *bytes);

/* Stage 1a: token scores I [B][T] (float32), Section 3.3 with the MLP scorer.
 * No workspace. */
arckv_status arckv_score(const arckv_problem *prob, const void *K, const void *V,
                         const arckv_indexer *ix, float *scores, hipStream_t stream);

/* The value-aware indexer of Appendix A.1 (eq. value_context,
 * indexer_projection, pairwise_index_score) with H_I = 8 index heads of width
 * d_I = 128 and a value head of width d_A = 128.  All matrices bfloat16,
 * row-major, per pair (B pairs in a call):
 *   L_q, L_k, L_c, L_v [B][1024][128];  U_q, U_k, U_v [B][128][128];
 *   L_x [B][8][d_x];  b_x [B][8] float32;
 *   X_ref [ceil(B / x_group)][n_pos][d_x]: the activation x_r of reference position r,
 *   shared by the query heads of a position and by the x_group consecutive
 *   pairs of one layer (its KV heads).
 * Q_ref rows are ordered [query head][position], so row i uses x_{i mod n_pos}. */
typedef struct {
  int32_t n_pos;      /* reference positions; n must be a multiple of n_pos */
  int32_t d_x;        /* activation width, >= 1 */
  int32_t x_group;    /* pairs sharing one X_ref block, >= 1 */
  float scale_a;      /* logit scale of the value head; <= 0 selects 1/sqrt(d_A) */
  const void *X_ref;
  const void *L_q, *L_k, *L_x;
  const float *b_x;
  const void *U_q, *U_k, *U_v;
  const void *L_c, *L_v;
} arckv_dsa_indexer;

/* Workspace for arckv_score_dsa with pair_chunk pairs in flight (0 = all B). */
arckv_status arckv_dsa_workspace_size(const arckv_problem *prob, int32_t pair_chunk, size_t *bytes);

/* Stage 1a with the value-aware indexer: pooled scores s_j of eq.
 * indexer_pooling, s_j = sqrt(mean_i softmax_j(I_i,:)_j^2), for every cached
 * token of every pair -> scores [B][T] float32 (rank them with arckv_select).
 * K, V, Q_ref bfloat16 only.  Intermediates (the value head's projections and
 * context, qbar, kbar) are stored in bfloat16; accumulation is float32. */
arckv_status arckv_score_dsa(const arckv_problem *prob, const void *K, const void *V,
                             const void *Q_ref, const arckv_dsa_indexer *ix, float *scores,
                             void *ws, size_t ws_bytes, hipStream_t stream);

/* Stage 1b: anchors S = TopK(scores, t) per pair (Section 3.3, eq.
 * persistent_support), written ascending to anchors [B][t].  Order: larger
 * score first, ties to the lower index, -0 equal to +0, NaN below every number.
 * Bit-exact by construction.  Needs 1 <= t <= T. */
arckv_status arckv_select(const arckv_problem *prob, const float *scores, int32_t t,
                          int32_t *anchors, void *ws, size_t ws_bytes, hipStream_t stream);

/* Per-pair budgets of eq. per_head_budget (host only, no GPU work):
 * t_out[i] = clip_[1,T](floor(a_i / sum(a) * P * t)) for P pairs with weights
 * a (host array, finite, >= 0, not all zero) and nominal per-pair budget t. */
arckv_status arckv_budgets(int32_t P, const double *a, int32_t t, int64_t T, int32_t *t_out);

/* Realised anchor count of chunked selection (Appendix A.3; host only):
 * sum over chunks c of length T_c of clip_[1,T_c](round(t T_c / T)) (rounded
 * half up) when chunk_len > 0 and T > 10,000, otherwise t. */
arckv_status arckv_select_count(int64_t T, int32_t t, int32_t chunk_len, int32_t *t_real);

/* Stage 1b, general form: per-pair budgets and/or chunked selection.
 *   t_pair     [B] device array of per-pair budgets (e.g. from arckv_budgets),
 *              or NULL for the uniform budget t; entries are clipped to [1, T].
 *   chunk_len  0 = global top-t; L > 0 = Appendix A.3 chunking when T > 10,000.
 *   anchors    [B][t_stride] output: each row holds the pair's anchors ascending,
 *              then -1 up to t_stride.  t_stride must cover every pair's realised
 *              count (arckv_select_count of its budget); rows are truncated, never
 *              overrun, if it does not.  With t_pair NULL a short t_stride is
 *              rejected (ARCKV_ERR_INVALID_ARG).
 * The order of S and the tie rules are those of arckv_select. */
arckv_status arckv_select_ex(const arckv_problem *prob, const float *scores, int32_t t,
                             const int32_t *t_pair, int32_t chunk_len, int32_t t_stride,
                             int32_t *anchors, hipStream_t stream);

/* Full-cache row statistics (Appendix A.9): with l_ij = s q_i.k_j,
 *   z [B][n]     z_i = max_j l_ij over the whole cache,
 *   m [B][n]     m_i = sum_j exp(l_ij - z_i)            (the mass targets Phi_K 1),
 *   Y [B][n][d]  Y_i = sum_j exp(l_ij - z_i) v_j / m_i   (full attention outputs).
 * No workspace. */
arckv_status arckv_rowstats(const arckv_problem *prob, const void *K, const void *V,
                            const void *Q_ref, float *z, float *m, float *Y, hipStream_t stream);

/* Stage 2: response-profile assignment and convex key merge (Section 3.4,
 * eq. response_profile, anchor_assignment, mass_centroid, key_merge).
 *   z        [B][n] row maxima from arckv_rowstats; max_i z_i is z_merge.
 *   anchors  [B][t] ascending anchor positions.
 *   C_k      [B][t][d] output; row r is the compact key of anchors[r], a convex
 *            combination of its group's keys with weights >= 0 summing to 1.
 *   assign   [B][T] output (may be NULL): the group r of every position;
 *            anchors are assigned to themselves, ties go to the lowest r.
 *   phi      [B][T] output (may be NULL): query-averaged mass exp(l - z_merge). */
arckv_status arckv_merge(const arckv_problem *prob, const void *K, const void *Q_ref,
                         const float *z, const int32_t *anchors, int32_t t, float lambda_m,
                         float *C_k, int32_t *assign, float *phi,
                         void *ws, size_t ws_bytes, hipStream_t stream);

/* Stage 3: mass bias (Appendix A.9, eq. mass_fit).  With
 * Phi_C = exp(s Q C_k^T - z 1^T): w~ solves (G + delta_beta tr(G)/t I) w = h,
 * G = Phi_C^T Phi_C, h = Phi_C^T m, by Cholesky (float32) plus refinement;
 * beta = clip(log max(max(w~, 0), eps_w), b_min, b_max).
 * With p->bias_mode = 1, w* instead minimises w^T (G + lam I) w / 2 - h^T w over
 * w >= 0 (lam the ridge settled by the factorisation above), found by block
 * principal pivoting: each iteration refactors the system restricted to the
 * current free set and solves it with refinement against the data.
 *   K, V  [B][T][d] the cache; read only when z or m is NULL.
 *   z, m  [B][n] row maxima and masses from arckv_rowstats, or NULL: both are then
 *         recomputed from K, V and Q_ref (arckv_rowstats) into the workspace.
 *   beta  [B][t] output.
 *   info  [B] output: 0 = ok; k > 0 = Cholesky pivot k failed after all ridge
 *         escalations; -1 = a non-finite value in z, m or C_k (the pair is not
 *         fitted); -2 = bias_mode 1 did not settle within nnls_max_iter
 *         iterations.  beta is NaN whenever info != 0.
 *   delta_used [B] output (may be NULL): the relative ridge actually used.
 * Ridge escalation: a pair whose factorisation fails, or whose refinement is
 * cut off (refine_steps), is refactored with the ridge raised tenfold (from
 * 1e-7 when delta_beta = 0), at most p->max_escalations times in all.  Before
 * each such round the call reads back one integer (the number of pairs to
 * refactor) and synchronises the stream; with max_escalations = 0 it never
 * synchronises. */
arckv_status arckv_fit_bias(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                            const float *C_k, int32_t t, const float *z, const float *m,
                            const arckv_fit_params *p, float *beta, int32_t *info, float *delta_used,
                            void *ws, size_t ws_bytes, hipStream_t stream);

/* Stage 4: compact values (Appendix A.9, eq. value_lstsq).  With
 * P_hat = softmax(s Q C_k^T + 1 beta^T): C_v solves
 * (A + delta_v tr(A)/t I) C_v = P_hat^T Y, A = P_hat^T P_hat.
 *   K, V  [B][T][d] the cache; read only when Y is NULL.
 *   Y     [B][n][d] full-attention outputs from arckv_rowstats, or NULL:
 *         recomputed from K, V and Q_ref into the workspace.
 *   C_v   [B][t][d] output.
 *   info  [B] output: 0 = ok; k > 0 = Cholesky pivot k failed after all ridge
 *         escalations; -1 = a non-finite value in Y, C_k or beta (a failed mass
 *         fit leaves beta NaN, so its pair reports -1 here).  C_v is NaN
 *         whenever info != 0.
 *   delta_used and the escalation rounds as for arckv_fit_bias. */
arckv_status arckv_fit_values(const arckv_problem *prob, const void *K, const void *V, const void *Q_ref,
                              const float *C_k, const float *beta, int32_t t, const float *Y,
                              const arckv_fit_params *p, float *C_v, int32_t *info, float *delta_used,
                              void *ws, size_t ws_bytes, hipStream_t stream);

/* The whole per-context path for B pairs: score, select, row statistics,
 * merge, mass fit, value fit.  t = arckv_budget(T, rho) (or, with
 * p->select_chunk, arckv_select_count of it) is written to *t_out (host
 * pointer) before any device work.  Outputs: anchors [B][t], C_k [B][t][d],
 * beta [B][t], C_v [B][t][d], info [B][2] (mass-fit, value-fit status as above;
 * a non-finite value anywhere in K, V or Q_ref reaches the row statistics and
 * the pair reports -1 in both).
 * Pairs are processed p->pair_chunk at a time (0 = all at once). */
arckv_status arckv_compact(const arckv_problem *prob, const void *K, const void *V,
                           const void *Q_ref, const arckv_indexer *ix, double rho,
                           const arckv_fit_params *p, int32_t *t_out, int32_t *anchors,
                           float *C_k, float *beta, float *C_v, int32_t *info,
                           void *ws, size_t ws_bytes, hipStream_t stream);

/* Decode-time attention over a compacted block followed by an optional
 * uncompressed block (eq. compact_attention; the joint form of Appendix A.7,
 * eq. concatenated_attention_preservation, which appends zero bias for the
 * uncompressed rows).  For each pair p (one sequence and KV head) and each of
 * its G query rows q (the query heads sharing that KV head):
 *   out[p][q] = softmax([s q C_k^T + beta, s q K_f^T]) [C_v; V_f]
 * with s = scale (<= 0 selects 1/sqrt(d)).  The consumer of arckv_compact's
 * output; with beta = NULL, C_k = K, C_v = V and F = 0 it is full-cache
 * attention.
 *   Q        [P][G][d] bfloat16, d = 128; G in {1, 2, 4, 8}.
 *   C_k, C_v [P][t][d] bfloat16 (may be NULL when t = 0).
 *   beta     [P][t] float32, or NULL for zero bias.
 *   K_f, V_f [P][F][d] bfloat16 (may be NULL when F = 0).
 *   out      [P][G][d] float32.
 * Requires t, F >= 0 and t + F >= 1; all arrays 16-byte aligned.  Workspace:
 * arckv_attend_workspace_size(P, G, t, F) bytes (per-chunk partial results).
 * Reads every key and value row once. */
arckv_status arckv_attend_workspace_size(int32_t P, int32_t G, int32_t t, int32_t F, size_t *bytes);
arckv_status arckv_attend(int32_t P, int32_t G, int32_t t, int32_t F, float scale, const void *Q,
                          const void *C_k, const float *beta, const void *C_v, const void *K_f,
                          const void *V_f, float *out, void *ws, size_t ws_bytes, hipStream_t stream);

/* arckv_attend for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same arguments and result, no workspace.  The split-key partials go to a
 * static device array of 64 MiB that the library holds on each GPU it runs
 * on until the process ends; the call itself allocates nothing.  Returns
 * ARCKV_ERR_WORKSPACE when arckv_attend_workspace_size(P, G, t, F) exceeds
 * 64 MiB (for instance P = 512, G = 4 allows t + F up to 16,128; use
 * arckv_attend with a workspace beyond that), ARCKV_ERR_HIP if the array's
 * device address cannot be obtained.  Every call on one GPU shares that GPU's
 * array, so calls that may overlap in time on one GPU (different streams or
 * host threads) race; calls ordered on one stream do not.  Nothing in the
 * array needs to start at zero. */
arckv_status arckv_attend_noalloc(int32_t P, int32_t G, int32_t t, int32_t F, float scale, const void *Q,
                                  const void *C_k, const float *beta, const void *C_v, const void *K_f,
                                  const void *V_f, float *out, hipStream_t stream);

/* arckv_compact with the scoring stage replaced by caller-supplied scores
 * [B][T] float32 (for instance from arckv_score_dsa): select, row statistics,
 * merge and both fits exactly as arckv_compact. */
arckv_status arckv_compact_scored(const arckv_problem *prob, const void *K, const void *V,
                                  const void *Q_ref, const float *scores, double rho,
                                  const arckv_fit_params *p, int32_t *t_out, int32_t *anchors,
                                  float *C_k, float *beta, float *C_v, int32_t *info,
                                  void *ws, size_t ws_bytes, hipStream_t stream);

/* Statistics of the key-to-anchor decision of the most recent arckv_merge,
 * arckv_compact or arckv_compact_scored call that used this workspace with
 * this problem and anchor count t (Section 3.4, eq. anchor_assignment).  The
 * argmax is decided in up to three passes: an fp16 (bf16 inputs) or fp32
 * contraction whose per-similarity rounding error is bounded, so every key
 * with a single anchor inside the bound is decided there; a refine pass over
 * the flagged keys' candidate anchors with logits accurate to about 1e-6; and
 * a float64 pass for the keys the refine pass cannot separate (equal float64
 * similarities go to the lowest r).  Copies [B][8] int32 to the device array
 * stats, per pair: [0] keys flagged after the first pass, [1] keys decided in
 * float64, [2] candidate anchors of the flagged keys (a whole anchor tile
 * counts its 256 (bf16) or 128 (float32) anchors), [3] keys left undecided
 * (no finite similarity reaches the first pass's bound, which takes a
 * non-finite input; such a key keeps the first pass's best), [4] and [5] the
 * undecided ones of the first and of the refine pass ([5] stays 0: the refine
 * pass sends every key's survivors, however many, to the float64 pass, and a
 * key whose candidates overflow the candidate pool goes there with all t
 * anchors), [6] keys sent to the refine pass, [7]
 * flagged keys with a whole anchor tile among their candidates.  Those
 * counters are the only workspace contents that outlive a call. */
arckv_status arckv_assign_stats(const arckv_problem *prob, int32_t t, const void *ws, size_t ws_bytes,
                                int32_t *stats, hipStream_t stream);

/* Human-readable name of a status code (static string). */
const char *arckv_status_string(arckv_status s);

/* Instrumentation.  When enabled (non-zero), entry points record HIP events
 * around each internal kernel stage on the call's stream; arckv_stage_times
 * then synchronises those events and returns per-stage milliseconds of the
 * most recent call, accumulated over calls since the last reset.
 *   names   receives up to max_stages static stage names (may be NULL),
 *   ms      receives the accumulated milliseconds,
 *   counts  receives how many launches were timed per stage (may be NULL).
 * Returns the number of stages via *n_stages.  Not thread-safe. */
arckv_status arckv_set_timing(int32_t enable);
arckv_status arckv_stage_times(int32_t max_stages, const char **names, double *ms,
                               int32_t *counts, int32_t *n_stages);
arckv_status arckv_reset_timing(void);

#ifdef __cplusplus
}
#endif
#endif /* ARCKV_H */
