"""Float64 CPU oracle for ARC-KV compaction (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package; the GPU library never does.
"""
from .core import *  # noqa: F401,F403
from .core import (DSAIndexer, rms_blocks, leaky_relu, dsa_logits, RMS_EPS, LEAKY_SLOPE, budget, budgets_per_pair, chunk_budgets, select_topt_chunked, CHUNK_THRESHOLD, gelu, score_mlp, pool_rms, select_topt, logits, global_logit_max,
                   response_profiles, assign, mass_weights, profiles_assign_phi, merge_keys,
                   rowstats, ridge_cholesky_solve, CholeskyFailure, phi_c, nnls_gram, fit_bias,
                   compact_probs, fit_values, round_to, attend_compact, attend_full, attend_joint, row_rel_err,
                   compact_pair, PairResult, BiasFit, ValueFit, LAMBDA_M, DELTA_BETA, DELTA_V,
                   EPS_W, B_MIN, B_MAX, MAX_ESCALATIONS)
