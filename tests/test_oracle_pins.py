"""Pins of the float64 oracle against things other than itself.

Each test checks the oracle against a brute-force loop written separately
(tests/brute.py), a closed form, an identity the paper states, a library
routine that solves the same problem another way, or a value printed in the
workload definitions.  No GPU involved.
"""
import dataclasses
import math
import os

import numpy as np
import pytest

import oracle
from tests import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.default_rng(seed)


def small_pair(seed=0, T=12, n=20, d=6, hidden=5, outlier=True):
    g = rng(seed)
    K = g.standard_normal((T, d))
    if outlier:
        K[:, 0] *= 3.0
    V = g.standard_normal((T, d))
    Q = g.standard_normal((n, d))
    W1 = g.uniform(-0.5, 0.5, (hidden, 2 * d))
    b1 = g.uniform(-0.5, 0.5, hidden)
    w2 = g.uniform(-0.5, 0.5, hidden)
    b2 = np.array([g.uniform(-0.5, 0.5)])
    return K, V, Q, W1, b1, w2, b2


# ----------------------------------------------------------------- O0 budget
def test_budget_golden():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "budgets.txt")) if l.strip() and not l.startswith("#")]
    assert rows
    for T, rho, t in rows:
        assert oracle.budget(int(T), float(rho)) == int(t)


def test_budget_edges():
    assert oracle.budget(10, 0.0) == 1            # clipped up to 1
    assert oracle.budget(10, 1.0) == 10
    assert oracle.budget(10, 5.0) == 10           # clipped down to T
    assert oracle.budget(10, 0.25) == 3           # 2.5 rounds half up
    assert oracle.budget(10, 0.24) == 2
    for T, rho in [(16384, 0.2), (16384, 0.1), (16384, 0.05), (16384, 0.02), (8192, 0.1), (32768, 0.1)]:
        t = oracle.budget(T, rho)
        assert abs(t - rho * T) <= 0.5


# ----------------------------------------------------------------- O1 score
def test_gelu_values():
    xs = np.array([-3.0, -1.0, -0.5, 0.0, 0.5, 1.0, 2.5])
    got = oracle.gelu(xs)
    for x, g in zip(xs, got):
        assert g == pytest.approx(0.5 * x * (1 + math.erf(x / math.sqrt(2))), rel=1e-15, abs=1e-300)
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    # GELU(x) - GELU(-x) = x for the erf form
    y = np.linspace(-6, 6, 101)
    np.testing.assert_allclose(oracle.gelu(y) - oracle.gelu(-y), y, rtol=0, atol=1e-14)


def test_score_bruteforce():
    K, V, Q, W1, b1, w2, b2 = small_pair(1)
    got = oracle.score_mlp(K, V, W1, b1, w2, b2)
    ref = brute.score(K.tolist(), V.tolist(), W1.tolist(), b1.tolist(), w2.tolist(), b2[0])
    np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-13)


def test_score_zero_weights_all_tie():
    K, V, Q, W1, b1, w2, b2 = small_pair(2)
    I = oracle.score_mlp(K, V, np.zeros_like(W1), b1, w2, b2)
    assert np.all(I == I[0])
    assert oracle.select_topt(I, 5).tolist() == [0, 1, 2, 3, 4]


def test_pool_rms_bruteforce_and_single_row():
    g = rng(3)
    I = g.standard_normal((7, 15)) * 2
    np.testing.assert_allclose(oracle.pool_rms(I), brute.pool_rms(I.tolist()), rtol=1e-13)
    # a query-independent scorer: identical rows -> s = softmax(I), same ranking as I
    row = g.standard_normal(15)
    s = oracle.pool_rms(np.tile(row, (4, 1)))
    e = np.exp(row - row.max())
    np.testing.assert_allclose(s, e / e.sum(), rtol=1e-13)
    assert oracle.select_topt(s, 6).tolist() == oracle.select_topt(row, 6).tolist()


# ----------------------------------------------------------------- O2 select
@pytest.mark.parametrize("seed", range(6))
def test_select_matches_exhaustive_sort(seed):
    g = rng(10 + seed)
    T = int(g.integers(1, 60))
    kind = seed % 3
    if kind == 0:
        s = g.standard_normal(T)
    elif kind == 1:
        s = g.integers(-3, 3, T).astype(np.float64)          # many duplicates
    else:
        s = g.choice([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, np.nan], T)
    for t in sorted({1, T, max(1, T // 3), max(1, T // 2)}):
        assert oracle.select_topt(s, t).tolist() == brute.select(s.tolist(), t)


def test_select_special_cases():
    s = np.array([1.0, 3.0, 3.0, -0.0, 0.0, np.nan, -np.inf])
    assert oracle.select_topt(s, 1).tolist() == [1]            # lowest-index argmax
    assert oracle.select_topt(s, 2).tolist() == [1, 2]
    assert oracle.select_topt(s, 4).tolist() == [0, 1, 2, 3]   # -0 ties +0; lower index wins
    assert oracle.select_topt(s, 6).tolist() == [0, 1, 2, 3, 4, 6]   # NaN below -inf
    assert oracle.select_topt(s, 7).tolist() == list(range(7))
    with pytest.raises(ValueError):
        oracle.select_topt(s, 0)


# ----------------------------------------------------------------- O3-O5
def test_profiles_bruteforce_and_invariants():
    K, V, Q, *_ = small_pair(4)
    s = 0.7
    E, U, zm = oracle.response_profiles(Q, K, s)
    Ub, phib, zmb = brute.profiles(Q.tolist(), K.tolist(), s)
    np.testing.assert_allclose(U.T, Ub, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(oracle.mass_weights(E), phib, rtol=1e-12)
    assert zm == pytest.approx(zmb, rel=1e-14)
    np.testing.assert_allclose(np.linalg.norm(U, axis=0), 1.0, rtol=1e-13)
    # profiles do not depend on the global shift
    _, U2, _ = oracle.response_profiles(Q, K, s, z_merge=zm - 3.0)
    np.testing.assert_allclose(U2, U, rtol=1e-12)


def test_assign_bruteforce_selfassign_and_partition():
    K, V, Q, *_ = small_pair(5, T=15)
    S = np.array([1, 4, 9, 13])
    _, U, _ = oracle.response_profiles(Q, K, 0.5)
    kap = oracle.assign(U, S)
    assert kap.tolist() == brute.assign(U.T.tolist(), S.tolist())
    assert kap[S].tolist() == list(range(len(S)))          # kappa(s_r) = r
    groups = [np.flatnonzero(kap == r) for r in range(len(S))]
    assert sum(len(gr) for gr in groups) == len(K)          # a partition of [T]
    assert all(len(gr) > 0 and S[r] in gr for r, gr in enumerate(groups))


def test_assign_ties_lowest_anchor_and_duplicate_keys():
    K, V, Q, *_ = small_pair(6, T=10)
    K[7] = K[2]                       # two anchors with identical keys -> identical profiles
    K[5] = K[3]                       # a duplicated non-anchor key
    S = np.array([2, 7])
    _, U, _ = oracle.response_profiles(Q, K, 0.5)
    kap = oracle.assign(U, S)
    assert kap[2] == 0 and kap[7] == 1
    others = [j for j in range(10) if j not in (2, 7)]
    assert all(kap[j] == 0 for j in others)   # every similarity ties -> lowest r
    S2 = np.array([0, 4, 8])
    kap2 = oracle.assign(U, S2)
    assert kap2[5] == kap2[3]


def test_chunked_path_equals_direct():
    K, V, Q, *_ = small_pair(7, T=40, n=9)
    S = np.array([0, 5, 17, 30, 39])
    E, U, zm = oracle.response_profiles(Q, K, 0.4)
    old = oracle.core._CHUNK_ELEMS
    try:
        oracle.core._CHUNK_ELEMS = 9 * 7                # 7 keys per chunk
        kap, phi, zm2 = oracle.profiles_assign_phi(Q, K, S, 0.4)
    finally:
        oracle.core._CHUNK_ELEMS = old
    assert kap.tolist() == oracle.assign(U, S).tolist()
    np.testing.assert_allclose(phi, oracle.mass_weights(E), rtol=1e-13)
    assert zm2 == zm


def test_merge_endpoints_and_bruteforce():
    K, V, Q, *_ = small_pair(8, T=14)
    S = np.array([0, 3, 6, 11])
    kap, phi, _ = oracle.profiles_assign_phi(Q, K, S, 0.5)
    # lambda_m = 0 leaves the anchors unmerged, bit for bit
    assert np.array_equal(oracle.merge_keys(K, phi, kap, S, 0.0), K[S])
    for lam in (0.25, 0.5, 1.0):
        got = oracle.merge_keys(K, phi, kap, S, lam)
        ref = brute.merge(K.tolist(), phi.tolist(), kap.tolist(), S.tolist(), lam)
        np.testing.assert_allclose(got, ref, rtol=1e-13, atol=1e-14)
    # t = 1: one group holding every key
    S1 = np.array([4])
    kap1, phi1, _ = oracle.profiles_assign_phi(Q, K, S1, 0.5)
    assert np.all(kap1 == 0)
    mu = (phi1[:, None] * K).sum(0) / phi1.sum()
    np.testing.assert_allclose(oracle.merge_keys(K, phi1, kap1, S1, 0.3)[0], 0.7 * K[4] + 0.3 * mu, rtol=1e-13)
    # t = T: singleton groups, C_k = K for every lambda
    SA = np.arange(len(K))
    kapA, phiA, _ = oracle.profiles_assign_phi(Q, K, SA, 0.5)
    np.testing.assert_allclose(oracle.merge_keys(K, phiA, kapA, SA, 0.6), K, rtol=1e-14, atol=1e-15)


def test_merge_convex_hull():
    K, V, Q, *_ = small_pair(9, T=30, n=25)
    S = np.array([2, 8, 15, 21, 27])
    kap, phi, _ = oracle.profiles_assign_phi(Q, K, S, 0.5)
    Ck = oracle.merge_keys(K, phi, kap, S, 0.6)
    probes = rng(99).standard_normal((50, K.shape[1]))
    for r in range(len(S)):
        G = K[kap == r]
        assert np.all(Ck[r] >= G.min(0) - 1e-12) and np.all(Ck[r] <= G.max(0) + 1e-12)
        lg = probes @ G.T
        lc = probes @ Ck[r]
        assert np.all(lc >= lg.min(1) - 1e-12) and np.all(lc <= lg.max(1) + 1e-12)


def test_merge_zero_mass_group_keeps_anchor():
    K = rng(1).standard_normal((4, 3))
    S = np.array([0, 2])
    kap = np.array([0, 0, 1, 1])
    phi = np.array([0.5, 0.5, 0.0, 0.0])
    Ck = oracle.merge_keys(K, phi, kap, S, 1.0)
    assert np.array_equal(Ck[1], K[2])


# ----------------------------------------------------------------- O6
def test_rowstats_bruteforce_and_bounds():
    K, V, Q, *_ = small_pair(10, T=11, n=7)
    z, m, Y = oracle.rowstats(Q, K, V, 0.6)
    zb, mb, Yb = brute.rowstats(Q.tolist(), K.tolist(), V.tolist(), 0.6)
    np.testing.assert_allclose(z, zb, rtol=1e-14)
    np.testing.assert_allclose(m, mb, rtol=1e-13)
    np.testing.assert_allclose(Y, Yb, rtol=1e-12, atol=1e-14)
    assert np.all(m >= 1.0 - 1e-15) and np.all(m <= len(K))
    assert np.all(Y >= V.min(0) - 1e-12) and np.all(Y <= V.max(0) + 1e-12)
    # T = 1: the single value comes back, m = 1
    z1, m1, Y1 = oracle.rowstats(Q, K[:1], V[:1], 0.6)
    np.testing.assert_allclose(m1, 1.0)
    np.testing.assert_allclose(Y1, np.tile(V[0], (len(Q), 1)), rtol=1e-15)
    np.testing.assert_allclose(z1, 0.6 * Q @ K[0], rtol=1e-14)


def test_rowstats_matches_library_softmax():
    from scipy.special import softmax
    K, V, Q, *_ = small_pair(11, T=50, n=13)
    _, _, Y = oracle.rowstats(Q, K, V, 0.3)
    np.testing.assert_allclose(Y, softmax(0.3 * Q @ K.T, axis=1) @ V, rtol=1e-12)


# ----------------------------------------------------------------- O7 mass fit
def test_mass_fit_single_anchor_closed_form():
    K, V, Q, *_ = small_pair(12, T=9, n=16)
    s = 0.5
    z, m, _ = oracle.rowstats(Q, K, V, s)
    Ck = K[3:4]
    bf = oracle.fit_bias(Q, Ck, z, m, s, delta=0.0)
    phi = np.exp(s * Q @ Ck[0] - z)
    assert bf.w_tilde[0] == pytest.approx(phi @ m / (phi @ phi), rel=1e-12)
    assert bf.beta[0] == pytest.approx(math.log(phi @ m / (phi @ phi)), rel=1e-12)


def test_mass_fit_matches_lstsq_without_ridge():
    K, V, Q, *_ = small_pair(13, T=25, n=60)
    s = 0.5
    z, m, _ = oracle.rowstats(Q, K, V, s)
    Ck = K[[1, 5, 9, 14, 20]] * 0.9
    bf = oracle.fit_bias(Q, Ck, z, m, s, delta=0.0)
    PhiC = np.exp(s * Q @ Ck.T - z[:, None])
    w_ls = np.linalg.lstsq(PhiC, m, rcond=None)[0]
    np.testing.assert_allclose(bf.w_tilde, w_ls, rtol=1e-8, atol=1e-10)
    np.testing.assert_allclose(bf.beta, np.clip(np.log(np.maximum(np.maximum(w_ls, 0), 1e-12)), -30, 30), rtol=1e-7)


def brute_nnls(G, h):
    t = len(h)
    best, bw = math.inf, None
    for mask in range(1 << t):
        P = [i for i in range(t) if mask >> i & 1]
        w = np.zeros(t)
        if P:
            w[P] = np.linalg.solve(G[np.ix_(P, P)], h[P])
            if np.any(w[P] < 0):
                continue
        f = 0.5 * w @ G @ w - h @ w
        if f < best - 1e-15:
            best, bw = f, w
    return bw


@pytest.mark.parametrize("seed", range(5))
def test_nnls_matches_bruteforce(seed):
    g = rng(40 + seed)
    t = int(g.integers(2, 9))
    A = g.standard_normal((3 * t, t))
    b = g.standard_normal(3 * t)
    G, h = A.T @ A, A.T @ b
    np.testing.assert_allclose(oracle.nnls_gram(G, h), brute_nnls(G, h), rtol=1e-9, atol=1e-11)


def test_nnls_mode_on_mass_fit():
    K, V, Q, *_ = small_pair(14, T=20, n=40)
    s = 0.8
    z, m, _ = oracle.rowstats(Q, K, V, s)
    Ck = K[[0, 2, 3, 7, 11, 12, 19]]
    bf0 = oracle.fit_bias(Q, Ck, z, m, s, delta=1e-8, mode=0)
    bf1 = oracle.fit_bias(Q, Ck, z, m, s, delta=1e-8, mode=1)
    t = len(Ck)
    Greg = bf1.G + 1e-8 * np.trace(bf1.G) / t * np.eye(t)
    np.testing.assert_allclose(bf1.w_star, brute_nnls(Greg, bf1.h), rtol=1e-7, atol=1e-10)
    if np.all(bf0.w_tilde >= 0):        # projected LS = NNLS when nothing is clipped
        np.testing.assert_allclose(bf0.w_star, bf1.w_star, rtol=1e-7)


def test_full_retention_mass_fit_is_exact():
    K, V, Q, *_ = small_pair(15, T=8, n=30)
    s = 0.5
    z, m, _ = oracle.rowstats(Q, K, V, s)
    bf = oracle.fit_bias(Q, K, z, m, s, delta=0.0)
    np.testing.assert_allclose(bf.w_tilde, 1.0, rtol=1e-9)
    np.testing.assert_allclose(bf.beta, 0.0, atol=1e-9)


def test_ridge_escalation():
    A = np.array([[1.0, 1.001], [1.001, 1.0]])          # indefinite by 1e-3
    X, d, attempts = oracle.ridge_cholesky_solve(A, np.ones(2), 1e-5)
    assert attempts == 4 and d == pytest.approx(1e-2)
    np.testing.assert_allclose((A + d * np.eye(2)) @ X, np.ones(2), rtol=1e-10)
    with pytest.raises(oracle.CholeskyFailure):
        oracle.ridge_cholesky_solve(A, np.ones(2), 1e-5, max_escalations=2)
    with pytest.raises(oracle.CholeskyFailure):
        oracle.ridge_cholesky_solve(np.zeros((2, 2)) - np.eye(2), np.ones(2), 0.0)


def test_row_rel_err_bruteforce():
    """The parity metric: per-row ||o - o_ref|| / ||o_ref||, against a loop.
    Rows differ in scale and the error sits in one row, so a wrong axis or a
    norm over the whole matrix fails."""
    g = np.random.default_rng(5)
    O_ref = g.standard_normal((7, 5)) * np.arange(1, 8)[:, None]
    O = O_ref.copy()
    O[3] += 0.01 * g.standard_normal(5)
    got = oracle.row_rel_err(O, O_ref)
    want = brute.row_rel_err(O, O_ref)
    assert got.shape == (7,)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)
    assert np.count_nonzero(got) == 1 and got[3] > 0
    np.testing.assert_allclose(oracle.row_rel_err(2 * O_ref, O_ref), 1.0)


def test_ridge_escalation_from_zero():
    """A zero ridge on a singular Gram (two equal columns) escalates from the
    floor: delta 0 fails at the second pivot, delta = 1e-7 succeeds."""
    A = np.array([[1.0, 1.0], [1.0, 1.0]])
    b = np.array([1.0, 2.0])
    X, d, attempts = oracle.ridge_cholesky_solve(A, b, 0.0)
    assert attempts == 2 and d == oracle.DELTA_FLOOR
    np.testing.assert_allclose((A + d * np.eye(2)) @ X, b, rtol=1e-6)
    with pytest.raises(oracle.CholeskyFailure):
        oracle.ridge_cholesky_solve(A, b, 0.0, max_escalations=0)


# ----------------------------------------------------------------- O8 value fit
def test_value_fit_matches_augmented_lstsq():
    K, V, Q, *_ = small_pair(16, T=30, n=50)
    s = 0.5
    z, m, Y = oracle.rowstats(Q, K, V, s)
    Ck = K[[0, 4, 9, 13, 22, 29]]
    beta = rng(0).uniform(-1, 1, 6)
    vf = oracle.fit_values(Q, Ck, beta, Y, s, delta=1e-3)
    P = oracle.compact_probs(Q, Ck, beta, s)
    lam = 1e-3 * np.trace(P.T @ P) / 6
    Aug = np.vstack([P, math.sqrt(lam) * np.eye(6)])
    rhs = np.vstack([Y, np.zeros((6, Y.shape[1]))])
    np.testing.assert_allclose(vf.C_v, np.linalg.lstsq(Aug, rhs, rcond=None)[0], rtol=1e-9, atol=1e-11)
    # normal-equation residual P^T (P C - Y) + lam C = 0
    res = P.T @ (P @ vf.C_v - Y) + lam * vf.C_v
    assert np.abs(res).max() < 1e-12 * max(1.0, np.abs(P.T @ Y).max())


def test_value_fit_linear_and_translation_equivariant():
    K, V, Q, *_ = small_pair(17, T=20, n=40)
    s = 0.5
    Ck = K[[1, 6, 12, 18]]
    beta = np.array([0.1, -0.2, 0.3, 0.0])
    Y1 = rng(1).standard_normal((40, 6))
    Y2 = rng(2).standard_normal((40, 6))
    f = lambda Y, dv: oracle.fit_values(Q, Ck, beta, Y, s, delta=dv).C_v
    np.testing.assert_allclose(f(2 * Y1 - 3 * Y2, 1e-3), 2 * f(Y1, 1e-3) - 3 * f(Y2, 1e-3), rtol=1e-9, atol=1e-12)
    c = rng(3).standard_normal(6)
    np.testing.assert_allclose(f(Y1 + c, 0.0), f(Y1, 0.0) + c, rtol=1e-8, atol=1e-10)


def test_compact_attention_bruteforce():
    g = rng(18)
    Q, Ck, Cv = g.standard_normal((5, 4)), g.standard_normal((3, 4)), g.standard_normal((3, 4))
    beta = g.standard_normal(3)
    np.testing.assert_allclose(oracle.attend_compact(Q, Ck, beta, Cv, 0.7),
                               brute.compact_attend(Q.tolist(), Ck.tolist(), beta.tolist(), Cv.tolist(), 0.7),
                               rtol=1e-13)


# ----------------------------------------------------------------- O9 end to end
def test_full_retention_reproduces_full_attention():
    K, V, Q, W1, b1, w2, b2 = small_pair(19, T=8, n=40)
    res = oracle.compact_pair(K, V, Q, W1, b1, w2, b2, t=8, scale=0.5, lambda_m=0.5,
                              delta_beta=0.0, delta_v=0.0)
    assert res.anchors.tolist() == list(range(8))
    np.testing.assert_allclose(res.C_k, K, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(res.beta, 0.0, atol=1e-8)
    np.testing.assert_allclose(res.C_v, V, rtol=1e-7, atol=1e-8)
    Qh = rng(20).standard_normal((15, K.shape[1]))
    np.testing.assert_allclose(oracle.attend_compact(Qh, res.C_k, res.beta, res.C_v, 0.5),
                               oracle.attend_full(Qh, K, V, 0.5), rtol=1e-7, atol=1e-8)
    # the joint objective with an uncompressed block (Appendix A.7) holds exactly too
    Kf, Vf = rng(21).standard_normal((3, K.shape[1])), rng(22).standard_normal((3, K.shape[1]))
    full = oracle.attend_full(Qh, np.vstack([K, Kf]), np.vstack([V, Vf]), 0.5)
    joint = oracle.attend_compact(Qh, np.vstack([res.C_k, Kf]), np.concatenate([res.beta, np.zeros(3)]),
                                  np.vstack([res.C_v, Vf]), 0.5)
    np.testing.assert_allclose(joint, full, rtol=1e-7, atol=1e-8)


def test_compaction_beats_hard_subset_on_heldout():
    """Trend check (Table 1 ordering): merged+fitted cache < hard subset error."""
    g = rng(23)
    T, n, d = 200, 160, 16
    K = g.standard_normal((T, d)); K[:, 0] *= 4
    V = g.standard_normal((T, d))
    Q = g.standard_normal((n, d))
    Qh = g.standard_normal((64, d))
    W1 = g.uniform(-.2, .2, (8, 2 * d)); b1 = g.uniform(-.2, .2, 8); w2 = g.uniform(-.3, .3, 8)
    res = oracle.compact_pair(K, V, Q, W1, b1, w2, np.zeros(1), rho=0.1, scale=0.25)
    O = oracle.attend_full(Qh, K, V, 0.25)
    fitted = oracle.row_rel_err(oracle.attend_compact(Qh, res.C_k, res.beta, res.C_v, 0.25), O).mean()
    S = res.anchors
    hard = oracle.row_rel_err(oracle.attend_compact(Qh, K[S], np.zeros(len(S)), V[S], 0.25), O).mean()
    assert fitted < hard


# ----------------------------------------------------------------- kernel-precision assignment
def test_round_to_matches_struct_rounding():
    g = rng(50)
    xs = np.concatenate([g.standard_normal(200) * 10.0 ** g.integers(-8, 8, 200),
                         [1.0, 1.00390625, 1.005859375, 1.0078125, -2.5, 0.0, 1e-40]])
    got = oracle.round_to(xs, "bf16")
    assert got.tolist() == [brute.round_bf16(float(x)) for x in xs]
    assert oracle.round_to(np.array([1.00390625]), "bf16")[0] == 1.0          # tie to even
    assert oracle.round_to(np.array([1.01171875]), "bf16")[0] == 1.015625      # tie to even (up)
    np.testing.assert_array_equal(oracle.round_to(xs, "f32"), xs.astype(np.float32).astype(np.float64))


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_assignment_in_storage_precision_bruteforce(dt):
    K, V, Q, *_ = small_pair(60, T=14, n=9)
    S = np.array([1, 5, 8, 12])
    rnd = brute.round_bf16 if dt == "bf16" else (lambda v: float(np.float32(v)))
    kap, _, _ = oracle.profiles_assign_phi(Q, K, S, 0.6, profile_dtype=dt)
    assert kap.tolist() == brute.assign_rounded(Q.tolist(), K.tolist(), S.tolist(), 0.6, rnd)


# ----------------------------------------------------------------- O10 joint decode attention
def _joint_case(seed, t=7, F=5, n=4, d=6):
    g = rng(seed)
    return (g.standard_normal((n, d)), g.standard_normal((t, d)), g.uniform(-2, 2, t), g.standard_normal((t, d)),
            g.standard_normal((F, d)), g.standard_normal((F, d)))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_joint_attention_bruteforce(seed):
    Q, Ck, b, Cv, Kf, Vf = _joint_case(seed)
    s = 0.7
    got = oracle.attend_joint(Q, Ck, b, Cv, Kf, Vf, s)
    ref = np.array(brute.joint_attend(Q.tolist(), Ck.tolist(), b.tolist(), Cv.tolist(), Kf.tolist(), Vf.tolist(), s))
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_joint_attention_block_decomposition():
    """softmax over two concatenated blocks = the mass-weighted mix of each block's
    own softmax output (Z_C O_C + Z_F O_F) / (Z_C + Z_F), with the masses of
    eq. block_attention_mass (Z_C includes the bias)."""
    Q, Ck, b, Cv, Kf, Vf = _joint_case(3, t=9, F=4)
    s = 0.5
    got = oracle.attend_joint(Q, Ck, b, Cv, Kf, Vf, s)
    for i, q in enumerate(Q):
        wc = np.array([math.exp(s * float(q @ c) + bb) for c, bb in zip(Ck, b)])
        wf = np.array([math.exp(s * float(q @ k)) for k in Kf])
        Oc, Of = wc @ Cv / wc.sum(), wf @ Vf / wf.sum()
        mix = (wc.sum() * Oc + wf.sum() * Of) / (wc.sum() + wf.sum())
        np.testing.assert_allclose(got[i], mix, rtol=1e-12, atol=1e-13)


def test_joint_attention_split_full_cache_is_full_attention():
    """With zero bias, a cache split into a 'compact' prefix and an uncompressed
    suffix attends exactly like the whole cache (row statistics' Y)."""
    g = rng(4)
    K, V, Q = g.standard_normal((13, 6)), g.standard_normal((13, 6)), g.standard_normal((5, 6))
    s = 0.8
    _, _, Y = oracle.rowstats(Q, K, V, s)
    for a in (0, 1, 6, 13):
        got = oracle.attend_joint(Q, K[:a], np.zeros(a), V[:a], K[a:], V[a:], s)
        np.testing.assert_allclose(got, Y, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(oracle.attend_joint(Q, K, None, V, None, None, s), Y, rtol=1e-12, atol=1e-13)


def test_joint_attention_bias_shift():
    """A constant c added to every beta leaves a lone compact block unchanged and,
    next to an uncompressed block, multiplies the compact block's mass by e^c."""
    Q, Ck, b, Cv, Kf, Vf = _joint_case(5)
    s, c = 0.6, 1.3
    np.testing.assert_allclose(oracle.attend_joint(Q, Ck, b + c, Cv, None, None, s),
                               oracle.attend_joint(Q, Ck, b, Cv, None, None, s), rtol=1e-12, atol=1e-13)
    got = oracle.attend_joint(Q, Ck, b + c, Cv, Kf, Vf, s)
    for i, q in enumerate(Q):
        wc = np.exp(s * (Ck @ q) + b)
        wf = np.exp(s * (Kf @ q))
        mix = (math.exp(c) * (wc @ Cv) + wf @ Vf) / (math.exp(c) * wc.sum() + wf.sum())
        np.testing.assert_allclose(got[i], mix, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------- O0/O2 per-pair budgets, chunked selection
def test_budgets_per_pair_closed_form():
    # uniform weights give every pair the nominal budget
    assert oracle.budgets_per_pair(np.ones(8), 819, 8192).tolist() == [819] * 8
    # a = (1, 2, 3, 4)/10, |P| t = 400: floor(40, 80, 120, 160)
    assert oracle.budgets_per_pair([1, 2, 3, 4], 100, 1000).tolist() == [40, 80, 120, 160]
    # floor then clip to [1, T]: a = (0, 0.5, 9.5)/10 with |P| t = 30 -> floor(0, 1.5, 28.5) -> (1, 1, 28), T = 20 -> 20
    assert oracle.budgets_per_pair([0, 0.5, 9.5], 10, 20).tolist() == [1, 1, 20]
    g = rng(3)
    a = g.uniform(0, 1, 256)
    tb = oracle.budgets_per_pair(a, 3277, 32768)
    assert 256 * 3277 - 256 <= tb.sum() <= 256 * 3277          # floor loses < 1 per pair
    with pytest.raises(ValueError):
        oracle.budgets_per_pair([0, 0], 10, 20)


def test_chunk_budgets_values():
    # below the threshold, or chunking off: one chunk with the nominal budget
    assert oracle.chunk_budgets(819, 8192, 8192) == [(0, 8192, 819)]
    assert oracle.chunk_budgets(3277, 32768, 0) == [(0, 32768, 3277)]
    # 32768 = 4 x 8192; 3277 * 8192 / 32768 = 819.25 -> 819 each
    assert oracle.chunk_budgets(3277, 32768, 8192) == [(0, 8192, 819), (8192, 8192, 819), (16384, 8192, 819),
                                                       (24576, 8192, 819)]
    # 131072 = 16 x 8192; 1311 / 16 = 81.94 -> 82 each, 1312 realised
    cb = oracle.chunk_budgets(1311, 131072, 8192)
    assert len(cb) == 16 and all(c[2] == 82 for c in cb)
    # ragged last chunk: 12000 = 8192 + 3808; 100 * 8192 / 12000 = 68.27 -> 68, 100 * 3808 / 12000 = 31.73 -> 32
    assert oracle.chunk_budgets(100, 12000, 8192) == [(0, 8192, 68), (8192, 3808, 32)]
    # a single chunk covering everything keeps t; tiny t is clipped up to one per chunk
    assert oracle.chunk_budgets(500, 12000, 20000) == [(0, 12000, 500)]
    assert [c[2] for c in oracle.chunk_budgets(1, 40000, 8192)] == [1] * 5
    # chunks tile [0, T)
    for T, L in [(10001, 8192), (131072, 8192), (50000, 7000)]:
        cb = oracle.chunk_budgets(T // 10, T, L)
        assert cb[0][0] == 0 and sum(c[1] for c in cb) == T
        assert all(a[0] + a[1] == b[0] for a, b in zip(cb, cb[1:]))


@pytest.mark.parametrize("T,t,L,seed", [(12000, 1200, 8192, 0), (20001, 77, 5000, 1), (9000, 900, 4096, 2)])
def test_chunked_select_bruteforce(T, t, L, seed):
    g = rng(seed)
    s = np.round(g.standard_normal(T), 2)          # many duplicates: ties resolved by position
    got = oracle.select_topt_chunked(s, t, L)
    ref = []
    for start, Tc, tc in oracle.chunk_budgets(t, T, L):
        idx = sorted(range(start, start + Tc), key=lambda j: (-s[j], j))[:tc]
        ref += sorted(idx)
    assert got.tolist() == ref
    assert np.all(np.diff(got) > 0)
    if T <= oracle.CHUNK_THRESHOLD:
        assert got.tolist() == oracle.select_topt(s, t).tolist()


# ----------------------------------------------------------------- O1' value-aware indexer
def _dsa_case(seed, n_pos=3, G=2, T=7, d=5, dx=6, H=2, dI=3, dA=4, zero_value=False):
    g = rng(seed)
    ix = oracle.DSAIndexer(
        L_q=g.standard_normal((H * dI, d)), L_k=g.standard_normal((H * dI, d)), L_x=g.standard_normal((H, dx)),
        b_x=g.standard_normal(H), U_q=g.standard_normal((dA, d)) / math.sqrt(d),
        U_k=g.standard_normal((dA, d)) / math.sqrt(d), U_v=g.standard_normal((dA, d)) / math.sqrt(d),
        L_c=np.zeros((H * dI, dA)) if zero_value else g.standard_normal((H * dI, dA)),
        L_v=np.zeros((H * dI, d)) if zero_value else g.standard_normal((H * dI, d)))
    Q = g.standard_normal((G * n_pos, d))
    X = g.standard_normal((n_pos, dx))
    K = g.standard_normal((T, d))
    V = g.standard_normal((T, d))
    return Q, X, K, V, ix, n_pos


@pytest.mark.parametrize("seed", [0, 1])
def test_dsa_logits_bruteforce(seed):
    Q, X, K, V, ix, n_pos = _dsa_case(seed)
    got = oracle.dsa_logits(Q, X, K, V, ix, n_pos, 0.5)
    P = {k: getattr(ix, k).tolist() for k in ("L_q", "L_k", "L_x", "b_x", "U_q", "U_k", "U_v", "L_c", "L_v")}
    ref = np.array(brute.dsa_logits(Q.tolist(), X.tolist(), K.tolist(), V.tolist(), P, n_pos, 0.5, ix.H_I, ix.d_I))
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)


def test_dsa_zero_value_path_reproduces_query_key_logits():
    """With L_c = L_v = 0 (their initialisation) the logits are those of the
    query-key-only scorer (Appendix A.1): sum_a w_a LeakyReLU(N(L_q q)_a . N(L_k k)_a / sqrt(d_I)),
    whatever U_q, U_k, U_v are."""
    Q, X, K, V, ix, n_pos = _dsa_case(2, T=9, zero_value=True)
    got = oracle.dsa_logits(Q, X, K, V, ix, n_pos, 1.0)
    H, dI = ix.H_I, ix.d_I
    ref = np.zeros_like(got)
    for i, q in enumerate(Q):
        w = ix.L_x @ X[i % n_pos] + ix.b_x
        qb = (ix.L_q @ q).reshape(H, dI)
        qb /= np.sqrt((qb ** 2).mean(axis=1, keepdims=True) + 1e-6)
        for j, k in enumerate(K):
            kb = (ix.L_k @ k).reshape(H, dI)
            kb /= np.sqrt((kb ** 2).mean(axis=1, keepdims=True) + 1e-6)
            sc = (qb * kb).sum(axis=1) / math.sqrt(dI)
            ref[i, j] = float(w @ np.maximum(sc, 0.1 * sc))
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # and the value head's weights do not enter
    ix2 = dataclasses.replace(ix, U_q=ix.U_q * 3.0, U_v=-ix.U_v)
    np.testing.assert_allclose(oracle.dsa_logits(Q, X, K, V, ix2, n_pos, 1.0), got, rtol=1e-12, atol=1e-12)


def test_dsa_building_blocks():
    g = rng(4)
    Z = g.standard_normal((5, 12)) * 7.0
    N = oracle.rms_blocks(Z, 3, 4).reshape(5, 3, 4)
    ms = (Z.reshape(5, 3, 4) ** 2).mean(axis=2)
    np.testing.assert_allclose((N ** 2).mean(axis=2), ms / (ms + 1e-6), rtol=1e-12)   # unit RMS up to the guard
    assert np.all(np.sign(N) == np.sign(Z.reshape(5, 3, 4)))
    x = np.array([-2.0, -0.5, 0.0, 0.5, 3.0])
    np.testing.assert_array_equal(oracle.leaky_relu(x), [-0.2, -0.05, 0.0, 0.5, 3.0])
    # the value context is the full attention of the projected cache (row statistics' Y)
    Q, X, K, V, ix, n_pos = _dsa_case(5, T=11)
    qa, ka, va = Q @ ix.U_q.T, K @ ix.U_k.T, V @ ix.U_v.T
    _, _, Y = oracle.rowstats(qa, ka, va, 0.7)
    A = np.exp(0.7 * qa @ ka.T)
    np.testing.assert_allclose((A / A.sum(axis=1, keepdims=True)) @ va, Y, rtol=1e-12)


def test_pool_rms_properties():
    g = rng(6)
    I = g.standard_normal((6, 9))
    s = oracle.pool_rms(I)
    pi = np.exp(I) / np.exp(I).sum(axis=1, keepdims=True)
    np.testing.assert_allclose(s, np.sqrt((pi ** 2).mean(axis=0)), rtol=1e-12)
    # identical rows reduce to that row's softmax (the query-independent scorer's case)
    row = g.standard_normal(9)
    np.testing.assert_allclose(oracle.pool_rms(np.tile(row, (4, 1))), np.exp(row) / np.exp(row).sum(), rtol=1e-12)
    # a constant added to a row leaves the pooled scores unchanged
    I2 = I.copy()
    I2[2] += 5.0
    np.testing.assert_allclose(oracle.pool_rms(I2), s, rtol=1e-12)


# ------------------------------------------- chunked key sweeps and Phi_C
@pytest.mark.parametrize("chunk_elems", [7, 60, 1 << 25])
def test_global_logit_max_and_rowstats_across_key_chunks(monkeypatch, chunk_elems):
    """eq. response_profile's z_merge and Appendix A.9's row statistics are
    streamed over key chunks; with chunks of 1..3 keys (several boundaries,
    a ragged last chunk) they must equal the brute-force loops over the whole
    logit matrix."""
    K, V, Q, *_ = small_pair(seed=7, T=17, n=9, d=5)
    s = 0.37
    monkeypatch.setattr(oracle.core, "_CHUNK_ELEMS", chunk_elems)
    L = brute.logits(Q, K, s)
    assert oracle.global_logit_max(Q, K, s) == pytest.approx(max(max(row) for row in L), rel=0, abs=1e-12)
    z, m, Y = oracle.rowstats(Q, K, V, s)
    zb, mb, Yb = brute.rowstats(Q, K, V, s)
    np.testing.assert_allclose(z, zb, rtol=0, atol=1e-12)
    np.testing.assert_allclose(m, mb, rtol=1e-12, atol=0)
    np.testing.assert_allclose(Y, Yb, rtol=1e-10, atol=1e-12)


def test_phi_c_closed_forms():
    """Appendix A.9's Phi_C = exp(s Q C_k^T - z): with C_k = K its row sums are
    the mass targets m (the definition of m); its entries match an explicit
    exponential loop; and for compact keys inside the convex hull of the keys
    every entry lies in (0, 1], because q . c is a convex combination of the
    q . k_j and z_i is their maximum."""
    K, V, Q, *_ = small_pair(seed=8, T=14, n=11, d=6)
    s = 0.41
    z, m, _ = oracle.rowstats(Q, K, V, s)
    P = oracle.phi_c(Q, K, z, s)
    np.testing.assert_allclose(P.sum(axis=1), m, rtol=1e-12, atol=0)
    L = brute.logits(Q, K, s)
    for i in range(Q.shape[0]):
        for j in range(K.shape[0]):
            assert P[i, j] == pytest.approx(math.exp(L[i][j] - z[i]), rel=1e-12)
    g = rng(9)
    A = g.dirichlet(np.ones(K.shape[0]), size=5)   # 5 convex combinations of the keys
    Pc = oracle.phi_c(Q, A @ K, z, s)
    assert np.all(Pc > 0.0) and np.all(Pc <= 1.0 + 1e-12)
