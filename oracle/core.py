"""Float64 CPU oracle for ARC-KV per-context compaction.

TEST INFRASTRUCTURE ONLY.  This module is the slow, plainly written reference
against which the GPU library is checked.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import it; the product path
never routes through it.  It shares no code with the GPU library.

Everything here works on one layer-KV-head pair (the paper treats pairs
independently, Method section and Appendix A.2) in float64 numpy, written
step by step from the paper's equations:

  O0  budget                 Appendix A.2 (per-head budget, eq. per_head_budget),
                             A.3 (chunk budgets)
  O1  token scores           the scoring MLP on concat(k_j, v_j); pooling by
                             eq. (indexer_pooling), Section 3.3
  O2  top-t anchors          S = TopK(s, t), Section 3.3 / eq. (persistent_support)
  O3  response profiles      eq. (response_profile), Section 3.4
  O4  anchor assignment      eq. (anchor_assignment)
  O5  convex key merge       eq. (mass_centroid) and eq. (key_merge)
  O6  full-cache row stats   Appendix A.9: z^fit, Phi_K 1, Y
  O7  mass bias fit          eq. (mass_fit), Appendix A.9
  O8  compact value fit      eq. (value_lstsq), Appendix A.9
  O9  compact attention      eq. (compact_attention), Section 3.1
  O1' value-aware indexer    eq. (value_context), (indexer_projection),
                             (pairwise_index_score) of Appendix A.1, pooled
                             by eq. (indexer_pooling)
  O10 joint decode attention eq. (concatenated_attention_preservation),
                             Appendix A.7: compact block with bias beta,
                             then an uncompressed block with zero bias

Readings where the paper is silent (budget rounding, tie rules, ridge
defaults, guards) are documented on the functions that take them.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# Parameter defaults (readings of the paper where it gives no value).
LAMBDA_M = 0.25          # Section 4.1 uses 0.25 on QuALITY and RULER
DELTA_BETA = 1e-6        # relative ridge of the mass fit (paper: unregularised LS)
DELTA_V = 1e-3           # lambda_v = DELTA_V * tr(A) / t (paper: lambda_v >= 0, no value)
EPS_W = 1e-12            # epsilon_w of eq. (mass_fit)
B_MIN, B_MAX = -30.0, 30.0
MAX_ESCALATIONS = 6      # ridge x10 retries when a Cholesky pivot fails
DELTA_FLOOR = 1e-7       # an escalation from a zero ridge starts here

_CHUNK_ELEMS = 1 << 25   # float64 elements per key chunk (256 MiB) in O3/O4/O6


# --------------------------------------------------------------------------- O0
def budget(T: int, rho: float) -> int:
    """t = clip_[1,T](floor(rho*T + 1/2)).

    The paper rounds with a ceiling in training, a floor in the per-head
    budget and 'round' in chunked selection (Section 3.5, Appendix A.2, A.3).
    Round-half-up is the reading used here.
    """
    t = int(math.floor(float(rho) * float(T) + 0.5))
    return min(int(T), max(1, t))


def budgets_per_pair(a, t: int, T: int) -> np.ndarray:
    """eq. (per_head_budget): t_p = clip_[1,T](floor(a_p |P| t)) with the weights
    a normalised to sum to 1 over the |P| pairs (Section 3.5)."""
    a = np.asarray(a, np.float64)
    if a.ndim != 1 or a.size == 0 or not np.all(np.isfinite(a)) or np.any(a < 0) or a.sum() <= 0:
        raise ValueError("weights must be finite, non-negative and not all zero")
    a = a / a.sum()
    return np.clip(np.floor(a * a.size * t), 1, T).astype(np.int64)


CHUNK_THRESHOLD = 10000   # chunking applies when T > 10,000 (Appendix A.3)


def chunk_budgets(t: int, T: int, chunk_len: int):
    """Appendix A.3: with chunks of chunk_len positions (when chunk_len > 0 and
    T > 10,000), chunk c of length T_c keeps t_c = clip_[1,T_c](round(t T_c / T))
    anchors; otherwise one chunk keeps t.  Returns [(start, T_c, t_c)].
    Reading: round() is round-half-up, as for the budget (O0)."""
    if chunk_len <= 0 or T <= CHUNK_THRESHOLD:
        return [(0, T, t)]
    out = []
    for start in range(0, T, chunk_len):
        Tc = min(chunk_len, T - start)
        tc = int(math.floor(t * Tc / T + 0.5))
        out.append((start, Tc, min(Tc, max(1, tc))))
    return out


# --------------------------------------------------------------------------- O1
def gelu(x: np.ndarray) -> np.ndarray:
    """Exact (erf) GELU: x * (1 + erf(x / sqrt 2)) / 2."""
    from scipy.special import erf
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def score_mlp(K, V, W1, b1, w2, b2) -> np.ndarray:
    """One logit per cached token: I_j = w2 . GELU(W1 [k_j; v_j] + b1) + b2.

    The scoring network is a 2-layer MLP (2d -> 64 -> 1) applied to the
    concatenation of each token's key and value; it is query-independent.
    """
    X = np.concatenate([np.asarray(K, np.float64), np.asarray(V, np.float64)], axis=1)
    H = gelu(X @ np.asarray(W1, np.float64).T + np.asarray(b1, np.float64)[None, :])
    return H @ np.asarray(w2, np.float64) + float(np.asarray(b2).reshape(-1)[0])


def pool_rms(I_rows: np.ndarray) -> np.ndarray:
    """eq. (indexer_pooling): s_j = sqrt(mean_i softmax_j(I_i,:)^2).

    With a query-independent scorer every row is the same logit vector, so
    s = softmax(I), a strictly increasing map of I; ranking on s or on I
    gives the same anchors.  The GPU ranks on I to avoid ties manufactured by
    rounding the exponentials.
    """
    I_rows = np.atleast_2d(np.asarray(I_rows, np.float64))
    zmax = I_rows.max(axis=1, keepdims=True)
    e = np.exp(I_rows - zmax)
    pi = e / e.sum(axis=1, keepdims=True)
    return np.sqrt(np.mean(pi * pi, axis=0))


# --------------------------------------------------------------------------- O1' value-aware indexer
@dataclasses.dataclass
class DSAIndexer:
    """Per-pair parameters of the value-aware indexer (Appendix A.1,
    eq. indexer_parameters and value_indexer_parameters):
    L_q, L_k [H_I d_I][d]; L_x [H_I][d_x]; b_x [H_I]; U_q, U_k, U_v [d_A][d];
    L_c [H_I d_I][d_A]; L_v [H_I d_I][d]."""
    L_q: np.ndarray
    L_k: np.ndarray
    L_x: np.ndarray
    b_x: np.ndarray
    U_q: np.ndarray
    U_k: np.ndarray
    U_v: np.ndarray
    L_c: np.ndarray
    L_v: np.ndarray

    @property
    def H_I(self):
        return self.L_x.shape[0]

    @property
    def d_I(self):
        return self.L_q.shape[0] // self.L_x.shape[0]


RMS_EPS = 1e-6        # eq. indexer_projection: N(z) = z / sqrt(||z||^2 / d_I + 1e-6)
LEAKY_SLOPE = 0.1     # eq. pairwise_index_score: LeakyReLU_{0.1}


def rms_blocks(Z: np.ndarray, H: int, dI: int) -> np.ndarray:
    """Parameter-free RMS normalisation of each width-d_I block of the rows of Z."""
    Zb = np.asarray(Z, np.float64).reshape(Z.shape[0], H, dI)
    return (Zb / np.sqrt((Zb * Zb).sum(axis=2, keepdims=True) / dI + RMS_EPS)).reshape(Z.shape[0], H * dI)


def leaky_relu(x, slope: float = LEAKY_SLOPE):
    return np.where(x >= 0, x, slope * x)


def dsa_logits(Q, X, K, V, ix: DSAIndexer, n_pos: int, scale_a: float, rnd=None) -> np.ndarray:
    """Indexer logits I [n][T] for reference rows i = (g, r) ordered [query
    head][position] (r = i mod n_pos), whose activation x_r (rows of X) is
    shared by the query heads at position r.

      value context   c_i = softmax_j(s_A (U_q q_i).(U_k k_j)) (U_v v_j)      eq. value_context
      projections     qbar_i = N(L_q q_i + L_c c_i), kbar_j = N(L_k k_j + L_v v_j),
                      w_i = L_x x_r + b_x                                    eq. indexer_projection
      logits          I_ij = sum_a w_ia LeakyReLU(qbar_ia . kbar_ja / sqrt(d_I))  eq. pairwise_index_score

    s_A is the logit scale of the value-attention head (reading: 1/sqrt(d_A),
    as for every attention logit here).  ``rnd`` (e.g. round_to(., "bf16"))
    is applied where a low-precision implementation stores intermediates: the
    projected q, k, v of the value head, the context c, and qbar, kbar."""
    r = rnd if rnd is not None else (lambda a: a)
    Q, X, K, V = (np.asarray(a, np.float64) for a in (Q, X, K, V))
    H, dI = ix.H_I, ix.d_I
    qa = r(Q @ ix.U_q.T)
    ka = r(K @ ix.U_k.T)
    va = r(V @ ix.U_v.T)
    Lg = scale_a * (qa @ ka.T)
    Lg -= Lg.max(axis=1, keepdims=True)
    A = np.exp(Lg)
    c = r((A / A.sum(axis=1, keepdims=True)) @ va)
    qbar = r(rms_blocks(Q @ ix.L_q.T + c @ ix.L_c.T, H, dI))
    kbar = r(rms_blocks(K @ ix.L_k.T + V @ ix.L_v.T, H, dI))
    w = (X @ ix.L_x.T + ix.b_x)[np.arange(Q.shape[0]) % n_pos]          # [n][H]
    I = np.zeros((Q.shape[0], K.shape[0]))
    for a in range(H):
        blk = slice(a * dI, (a + 1) * dI)
        I += w[:, a:a + 1] * leaky_relu(qbar[:, blk] @ kbar[:, blk].T / math.sqrt(dI))
    return I


# --------------------------------------------------------------------------- O2
def select_topt(scores, t: int) -> np.ndarray:
    """S = TopK(s, t), returned in ascending position order.

    Total order: larger score first, ties to the lower index.  -0 counts as
    +0 and NaN ranks below every number (including -inf).
    """
    s = np.asarray(scores, np.float64).copy()
    T = s.shape[0]
    if not 1 <= t <= T:
        raise ValueError("t must lie in [1, T]")
    s[s == 0.0] = 0.0
    nan = np.isnan(s)
    # primary key: NaN last, then -score; secondary: index (lexsort: last key primary)
    order = np.lexsort((np.arange(T), np.where(nan, 0.0, -s), nan))
    return np.sort(order[:t]).astype(np.int64)


def select_topt_chunked(scores, t: int, chunk_len: int) -> np.ndarray:
    """Appendix A.3: the union of each chunk's local top-t_c (chunk_budgets),
    ascending; the global top-t when chunking does not apply."""
    s = np.asarray(scores, np.float64)
    parts = [start + select_topt(s[start:start + Tc], tc) for start, Tc, tc in chunk_budgets(t, s.shape[0], chunk_len)]
    return np.concatenate(parts).astype(np.int64)


# --------------------------------------------------------------------------- O3-O5
def logits(Q, K, scale: float) -> np.ndarray:
    """l_ij = scale * q_i . k_j (the paper writes the unscaled form)."""
    return scale * (np.asarray(Q, np.float64) @ np.asarray(K, np.float64).T)


def _key_chunks(T: int, n: int):
    step = max(1, _CHUNK_ELEMS // max(1, n))
    for j0 in range(0, T, step):
        yield j0, min(T, j0 + step)


def global_logit_max(Q, K, scale: float) -> float:
    """z_merge = max_{i,j} l_ij (eq. response_profile)."""
    z = -np.inf
    for j0, j1 in _key_chunks(K.shape[0], Q.shape[0]):
        z = max(z, float(logits(Q, K[j0:j1], scale).max()))
    return z


def response_profiles(Q, K, scale: float, z_merge=None):
    """eq. (response_profile): u_j = e_j / ||e_j||, e_ij = exp(l_ij - z_merge).

    Returns (E, U, z_merge) with E, U of shape [n, T].  A column whose norm
    underflows to zero gets u_j = 0 (reading: all its similarities then tie).
    """
    L = logits(Q, K, scale)
    if z_merge is None:
        z_merge = float(L.max())
    E = np.exp(L - z_merge)
    norms = np.linalg.norm(E, axis=0)
    U = np.divide(E, norms[None, :], out=np.zeros_like(E), where=norms[None, :] > 0)
    return E, U, z_merge


def assign(U: np.ndarray, S: np.ndarray) -> np.ndarray:
    """eq. (anchor_assignment): kappa(s_r) = r; otherwise argmax_r u_j . u_{s_r}.

    Ties go to the lowest r (the paper fixes a deterministic rule without
    naming it).
    """
    S = np.asarray(S)
    sim = U.T @ U[:, S]                      # [T, t]
    kappa = np.argmax(sim, axis=1)           # first maximum = lowest r
    kappa[S] = np.arange(S.shape[0])
    return kappa.astype(np.int64)


def mass_weights(E: np.ndarray) -> np.ndarray:
    """eq. (mass_centroid): phi_j = (1/n) sum_i exp(l_ij - z_merge)."""
    return E.mean(axis=0)


def round_to(x: np.ndarray, dtype) -> np.ndarray:
    """Round float64 values to bfloat16 ("bf16", nearest even) or float32 ("f32")."""
    x = np.asarray(x, np.float64)
    if dtype is None:
        return x
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        u = x.astype(np.float32).view(np.uint32).astype(np.uint64)
        lsb = (u >> np.uint64(16)) & np.uint64(1)
        r = ((u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
        return r.view(np.float32).astype(np.float64)
    raise ValueError(dtype)


def profiles_assign_phi(Q, K, S, scale: float, profile_dtype=None):
    """O3-O5 inputs for a whole pair, chunked over keys to bound memory.

    Each chunk holds whole key columns, so every column's profile,
    similarity row and mass weight is computed exactly as in the
    unchunked definition.  Returns (kappa, phi, z_merge).

    profile_dtype: None computes the argmax of eq. (anchor_assignment) in
    float64.  "bf16" / "f32" take that integer decision in the precision in
    which a compared implementation stores the profiles: exp(l - z_merge) and
    the normalised anchor profiles are rounded to that type before the
    similarities are formed (in float64).  phi is never rounded.
    """
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    S = np.asarray(S)
    z_merge = global_logit_max(Q, K, scale)
    if profile_dtype is None:
        _, US, _ = response_profiles(Q, K[S], scale, z_merge)       # [n, t]
    else:
        ES = round_to(np.exp(logits(Q, K[S], scale) - z_merge), profile_dtype)
        nrm = np.linalg.norm(ES, axis=0)
        US = round_to(np.divide(ES, nrm[None, :], out=np.zeros_like(ES), where=nrm[None, :] > 0), profile_dtype)
    T = K.shape[0]
    kappa = np.empty(T, np.int64)
    phi = np.empty(T, np.float64)
    for j0, j1 in _key_chunks(T, Q.shape[0]):
        E, U, _ = response_profiles(Q, K[j0:j1], scale, z_merge)
        if profile_dtype is not None:
            Er = round_to(E, profile_dtype)
            nr = np.linalg.norm(Er, axis=0)
            U = np.divide(Er, nr[None, :], out=np.zeros_like(Er), where=nr[None, :] > 0)
        kappa[j0:j1] = np.argmax(U.T @ US, axis=1)
        phi[j0:j1] = mass_weights(E)
    kappa[S] = np.arange(S.shape[0])
    return kappa, phi, z_merge


def merge_keys(K, phi, kappa, S, lambda_m: float) -> np.ndarray:
    """eq. (mass_centroid) + eq. (key_merge).

    mu_r = sum_{j in G_r} phi_j k_j / sum_{j in G_r} phi_j and
    c_r = (1 - lambda_m) k_{s_r} + lambda_m mu_r.  If a group's mass
    underflows to zero, mu_r = k_{s_r} (reading).
    """
    K = np.asarray(K, np.float64)
    S = np.asarray(S)
    t = S.shape[0]
    kappa = np.asarray(kappa)
    phi = np.asarray(phi, np.float64)
    num = np.zeros((t, K.shape[1]))
    den = np.zeros(t)
    np.add.at(num, kappa, phi[:, None] * K)
    np.add.at(den, kappa, phi)
    mu = K[S].copy()
    ok = den > 0
    mu[ok] = num[ok] / den[ok, None]
    return (1.0 - lambda_m) * K[S] + lambda_m * mu


# --------------------------------------------------------------------------- O6
def rowstats(Q, K, V, scale: float):
    """Appendix A.9: z_i = max_j l_ij, m = Phi_K 1, Y = softmax(l) V.

    z is the row maximum over the full cache (it weights each row of the
    mass fit, so it is not a free shift).  Chunked over keys; the row
    maximum is taken first so every chunk uses the final z.
    """
    Q = np.asarray(Q, np.float64)
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    n = Q.shape[0]
    z = np.full(n, -np.inf)
    for j0, j1 in _key_chunks(K.shape[0], n):
        z = np.maximum(z, logits(Q, K[j0:j1], scale).max(axis=1))
    m = np.zeros(n)
    num = np.zeros((n, V.shape[1]))
    for j0, j1 in _key_chunks(K.shape[0], n):
        PhiK = np.exp(logits(Q, K[j0:j1], scale) - z[:, None])
        m += PhiK.sum(axis=1)
        num += PhiK @ V[j0:j1]
    return z, m, num / m[:, None]


# --------------------------------------------------------------------------- O7-O8
class CholeskyFailure(np.linalg.LinAlgError):
    pass


def ridge_cholesky_solve(A: np.ndarray, B: np.ndarray, delta: float,
                         max_escalations: int = MAX_ESCALATIONS):
    """Solve (A + delta * tr(A)/t * I) X = B by Cholesky.

    If a pivot is not positive the relative ridge is multiplied by 10 (a
    zero ridge is raised to DELTA_FLOOR), at most ``max_escalations`` times
    (reading: the paper states no regulariser for the mass fit and a free
    lambda_v >= 0 for the values).  Returns (X, delta_used, attempts).
    """
    import scipy.linalg as sla
    t = A.shape[0]
    abar = np.trace(A) / t
    d = float(delta)
    for attempt in range(max_escalations + 1):
        M = A + (d * abar) * np.eye(t)
        try:
            c = sla.cho_factor(M, lower=True, check_finite=True)
        except np.linalg.LinAlgError:
            if attempt == max_escalations:
                raise CholeskyFailure(f"Cholesky failed at delta={d:g}")
            d = max(10.0 * d, DELTA_FLOOR)
            continue
        return sla.cho_solve(c, B), d, attempt + 1
    raise CholeskyFailure("unreachable")


def phi_c(Q, C_k, z, scale: float) -> np.ndarray:
    """Phi_C = exp(Q C_k^T - z 1^T) with the full-cache row maxima z."""
    return np.exp(logits(Q, C_k, scale) - np.asarray(z, np.float64)[:, None])


def nnls_gram(G: np.ndarray, h: np.ndarray, tol: float = 1e-12, max_iter: int = None) -> np.ndarray:
    """Lawson-Hanson active-set NNLS in normal-equation form.

    Minimises w^T G w / 2 - h^T w subject to w >= 0, which for G = A^T A and
    h = A^T b is min ||A w - b||^2, w >= 0 (Lawson & Hanson, Solving Least
    Squares Problems, 1974, ch. 23).  G must be positive definite.
    """
    t = G.shape[0]
    max_iter = max_iter or 3 * t + 10
    w = np.zeros(t)
    passive = np.zeros(t, dtype=bool)
    scale = max(1.0, float(np.abs(h).max()) if t else 1.0)
    for _ in range(max_iter):
        grad = h - G @ w                       # negative gradient
        cand = (~passive) & (grad > tol * scale)
        if not cand.any():
            break
        passive[np.argmax(np.where(cand, grad, -np.inf))] = True
        while True:
            idx = np.flatnonzero(passive)
            z = np.zeros(t)
            z[idx] = np.linalg.solve(G[np.ix_(idx, idx)], h[idx])
            if (z[idx] > 0).all():
                w = z
                break
            neg = idx[z[idx] <= 0]
            ratios = w[neg] / (w[neg] - z[neg])
            alpha = float(np.min(ratios))
            w = w + alpha * (z - w)
            w[neg[ratios <= alpha]] = 0.0     # the blocking coordinates leave
            passive &= w > 0.0
            w[~passive] = 0.0
    return w


@dataclasses.dataclass
class BiasFit:
    beta: np.ndarray
    w_tilde: np.ndarray
    w_star: np.ndarray
    delta_used: float
    G: np.ndarray
    h: np.ndarray
    PhiC: np.ndarray


def fit_bias(Q, C_k, z, m, scale: float, delta: float = DELTA_BETA, eps_w: float = EPS_W,
             b_min: float = B_MIN, b_max: float = B_MAX, mode: int = 0,
             max_escalations: int = MAX_ESCALATIONS) -> BiasFit:
    """eq. (mass_fit).

    mode 0 (the paper's): w~ = argmin ||Phi_C w - m||^2 through the normal
    equations G w = h with G = Phi_C^T Phi_C, h = Phi_C^T m and a relative
    ridge delta * tr(G)/t; then w* = max(w~, 0).
    mode 1: exact non-negative least squares on the same ridged system.
    beta = clip(log max(w*, eps_w), b_min, b_max).
    """
    PhiC = phi_c(Q, C_k, z, scale)
    G = PhiC.T @ PhiC
    h = PhiC.T @ np.asarray(m, np.float64)
    w_tilde, d_used, _ = ridge_cholesky_solve(G, h, delta, max_escalations)
    if mode == 0:
        w_star = np.maximum(w_tilde, 0.0)
    elif mode == 1:
        t = G.shape[0]
        w_star = nnls_gram(G + d_used * np.trace(G) / t * np.eye(t), h)
    else:
        raise ValueError("mode must be 0 or 1")
    beta = np.clip(np.log(np.maximum(w_star, eps_w)), b_min, b_max)
    return BiasFit(beta, w_tilde, w_star, d_used, G, h, PhiC)


def compact_probs(Q, C_k, beta, scale: float) -> np.ndarray:
    """P_hat = softmax(Q C_k^T + 1 beta^T), normalised with its own row max."""
    X = logits(Q, C_k, scale) + np.asarray(beta, np.float64)[None, :]
    X -= X.max(axis=1, keepdims=True)
    E = np.exp(X)
    return E / E.sum(axis=1, keepdims=True)


@dataclasses.dataclass
class ValueFit:
    C_v: np.ndarray
    delta_used: float
    A: np.ndarray
    B: np.ndarray
    P: np.ndarray


def fit_values(Q, C_k, beta, Y, scale: float, delta: float = DELTA_V,
               max_escalations: int = MAX_ESCALATIONS) -> ValueFit:
    """eq. (value_lstsq): C_v = argmin ||P_hat C - Y||_F^2 + lambda_v ||C||_F^2.

    Solved through (A + lambda_v I) C_v = P_hat^T Y with A = P_hat^T P_hat
    and lambda_v = delta * tr(A) / t.
    """
    P = compact_probs(Q, C_k, beta, scale)
    A = P.T @ P
    B = P.T @ np.asarray(Y, np.float64)
    C_v, d_used, _ = ridge_cholesky_solve(A, B, delta, max_escalations)
    return ValueFit(C_v, d_used, A, B, P)


# --------------------------------------------------------------------------- O9
def attend_compact(Q, C_k, beta, C_v, scale: float) -> np.ndarray:
    """eq. (compact_attention): softmax(Q C_k^T + 1 beta^T) C_v."""
    return compact_probs(Q, C_k, beta, scale) @ np.asarray(C_v, np.float64)


def attend_full(Q, K, V, scale: float) -> np.ndarray:
    """eq. (full_attention): softmax(Q K^T) V."""
    return rowstats(Q, K, V, scale)[2]


def attend_joint(Q, C_k, beta, C_v, K_f, V_f, scale: float) -> np.ndarray:
    """eq. (concatenated_attention_preservation), right-hand side: one softmax
    over the concatenated logits [s Q C_k^T + 1 beta^T, s Q K_f^T] (zero bias on
    the uncompressed rows) applied to [C_v; V_f].  Either block may be empty
    (t = 0 or F = 0 rows); beta = None means zero bias."""
    Q = np.asarray(Q, np.float64)
    d = Q.shape[1]
    C_k = np.zeros((0, d)) if C_k is None else np.asarray(C_k, np.float64)
    C_v = np.zeros((0, d)) if C_v is None else np.asarray(C_v, np.float64)
    K_f = np.zeros((0, d)) if K_f is None else np.asarray(K_f, np.float64)
    V_f = np.zeros((0, d)) if V_f is None else np.asarray(V_f, np.float64)
    b = np.zeros(C_k.shape[0]) if beta is None else np.asarray(beta, np.float64)
    X = np.concatenate([scale * (Q @ C_k.T) + b[None, :], scale * (Q @ K_f.T)], axis=1)
    X -= X.max(axis=1, keepdims=True)
    E = np.exp(X)
    return (E / E.sum(axis=1, keepdims=True)) @ np.concatenate([C_v, V_f], axis=0)


def row_rel_err(O_test, O_ref) -> np.ndarray:
    """Per-row ||o_test - o_ref|| / ||o_ref|| (the per-row form of eq. output_loss)."""
    O_test = np.asarray(O_test, np.float64)
    O_ref = np.asarray(O_ref, np.float64)
    return np.linalg.norm(O_test - O_ref, axis=1) / np.linalg.norm(O_ref, axis=1)


# --------------------------------------------------------------------------- whole pair
@dataclasses.dataclass
class PairResult:
    t: int
    scores: np.ndarray
    anchors: np.ndarray
    kappa: np.ndarray
    phi: np.ndarray
    z_merge: float
    C_k: np.ndarray
    z: np.ndarray
    m: np.ndarray
    Y: np.ndarray
    beta: np.ndarray
    w_tilde: np.ndarray
    delta_beta_used: float
    C_v: np.ndarray
    delta_v_used: float


def compact_pair(K, V, Q, W1, b1, w2, b2, rho: float = None, t: int = None, scale: float = None,
                 lambda_m: float = LAMBDA_M, delta_beta: float = DELTA_BETA,
                 delta_v: float = DELTA_V, eps_w: float = EPS_W, b_min: float = B_MIN,
                 b_max: float = B_MAX, bias_mode: int = 0, scores=None,
                 anchors=None, kappa=None, profile_dtype=None) -> PairResult:
    """The four stages in order: score, select, merge, fit (Section 3.2).

    ``scores`` / ``anchors`` / ``kappa`` may be supplied to run the later
    stages on given upstream values (stage-wise checking); ``profile_dtype``
    is passed to the assignment (see profiles_assign_phi).
    """
    K = np.asarray(K, np.float64)
    V = np.asarray(V, np.float64)
    Q = np.asarray(Q, np.float64)
    T, d = K.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if t is None:
        t = budget(T, rho)
    if scores is None:
        scores = score_mlp(K, V, W1, b1, w2, b2)
    if anchors is None:
        anchors = select_topt(scores, t)
    anchors = np.asarray(anchors, np.int64)
    kap, phi, z_merge = profiles_assign_phi(Q, K, anchors, scale, profile_dtype)
    if kappa is None:
        kappa = kap
    kappa = np.asarray(kappa, np.int64)
    C_k = merge_keys(K, phi, kappa, anchors, lambda_m)
    z, m, Y = rowstats(Q, K, V, scale)
    bf = fit_bias(Q, C_k, z, m, scale, delta_beta, eps_w, b_min, b_max, bias_mode)
    vf = fit_values(Q, C_k, bf.beta, Y, scale, delta_v)
    return PairResult(t, np.asarray(scores, np.float64), anchors, kappa, phi, z_merge, C_k,
                      z, m, Y, bf.beta, bf.w_tilde, bf.delta_used, vf.C_v, vf.delta_used)
