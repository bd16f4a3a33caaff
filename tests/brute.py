"""Pure-Python loop versions of the paper's definitions, for tiny inputs.

These pin the float64 oracle: each function is written independently of
``oracle/`` (plain loops over Python floats, the ``math`` module only), so a
dropped term, wrong sign or transposed operand in either one shows up as a
mismatch.
"""
import math


def gelu(x):
    return 0.5 * x * (1.0 + math.erf(x / math.sqrt(2.0)))


def score(K, V, W1, b1, w2, b2):
    T, d = len(K), len(K[0])
    out = []
    for j in range(T):
        x = list(K[j]) + list(V[j])
        acc = float(b2)
        for a in range(len(W1)):
            pre = float(b1[a])
            for c in range(2 * d):
                pre += float(W1[a][c]) * float(x[c])
            acc += float(w2[a]) * gelu(pre)
        out.append(acc)
    return out


def pool_rms(I_rows):
    n, T = len(I_rows), len(I_rows[0])
    s = [0.0] * T
    for i in range(n):
        mx = max(I_rows[i])
        den = sum(math.exp(v - mx) for v in I_rows[i])
        for j in range(T):
            p = math.exp(I_rows[i][j] - mx) / den
            s[j] += p * p / n
    return [math.sqrt(v) for v in s]


def select(scores, t):
    def key(j):
        v = scores[j]
        if v != v:            # NaN: after every number
            return (1, 0.0, j)
        if v == 0.0:
            v = 0.0
        return (0, -v, j)
    order = sorted(range(len(scores)), key=key)
    return sorted(order[:t])


def dot(a, b):
    return sum(float(x) * float(y) for x, y in zip(a, b))


def logits(Q, K, scale):
    return [[scale * dot(q, k) for k in K] for q in Q]


def profiles(Q, K, scale):
    L = logits(Q, K, scale)
    n, T = len(Q), len(K)
    zm = max(max(row) for row in L)
    E = [[math.exp(L[i][j] - zm) for j in range(T)] for i in range(n)]
    U = []
    for j in range(T):
        col = [E[i][j] for i in range(n)]
        nrm = math.sqrt(sum(v * v for v in col))
        U.append([v / nrm if nrm > 0 else 0.0 for v in col])
    phi = [sum(E[i][j] for i in range(n)) / n for j in range(T)]
    return U, phi, zm


def assign(U, S):
    T = len(U)
    pos = {s: r for r, s in enumerate(S)}
    kappa = []
    for j in range(T):
        if j in pos:
            kappa.append(pos[j])
            continue
        best, br = -math.inf, -1
        for r, s in enumerate(S):
            v = dot(U[j], U[s])
            if v > best:
                best, br = v, r
        kappa.append(br)
    return kappa


def merge(K, phi, kappa, S, lam):
    d = len(K[0])
    out = []
    for r, s in enumerate(S):
        num = [0.0] * d
        den = 0.0
        for j in range(len(K)):
            if kappa[j] == r:
                den += phi[j]
                for c in range(d):
                    num[c] += phi[j] * float(K[j][c])
        mu = [v / den for v in num] if den > 0 else [float(v) for v in K[s]]
        out.append([(1 - lam) * float(K[s][c]) + lam * mu[c] for c in range(d)])
    return out


def rowstats(Q, K, V, scale):
    L = logits(Q, K, scale)
    z, m, Y = [], [], []
    for i in range(len(Q)):
        zi = max(L[i])
        w = [math.exp(v - zi) for v in L[i]]
        mi = sum(w)
        y = [sum(w[j] * float(V[j][c]) for j in range(len(K))) / mi for c in range(len(V[0]))]
        z.append(zi)
        m.append(mi)
        Y.append(y)
    return z, m, Y


def compact_attend(Q, C_k, beta, C_v, scale):
    out = []
    for q in Q:
        x = [scale * dot(q, c) + b for c, b in zip(C_k, beta)]
        mx = max(x)
        w = [math.exp(v - mx) for v in x]
        s = sum(w)
        out.append([sum(w[r] * C_v[r][c] for r in range(len(C_k))) / s for c in range(len(C_v[0]))])
    return out


def row_rel_err(O_test, O_ref):
    """Per-row relative Euclidean error, one row and one element at a time."""
    out = []
    for a, b in zip(O_test, O_ref):
        num = math.sqrt(sum((float(x) - float(y)) ** 2 for x, y in zip(a, b)))
        den = math.sqrt(sum(float(y) ** 2 for y in b))
        out.append(num / den)
    return out


def joint_attend(Q, C_k, beta, C_v, K_f, V_f, scale):
    """One softmax over the compact keys (logit + beta_r) followed by the
    uncompressed keys (logit + 0), by explicit loops."""
    keys = [(c, b, v) for c, b, v in zip(C_k, beta, C_v)] + [(k, 0.0, v) for k, v in zip(K_f, V_f)]
    out = []
    for q in Q:
        x = [scale * dot(q, k) + b for k, b, _ in keys]
        mx = max(x)
        w = [math.exp(v - mx) for v in x]
        s = sum(w)
        d = len(keys[0][2])
        out.append([sum(w[j] * float(keys[j][2][c]) for j in range(len(keys))) / s for c in range(d)])
    return out


def dsa_logits(Q, X, K, V, P, n_pos, scale_a, H, dI):
    """Value-aware indexer logits by explicit loops (P: dict of parameter lists)."""
    def mat(Mx, x):
        return [sum(float(Mx[o][c]) * float(x[c]) for c in range(len(x))) for o in range(len(Mx))]
    n, T = len(Q), len(K)
    qa = [mat(P["U_q"], q) for q in Q]
    ka = [mat(P["U_k"], k) for k in K]
    va = [mat(P["U_v"], v) for v in V]
    cs = []
    for i in range(n):
        lg = [scale_a * dot(qa[i], ka[j]) for j in range(T)]
        mx = max(lg)
        e = [math.exp(x - mx) for x in lg]
        z = sum(e)
        cs.append([sum(e[j] * va[j][c] for j in range(T)) / z for c in range(len(va[0]))])

    def rms(z):
        out = []
        for a in range(H):
            blk = z[a * dI:(a + 1) * dI]
            den = math.sqrt(sum(x * x for x in blk) / dI + 1e-6)
            out += [x / den for x in blk]
        return out
    qbar = [rms([u + w for u, w in zip(mat(P["L_q"], Q[i]), mat(P["L_c"], cs[i]))]) for i in range(n)]
    kbar = [rms([u + w for u, w in zip(mat(P["L_k"], K[j]), mat(P["L_v"], V[j]))]) for j in range(T)]
    out = []
    for i in range(n):
        x = X[i % n_pos]
        w = [sum(float(P["L_x"][a][c]) * float(x[c]) for c in range(len(x))) + float(P["b_x"][a]) for a in range(H)]
        row = []
        for j in range(T):
            tot = 0.0
            for a in range(H):
                sc = sum(qbar[i][a * dI + c] * kbar[j][a * dI + c] for c in range(dI)) / math.sqrt(dI)
                tot += w[a] * (sc if sc >= 0 else 0.1 * sc)
            row.append(tot)
        out.append(row)
    return out


def round_bf16(x):
    """Nearest-even bfloat16 value of float x (via its float32 bit pattern)."""
    import struct
    u = struct.unpack("<I", struct.pack("<f", x))[0]
    lower = u & 0xFFFF0000
    rem = u & 0xFFFF
    if rem > 0x8000 or (rem == 0x8000 and (u >> 16) & 1):
        lower += 0x10000
    return struct.unpack("<f", struct.pack("<I", lower & 0xFFFFFFFF))[0]


def assign_rounded(Q, K, S, scale, rnd):
    """eq. anchor_assignment with exp-profiles and anchor profiles rounded by rnd."""
    L = logits(Q, K, scale)
    n, T = len(Q), len(K)
    zm = max(max(row) for row in L)
    E = [[rnd(math.exp(L[i][j] - zm)) for j in range(T)] for i in range(n)]
    US = []
    for s in S:
        col = [E[i][s] for i in range(n)]
        nrm = math.sqrt(sum(v * v for v in col))
        US.append([rnd(v / nrm) for v in col])
    pos = {s: r for r, s in enumerate(S)}
    kappa = []
    for j in range(T):
        if j in pos:
            kappa.append(pos[j])
            continue
        col = [E[i][j] for i in range(n)]
        nrm = math.sqrt(sum(v * v for v in col))
        best, br = -math.inf, -1
        for r in range(len(S)):
            v = sum(col[i] / nrm * US[r][i] for i in range(n))
            if v > best:
                best, br = v, r
        kappa.append(br)
    return kappa
