"""GPU parity of the exact non-negative mass fit (bias_mode 1).

The oracle solves the same ridged problem, min ||Phi_C w - m||^2 + lam ||w||^2
over w >= 0, with Lawson-Hanson active sets; the GPU with block principal
pivoting.  The ridged Gram is positive definite, so the minimiser is unique and
both must reach it.  Checked, in float64 on the oracle's Phi_C:

  * the objective of the GPU's w against the oracle's (relative gap),
  * the KKT conditions of the GPU's w (gradient ~0 on its support, >= 0 off it),
    which certify optimality by themselves at sizes the oracle's NNLS cannot
    reach,
  * that the exact fit never does worse than the projected fit (bias_mode 0).

Tolerances: as the projected fit's (1e-4 relative for fp32 inputs, 5e-3 for
bf16, whose compact keys enter as hi/lo bf16 pairs); KKT residuals relative to
max |h|.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import TOL_OUT, certify_flips, gpu_assignment, log_assign_stats, make_inputs, np64, scale_of

pytestmark = pytest.mark.gpu

CASES = [
    synth.WORKLOADS["tiny_f32_T1024"],
    synth.custom("bf16_T2600_n520", kv_heads=3, T=2600, q_heads_per_kv=4, n_pos=130, rho=0.12, dtype="bf16",
                 rope=True),
    synth.custom("f32_T777_n200", kv_heads=2, T=777, q_heads_per_kv=2, n_pos=100, rho=0.2, dtype="f32",
                 rope=True),
]
IDS = [c.name for c in CASES]
OBJ_TOL = {"f32": 1e-4, "bf16": 5e-3}
KKT_TOL = {"f32": 1e-4, "bf16": 2e-3}


def A():
    from paper_2609_36835_amd import arckv
    return arckv


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_weights(beta, eps_w):
    """w from beta = log max(w, eps_w); entries at the floor are the bound ones."""
    w = np.exp(np.asarray(beta, np.float64))
    w[beta <= np.log(eps_w) + 1e-4] = 0.0
    return w


def mass_problem(Q, Ck, z, m, s, delta_used):
    PhiC = oracle.phi_c(Q, Ck, z, s)
    G = PhiC.T @ PhiC
    h = PhiC.T @ m
    lam = float(delta_used) * np.trace(G) / G.shape[0]
    return PhiC, G, h, lam


def objective(PhiC, m, lam, w):
    r = PhiC @ w - m
    return float(r @ r + lam * (w @ w))


def kkt(G, h, lam, w):
    """Largest violation of the optimality conditions, relative to max |h|."""
    g = G @ w + lam * w - h
    sc = np.abs(h).max()
    free = w > 0
    on = np.abs(g[free]).max() / sc if free.any() else 0.0
    off = max(0.0, -g[~free].min()) / sc if (~free).any() else 0.0
    return on, off, int(free.sum())


@pytest.fixture(scope="module", params=CASES, ids=IDS)
def case(request):
    wl = request.param
    log(f"[case] {wl.name}: B={wl.pairs} T={wl.T} n={wl.n} rho={wl.rho} dtype={wl.dtype}")
    dev, host = make_inputs(wl)
    s = scale_of(wl)
    t = oracle.budget(wl.T, wl.rho)
    ref = [oracle.compact_pair(host["K"][b], host["V"][b], host["Q"][b], host["W1"][b], host["b1"][b],
                               host["w2"][b], host["b2"][b], t=t, scale=s)
           for b in range(wl.pairs)]
    return wl, dev, host, s, t, ref


def test_nnls_fit_matches_oracle(case):
    wl, dev, host, s, t, ref = case
    Ck = np.stack([r.C_k for r in ref]).astype(np.float32)
    z = np.stack([r.z for r in ref]).astype(np.float32)
    m = np.stack([r.m for r in ref]).astype(np.float32)
    args = (dev["Q"], torch.from_numpy(Ck).cuda(), torch.from_numpy(z).cuda(), torch.from_numpy(m).cuda())
    p1 = A().default_params(bias_mode=1)
    beta1, info1, dused1 = A().fit_bias(*args, params=p1, scale=s, T=wl.T)
    beta0, info0, _ = A().fit_bias(*args, scale=s, T=wl.T)
    beta1, beta0 = np64(beta1), np64(beta0)
    info1, info0, dused1 = info1.cpu().numpy(), info0.cpu().numpy(), dused1.cpu().numpy()
    assert np.all(info1 == 0) and np.all(info0 == 0), (info1, info0)
    n_bound_total = 0
    for b in range(wl.pairs):
        Q = host["Q"][b]
        zz, mm, ck = z[b].astype(np.float64), m[b].astype(np.float64), Ck[b].astype(np.float64)
        bf = oracle.fit_bias(Q, ck, zz, mm, s, mode=1)
        assert dused1[b] == pytest.approx(bf.delta_used, rel=1e-6)
        PhiC, G, h, lam = mass_problem(Q, ck, zz, mm, s, bf.delta_used)
        w1 = gpu_weights(beta1[b], p1.eps_w)
        w0 = gpu_weights(beta0[b], p1.eps_w)
        f_gpu, f_ref = objective(PhiC, mm, lam, w1), objective(PhiC, mm, lam, bf.w_star)
        f_proj = objective(PhiC, mm, lam, w0)
        on, off, n_free = kkt(G, h, lam, w1)
        n_bound_total += t - n_free
        ref_free = int((bf.w_star > 0).sum())
        log(f"  pair {b}: objective gpu {f_gpu:.8e} oracle {f_ref:.8e} projected {f_proj:.8e}; "
            f"KKT on {on:.2e} off {off:.2e}; free {n_free}/{t} (oracle {ref_free})")
        assert f_gpu >= f_ref * (1 - 1e-9) - 1e-300   # the oracle's w is the minimiser
        assert f_gpu - f_ref <= OBJ_TOL[wl.dtype] * f_ref, (b, f_gpu, f_ref)
        assert on <= KKT_TOL[wl.dtype] and off <= KKT_TOL[wl.dtype], (b, on, off)
        assert f_gpu <= f_proj * (1 + OBJ_TOL[wl.dtype]), (b, f_gpu, f_proj)
        big = bf.w_star > 1e-2 * bf.w_star.max()
        rel = np.abs(w1[big] - bf.w_star[big]) / bf.w_star[big]
        log(f"    large weights: {int(big.sum())}, rel err median {np.median(rel):.2e} max {rel.max():.2e}")
    assert n_bound_total > 0, "the constraints never bind: the case does not exercise the pivoting"


def test_nnls_iteration_cap_reports_unsettled_pairs(case):
    """With one pivoting iteration (F = all keys with h > 0, one solve) a pair
    whose unconstrained solution has negative entries cannot settle: info = -2
    and beta NaN; pairs that do settle match the uncapped fit."""
    wl, dev, host, s, t, ref = case
    Ck = np.stack([r.C_k for r in ref]).astype(np.float32)
    z = np.stack([r.z for r in ref]).astype(np.float32)
    m = np.stack([r.m for r in ref]).astype(np.float32)
    args = (dev["Q"], torch.from_numpy(Ck).cuda(), torch.from_numpy(z).cuda(), torch.from_numpy(m).cuda())
    beta_c, info_c, _ = A().fit_bias(*args, params=A().default_params(bias_mode=1, nnls_max_iter=1), scale=s, T=wl.T)
    beta_f, info_f, _ = A().fit_bias(*args, params=A().default_params(bias_mode=1), scale=s, T=wl.T)
    beta_c, beta_f, info_c = np64(beta_c), np64(beta_f), info_c.cpu().numpy()
    for b in range(wl.pairs):
        bf0 = oracle.fit_bias(host["Q"][b], Ck[b].astype(np.float64), z[b].astype(np.float64),
                              m[b].astype(np.float64), s, mode=0)
        # clearly negative entries of the unconstrained solution cannot be feasible
        negative = bool((bf0.w_tilde < -1e-3 * np.abs(bf0.w_tilde).max()).any())
        log(f"  pair {b}: capped info {info_c[b]}, unconstrained LS clearly negative: {negative}")
        if info_c[b] == -2:
            assert np.all(np.isnan(beta_c[b]))
        else:
            assert info_c[b] == 0 and not negative
            np.testing.assert_allclose(beta_c[b], beta_f[b], rtol=0, atol=1e-5)
    assert np.any(info_c == -2), "every pair settled in one iteration"


def test_compact_with_nnls_end_to_end(case):
    wl, dev, host, s, t, ref = case
    params = A().default_params(bias_mode=1)
    anchors_d, Ck, beta, Cv, info = A().compact(dev["K"], dev["V"], dev["Q"], dev["W1"], dev["b1"], dev["w2"],
                                                dev["b2"], wl.rho, scale=s, params=params)
    anchors, Ck, beta, Cv, info = anchors_d.cpu().numpy(), np64(Ck), np64(beta), np64(Cv), info.cpu().numpy()
    assert np.all(info == 0), info
    for b in range(wl.pairs):
        Q, K = host["Q"][b], host["K"][b]
        S = anchors[b].astype(np.int64)
        kap_gpu, st = gpu_assignment(dev["K"][b:b + 1].contiguous(), dev["V"][b:b + 1].contiguous(),
                                     dev["Q"][b:b + 1].contiguous(), anchors_d[b:b + 1].contiguous(), s)
        log_assign_stats(st, wl.T, t, log=log)
        rr = oracle.compact_pair(K, host["V"][b], Q, host["W1"][b], host["b1"][b], host["w2"][b], host["b2"][b],
                                 t=t, scale=s, anchors=S, bias_mode=1)
        if certify_flips(kap_gpu, rr.kappa, Q, K, S, s, log=log):
            rr = oracle.compact_pair(K, host["V"][b], Q, host["W1"][b], host["b1"][b], host["w2"][b], host["b2"][b],
                                     t=t, scale=s, anchors=S, kappa=kap_gpu, bias_mode=1)
        err = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s),
                                 oracle.attend_compact(Q, rr.C_k, rr.beta, rr.C_v, s))
        O = oracle.attend_full(Q, K, host["V"][b], s)
        e_gpu = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s), O).mean()
        e_ref = oracle.row_rel_err(oracle.attend_compact(Q, rr.C_k, rr.beta, rr.C_v, s), O).mean()
        log(f"  pair {b}: O(Q_ref) max row rel err vs oracle {err.max():.3e}; error vs full attention "
            f"gpu {e_gpu:.4f} oracle {e_ref:.4f}")
        assert err.max() <= TOL_OUT[wl.dtype], (b, err.max())


def test_nnls_kkt_at_full_shape():
    """Eight pairs of the 32K-context workload (T = 32768, n = 4096, 10% kept):
    row statistics, then the exact fit on the anchors' keys; the KKT conditions
    of two sampled pairs' solutions are checked in float64."""
    wl = synth.WORKLOADS["llama8b_bf16_T32768"]
    idx = list(range(8))
    log(f"[case] {wl.name} pairs {idx}: T={wl.T} n={wl.n} rho={wl.rho}")
    arr = synth.workload_arrays(wl, pairs=idx, threads=16)
    td = torch.bfloat16
    K = torch.from_numpy(arr["K"]).cuda().to(td)
    V = torch.from_numpy(arr["V"]).cuda().to(td)
    Q = torch.from_numpy(arr["Q"]).cuda().to(td)
    s = 1.0 / np.sqrt(wl.d)
    t = oracle.budget(wl.T, wl.rho)
    sc = A().score(K, V, torch.from_numpy(arr["W1"]).cuda().to(td), torch.from_numpy(arr["b1"]).cuda(),
                   torch.from_numpy(arr["w2"]).cuda(), torch.from_numpy(arr["b2"][:, 0]).cuda())
    anchors = A().select(sc, t)
    z, m, Y = A().rowstats(K, V, Q, scale=s)
    Ck, _, _ = A().merge(K, Q, z, anchors, scale=s)
    p1 = A().default_params(bias_mode=1)
    beta, info, dused = A().fit_bias(Q, Ck, z, m, params=p1, scale=s, T=wl.T)
    torch.cuda.synchronize()
    info = info.cpu().numpy()
    assert np.all(info == 0), info
    beta, dused = np64(beta), dused.cpu().numpy()
    Qh, Ckh, zh, mh = np64(Q.float()), np64(Ck), np64(z), np64(m)
    for b in (0, 5):
        PhiC, G, h, lam = mass_problem(Qh[b], Ckh[b], zh[b], mh[b], s, dused[b])
        w = gpu_weights(beta[b], p1.eps_w)
        on, off, n_free = kkt(G, h, lam, w)
        log(f"  pair {b}: t={t}, free {n_free}, KKT on {on:.2e} off {off:.2e}")
        assert 0 < n_free < t
        assert on <= KKT_TOL["bf16"] and off <= KKT_TOL["bf16"], (b, on, off)


def test_nnls_chunk_invariant(case):
    """The exact fit in pair chunks of one (each chunk sizes its own compressed
    system) gives the same compaction as all pairs together."""
    wl, dev, host, s, t, ref = case
    if wl.pairs < 2:
        pytest.skip("needs two pairs")
    args = (dev["K"], dev["V"], dev["Q"], dev["W1"], dev["b1"], dev["w2"], dev["b2"], wl.rho)
    out_all = A().compact(*args, scale=s, params=A().default_params(bias_mode=1))
    out_one = A().compact(*args, scale=s, params=A().default_params(bias_mode=1, pair_chunk=1))
    names = ("anchors", "C_k", "beta", "C_v", "info")
    for name, a, b in zip(names, out_all, out_one):
        a, b = a.cpu().numpy(), b.cpu().numpy()
        if name in ("anchors", "info"):
            np.testing.assert_array_equal(a, b, err_msg=name)
        else:
            np.testing.assert_allclose(a, b, rtol=0, atol=1e-6 * max(1.0, float(np.abs(a).max())), err_msg=name)
    log(f"  {wl.name}: chunked and unchunked exact fits agree")
