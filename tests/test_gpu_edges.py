"""GPU edge cases: full retention, a single anchor, tiny and ragged caches against
the oracle, lambda_m = 0, Cholesky failure and ridge escalation (also at the
32K-context shape), non-finite inputs, recomputed row statistics, the exact
fit where it cannot bind, and keys tied with many anchors."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import TOL_OUT, certify_flips, gpu_assignment, make_inputs, np64

pytestmark = pytest.mark.gpu


def A():
    from paper_2609_36835_amd import arckv
    return arckv


def run(wl, rho, **params):
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    out = A().compact(dev["K"], dev["V"], dev["Q"], dev["W1"], dev["b1"], dev["w2"], dev["b2"], rho, scale=s,
                      params=A().default_params(**params))
    return dev, host, s, [o.cpu() for o in out]


def test_full_retention_reproduces_attention_fp32():
    wl = synth.custom("full", kv_heads=2, T=48, q_heads_per_kv=2, n_pos=64, dtype="f32", rope=True)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, 1.0, delta_beta=0.0, delta_v=0.0)
    assert np.all(info.numpy() == 0)
    for b in range(wl.pairs):
        K, V, Q = host["K"][b], host["V"][b], host["Q"][b]
        assert anchors[b].tolist() == list(range(wl.T))
        assert np.array_equal(Ck[b].numpy().astype(np.float64), K)      # singleton groups keep the key exactly
        Qh = synth.heldout_queries(wl, 0, b).astype(np.float64)
        O = oracle.attend_full(Qh, K, V, s)
        Oc = oracle.attend_compact(Qh, np64(Ck[b]), np64(beta[b]), np64(Cv[b]), s)
        err = oracle.row_rel_err(Oc, O).max()
        print(f"  pair {b}: full retention, held-out max row rel err {err:.2e}", flush=True)
        assert err <= TOL_OUT["f32"], err


def test_single_anchor_closed_form():
    wl = synth.custom("t1", kv_heads=1, T=300, q_heads_per_kv=1, n_pos=64, dtype="f32", rope=False)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, 0.001)
    assert anchors.shape[1] == 1 and np.all(info.numpy() == 0)
    K, V, Q = host["K"][0], host["V"][0], host["Q"][0]
    r = oracle.compact_pair(K, V, Q, host["W1"][0], host["b1"][0], host["w2"][0], host["b2"][0], t=1, scale=s)
    assert anchors[0].tolist() == r.anchors.tolist()
    np.testing.assert_allclose(np64(Ck[0]), r.C_k, rtol=0, atol=1e-5 * np.abs(K).max())
    z, m, _ = oracle.rowstats(Q, K, V, s)
    phi = np.exp(s * Q @ np64(Ck[0])[0] - z)
    w = phi @ m / (phi @ phi)
    assert np64(beta[0])[0] == pytest.approx(math.log(w), abs=1e-3)


@pytest.mark.parametrize("T,n_pos,rho", [(7, 3, 0.5), (64, 64, 0.25), (257, 33, 0.1), (513, 1, 0.9)])
def test_tiny_and_ragged_shapes(T, n_pos, rho):
    """Tiny and ragged caches (several with t > n, where the fits are
    rank-deficient and the ridge decides) against the float64 oracle's own
    compaction: assignment and the compact-attention output on Q_ref."""
    wl = synth.custom(f"s{T}", kv_heads=2, T=T, q_heads_per_kv=1, n_pos=n_pos, dtype="bf16", rope=True)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, rho)
    t = oracle.budget(T, rho)
    assert anchors.shape == (2, t)
    for b in range(2):
        K, V, Q = host["K"][b], host["V"][b], host["Q"][b]
        a = anchors[b].numpy()
        assert np.all(np.diff(a) > 0) and a.min() >= 0 and a.max() < T
        # the oracle on the GPU's anchors (score near-ties at the selection
        # boundary are the selection tests' subject, not this one's)
        r = oracle.compact_pair(K, V, Q, host["W1"][b], host["b1"][b], host["w2"][b], host["b2"][b], t=t,
                                scale=s, anchors=a)
        kap, st = gpu_assignment(dev["K"][b:b + 1].contiguous(), dev["V"][b:b + 1].contiguous(),
                                 dev["Q"][b:b + 1].contiguous(), torch.from_numpy(a[None].astype(np.int32)).cuda(), s)
        certify_flips(kap, r.kappa, Q, K, r.anchors, s)
        assert st[3] == 0, st
        assert np.all(info[b].numpy() == 0), info[b]
        err = oracle.row_rel_err(oracle.attend_compact(Q, np64(Ck[b]), np64(beta[b]), np64(Cv[b]), s),
                                 oracle.attend_compact(Q, r.C_k, r.beta, r.C_v, s)).max()
        print(f"  T={T} n={wl.n} t={t} pair {b}: O(Q_ref) max row rel err {err:.2e}", flush=True)
        assert err <= TOL_OUT["bf16"], (b, err)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_lambda_zero_keeps_anchor_keys(dtype):
    """lambda_m = 0 in eq. key_merge: each compact key is its anchor's key, bit for bit."""
    wl = synth.custom(f"lam0{dtype}", kv_heads=2, T=700, q_heads_per_kv=2, n_pos=64, rho=0.1, dtype=dtype, rope=True)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, wl.rho, lambda_m=0.0)
    for b in range(wl.pairs):
        assert np.array_equal(np64(Ck[b]), host["K"][b][anchors[b].numpy()]), b


def _pair_refs(wl, host, s):
    t = oracle.budget(wl.T, wl.rho)
    return [oracle.compact_pair(host["K"][b], host["V"][b], host["Q"][b], host["W1"][b], host["b1"][b],
                                host["w2"][b], host["b2"][b], t=t, scale=s) for b in range(wl.pairs)]


def _f32(x):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, np.float32))).cuda()


def test_cholesky_failure_reports_info_and_nan():
    """Grams that are singular at any ridge relative to their trace, made exactly
    so in float32 and float64 alike:
    mass fit: z raised by 1e4 for pair 0 makes every Phi_C entry underflow to
    0, so G = 0 and the first pivot is 0 (info = 1) whatever the escalation;
    value fit: beta_1 = -1e4 for pair 0 zeroes column 1 of P_hat, so with
    lambda_v = 0 and no escalation the second pivot is exactly 0 (info = 2).
    The failing pair's outputs are NaN; the other pair is unaffected, bit for bit."""
    wl = synth.custom("fail", kv_heads=2, T=600, q_heads_per_kv=2, n_pos=64, rho=0.1, dtype="f32", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    refs = _pair_refs(wl, host, s)
    Ck = _f32(np.stack([r.C_k for r in refs]))
    z, m, Y = (_f32(np.stack([getattr(r, k) for r in refs])) for k in ("z", "m", "Y"))
    beta_ok = _f32(np.stack([r.beta for r in refs]))

    p = A().default_params(delta_beta=0.0, max_escalations=3)
    b_ok, i_ok, _ = A().fit_bias(dev["Q"], Ck, z, m, params=p, scale=s, T=wl.T)
    z_bad = z.clone()
    z_bad[0] += 1e4
    beta, info, _ = A().fit_bias(dev["Q"], Ck, z_bad, m, params=p, scale=s, T=wl.T)
    info = info.cpu().numpy()
    assert info[0] == 1 and torch.isnan(beta[0]).all(), info
    assert info[1] == i_ok[1].item() == 0 and torch.equal(beta[1], b_ok[1])
    with pytest.raises(oracle.CholeskyFailure):
        oracle.fit_bias(host["Q"][0], refs[0].C_k, refs[0].z + 1e4, refs[0].m, s, delta=0.0, max_escalations=3)

    p = A().default_params(delta_v=0.0, max_escalations=0)
    c_ok, j_ok, _ = A().fit_values(dev["Q"], Ck, beta_ok, Y, params=p, scale=s, T=wl.T)
    beta_bad = beta_ok.clone()
    beta_bad[0, 1] = -1e4
    Cv, info, _ = A().fit_values(dev["Q"], Ck, beta_bad, Y, params=p, scale=s, T=wl.T)
    info = info.cpu().numpy()
    assert info[0] == 2 and torch.isnan(Cv[0]).all(), info
    assert info[1] == j_ok[1].item() == 0 and torch.equal(Cv[1], c_ok[1])
    bb = refs[0].beta.copy()
    bb[1] = -1e4
    with pytest.raises(oracle.CholeskyFailure):
        oracle.fit_values(host["Q"][0], refs[0].C_k, bb, refs[0].Y, s, delta=0.0, max_escalations=0)


@pytest.mark.parametrize("name,T,n_pos,rho", [("esc0", 600, 32, 0.2), ("llama8b_bf16_T32768", 32768, 1024, 0.1)])
def test_escalation_from_zero_ridge(name, T, n_pos, rho):
    """lambda_v = 0 with column 1 of P_hat zeroed (beta_1 = -1e4): the first
    factorisation fails exactly, the ridge is raised to the 1e-7 floor (x10 per
    further retry) and only the failing pairs are refactored.  The values must
    agree with the float64 fit at the ridge the library reports (compact-attention
    output on Q_ref; ridge ~1e-7 of the mean diagonal, so the bar is 1e-3).
    The second case is the 32K-context shape (t = 3277, n = 4096).  At the small
    shape t > n, so the mass-fit Gram is singular too: with delta_beta = 0 it must
    also escalate and end finite."""
    if name in synth.WORKLOADS:
        wl = synth.WORKLOADS[name]
        arr = synth.workload_arrays(wl, pairs=[0, 5], threads=16)
        dev = {k: torch.from_numpy(arr[k]).to("cuda", torch.bfloat16).contiguous() for k in ("K", "V", "Q")}
        host = {k: arr[k].astype(np.float64) for k in ("K", "V", "Q")}
    else:
        wl = synth.custom(name, kv_heads=2, T=T, q_heads_per_kv=2, n_pos=n_pos, rho=rho, dtype="bf16", rope=True)
        dev, host = make_inputs(wl)
    B = dev["K"].shape[0]
    s = 1.0 / math.sqrt(128)
    t = oracle.budget(T, rho)
    z, m, Y = A().rowstats(dev["K"], dev["V"], dev["Q"], scale=s)
    S = np.linspace(0, T - 1, t).astype(np.int64)          # compact keys: evenly spaced cache keys
    Ck = np.stack([host["K"][b][S] for b in range(B)])
    beta = np.zeros((B, t))
    beta[:, 1] = -1e4
    p = A().default_params(delta_v=0.0, max_escalations=3)
    Cv, info, dused = A().fit_values(dev["Q"], _f32(Ck), _f32(beta), Y, params=p, scale=s, T=T)
    Cv, info, dused = np64(Cv), info.cpu().numpy(), dused.cpu().numpy()
    assert np.all(info == 0), info
    assert np.all(dused >= np.float32(oracle.DELTA_FLOOR)), dused
    Yh = np64(Y)
    for b in range(B):
        Q = host["Q"][b]
        vf = oracle.fit_values(Q, Ck[b], beta[b], Yh[b], s, delta=float(dused[b]), max_escalations=0)
        err = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s),
                                 oracle.attend_compact(Q, Ck[b], beta[b], vf.C_v, s)).max()
        print(f"  {name} pair {b}: t={t} n={Q.shape[0]}, ridge raised from 0 to {dused[b]:.1e}; output max row "
              f"rel err {err:.2e}", flush=True)
        assert err <= 1e-3, (b, err)
    if t > Q.shape[0]:
        p = A().default_params(delta_beta=0.0, max_escalations=6)
        bt, info, dused = A().fit_bias(dev["Q"], _f32(Ck), z, m, params=p, scale=s, T=T)
        info, dused = info.cpu().numpy(), dused.cpu().numpy()
        assert np.all(info == 0) and np.all(dused > 0), (info, dused)
        assert torch.isfinite(bt).all()


@pytest.mark.parametrize("where", ["K", "V", "Q"])
def test_nonfinite_input_reports_minus_one(where):
    """A NaN in one pair's K, V or Q_ref reaches that pair's row statistics:
    both fits report info = -1 with NaN outputs; the other pairs are
    unaffected (bit for bit, pairs are independent)."""
    wl = synth.custom("nan", kv_heads=3, T=500, q_heads_per_kv=2, n_pos=48, rho=0.1, dtype="bf16", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    ref = [o.cpu() for o in A().compact(dev["K"], dev["V"], dev["Q"], dev["W1"], dev["b1"], dev["w2"], dev["b2"],
                                        wl.rho, scale=s)]
    X = dev[where].clone()
    X[1, 7, 3] = float("nan")
    args = {k: (X if k == where else dev[k]) for k in ("K", "V", "Q")}
    out = [o.cpu() for o in A().compact(args["K"], args["V"], args["Q"], dev["W1"], dev["b1"], dev["w2"], dev["b2"],
                                        wl.rho, scale=s)]
    info = out[4].numpy()
    assert info[1].tolist() == [-1, -1], info
    assert torch.isnan(out[2][1]).all() and torch.isnan(out[3][1]).all()
    for b in (0, 2):
        assert info[b].tolist() == [0, 0]
        for x, y in zip(out[:4], ref[:4]):
            assert torch.equal(x[b], y[b]), b


def test_fits_recompute_row_statistics_when_null():
    """z and m (mass fit) and Y (value fit) passed as NULL are recomputed from
    K and V: the results equal those with the row statistics given, bit for bit."""
    wl = synth.custom("null", kv_heads=2, T=900, q_heads_per_kv=2, n_pos=64, rho=0.1, dtype="bf16", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    t = oracle.budget(wl.T, wl.rho)
    z, m, Y = A().rowstats(dev["K"], dev["V"], dev["Q"], scale=s)
    S = torch.from_numpy(np.stack([np.linspace(0, wl.T - 1, t).astype(np.int32)] * wl.pairs)).cuda()
    Ck, _, _ = A().merge(dev["K"], dev["Q"], z, S, scale=s)
    b1, i1, _ = A().fit_bias(dev["Q"], Ck, z, m, scale=s, T=wl.T)
    b2, i2, _ = A().fit_bias(dev["Q"], Ck, None, None, scale=s, K=dev["K"], V=dev["V"])
    assert torch.equal(b1, b2) and torch.equal(i1, i2)
    c1, j1, _ = A().fit_values(dev["Q"], Ck, b1, Y, scale=s, T=wl.T)
    c2, j2, _ = A().fit_values(dev["Q"], Ck, b1, None, scale=s, K=dev["K"], V=dev["V"])
    assert torch.equal(c1, c2) and torch.equal(j1, j2)


def test_escalated_value_fit_matches_oracle_at_used_ridge():
    """More compact keys than reference queries (t = 600 > n = 256) makes the
    value-fit Gram rank-deficient; with a 1e-9 relative ridge the float32
    factorisation fails and the ridge is escalated (x10 per retry).  The solve
    that follows must use the escalated factor: compare with the float64 fit
    at the ridge the library reports.  Ill-conditioned (ridge ~1e-5 of the
    mean diagonal), so the bar is 1e-3 rather than the well-posed 1e-4."""
    wl = synth.custom("esc", kv_heads=2, T=2000, q_heads_per_kv=2, n_pos=128, rho=0.3, dtype="f32", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    t = oracle.budget(wl.T, wl.rho)
    assert t > wl.n
    refs = [oracle.compact_pair(host["K"][b], host["V"][b], host["Q"][b], host["W1"][b], host["b1"][b],
                                host["w2"][b], host["b2"][b], t=t, scale=s) for b in range(wl.pairs)]
    Ck = np.stack([r.C_k for r in refs]).astype(np.float32)
    beta = np.stack([r.beta for r in refs]).astype(np.float32)
    Y = np.stack([r.Y for r in refs]).astype(np.float32)
    params = A().default_params(delta_v=1e-9, max_escalations=6)
    Cv, info, dused = A().fit_values(dev["Q"], torch.from_numpy(Ck).cuda(), torch.from_numpy(beta).cuda(),
                                     torch.from_numpy(Y).cuda(), params=params, scale=s, T=wl.T)
    Cv, info, dused = np64(Cv), info.cpu().numpy(), dused.cpu().numpy()
    assert np.all(info == 0), info
    assert np.all(dused > 1e-9), dused        # every pair went through the escalation path
    for b in range(wl.pairs):
        Q = host["Q"][b]
        vf = oracle.fit_values(Q, Ck[b].astype(np.float64), beta[b].astype(np.float64), Y[b].astype(np.float64), s,
                               delta=float(dused[b]))
        err = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s),
                                 oracle.attend_compact(Q, Ck[b], beta[b], vf.C_v, s)).max()
        print(f"  pair {b}: ridge escalated to {dused[b]:.1e}; output max row rel err {err:.3e}", flush=True)
        assert err <= 1e-3, (b, err)


def test_value_fit_tiny_ridge_well_posed():
    """A full-rank value-fit Gram (t = 600 < n = 1024, three 256-row blocks)
    with a 1e-12 relative ridge: no escalation, but the a-priori bound
    ||R_c|| / sqrt(lam) that scales the forward solve's fp16 operand is far
    above the solution, so the solve must fall back to its fp32 form (or keep
    enough bits) and still match the float64 fit at that ridge (eq.
    value_lstsq) to the fp32 bar of 1e-4."""
    wl = synth.custom("vtiny", kv_heads=2, T=3000, q_heads_per_kv=4, n_pos=256, rho=0.2, dtype="f32", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(128)
    t = oracle.budget(wl.T, wl.rho)
    assert 512 < t < wl.n
    refs = [oracle.compact_pair(host["K"][b], host["V"][b], host["Q"][b], host["W1"][b], host["b1"][b],
                                host["w2"][b], host["b2"][b], t=t, scale=s) for b in range(wl.pairs)]
    Ck = np.stack([r.C_k for r in refs]).astype(np.float32)
    beta = np.stack([r.beta for r in refs]).astype(np.float32)
    Y = np.stack([r.Y for r in refs]).astype(np.float32)
    params = A().default_params(delta_v=1e-12, max_escalations=0)
    Cv, info, dused = A().fit_values(dev["Q"], torch.from_numpy(Ck).cuda(), torch.from_numpy(beta).cuda(),
                                     torch.from_numpy(Y).cuda(), params=params, scale=s, T=wl.T)
    Cv, info, dused = np64(Cv), info.cpu().numpy(), dused.cpu().numpy()
    assert np.all(info == 0), info
    for b in range(wl.pairs):
        Q = host["Q"][b]
        vf = oracle.fit_values(Q, Ck[b].astype(np.float64), beta[b].astype(np.float64), Y[b].astype(np.float64), s,
                               delta=float(dused[b]))
        err = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s),
                                 oracle.attend_compact(Q, Ck[b], beta[b], vf.C_v, s)).max()
        print(f"  pair {b}: ridge {dused[b]:.1e}; output max row rel err {err:.3e}", flush=True)
        assert err <= 1e-4, (b, err)


def test_exact_fit_degenerate_cases():
    """The exact non-negative fit where the constraints cannot bind: full
    retention (C_k = K, so w = 1 fits the mass exactly: beta = 0) and a single
    anchor (a scalar least-squares weight, positive): both must agree with the
    projected fit."""
    wl = synth.custom("full1", kv_heads=2, T=48, q_heads_per_kv=2, n_pos=64, dtype="f32", rope=True)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, 1.0, delta_beta=0.0, delta_v=0.0, bias_mode=1)
    assert np.all(info.numpy() == 0), info
    assert np.abs(np64(beta)).max() < 1e-3, np.abs(np64(beta)).max()
    for b in range(wl.pairs):
        K, V = host["K"][b], host["V"][b]
        Qh = synth.heldout_queries(wl, 0, b).astype(np.float64)
        Oc = oracle.attend_compact(Qh, np64(Ck[b]), np64(beta[b]), np64(Cv[b]), s)
        assert oracle.row_rel_err(Oc, oracle.attend_full(Qh, K, V, s)).max() < 1e-3
    wl = synth.custom("t1e", kv_heads=1, T=300, q_heads_per_kv=1, n_pos=64, dtype="f32", rope=False)
    _, _, _, out0 = run(wl, 0.001)
    _, _, _, out1 = run(wl, 0.001, bias_mode=1)
    assert np.all(out1[4].numpy() == 0)
    np.testing.assert_allclose(np64(out1[2]), np64(out0[2]), rtol=0, atol=1e-5)


@pytest.mark.parametrize("n_dup_anchors", [40, 70])
def test_key_tied_with_many_anchors(n_dup_anchors):
    """Keys whose row repeats in more than 31 anchors (eq. anchor_assignment):
    every tied anchor survives the refine pass, the float64 pass splits the key
    over several entries, and the merged decision is the lowest tied r (ties to
    the lowest r).  The other keys match the float64 oracle up to certified
    near-ties."""
    rng = np.random.default_rng(11 + n_dup_anchors)
    T, n, t = 640, 256, 160
    s = 1.0 / math.sqrt(128)
    K = rng.standard_normal((T, 128)).astype(np.float32)
    V = rng.standard_normal((T, 128)).astype(np.float32)
    Q = rng.standard_normal((n, 128)).astype(np.float32)
    dup = np.sort(rng.choice(T, n_dup_anchors + 24, replace=False))
    K[dup] = K[dup[0]]
    others = np.setdiff1d(np.arange(T), dup)
    S = np.sort(np.concatenate([dup[:n_dup_anchors], rng.choice(others, t - n_dup_anchors, replace=False)]))
    Kb, Vb, Qb = (torch.from_numpy(x).to(torch.bfloat16) for x in (K, V, Q))
    kap, st = gpu_assignment(Kb[None].cuda().contiguous(), Vb[None].cuda().contiguous(),
                             Qb[None].cuda().contiguous(), torch.from_numpy(S.astype(np.int32))[None].cuda(), s)
    r_dup = np.searchsorted(S, dup[:n_dup_anchors])      # the tied anchors' indices r
    for j in dup[n_dup_anchors:]:                          # the tied keys that are not anchors
        assert kap[j] == r_dup.min(), (j, kap[j], r_dup.min())
    assert st[1] >= len(dup) - n_dup_anchors               # they went to the float64 pass
    assert np.all(kap[S] == np.arange(t))
    K64, Q64 = np64(Kb), np64(Qb)
    ref, _, _ = oracle.profiles_assign_phi(Q64, K64, S, s)
    ref[dup] = kap[dup]   # checked above against the exact tie rule
    certify_flips(kap, ref, Q64, K64, S, s)


@pytest.mark.parametrize("t", [16384, 17000])
def test_merge_many_groups(t):
    """The grouping of keys by anchor (a stable counting sort inside arckv_merge)
    with as many groups as its LDS cursors hold (t = 16384) and more (t = 17000,
    cursors in global scratch): every anchor keeps itself and the merged keys
    equal eq. key_merge on the GPU's assignment and mass weights."""
    rng = np.random.default_rng(t)
    T, n = 20000, 64
    s = 1.0 / math.sqrt(128)
    K = rng.standard_normal((T, 128)).astype(np.float32)
    V = rng.standard_normal((T, 128)).astype(np.float32)
    Q = rng.standard_normal((n, 128)).astype(np.float32)
    S = np.sort(rng.choice(T, t, replace=False))
    Kb, Vb, Qb = (torch.from_numpy(x).to(torch.bfloat16)[None].cuda().contiguous() for x in (K, V, Q))
    from paper_2609_36835_amd import arckv
    z, _, _ = arckv.rowstats(Kb, Vb, Qb, scale=s)
    Ck, kappa, phi, st = arckv.merge(Kb, Qb, z, torch.from_numpy(S.astype(np.int32))[None].cuda(),
                                     lambda_m=oracle.LAMBDA_M, scale=s, return_stats=True)
    kap = kappa[0].cpu().numpy().astype(np.int64)
    assert np.all(kap[S] == np.arange(t))
    assert kap.min() >= 0 and kap.max() < t
    assert st[0].cpu().numpy()[3] == 0
    K64 = np64(Kb)[0]
    ref = oracle.merge_keys(K64, np64(phi)[0], kap, S, oracle.LAMBDA_M)
    np.testing.assert_allclose(np64(Ck)[0], ref, rtol=0, atol=2e-5 * np.abs(K64).max())
