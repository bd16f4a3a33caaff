"""Chunked anchor selection (Appendix A.3) and per-pair budgets (eq.
per_head_budget) on the GPU: bit-exact against the oracle on the same float32
scores, rows padded with -1; and arckv_compact with chunked selection end to
end."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import TOL_OUT, certify_flips, gpu_assignment, log_assign_stats, make_inputs, np64

pytestmark = pytest.mark.gpu


def A():
    from paper_2609_36835_amd import arckv
    return arckv


def scores_of(B, T, seed, dup):
    g = np.random.default_rng(seed)
    s = g.standard_normal((B, T)).astype(np.float32)
    if dup:
        s = np.round(s * 4) / 4      # heavy ties: resolved by position
    return s


@pytest.mark.parametrize("B,T,t,L,dup", [(3, 12000, 1200, 8192, False), (2, 20001, 77, 5000, True),
                                         (2, 40000, 4000, 8192, True), (2, 9000, 900, 4096, False),
                                         (1, 131072, 1311, 8192, False)])
def test_chunked_select_bitexact(B, T, t, L, dup):
    s = scores_of(B, T, seed=T + t, dup=dup)
    print(f"chunked select B={B} T={T} t={t} L={L}", flush=True)
    got = A().select_ex(torch.from_numpy(s).cuda(), t, chunk_len=L).cpu().numpy()
    tr = A().select_count(T, t, L)
    assert got.shape == (B, tr)
    for b in range(B):
        ref = oracle.select_topt_chunked(s[b].astype(np.float64), t, L)
        assert got[b].tolist() == ref.tolist(), b


@pytest.mark.parametrize("chunk", [0, 8192])
def test_per_pair_budgets(chunk):
    B, T = 6, 14000
    a = np.random.default_rng(5).uniform(0.2, 3.0, B)
    tb = A().budgets(list(a), 700, T)
    assert tb == oracle.budgets_per_pair(a, 700, T).tolist()
    s = scores_of(B, T, seed=9, dup=True)
    stride = max(A().select_count(T, x, chunk) for x in tb) + 3
    print(f"per-pair budgets {tb} chunk={chunk} stride={stride}", flush=True)
    got = A().select_ex(torch.from_numpy(s).cuda(), 700, t_pair=torch.tensor(tb, dtype=torch.int32).cuda(),
                        chunk_len=chunk, t_stride=stride).cpu().numpy()
    for b in range(B):
        ref = oracle.select_topt_chunked(s[b].astype(np.float64), tb[b], chunk)
        assert got[b, :len(ref)].tolist() == ref.tolist(), b
        assert np.all(got[b, len(ref):] == -1), b


def test_compact_with_chunked_selection():
    # n = 512 reference queries > t = 360 anchors, so both fits are determined (as in every workload)
    wl = synth.custom("bf16_T12000_chunked", kv_heads=2, T=12000, q_heads_per_kv=2, n_pos=256, rho=0.03,
                      dtype="bf16", rope=True)
    dev, host = make_inputs(wl)
    s = 1.0 / math.sqrt(wl.d)
    L = 8192
    params = A().default_params(select_chunk=L)
    t_nom = oracle.budget(wl.T, wl.rho)
    t = A().select_count(wl.T, t_nom, L)
    print(f"compact with chunked selection: T={wl.T} t={t_nom} -> {t}", flush=True)
    anchors_d, Ck, beta, Cv, info = A().compact(dev["K"], dev["V"], dev["Q"], dev["W1"], dev["b1"], dev["w2"],
                                                dev["b2"], wl.rho, scale=s, params=params)
    assert anchors_d.shape[1] == t
    assert np.all(info.cpu().numpy() == 0)
    scores = A().score(dev["K"], dev["V"], dev["W1"], dev["b1"], dev["w2"], dev["b2"]).cpu().numpy()
    anchors, Ck, beta, Cv = anchors_d.cpu().numpy(), np64(Ck), np64(beta), np64(Cv)
    for b in range(wl.pairs):
        S = oracle.select_topt_chunked(scores[b].astype(np.float64), t_nom, L)
        assert anchors[b].tolist() == S.tolist(), b
        Q, K = host["Q"][b], host["K"][b]
        kap_gpu, st = gpu_assignment(dev["K"][b:b + 1].contiguous(), dev["V"][b:b + 1].contiguous(),
                                     dev["Q"][b:b + 1].contiguous(), anchors_d[b:b + 1].contiguous(), s)
        log_assign_stats(st, wl.T, t)
        rr = oracle.compact_pair(K, host["V"][b], Q, host["W1"][b], host["b1"][b], host["w2"][b], host["b2"][b],
                                 t=t, scale=s, anchors=S)
        if certify_flips(kap_gpu, rr.kappa, Q, K, S, s):
            rr = oracle.compact_pair(K, host["V"][b], Q, host["W1"][b], host["b1"][b], host["w2"][b], host["b2"][b],
                                     t=t, scale=s, anchors=S, kappa=kap_gpu)
        err = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s),
                                 oracle.attend_compact(Q, rr.C_k, rr.beta, rr.C_v, s))
        print(f"  pair {b}: O(Q_ref) max row rel err {err.max():.3e}", flush=True)
        assert err.max() <= TOL_OUT[wl.dtype], (b, err.max())
