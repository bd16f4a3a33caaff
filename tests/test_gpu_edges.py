"""GPU edge cases: full retention, a single anchor, tiny caches, ridge-free fits."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import make_inputs, np64

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
        assert oracle.row_rel_err(Oc, O).max() < 1e-3


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
    wl = synth.custom(f"s{T}", kv_heads=2, T=T, q_heads_per_kv=1, n_pos=n_pos, dtype="bf16", rope=True)
    dev, host, s, (anchors, Ck, beta, Cv, info) = run(wl, rho)
    t = oracle.budget(T, rho)
    assert anchors.shape == (2, t)
    for b in range(2):
        a = anchors[b].numpy()
        assert np.all(np.diff(a) > 0) and a.min() >= 0 and a.max() < T
        assert np.isfinite(np64(Ck[b])).all()
        if info[b, 0] == 0:
            assert np.isfinite(np64(beta[b])).all()
        if info[b, 1] == 0:
            assert np.isfinite(np64(Cv[b])).all()
