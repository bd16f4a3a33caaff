"""Decode attention over a compact block (+ an uncompressed block) on the GPU
against the float64 oracle (eq. compact_attention and the joint form of
Appendix A.7).  Inputs are bf16 (bias fp32), so the products are exact and only
fp32 summation, the exponential and the split-key merge differ: per-row relative
error <= 1e-4."""
import math

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

TOL = 1e-4


def bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to("cuda", torch.bfloat16)


def run_case(P, G, t, F, seed, beta_range=3.0, with_beta=True, scale=None):
    from paper_2609_36835_amd import arckv
    g = np.random.default_rng(seed)
    d = 128
    Q = bf16(g.standard_normal((P, G, d)))
    Ck = bf16(g.standard_normal((P, t, d))) if t else None
    Cv = bf16(g.standard_normal((P, t, d))) if t else None
    Kf = bf16(g.standard_normal((P, F, d))) if F else None
    Vf = bf16(g.standard_normal((P, F, d))) if F else None
    beta = (torch.from_numpy(g.uniform(-beta_range, beta_range, (P, t)).astype(np.float32)).cuda()
            if (t and with_beta) else None)
    print(f"attend P={P} G={G} t={t} F={F} seed={seed}", flush=True)
    out = arckv.attend(Q, Ck, beta, Cv, Kf, Vf, scale=scale).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    s = scale if scale else 1.0 / math.sqrt(d)
    h = lambda x: None if x is None else x.float().cpu().numpy().astype(np.float64)
    Qh, Ckh, Cvh, Kfh, Vfh, bh = h(Q), h(Ck), h(Cv), h(Kf), h(Vf), h(beta)
    worst = 0.0
    for p in range(P):
        ref = oracle.attend_joint(Qh[p], None if Ckh is None else Ckh[p], None if bh is None else bh[p],
                                  None if Cvh is None else Cvh[p], None if Kfh is None else Kfh[p],
                                  None if Vfh is None else Vfh[p], s)
        worst = max(worst, float(oracle.row_rel_err(out[p], ref).max()))
    print(f"    max row rel err {worst:.2e}", flush=True)
    assert worst <= TOL, worst


@pytest.mark.parametrize("P,G,t,F", [(3, 4, 1, 0), (2, 1, 300, 0), (5, 4, 257, 33), (2, 8, 0, 70),
                                     (4, 2, 1000, 1), (3, 4, 511, 0), (2, 4, 256, 256)])
def test_attend_matches_oracle(P, G, t, F):
    run_case(P, G, t, F, seed=P * 1000 + t + F)


def test_attend_extreme_bias_and_scale():
    run_case(3, 4, 700, 50, seed=7, beta_range=30.0)
    run_case(2, 4, 300, 20, seed=8, scale=1.0)


def test_attend_without_bias_is_full_attention():
    run_case(4, 4, 900, 0, seed=9, with_beta=False)


def test_attend_decode_shape_32k_at_20_percent():
    # one pair of the 32K-context decode workload: t = round(0.2 * 32768) = 6554 compact rows
    run_case(2, 4, 6554, 0, seed=11)


@pytest.mark.parametrize("label", ["full", "compact"])
def test_attend_bench_launch_sampled_pairs(label):
    """The decode launch the benchmark times: batch 64 x 8 KV heads = 512 pairs, 4 query heads per KV head,
    a 32K context either whole (L = 32768, no bias) or compacted at rho = 0.2 (t = 6554, bias in [-3, 3]).
    Inputs drawn on the device as the benchmark draws them; sampled pairs (first, last, and six more spread
    over the batch) are checked against the float64 oracle one by one."""
    from paper_2609_36835_amd import arckv
    P, G, d, T = 512, 4, 128, 32768
    L = T if label == "full" else arckv.budget(T, 0.2)
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    K = torch.randn(P, L, d, device=dev, dtype=torch.bfloat16, generator=g)
    V = torch.randn(P, L, d, device=dev, dtype=torch.bfloat16, generator=g)
    Q = torch.randn(P, G, d, device=dev, dtype=torch.bfloat16, generator=g)
    beta = (torch.rand(P, L, device=dev, generator=g) * 6 - 3) if label == "compact" else None
    print(f"attend bench launch {label}: P={P} G={G} L={L}", flush=True)
    att = arckv.Attender(P, G, L, 0, dev)
    out = att(Q, K, beta, V).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    s = 1.0 / math.sqrt(d)
    worst = 0.0
    for p in (0, 1, 97, 200, 255, 256, 421, P - 1):
        h = lambda x: x[p].float().cpu().numpy().astype(np.float64)
        ref = oracle.attend_joint(h(Q), h(K), None if beta is None else h(beta), h(V), None, None, s)
        worst = max(worst, float(oracle.row_rel_err(out[p], ref).max()))
    print(f"    max row rel err over sampled pairs {worst:.2e}", flush=True)
    assert worst <= TOL, worst
    assert np.isfinite(out).all()
