"""Shared helpers for the GPU parity tests: seeded inputs on device + float64 views."""
import math

import numpy as np
import torch

import synth

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}

# Tolerances (per-row relative l2 of compact-attention outputs on Q_ref; the
# fp32 and bf16-input bars of the benchmark spec).
TOL_OUT = {"f32": 1e-4, "bf16": 2e-2}


def make_inputs(wl, seed=0, pairs=None, device="cuda"):
    """Device tensors [B][...] plus the float64 host copies the oracle uses."""
    arr = synth.workload_arrays(wl, seed=seed, pairs=pairs)
    td = TORCH_DTYPE[wl.dtype]
    dev = {
        "K": torch.from_numpy(arr["K"]).to(device=device, dtype=td).contiguous(),
        "V": torch.from_numpy(arr["V"]).to(device=device, dtype=td).contiguous(),
        "Q": torch.from_numpy(arr["Q"]).to(device=device, dtype=td).contiguous(),
        "W1": torch.from_numpy(arr["W1"]).to(device=device, dtype=td).contiguous(),
        "b1": torch.from_numpy(arr["b1"]).to(device=device).contiguous(),
        "w2": torch.from_numpy(arr["w2"]).to(device=device).contiguous(),
        "b2": torch.from_numpy(arr["b2"][:, 0]).to(device=device).contiguous(),
    }
    host = {k: v.astype(np.float64) for k, v in arr.items()}
    host["b2"] = host["b2"][:, 0]
    # the device values are exactly the host values (bf16-representable for bf16)
    assert np.array_equal(dev["K"].float().cpu().numpy().astype(np.float64), host["K"])
    return dev, host


def scale_of(wl):
    return 1.0 / math.sqrt(wl.d)


def np64(x):
    return x.detach().float().cpu().numpy().astype(np.float64)


# An assignment difference between the GPU and the float64 oracle is accepted
# only at a float64 near-tie: the library's last pass decides in float64
# (logits from exact products, exponentials, norms and dot products in float64),
# so the two can disagree only where the two anchors' float64 similarities
# agree to within their rounding, about n 2^-52 relative (1e-12 at n = 4096).
TIE_F64 = 1e-10


def assignment_gap(Q, K, S, scale, j, r_gpu, r_ref):
    """Relative float64 gap of eq. anchor_assignment between the oracle's anchor
    r_ref and the GPU's r_gpu for key j (>= 0 when r_ref is the argmax)."""
    import oracle
    zm = oracle.global_logit_max(Q, K, scale)
    _, US, _ = oracle.response_profiles(Q, K[np.asarray(S)[[r_gpu, r_ref]]], scale, zm)
    e = np.exp(oracle.logits(Q, K[j:j + 1], scale) - zm)[:, 0]
    sim = e @ US
    return (sim[1] - sim[0]) / max(abs(sim[1]), 1e-300)


def gpu_assignment(K, V, Q, anchors, scale):
    """kappa and the assignment counters (arckv_assign_stats) as arckv_compact
    computes them for one pair: the GPU row maxima z (arckv_rowstats) feed
    arckv_merge on the given anchors.  K, V, Q: [1][...] device tensors,
    anchors [1][t] int32."""
    from paper_2609_36835_amd import arckv
    import oracle
    z, _, _ = arckv.rowstats(K, V, Q, scale=scale)
    _, kappa, _, st = arckv.merge(K, Q, z, anchors, lambda_m=oracle.LAMBDA_M, scale=scale, return_stats=True)
    return kappa[0].cpu().numpy().astype(np.int64), st[0].cpu().numpy()


def certify_flips(kappa_gpu, kappa_ref, Q, K, anchors, scale, log=print):
    """Every assignment difference from the float64 definition must be a float64
    near-tie (TIE_F64).  Returns the number of differences."""
    flips = np.flatnonzero(kappa_gpu != kappa_ref)
    for j in flips:
        gap = assignment_gap(Q, K, anchors, scale, j, kappa_gpu[j], kappa_ref[j])
        log(f"    key {j}: gpu anchor {kappa_gpu[j]}, oracle anchor {kappa_ref[j]}, float64 relative gap {gap:.2e}")
        assert abs(gap) <= TIE_F64, (j, gap)
    return len(flips)


def log_assign_stats(st, T, t, log=print):
    """Counters of the three assignment passes; no key may be left undecided."""
    keys = max(1, T - t)
    log(f"    assignment: {st[0]} keys flagged by the fp16 bound ({st[0] / keys:.2%}; {st[6]} refined, {st[7]} with "
        f"a whole tile), {st[1]} decided in float64 ({st[1] / keys:.3%}), {st[2]} candidates, {st[3]} undecided")
    assert st[3] == 0, st
