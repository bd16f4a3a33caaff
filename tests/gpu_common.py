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


def profile_dtype(wl):
    """The precision the GPU stores response profiles in (bf16 or fp32 inputs)."""
    return "bf16" if wl.dtype == "bf16" else "f32"


def assignment_gap(Q, K, S, scale, j, pdt):
    """Relative gap between key j's best and runner-up anchor similarity,
    with profiles rounded to the storage precision pdt."""
    import oracle
    zm = oracle.global_logit_max(Q, K, scale)
    ES = oracle.round_to(np.exp(oracle.logits(Q, K[S], scale) - zm), pdt)
    US = oracle.round_to(ES / np.linalg.norm(ES, axis=0)[None, :], pdt)
    ej = oracle.round_to(np.exp(oracle.logits(Q, K[j:j + 1], scale) - zm), pdt)[:, 0]
    sim = ej @ US
    top = np.sort(sim)[::-1]
    return 0.0 if len(top) < 2 else (top[0] - top[1]) / max(abs(top[0]), 1e-300)


def gpu_assignment(K, V, Q, anchors, scale):
    """kappa as arckv_compact computes it for one pair: the GPU row maxima z
    (arckv_rowstats) feed arckv_merge on the GPU's anchors.  K, V, Q: [1][...]
    device tensors, anchors [1][t] int32."""
    from paper_2609_36835_amd import arckv
    import oracle
    z, _, _ = arckv.rowstats(K, V, Q, scale=scale)
    _, kappa, _ = arckv.merge(K, Q, z, anchors, lambda_m=oracle.LAMBDA_M, scale=scale)
    return kappa[0].cpu().numpy().astype(np.int64)


def certify_flips(kappa_gpu, kappa_ref, Q, K, anchors, scale, pdt, log=print):
    """Assignment differences must be near-ties within one storage-precision
    rounding term (2^-7 relative for bf16 profiles, 2^-23 + n 2^-24 for fp32)
    and rare (at most max(1, T/1000))."""
    rel_tie = 2.0 ** -7 if pdt == "bf16" else 2.0 ** -23 + Q.shape[0] * 2.0 ** -24
    flips = np.flatnonzero(kappa_gpu != kappa_ref)
    for j in flips:
        gap = assignment_gap(Q, K, anchors, scale, j, pdt)
        log(f"    key {j}: gpu anchor {kappa_gpu[j]}, oracle anchor {kappa_ref[j]}, relative gap {gap:.2e}")
        assert gap <= rel_tie, (j, gap)
    assert len(flips) <= max(1, len(K) // 1000), len(flips)
    return len(flips)
