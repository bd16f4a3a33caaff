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


def assignment_near_tie(Q, K, S, scale, j, rel):
    """True if key j's best and runner-up anchor similarities are within rel."""
    import oracle
    zm = oracle.global_logit_max(Q, K, scale)
    _, US, _ = oracle.response_profiles(Q, K[S], scale, zm)
    _, uj, _ = oracle.response_profiles(Q, K[j:j + 1], scale, zm)
    sim = (uj.T @ US)[0]
    top = np.sort(sim)[::-1]
    return len(top) < 2 or (top[0] - top[1]) <= rel * max(abs(top[0]), 1e-300)
