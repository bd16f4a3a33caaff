"""Seeded synthetic inputs for ARC-KV per-context compaction.

This module only draws inputs: Gaussian key/value/query caches shaped like
Llama-3.1-8B attention (head_dim 128, grouped-query attention with 4 query
heads per KV head), a few large-magnitude key channels, rotary position
embedding on keys and queries, and random weights for the token-scoring MLP.
It contains none of the compaction arithmetic, so both the float64 oracle and
the GPU path can use it without sharing any of the method's code.

Every (layer, head, stream) triple has its own generator, so any single pair
can be regenerated on its own:
``numpy.random.default_rng(SeedSequence([seed, layer, head, stream]))`` with
stream 0 = K, 1 = V, 2 = Q_ref, 3 = indexer weights, 4 = held-out queries.

Values for bf16 workloads are rounded once to bfloat16 (round to nearest even)
and returned as float32 arrays holding exactly representable values, so the
GPU receives them bit-exactly after ``.to(torch.bfloat16)`` and the oracle
upcasts them to float64 without further rounding.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HEAD_DIM = 128
HIDDEN = 64
OUTLIER_CHANNELS = (60, 61, 62, 63)
OUTLIER_SCALE = 8.0
ROPE_THETA = 500000.0

STREAM_K, STREAM_V, STREAM_Q, STREAM_W, STREAM_HELD = 0, 1, 2, 3, 4


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic compaction workload (all pairs share T, n and rho)."""

    name: str
    layers: int
    kv_heads: int
    T: int
    q_heads_per_kv: int
    n_pos: int
    rho: float
    dtype: str          # "f32" or "bf16"
    rope: bool
    d: int = HEAD_DIM

    @property
    def pairs(self) -> int:
        return self.layers * self.kv_heads

    @property
    def n(self) -> int:
        return self.q_heads_per_kv * self.n_pos


WORKLOADS = {
    # single pair, fp32, no rotary embedding, 256 reference queries
    "tiny_f32_T1024": Workload("tiny_f32_T1024", 1, 1, 1024, 1, 256, 0.10, "f32", False),
    # one Llama-3.1-8B layer: 8 KV heads x 4 query heads, T = 8192
    "layer_bf16_T8192": Workload("layer_bf16_T8192", 1, 8, 8192, 4, 1024, 0.10, "bf16", True),
    # full 32-layer x 8-head cache at T = 32768, 10% kept
    "llama8b_bf16_T32768": Workload("llama8b_bf16_T32768", 32, 8, 32768, 4, 1024, 0.10, "bf16", True),
    # retention sweep at T = 16384
    "llama8b_bf16_T16384_r20": Workload("llama8b_bf16_T16384_r20", 32, 8, 16384, 4, 1024, 0.20, "bf16", True),
    "llama8b_bf16_T16384_r10": Workload("llama8b_bf16_T16384_r10", 32, 8, 16384, 4, 1024, 0.10, "bf16", True),
    "llama8b_bf16_T16384_r05": Workload("llama8b_bf16_T16384_r05", 32, 8, 16384, 4, 1024, 0.05, "bf16", True),
    "llama8b_bf16_T16384_r02": Workload("llama8b_bf16_T16384_r02", 32, 8, 16384, 4, 1024, 0.02, "bf16", True),
    # long context: one layer, T = 131072, 8192 reference queries, 1% kept
    "long_bf16_T131072": Workload("long_bf16_T131072", 1, 8, 131072, 4, 2048, 0.01, "bf16", True),
}


def custom(name: str, *, layers=1, kv_heads=1, T=256, q_heads_per_kv=1, n_pos=64,
           rho=0.1, dtype="f32", rope=False) -> Workload:
    """A small workload for tests (ragged sizes, edge cases)."""
    return Workload(name, layers, kv_heads, T, q_heads_per_kv, n_pos, rho, dtype, rope)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def _rng(seed: int, layer: int, head: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, layer, head, stream]))


def llama3_inv_freq(d: int = HEAD_DIM, theta: float = ROPE_THETA, factor: float = 8.0,
                    low_freq_factor: float = 1.0, high_freq_factor: float = 4.0,
                    original_max_position: int = 8192) -> np.ndarray:
    """Rotary inverse frequencies with Llama-3.1's long-context rescaling."""
    inv = 1.0 / theta ** (np.arange(0, d, 2, dtype=np.float64) / d)
    low_wavelen = original_max_position / low_freq_factor
    high_wavelen = original_max_position / high_freq_factor
    wavelen = 2.0 * math.pi / inv
    out = np.where(wavelen > low_wavelen, inv / factor, inv)
    smooth = (original_max_position / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    mid = (wavelen >= high_wavelen) & (wavelen <= low_wavelen)
    out = np.where(mid, (1.0 - smooth) * inv / factor + smooth * inv, out)
    return out


def apply_rope(x: np.ndarray, positions: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding (channel c pairs with c + d/2)."""
    d = x.shape[-1]
    ang = positions.astype(np.float64)[:, None] * llama3_inv_freq(d)[None, :]
    cos = np.cos(ang).astype(np.float32)
    sin = np.sin(ang).astype(np.float32)
    x1, x2 = x[:, : d // 2], x[:, d // 2:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=1).astype(np.float32)


def _cast(wl: Workload, x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return round_bf16(x) if wl.dtype == "bf16" else x


def query_positions(wl: Workload) -> np.ndarray:
    """Position of each reference-query row, ordered [query head][position]."""
    r = np.arange(wl.n_pos, dtype=np.int64)
    pos = (r * wl.T) // wl.n_pos
    return np.tile(pos, wl.q_heads_per_kv)


def pair_inputs(wl: Workload, layer: int, head: int, seed: int = 0) -> dict:
    """K, V [T, d], Q_ref [n, d] and the scoring-MLP weights of one pair."""
    d = wl.d
    k0 = _rng(seed, layer, head, STREAM_K).standard_normal((wl.T, d), dtype=np.float32)
    k0[:, list(OUTLIER_CHANNELS)] *= np.float32(OUTLIER_SCALE)
    v = _rng(seed, layer, head, STREAM_V).standard_normal((wl.T, d), dtype=np.float32)
    q = _rng(seed, layer, head, STREAM_Q).standard_normal((wl.n, d), dtype=np.float32)
    if wl.rope:
        k0 = apply_rope(k0, np.arange(wl.T))
        q = apply_rope(q, query_positions(wl))
    out = {"K": _cast(wl, k0), "V": _cast(wl, v), "Q": _cast(wl, q)}
    out.update(indexer_weights(wl, layer, head, seed))
    return out


def indexer_weights(wl: Workload, layer: int, head: int, seed: int = 0) -> dict:
    """Random init of the 2d -> 64 -> 1 scoring MLP (uniform fan-in bounds)."""
    rng = _rng(seed, layer, head, STREAM_W)
    a1 = 1.0 / math.sqrt(2 * wl.d)
    a2 = 1.0 / math.sqrt(HIDDEN)
    W1 = rng.uniform(-a1, a1, (HIDDEN, 2 * wl.d)).astype(np.float32)
    b1 = rng.uniform(-a1, a1, HIDDEN).astype(np.float32)
    w2 = rng.uniform(-a2, a2, HIDDEN).astype(np.float32)
    b2 = np.float32(rng.uniform(-a2, a2))
    if wl.dtype == "bf16":
        W1 = round_bf16(W1)
    return {"W1": W1, "b1": b1, "w2": w2, "b2": np.array([b2], dtype=np.float32)}


def heldout_queries(wl: Workload, layer: int, head: int, rows: int = 256, seed: int = 0) -> np.ndarray:
    """Queries disjoint from Q_ref (own stream), same distribution and positions."""
    q = _rng(seed, layer, head, STREAM_HELD).standard_normal((rows, wl.d), dtype=np.float32)
    if wl.rope:
        pos = (np.arange(rows, dtype=np.int64) * wl.T) // rows
        q = apply_rope(q, pos)
    return _cast(wl, q)


def pair_index(wl: Workload, b: int) -> tuple:
    """Pair b of the flattened [layer][kv_head] order -> (layer, head)."""
    return divmod(b, wl.kv_heads)


def workload_arrays(wl: Workload, seed: int = 0, pairs=None, threads: int = 8) -> dict:
    """Stacked inputs for the given pairs (default: all), in [B][...] layout."""
    idx = list(range(wl.pairs)) if pairs is None else list(pairs)

    def one(b):
        layer, head = pair_index(wl, b)
        return pair_inputs(wl, layer, head, seed)

    with ThreadPoolExecutor(max_workers=max(1, threads)) as ex:
        parts = list(ex.map(one, idx))
    return {key: np.stack([p[key] for p in parts]) for key in parts[0]}
