"""Throughput of ARC-KV per-context compaction on one MI355X.

One step = one arckv_compact call over every layer-KV-head pair of the
workload (score, select, row statistics, assignment and merge, mass fit,
value fit), inputs resident in HBM.  Prints ONE JSON line.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HEADLINE = "llama8b_bf16_T32768"
PEAK_BF16_TFLOPS = 2500.0        # MI355X dense bf16 / fp16 MFMA
PEAK_FP32_TFLOPS = 157.3


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def load_inputs(wl, device):
    """Generate the seeded workload layer by layer and upload it (bf16 / fp32)."""
    import torch
    td = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    B, T, n, d = wl.pairs, wl.T, wl.n, wl.d
    K = torch.empty(B, T, d, dtype=td, device=device)
    V = torch.empty(B, T, d, dtype=td, device=device)
    Q = torch.empty(B, n, d, dtype=td, device=device)
    W1 = torch.empty(B, 64, 2 * d, dtype=td, device=device)
    b1 = torch.empty(B, 64, dtype=torch.float32, device=device)
    w2 = torch.empty(B, 64, dtype=torch.float32, device=device)
    b2 = torch.empty(B, dtype=torch.float32, device=device)
    step = wl.kv_heads
    threads = min(16, os.cpu_count() or 1)
    t0 = time.time()
    for b0 in range(0, B, step):
        idx = list(range(b0, min(B, b0 + step)))
        arr = synth.workload_arrays(wl, pairs=idx, threads=threads)
        sl = slice(idx[0], idx[-1] + 1)
        K[sl] = torch.from_numpy(arr["K"]).to(device).to(td)
        V[sl] = torch.from_numpy(arr["V"]).to(device).to(td)
        Q[sl] = torch.from_numpy(arr["Q"]).to(device).to(td)
        W1[sl] = torch.from_numpy(arr["W1"]).to(device).to(td)
        b1[sl] = torch.from_numpy(arr["b1"]).to(device)
        w2[sl] = torch.from_numpy(arr["w2"]).to(device)
        b2[sl] = torch.from_numpy(arr["b2"][:, 0]).to(device)
        if (b0 // step) % 8 == 0:
            log(f"[inputs] pairs {idx[-1] + 1}/{B} generated ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    return K, V, Q, W1, b1, w2, b2


def assign_flops(wl, t):
    """Algorithmic flops of the key-to-anchor assignment, all pairs: 2 n (T - t) t each."""
    return 2.0 * wl.n * (wl.T - t) * t * wl.pairs


def blas_info():
    """The BLAS numpy links (vendor, version, threading) and its thread count."""
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if pools:
            p = pools[0]
            return {"vendor": p.get("internal_api"), "version": p.get("version"),
                    "threading": p.get("threading_layer"), "threads": p.get("num_threads")}
    except Exception:   # threadpoolctl missing or unable to inspect
        pass
    return {"vendor": "unknown"}


def cpu_baseline(wl, t, budget_s=30.0):
    """The float64 oracle timed on the host cores: one whole layer (every KV head of layer 0) of the same workload,
    scaled to all pairs, plus the 1-pair fp32 workload on all threads and on one thread."""
    import oracle
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    s = 1.0 / math.sqrt(wl.d)
    blas = blas_info()
    done, t_used = 0, 0.0
    while done < min(wl.kv_heads, wl.pairs):
        layer, head = synth.pair_index(wl, done)
        p = synth.pair_inputs(wl, layer, head)
        h = {k: v.astype(np.float64) for k, v in p.items()}
        t0 = time.perf_counter()
        oracle.compact_pair(h["K"], h["V"], h["Q"], h["W1"], h["b1"], h["w2"], h["b2"][0], t=t, scale=s)
        t_used += time.perf_counter() - t0
        done += 1
        log(f"[cpu_baseline] oracle pair {done}: {t_used:.1f}s cumulative")
        if t_used >= budget_s * 2:
            break
    per_pair = t_used / done
    value = wl.T / (per_pair * wl.pairs)

    def tiny_time():
        w1 = synth.WORKLOADS["tiny_f32_T1024"]
        p = synth.pair_inputs(w1, 0, 0)
        h = {k: v.astype(np.float64) for k, v in p.items()}
        t0 = time.perf_counter()
        oracle.compact_pair(h["K"], h["V"], h["Q"], h["W1"], h["b1"], h["w2"], h["b2"][0],
                            t=oracle.budget(w1.T, w1.rho), scale=s)
        return time.perf_counter() - t0
    tiny_all = tiny_time()
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            tiny_one = tiny_time()
    except Exception:   # no thread control: report none
        tiny_one = None
    return {"value": value, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} of {wl.pairs} pairs (layer 0, every KV head) of the same workload, float64 numpy "
                      f"oracle, {per_pair:.2f} s/pair, extrapolated to all {wl.pairs} pairs",
            "blas": blas, "seconds_per_pair": round(per_pair, 3),
            "tiny_f32_T1024_seconds": {"all_threads": round(tiny_all, 4),
                                       "one_thread": None if tiny_one is None else round(tiny_one, 4)}}


COPY_BYTES = 1 << 30
PEAK_HBM_GBS = 8000.0            # MI355X HBM3E
# Counter-derived HBM traffic per launch, committed under profiles/ together with
# the hash of the sources of the kernels they were taken on.
TRAFFIC = {
    "assign": (os.path.join(ROOT, "profiles", "assign_gemm_llama8b_bf16_T32768_traffic.json"),
               ("paper_2609_36835_amd/csrc/gemm_big.hpp", "paper_2609_36835_amd/csrc/gemm.hip",
                "paper_2609_36835_amd/csrc/common.hpp")),
    "score_select": (os.path.join(ROOT, "profiles", "score_select_llama8b_bf16_T32768_traffic.json"),
                     ("paper_2609_36835_amd/csrc/score.hip", "paper_2609_36835_amd/csrc/select.hip",
                      "paper_2609_36835_amd/csrc/common.hpp")),
}


def copy_calibration():
    """A plain device copy of known size: its counter readings scale FETCH_SIZE / WRITE_SIZE to bytes."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": COPY_BYTES}), flush=True)


def sources_sha256(sources):
    import hashlib
    hsh = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(ROOT, rel), "rb") as f:
            hsh.update(f.read())
    return hsh.hexdigest()


def measured_traffic(which, wl):
    """HBM bytes per launch from the committed counter runs, or None when the kernels' sources have changed
    since they were taken (or the workload differs)."""
    path, sources = TRAFFIC[which]
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != wl.name or rec.get("source_sha256") != sources_sha256(sources):
        return None
    return rec.get("traffic_bytes_per_launch")


def stage_rooflines(wl, t, stages, steps, refine_steps=2, bias_mode=0, value_refine_steps=1):
    """Per-stage roofline.  `algorithmic_*` is the method's own work for all pairs (the flops of a contraction,
    or the HBM bytes a stage must move), and `frac` prices it at the arithmetic's peak over the stage's
    event-timed duration per step.  Where the implementation issues more than that, `issued_*` / `issued_frac`
    report what it runs:
      - the Grams and the value right-hand side on split bf16 operands issue three bf16 products per term;
      - the Cholesky factorisations run their bulk (the left-looking updates and the strip below each diagonal
        block) on split fp16 planes of L, three fp16 products per term, so they are priced at the fp16 peak;
      - the two solves include `refine_steps` (mass fit) and `value_refine_steps` refinement steps against the
        data (each a residual and another solve), which the method itself does not need: its solve is one forward and one backward triangular
        sweep (mass fit: L read twice, 4 t^2 bytes per pair; value fit: 2 t^2 d flops per pair);
      - the profile pass materialises E^T (2 bytes per entry) for the assignment contraction: its algorithmic work
        is the logit contraction (2 n T d flops), the store is the implementation's.
    The assignment passes after the contraction (finalize, refine, exact) and the precise anchor profiles are
    the certification of the argmax; they are reported by time.  With the exact non-negative fit (bias_mode 1)
    the beta solve is a data-dependent number of pivoting iterations and is not priced."""
    B, T, n, d = wl.pairs, wl.T, wl.n, wl.d
    esz = 2 if wl.dtype == "bf16" else 4
    r, rv = refine_steps, value_refine_steps
    split = 3.0 if wl.dtype == "bf16" else 1.0
    work = {   # stage: (unit, algorithmic amount for all pairs, peak, issued amount or None)
        "rowstats": ("flop", 4.0 * n * T * d * B, PEAK_BF16_TFLOPS, None),
        "profiles": ("flop", 2.0 * n * T * d * B, PEAK_BF16_TFLOPS, None),
        "anchor_profiles": ("flop", 2.0 * n * t * d * B, PEAK_BF16_TFLOPS, None),
        "assign_gemm": ("flop", assign_flops(wl, t), PEAK_BF16_TFLOPS, None),
        "merge": ("byte", (T * d * esz + 8 * T + 2 * t * d * 4) * B, PEAK_HBM_GBS, None),
        "phic": ("flop", 2.0 * n * t * d * B, PEAK_BF16_TFLOPS, None),
        "gram_G": ("flop", 1.0 * n * t * (t + 1) * B, PEAK_BF16_TFLOPS, split * n * t * (t + 1) * B),
        "chol_G": ("flop", t ** 3 / 3.0 * B, PEAK_BF16_TFLOPS, 3.0 * t ** 3 / 3.0 * B),
        "solve_beta": ("byte", 4.0 * t * t * B, PEAK_HBM_GBS,
                       ((r + 1) * 4.0 * t * t + r * 2 * 4.0 * t * n) * B),
        "phat": ("byte", (2 * 4.0 * t * n + 4 * 2.0 * t * n) * B, PEAK_HBM_GBS, None),
        "gram_A": ("flop", 1.0 * n * t * (t + 1) * B, PEAK_BF16_TFLOPS, split * n * t * (t + 1) * B),
        "rhs_B": ("flop", 2.0 * n * t * d * B, PEAK_BF16_TFLOPS, split * 2.0 * n * t * d * B),
        "chol_A": ("flop", t ** 3 / 3.0 * B, PEAK_BF16_TFLOPS, 3.0 * t ** 3 / 3.0 * B),
        "solve_values": ("flop", 2.0 * t * t * d * B, PEAK_FP32_TFLOPS,
                         ((rv + 1) * 2.0 * t * t * d + rv * 2 * 2.0 * n * t * d) * B),
    }
    out = {}
    if bias_mode == 1:
        del work["solve_beta"]
        ms, cnt = stages.get("solve_beta", (0.0, 0))
        if cnt:
            out["solve_beta"] = {"ms": round(ms / steps, 3),
                                 "note": "exact NNLS: pivoting iterations depend on the data; not priced"}
    for name, (unit, amount, peak, issued) in work.items():
        ms, cnt = stages.get(name, (0.0, 0))
        if not cnt:
            continue
        sec = ms / 1e3 / steps
        scale, u, b = (1e12, "TFLOP/s", "mfma") if unit == "flop" else (1e9, "GB/s", "hbm")
        ach = amount / sec / scale
        key = "algorithmic_tflop" if unit == "flop" else "algorithmic_gb"
        e = {"bound": b, "ms": round(ms / steps, 3), key: round(amount / scale, 3), "achieved": round(ach, 1),
             "peak": peak, "unit": u, "frac": round(ach / peak, 4)}
        if issued is not None:
            e["issued_" + key.split("_")[1]] = round(issued / scale, 3)
            e["issued_frac"] = round(issued / sec / scale / peak, 4)
        out[name] = e
    for name in ("assign_finalize", "assign_refine", "assign_exact", "zmax", "score", "select"):
        ms, cnt = stages.get(name, (0.0, 0))
        if cnt and name not in out:
            out[name] = {"ms": round(ms / steps, 3)}
    return out


def quality(wl, t, outs, pairs=(0, -1)):
    """Diagnostics of the compaction on sampled pairs (float64, from the GPU's outputs; not gated):
    the mass-fit residual E_mass = ||Phi_C w* - m|| / ||m|| (w* = exp(beta)) of eq. mass_fit, the mean per-row
    relative l2 error against full attention on Q_ref and on 256 held-out queries, and the same errors of the
    hard-subset baseline (attention over the t selected tokens' own keys and values, no bias)."""
    import oracle
    anchors = outs[0].cpu().numpy().astype(np.int64)
    Ck, beta, Cv = (x.cpu().double().numpy() for x in outs[1:])
    s = 1.0 / math.sqrt(wl.d)
    res = []
    for b in pairs:
        b = b % wl.pairs
        layer, head = synth.pair_index(wl, b)
        p = synth.pair_inputs(wl, layer, head)
        K, V, Q = (p[k].astype(np.float64) for k in ("K", "V", "Q"))
        Qh = synth.heldout_queries(wl, layer, head).astype(np.float64)
        z, m, Y = oracle.rowstats(Q, K, V, s)
        Oh = oracle.attend_full(Qh, K, V, s)
        PhiC = oracle.phi_c(Q, Ck[b], z, s)
        e_mass = float(np.linalg.norm(PhiC @ np.exp(beta[b]) - m) / np.linalg.norm(m))
        S = anchors[b]
        comp_ref = oracle.row_rel_err(oracle.attend_compact(Q, Ck[b], beta[b], Cv[b], s), Y).mean()
        comp_held = oracle.row_rel_err(oracle.attend_compact(Qh, Ck[b], beta[b], Cv[b], s), Oh).mean()
        hard_ref = oracle.row_rel_err(oracle.attend_full(Q, K[S], V[S], s), Y).mean()
        hard_held = oracle.row_rel_err(oracle.attend_full(Qh, K[S], V[S], s), Oh).mean()
        res.append({"pair": b, "E_mass": round(e_mass, 5), "rel_l2_ref": round(float(comp_ref), 5),
                    "rel_l2_heldout": round(float(comp_held), 5), "hard_subset_rel_l2_ref": round(float(hard_ref), 5),
                    "hard_subset_rel_l2_heldout": round(float(hard_held), 5)})
        log(f"[quality] pair {b}: {res[-1]}")
    return res


def score_select_bytes(wl, t):
    """Algorithmic HBM bytes of scoring + selection for all pairs: read K and V, write the scores, read them
    back, write the anchors."""
    esz = 2 if wl.dtype == "bf16" else 4
    return wl.pairs * (wl.T * (2 * wl.d * esz + 4 + 4) + 4 * t)


DECODE_CONTEXTS = (4096, 8192, 16384, 32768)


def decode_bench(reps=20, warmup=3):
    """One decode step of attention for one layer at batch 64 (64 sequences x 8 KV heads = 512 pairs, 4 query
    heads per KV head): full-cache attention (C_k = K, C_v = V, no bias) against the compact cache at rho = 0.2
    with its bias, both through arckv_attend.  Synthetic bf16 caches; returns one JSON-able dict."""
    import torch
    from paper_2609_36835_amd import arckv
    dev = torch.device("cuda:0")
    P, G, d = 64 * 8, 4, 128
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    rows = []
    for T in DECODE_CONTEXTS:
        t = arckv.budget(T, 0.2)
        res = {"context": T, "t": t}
        for label, L, with_beta in (("full", T, False), ("compact", t, True)):
            K = torch.randn(P, L, d, device=dev, dtype=torch.bfloat16, generator=g)
            V = torch.randn(P, L, d, device=dev, dtype=torch.bfloat16, generator=g)
            Q = torch.randn(P, G, d, device=dev, dtype=torch.bfloat16, generator=g)
            beta = (torch.rand(P, L, device=dev, generator=g) * 6 - 3) if with_beta else None
            att = arckv.Attender(P, G, L, 0, dev)
            for _ in range(warmup):
                att(Q, K, beta, V)
            torch.cuda.synchronize()
            arckv.reset_timing()
            arckv.set_timing(True)
            for _ in range(reps):
                att(Q, K, beta, V)
            torch.cuda.synchronize()
            arckv.set_timing(False)
            ms, cnt = arckv.stage_times()["attend"]
            us = 1e3 * ms / cnt
            nbytes = P * L * d * 2 * 2 + (P * L * 4 if with_beta else 0) + P * G * d * (2 + 4)
            res[f"{label}_us"] = round(us, 2)
            res[f"{label}_GBps"] = round(nbytes / (us * 1e-6) / 1e9, 1)
            res[f"{label}_hbm_frac"] = round(nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)
            log(f"[decode] T={T} {label}: L={L} {us:.1f} us/layer, {res[f'{label}_GBps']:.0f} GB/s")
            del K, V, Q, beta, att
            torch.cuda.empty_cache()
        res["speedup"] = round(res["full_us"] / res["compact_us"], 3)
        res["ms_per_token_32_layers"] = {"full": round(32 * res["full_us"] / 1e3, 3),
                                         "compact": round(32 * res["compact_us"] / 1e3, 3)}
        rows.append(res)
    return {"metric": "decode attention latency per layer (batch 64, Llama-3.1-8B shapes, rho = 0.2 compact cache "
                      "with fitted bias vs full cache)", "unit": "us", "higher_is_better": False, "n_gpus": 1,
            "dtype": "bf16", "data": "synthetic (random bf16 caches and queries)",
            "config": {"workload": "decode_b64_llama8b", "pairs": P, "query_heads_per_kv": G, "rho": 0.2},
            "kernel": "k_attend_partial<4> + k_attend_combine", "peak_hbm_GBps": PEAK_HBM_GBS, "rows": rows}


def dsa_bench(wl, steps=3, warmup=1):
    """The value-aware indexer (Appendix A.1, H_I = 8, d_I = d_A = 128, d_x = 4096) on the workload's caches:
    pooled scores for every pair, then the whole compaction on those scores.  Random weights (std 1/sqrt(fan-in),
    value path active) and random activations X_ref [layers][n_pos][4096]."""
    import torch
    from paper_2609_36835_amd import arckv
    dev = torch.device("cuda:0")
    K, V, Q, _, _, _, _ = load_inputs(wl, dev)
    B, T, n, d = wl.pairs, wl.T, wl.n, wl.d
    dx, n_pos = 4096, wl.n_pos
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    r = lambda *sh, std: (torch.randn(*sh, device=dev, generator=g) * std).to(torch.bfloat16)
    P = {"L_q": r(B, 1024, d, std=d ** -0.5), "L_k": r(B, 1024, d, std=d ** -0.5), "L_x": r(B, 8, dx, std=dx ** -0.5),
         "b_x": torch.zeros(B, 8, device=dev), "U_q": r(B, 128, d, std=d ** -0.5), "U_k": r(B, 128, d, std=d ** -0.5),
         "U_v": r(B, 128, d, std=d ** -0.5), "L_c": r(B, 1024, 128, std=128 ** -0.5),
         "L_v": r(B, 1024, d, std=d ** -0.5)}
    X = r(wl.layers, n_pos, dx, std=1.0)
    prob = arckv.problem(K, Q)
    ix = arckv.dsa_indexer(X, P, n_pos, x_group=wl.kv_heads)
    ws_bytes = arckv.dsa_workspace_size(prob)
    ws = arckv._workspace(ws_bytes, dev)
    scores = torch.empty(B, T, dtype=torch.float32, device=dev)
    import ctypes
    call = lambda: arckv._check(arckv.lib().arckv_score_dsa(ctypes.byref(prob), arckv._ptr(K), arckv._ptr(V),
                                                              arckv._ptr(Q), ctypes.byref(ix), arckv._ptr(scores),
                                                              arckv._ptr(ws), ws_bytes, arckv._stream()),
                                "arckv_score_dsa")
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    arckv.reset_timing()
    arckv.set_timing(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    score_ms = (time.perf_counter() - t0) / steps * 1e3
    arckv.set_timing(False)
    st = {k: v[0] / steps for k, v in arckv.stage_times().items() if v[1]}
    index_flops = 2 * 2.0 * n * T * 1024 * B          # two passes of n x T x (H_I d_I) multiply-adds
    idx_tf = index_flops / (st["dsa_index"] / 1e3) / 1e12
    del ws
    torch.cuda.empty_cache()
    # the compaction on these scores
    comp = arckv.Compactor(B, T, n, wl.rho, K.dtype, dev, scale=1.0 / math.sqrt(d))
    import ctypes as C
    def compact_call():
        t_out = C.c_int32()
        arckv._check(arckv.lib().arckv_compact_scored(C.byref(comp.prob), arckv._ptr(K), arckv._ptr(V), arckv._ptr(Q),
                                                       arckv._ptr(scores), comp.rho, C.byref(comp.params),
                                                       C.byref(t_out), arckv._ptr(comp.anchors), arckv._ptr(comp.C_k),
                                                       arckv._ptr(comp.beta), arckv._ptr(comp.C_v),
                                                       arckv._ptr(comp.info), arckv._ptr(comp.ws), comp.ws_bytes,
                                                       arckv._stream()), "arckv_compact_scored")
    compact_call()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        compact_call()
    torch.cuda.synchronize()
    comp_ms = (time.perf_counter() - t0) / steps * 1e3
    total = score_ms + comp_ms
    return {"metric": "full-cache tokens compacted/sec per MI355X with the value-aware indexer "
                      "(Llama-3.1-8B shapes, 10% kept)", "value": round(T / (total / 1e3), 2), "unit": "tokens/s",
            "n_gpus": 1, "steps": steps, "ms_per_step": round(total, 3), "higher_is_better": True, "dtype": "bf16",
            "data": "synthetic caches; random indexer weights and activations",
            "config": {"workload": wl.name + "_dsa", "pairs": B, "T": T, "n_ref": n, "d_x": dx, "H_I": 8, "d_I": 128},
            "score_ms": round(score_ms, 3), "compact_ms": round(comp_ms, 3),
            "stage_ms": {k: round(v, 3) for k, v in st.items()},
            "roofline_index": {"bound": "mfma", "kernel": "k_dsa_index<1> + k_dsa_index<2>",
                               "achieved": round(idx_tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                               "frac": round(idx_tf / PEAK_BF16_TFLOPS, 4),
                               "algorithmic_flops_per_step": index_flops}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default=HEADLINE, choices=sorted(synth.WORKLOADS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pair-chunk", type=int, default=0)
    ap.add_argument("--select-chunk", type=int, default=0,
                    help="chunked anchor selection (chunks of this many positions when T > 10000); 0 = global top-t")
    ap.add_argument("--bias-mode", type=int, default=0, choices=(0, 1),
                    help="mass fit: 0 = projected least squares (the paper's), 1 = exact non-negative least squares")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (3 times), the reference kernel that scales the "
                         "FETCH_SIZE / WRITE_SIZE counters to bytes")
    ap.add_argument("--decode", action="store_true",
                    help="instead of compaction, time decode attention over full and compact caches (batch 64)")
    ap.add_argument("--dsa", action="store_true",
                    help="score with the value-aware indexer (arckv_score_dsa) and compact on those scores")
    args = ap.parse_args()
    if args.dsa:
        import synth as _s
        print(json.dumps(dsa_bench(_s.WORKLOADS[args.workload])), flush=True)
        return
    if args.decode:
        print(json.dumps(decode_bench()), flush=True)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one MI355X: the compaction path has no multi-GPU mode "
              "(pairs shard across GPUs with no communication); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_36835_amd import arckv

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wl = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    log(f"[bench] workload {wl.name}: pairs={wl.pairs} T={wl.T} n={wl.n} rho={wl.rho} dtype={wl.dtype}")
    K, V, Q, W1, b1, w2, b2 = load_inputs(wl, dev)
    params = arckv.default_params(pair_chunk=args.pair_chunk, select_chunk=args.select_chunk,
                                  bias_mode=args.bias_mode)
    comp = arckv.Compactor(wl.pairs, wl.T, wl.n, wl.rho, K.dtype, dev, scale=1.0 / math.sqrt(wl.d), params=params)
    t = comp.t
    log(f"[bench] t={t}, workspace {comp.ws_bytes / 2**30:.1f} GiB")

    for i in range(args.warmup):
        comp(K, V, Q, W1, b1, w2, b2)
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    info = comp.info.cpu()
    if int(info.abs().sum()) != 0:
        log(f"[bench] WARNING: nonzero fit status in {int((info != 0).sum())} entries")

    arckv.reset_timing()
    arckv.set_timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        comp(K, V, Q, W1, b1, w2, b2)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    arckv.set_timing(False)
    stages = arckv.stage_times()
    ms_per_step = 1e3 * elapsed / args.steps
    value = wl.T * args.steps / elapsed
    log(f"[bench] {args.steps} steps in {elapsed:.3f}s: {ms_per_step:.2f} ms/step, {value:.1f} tokens/s")
    for name, (ms, cnt) in stages.items():
        if cnt:
            log(f"    {name:16s} {ms / args.steps:9.3f} ms/step  ({cnt} launches)")

    ms_assign, cnt_assign = stages["assign_gemm"]
    avg_launch_s = ms_assign / 1e3 / max(cnt_assign, 1)
    launches_per_step = max(cnt_assign // args.steps, 1)
    flops_per_launch = assign_flops(wl, t) / launches_per_step
    achieved = flops_per_launch / avg_launch_s / 1e12
    roofline = {"bound": "mfma", "kernel": "k_gemm_big<4,2,2,4,64,1,1,2,f16,EpiArgmaxBig> (key-to-anchor assignment, "
                                      "fp16 operands)",
                "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic("assign", wl),
                "avg_launch_ms": round(avg_launch_s * 1e3, 3),
                "algorithmic_flops_per_launch": flops_per_launch}
    # scoring + selection against HBM: algorithmic bytes / (score + select launch durations)
    ms_sc, cnt_sc = stages["score"]
    ms_se, cnt_se = stages["select"]
    ss_s = (ms_sc / max(cnt_sc, 1) + ms_se / max(cnt_se, 1)) / 1e3
    ss_bytes = score_select_bytes(wl, t)
    ss_gbs = ss_bytes / ss_s / 1e9
    roofline_ss = {"bound": "hbm", "kernel": "k_score_bf16 + k_select_topt (scoring and top-t selection)",
                   "achieved": round(ss_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                   "frac": round(ss_gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("score_select", wl),
                   "avg_launch_ms": round(ss_s * 1e3, 4), "algorithmic_bytes_per_launch": ss_bytes}

    st = comp.assign_stats().cpu().numpy()
    keys = wl.pairs * max(1, wl.T - t)
    assign_stats = {"flagged_frac": round(float(st[:, 0].sum()) / keys, 5),
                    "float64_frac": round(float(st[:, 1].sum()) / keys, 6),
                    "candidates_per_flagged": round(float(st[:, 2].sum()) / max(1, int(st[:, 0].sum())), 3),
                    "undecided": int(st[:, 3].sum())}
    outs = [x.clone() for x in (comp.anchors, comp.C_k, comp.beta, comp.C_v)]
    cpu = None
    qual = None
    if not args.no_cpu_baseline:
        del K, V, Q, comp
        torch.cuda.empty_cache()
        qual = quality(wl, t, outs)
        cpu = cpu_baseline(wl, t)

    out = {
        "metric": "full-cache tokens compacted/sec per MI355X (Llama-3.1-8B shapes, 10% kept)",
        "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic (seeded Gaussian K/V/Q_ref with RoPE and outlier key channels; "
                                  "random-init scoring MLP)",
        "config": {"workload": wl.name, "pairs": wl.pairs, "layers": wl.layers, "kv_heads": wl.kv_heads,
                   "T": wl.T, "n_ref": wl.n, "t": t, "rho": wl.rho, "head_dim": wl.d,
                   "pair_chunk": args.pair_chunk or wl.pairs, "select_chunk": args.select_chunk,
                   "bias_mode": args.bias_mode},
        "roofline": roofline,
        "roofline_score_select": roofline_ss,
        "cpu_baseline": cpu,
        "stage_ms_per_step": {k: round(v[0] / args.steps, 3) for k, v in stages.items() if v[1]},
        "stage_roofline": stage_rooflines(wl, t, stages, args.steps, params.refine_steps, args.bias_mode,
                                          params.value_refine_steps),
        "assignment": assign_stats,
        "quality": qual,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
