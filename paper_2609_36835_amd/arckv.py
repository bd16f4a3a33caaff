"""Python binding of libarckv.so (ctypes): argument marshalling only.

Every function mirrors the C entry point of the same name in include/arckv.h.
Tensors must be CUDA (HIP) tensors, contiguous, of the documented dtype; the
work is enqueued on torch's current stream.  Nothing here computes any part
of the compaction: if the library is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libarckv.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, 1, 2, 3, 4
F32, BF16 = 0, 1

# Every entry point declared in include/arckv.h.
ENTRY_POINTS = (
    "arckv_default_params", "arckv_budget", "arckv_workspace_size", "arckv_score", "arckv_select",
    "arckv_rowstats", "arckv_merge", "arckv_fit_bias", "arckv_fit_values", "arckv_compact",
    "arckv_status_string", "arckv_set_timing", "arckv_stage_times", "arckv_reset_timing",
    "arckv_attend_workspace_size", "arckv_attend", "arckv_budgets", "arckv_select_count", "arckv_select_ex",
    "arckv_dsa_workspace_size", "arckv_score_dsa", "arckv_compact_scored", "arckv_assign_stats",
    "arckv_attend_noalloc",
)


class ArckvError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} (status {status})")
        self.status = status


class Problem(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("T", ctypes.c_int32), ("n", ctypes.c_int32), ("d", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("scale", ctypes.c_float)]


class Indexer(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("w1_dtype", ctypes.c_int32), ("W1", ctypes.c_void_p),
                ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p), ("b2", ctypes.c_void_p)]


class FitParams(ctypes.Structure):
    _fields_ = [("lambda_m", ctypes.c_float), ("delta_beta", ctypes.c_float), ("delta_v", ctypes.c_float),
                ("eps_w", ctypes.c_float), ("b_min", ctypes.c_float), ("b_max", ctypes.c_float),
                ("bias_mode", ctypes.c_int32), ("max_escalations", ctypes.c_int32),
                ("refine_steps", ctypes.c_int32), ("pair_chunk", ctypes.c_int32),
                ("select_chunk", ctypes.c_int32), ("nnls_max_iter", ctypes.c_int32),
                ("value_refine_steps", ctypes.c_int32)]


class DSAIndexer(ctypes.Structure):
    _fields_ = [("n_pos", ctypes.c_int32), ("d_x", ctypes.c_int32), ("x_group", ctypes.c_int32),
                ("scale_a", ctypes.c_float), ("X_ref", ctypes.c_void_p), ("L_q", ctypes.c_void_p),
                ("L_k", ctypes.c_void_p), ("L_x", ctypes.c_void_p), ("b_x", ctypes.c_void_p),
                ("U_q", ctypes.c_void_p), ("U_k", ctypes.c_void_p), ("U_v", ctypes.c_void_p),
                ("L_c", ctypes.c_void_p), ("L_v", ctypes.c_void_p)]


_LIB = None


def lib():
    """Load libarckv.so (built in-tree by paper_2609_36835_amd.build)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run `python -m paper_2609_36835_amd.build` first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        P = ctypes.POINTER
        L.arckv_default_params.argtypes = [P(FitParams)]
        L.arckv_budget.argtypes = [ctypes.c_int64, ctypes.c_double, P(i32)]
        L.arckv_workspace_size.argtypes = [P(Problem), i32, P(FitParams), P(sz)]
        L.arckv_score.argtypes = [P(Problem), vp, vp, P(Indexer), vp, vp]
        L.arckv_select.argtypes = [P(Problem), vp, i32, vp, vp, sz, vp]
        L.arckv_rowstats.argtypes = [P(Problem), vp, vp, vp, vp, vp, vp, vp]
        L.arckv_merge.argtypes = [P(Problem), vp, vp, vp, vp, i32, ctypes.c_float, vp, vp, vp, vp, sz, vp]
        L.arckv_fit_bias.argtypes = [P(Problem), vp, vp, vp, vp, i32, vp, vp, P(FitParams), vp, vp, vp, vp, sz, vp]
        L.arckv_fit_values.argtypes = [P(Problem), vp, vp, vp, vp, vp, i32, vp, P(FitParams), vp, vp, vp, vp, sz,
                                       vp]
        L.arckv_compact.argtypes = [P(Problem), vp, vp, vp, P(Indexer), ctypes.c_double, P(FitParams), P(i32),
                                    vp, vp, vp, vp, vp, vp, sz, vp]
        L.arckv_status_string.argtypes = [ctypes.c_int]
        L.arckv_status_string.restype = ctypes.c_char_p
        L.arckv_set_timing.argtypes = [i32]
        L.arckv_stage_times.argtypes = [i32, P(ctypes.c_char_p), P(ctypes.c_double), P(i32), P(i32)]
        L.arckv_reset_timing.argtypes = []
        L.arckv_attend_workspace_size.argtypes = [i32, i32, i32, i32, P(sz)]
        L.arckv_budgets.argtypes = [i32, P(ctypes.c_double), i32, ctypes.c_int64, P(i32)]
        L.arckv_select_count.argtypes = [ctypes.c_int64, i32, i32, P(i32)]
        L.arckv_select_ex.argtypes = [P(Problem), vp, i32, vp, i32, i32, vp, vp]
        L.arckv_dsa_workspace_size.argtypes = [P(Problem), i32, P(sz)]
        L.arckv_score_dsa.argtypes = [P(Problem), vp, vp, vp, P(DSAIndexer), vp, vp, sz, vp]
        L.arckv_compact_scored.argtypes = [P(Problem), vp, vp, vp, vp, ctypes.c_double, P(FitParams), P(i32),
                                           vp, vp, vp, vp, vp, vp, sz, vp]
        L.arckv_attend.argtypes = [i32, i32, i32, i32, ctypes.c_float, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.arckv_attend_noalloc.argtypes = [i32, i32, i32, i32, ctypes.c_float, vp, vp, vp, vp, vp, vp, vp, vp]
        L.arckv_assign_stats.argtypes = [P(Problem), i32, vp, sz, vp, vp]
        for name in ENTRY_POINTS:
            getattr(L, name).restype = ctypes.c_int if name != "arckv_status_string" else ctypes.c_char_p
        _LIB = L
    return _LIB


def status_string(status: int) -> str:
    return lib().arckv_status_string(int(status)).decode()


def _check(status: int, where: str):
    if status != OK:
        raise ArckvError(status, where)


def default_params(**overrides) -> FitParams:
    p = FitParams()
    _check(lib().arckv_default_params(ctypes.byref(p)), "arckv_default_params")
    for k, v in overrides.items():
        if not hasattr(p, k):
            raise KeyError(k)
        setattr(p, k, v)
    return p


def budget(T: int, rho: float) -> int:
    t = ctypes.c_int32()
    _check(lib().arckv_budget(int(T), float(rho), ctypes.byref(t)), "arckv_budget")
    return t.value


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return BF16
    if dt == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {dt}")


def problem(K: torch.Tensor, Q: torch.Tensor, scale: Optional[float] = None) -> Problem:
    B, T, d = K.shape
    n = Q.shape[1]
    return Problem(B, T, n, d, _dtype_code(K.dtype), float(scale) if scale else 0.0)


def problem_from_dims(B: int, T: int, n: int, d: int = 128, dtype: int = BF16, scale: float = 0.0) -> Problem:
    return Problem(B, T, n, d, dtype, scale)


def workspace_size(prob: Problem, t: int, params: Optional[FitParams] = None) -> int:
    out = ctypes.c_size_t()
    pp = ctypes.byref(params) if params is not None else None
    _check(lib().arckv_workspace_size(ctypes.byref(prob), int(t), pp, ctypes.byref(out)), "arckv_workspace_size")
    return out.value


def _ptr(x: Optional[torch.Tensor]):
    if x is None:
        return None
    if not x.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not x.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(x.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _workspace(nbytes: int, device) -> torch.Tensor:
    ws = torch.empty(max(nbytes, 256) + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + max(nbytes, 256)]


def indexer(W1, b1, w2, b2) -> Indexer:
    return Indexer(W1.shape[1], _dtype_code(W1.dtype), _ptr(W1), _ptr(b1), _ptr(w2), _ptr(b2))


def score(K, V, W1, b1, w2, b2, scale=None) -> torch.Tensor:
    prob = problem(K, K[:, :1], scale)
    out = torch.empty(K.shape[0], K.shape[1], dtype=torch.float32, device=K.device)
    ix = indexer(W1, b1, w2, b2)
    _check(lib().arckv_score(ctypes.byref(prob), _ptr(K), _ptr(V), ctypes.byref(ix), _ptr(out), _stream()),
           "arckv_score")
    return out


def select(scores: torch.Tensor, t: int) -> torch.Tensor:
    B, T = scores.shape
    prob = Problem(B, T, 1, 128, F32, 0.0)
    out = torch.empty(B, t, dtype=torch.int32, device=scores.device)
    _check(lib().arckv_select(ctypes.byref(prob), _ptr(scores), int(t), _ptr(out), None, 0, _stream()),
           "arckv_select")
    return out


def budgets(a, t: int, T: int):
    """eq. per_head_budget: per-pair budgets (host list) from weights a."""
    n = len(a)
    arr = (ctypes.c_double * n)(*[float(x) for x in a])
    out = (ctypes.c_int32 * n)()
    _check(lib().arckv_budgets(n, arr, int(t), int(T), out), "arckv_budgets")
    return list(out)


def select_count(T: int, t: int, chunk_len: int) -> int:
    out = ctypes.c_int32()
    _check(lib().arckv_select_count(int(T), int(t), int(chunk_len), ctypes.byref(out)), "arckv_select_count")
    return out.value


def select_ex(scores: torch.Tensor, t: int, t_pair: Optional[torch.Tensor] = None, chunk_len: int = 0,
              t_stride: Optional[int] = None) -> torch.Tensor:
    """Per-pair budgets (t_pair, int32 [B] on the GPU) and/or chunked selection; rows padded with -1."""
    B, T = scores.shape
    if t_stride is None:
        tmax = int(t_pair.max().item()) if t_pair is not None else t
        t_stride = select_count(T, tmax, chunk_len) + (B if t_pair is not None and chunk_len else 0)
    prob = Problem(B, T, 1, 128, F32, 0.0)
    out = torch.empty(B, t_stride, dtype=torch.int32, device=scores.device)
    _check(lib().arckv_select_ex(ctypes.byref(prob), _ptr(scores), int(t), _ptr(t_pair), int(chunk_len),
                                 int(t_stride), _ptr(out), _stream()), "arckv_select_ex")
    return out


def rowstats(K, V, Q, scale=None):
    prob = problem(K, Q, scale)
    B, n = Q.shape[0], Q.shape[1]
    z = torch.empty(B, n, dtype=torch.float32, device=K.device)
    m = torch.empty_like(z)
    Y = torch.empty(B, n, K.shape[2], dtype=torch.float32, device=K.device)
    _check(lib().arckv_rowstats(ctypes.byref(prob), _ptr(K), _ptr(V), _ptr(Q), _ptr(z), _ptr(m), _ptr(Y),
                                _stream()), "arckv_rowstats")
    return z, m, Y


def assign_stats(prob: Problem, t: int, ws: torch.Tensor, ws_bytes: int) -> torch.Tensor:
    """arckv_assign_stats: [B][8] int32 counters of the last assignment run on ws (include/arckv.h)."""
    out = torch.empty(prob.B, 8, dtype=torch.int32, device=ws.device)
    _check(lib().arckv_assign_stats(ctypes.byref(prob), int(t), _ptr(ws), int(ws_bytes), _ptr(out), _stream()),
           "arckv_assign_stats")
    return out


def merge(K, Q, z, anchors, lambda_m=0.25, scale=None, ws_bytes: Optional[int] = None, return_stats=False):
    prob = problem(K, Q, scale)
    t = anchors.shape[1]
    B, T, d = K.shape
    Ck = torch.empty(B, t, d, dtype=torch.float32, device=K.device)
    kappa = torch.empty(B, T, dtype=torch.int32, device=K.device)
    phi = torch.empty(B, T, dtype=torch.float32, device=K.device)
    nbytes = ws_bytes if ws_bytes is not None else workspace_size(prob, t)
    ws = _workspace(nbytes, K.device)
    _check(lib().arckv_merge(ctypes.byref(prob), _ptr(K), _ptr(Q), _ptr(z), _ptr(anchors), int(t), float(lambda_m),
                             _ptr(Ck), _ptr(kappa), _ptr(phi), _ptr(ws), nbytes, _stream()), "arckv_merge")
    if return_stats:
        return Ck, kappa, phi, assign_stats(prob, t, ws, nbytes)
    return Ck, kappa, phi


def fit_bias(Q, C_k, z, m, params: Optional[FitParams] = None, scale=None, T: Optional[int] = None, K=None, V=None):
    """arckv_fit_bias; z and m may be None when K and V are given (recomputed)."""
    B, n, d = Q.shape
    t = C_k.shape[1]
    if K is not None:
        T = K.shape[1]
    prob = Problem(B, T or max(t, 1), n, d, _dtype_code(Q.dtype), float(scale) if scale else 0.0)
    params = params or default_params()
    beta = torch.empty(B, t, dtype=torch.float32, device=Q.device)
    info = torch.empty(B, dtype=torch.int32, device=Q.device)
    dused = torch.empty(B, dtype=torch.float32, device=Q.device)
    nbytes = workspace_size(prob, t, params)
    ws = _workspace(nbytes, Q.device)
    _check(lib().arckv_fit_bias(ctypes.byref(prob), _ptr(K), _ptr(V), _ptr(Q), _ptr(C_k), int(t), _ptr(z), _ptr(m),
                                ctypes.byref(params), _ptr(beta), _ptr(info), _ptr(dused), _ptr(ws), nbytes,
                                _stream()), "arckv_fit_bias")
    return beta, info, dused


def fit_values(Q, C_k, beta, Y, params: Optional[FitParams] = None, scale=None, T: Optional[int] = None, K=None,
               V=None):
    """arckv_fit_values; Y may be None when K and V are given (recomputed)."""
    B, n, d = Q.shape
    t = C_k.shape[1]
    if K is not None:
        T = K.shape[1]
    prob = Problem(B, T or max(t, 1), n, d, _dtype_code(Q.dtype), float(scale) if scale else 0.0)
    params = params or default_params()
    Cv = torch.empty(B, t, d, dtype=torch.float32, device=Q.device)
    info = torch.empty(B, dtype=torch.int32, device=Q.device)
    dused = torch.empty(B, dtype=torch.float32, device=Q.device)
    nbytes = workspace_size(prob, t, params)
    ws = _workspace(nbytes, Q.device)
    _check(lib().arckv_fit_values(ctypes.byref(prob), _ptr(K), _ptr(V), _ptr(Q), _ptr(C_k), _ptr(beta), int(t),
                                  _ptr(Y), ctypes.byref(params), _ptr(Cv), _ptr(info), _ptr(dused), _ptr(ws), nbytes,
                                  _stream()), "arckv_fit_values")
    return Cv, info, dused


def attend_workspace_size(P: int, G: int, t: int, F: int) -> int:
    out = ctypes.c_size_t()
    _check(lib().arckv_attend_workspace_size(int(P), int(G), int(t), int(F), ctypes.byref(out)),
           "arckv_attend_workspace_size")
    return out.value


class Attender:
    """Holds the output and workspace for repeated arckv_attend calls of one shape."""

    def __init__(self, P, G, t, F=0, device="cuda", scale=None):
        self.P, self.G, self.t, self.F = int(P), int(G), int(t), int(F)
        self.scale = float(scale) if scale else 0.0
        dev = torch.device(device)
        self.out = torch.empty(self.P, self.G, 128, dtype=torch.float32, device=dev)
        self.ws_bytes = attend_workspace_size(self.P, self.G, self.t, self.F)
        self.ws = _workspace(self.ws_bytes, dev)

    def __call__(self, Q, C_k, beta, C_v, K_f=None, V_f=None):
        _check(lib().arckv_attend(self.P, self.G, self.t, self.F, self.scale, _ptr(Q), _ptr(C_k), _ptr(beta),
                                  _ptr(C_v), _ptr(K_f), _ptr(V_f), _ptr(self.out), _ptr(self.ws), self.ws_bytes,
                                  _stream()), "arckv_attend")
        return self.out


def attend(Q, C_k, beta, C_v, K_f=None, V_f=None, scale=None) -> torch.Tensor:
    """Decode attention softmax([s Q C_k^T + beta, s Q K_f^T]) [C_v; V_f] per pair:
    Q [P][G][128], C_k/C_v [P][t][128], beta [P][t] or None, K_f/V_f [P][F][128] or None (bf16; beta fp32)."""
    P, G, _ = Q.shape
    t = C_k.shape[1] if C_k is not None else 0
    F = K_f.shape[1] if K_f is not None else 0
    return Attender(P, G, t, F, Q.device, scale)(Q, C_k, beta, C_v, K_f, V_f)


def attend_noalloc(Q, C_k, beta, C_v, K_f=None, V_f=None, scale=None, out=None) -> torch.Tensor:
    """arckv_attend_noalloc: attend() without a workspace (the library's static per-GPU scratch holds the
    partials).  out [P][G][128] float32 may be given; else it is allocated here, by the caller's side."""
    P, G, _ = Q.shape
    t = C_k.shape[1] if C_k is not None else 0
    F = K_f.shape[1] if K_f is not None else 0
    if out is None:
        out = torch.empty(P, G, 128, dtype=torch.float32, device=Q.device)
    _check(lib().arckv_attend_noalloc(int(P), int(G), int(t), int(F), float(scale) if scale else 0.0, _ptr(Q),
                                      _ptr(C_k), _ptr(beta), _ptr(C_v), _ptr(K_f), _ptr(V_f), _ptr(out), _stream()),
           "arckv_attend_noalloc")
    return out


DSA_FIELDS = ("L_q", "L_k", "L_x", "b_x", "U_q", "U_k", "U_v", "L_c", "L_v")


def dsa_indexer(X_ref, params: dict, n_pos: int, x_group: int = 1, scale_a: Optional[float] = None) -> DSAIndexer:
    """params: tensors L_q, L_k, L_c, L_v [B][1024][128], U_q/U_k/U_v [B][128][128], L_x [B][8][d_x] (bf16) and
    b_x [B][8] (fp32); X_ref [B / x_group][n_pos][d_x] bf16."""
    return DSAIndexer(int(n_pos), int(X_ref.shape[-1]), int(x_group), float(scale_a) if scale_a else 0.0,
                      _ptr(X_ref), *[_ptr(params[k]) for k in DSA_FIELDS])


def dsa_workspace_size(prob: Problem, pair_chunk: int = 0) -> int:
    out = ctypes.c_size_t()
    _check(lib().arckv_dsa_workspace_size(ctypes.byref(prob), int(pair_chunk), ctypes.byref(out)),
           "arckv_dsa_workspace_size")
    return out.value


def score_dsa(K, V, Q, X_ref, params: dict, n_pos: int, x_group: int = 1, scale_a=None, pair_chunk: int = 0):
    """Pooled value-aware-indexer scores [B][T] (arckv_score_dsa)."""
    prob = problem(K, Q)
    ix = dsa_indexer(X_ref, params, n_pos, x_group, scale_a)
    out = torch.empty(K.shape[0], K.shape[1], dtype=torch.float32, device=K.device)
    nbytes = dsa_workspace_size(prob, pair_chunk)
    ws = _workspace(nbytes, K.device)
    _check(lib().arckv_score_dsa(ctypes.byref(prob), _ptr(K), _ptr(V), _ptr(Q), ctypes.byref(ix), _ptr(out), _ptr(ws),
                                 nbytes, _stream()), "arckv_score_dsa")
    return out


def compact_scored(K, V, Q, scores, rho, scale=None, params: Optional[FitParams] = None):
    """arckv_compact_scored: the compaction path on given scores; returns (anchors, C_k, beta, C_v, info)."""
    B, T, _ = K.shape
    c = Compactor(B, T, Q.shape[1], rho, K.dtype, K.device, scale, params)
    t_out = ctypes.c_int32()
    _check(lib().arckv_compact_scored(ctypes.byref(c.prob), _ptr(K), _ptr(V), _ptr(Q), _ptr(scores), c.rho,
                                      ctypes.byref(c.params), ctypes.byref(t_out), _ptr(c.anchors), _ptr(c.C_k),
                                      _ptr(c.beta), _ptr(c.C_v), _ptr(c.info), _ptr(c.ws), c.ws_bytes, _stream()),
           "arckv_compact_scored")
    return c.anchors, c.C_k, c.beta, c.C_v, c.info


class Compactor:
    """Holds output buffers and the workspace for repeated arckv_compact calls."""

    def __init__(self, B, T, n, rho, dtype=torch.bfloat16, device="cuda", scale=None,
                 params: Optional[FitParams] = None):
        self.prob = Problem(B, T, n, 128, _dtype_code(dtype), float(scale) if scale else 0.0)
        self.rho = float(rho)
        self.params = params or default_params()
        self.t = budget(T, rho)
        if self.params.select_chunk:
            self.t = select_count(T, self.t, self.params.select_chunk)
        dev = torch.device(device)
        self.anchors = torch.empty(B, self.t, dtype=torch.int32, device=dev)
        self.C_k = torch.empty(B, self.t, 128, dtype=torch.float32, device=dev)
        self.beta = torch.empty(B, self.t, dtype=torch.float32, device=dev)
        self.C_v = torch.empty(B, self.t, 128, dtype=torch.float32, device=dev)
        self.info = torch.empty(B, 2, dtype=torch.int32, device=dev)
        self.ws_bytes = workspace_size(self.prob, self.t, self.params)
        self.ws = _workspace(self.ws_bytes, dev)

    def __call__(self, K, V, Q, W1, b1, w2, b2):
        ix = indexer(W1, b1, w2, b2)
        t_out = ctypes.c_int32()
        _check(lib().arckv_compact(ctypes.byref(self.prob), _ptr(K), _ptr(V), _ptr(Q), ctypes.byref(ix), self.rho,
                                   ctypes.byref(self.params), ctypes.byref(t_out), _ptr(self.anchors),
                                   _ptr(self.C_k), _ptr(self.beta), _ptr(self.C_v), _ptr(self.info),
                                   _ptr(self.ws), self.ws_bytes, _stream()), "arckv_compact")
        assert t_out.value == self.t
        return self.anchors, self.C_k, self.beta, self.C_v, self.info

    def assign_stats(self) -> torch.Tensor:
        """[B][8] assignment counters of the last call (arckv_assign_stats)."""
        return assign_stats(self.prob, self.t, self.ws, self.ws_bytes)


def compact(K, V, Q, W1, b1, w2, b2, rho, scale=None, params: Optional[FitParams] = None, return_stats=False):
    """One-shot arckv_compact: returns (anchors, C_k, beta, C_v, info) (+ assignment stats)."""
    B, T, _ = K.shape
    c = Compactor(B, T, Q.shape[1], rho, K.dtype, K.device, scale, params)
    out = c(K, V, Q, W1, b1, w2, b2)
    return (*out, c.assign_stats()) if return_stats else out


def set_timing(enable: bool):
    _check(lib().arckv_set_timing(1 if enable else 0), "arckv_set_timing")


def reset_timing():
    _check(lib().arckv_reset_timing(), "arckv_reset_timing")


def stage_times() -> dict:
    n = 64
    names = (ctypes.c_char_p * n)()
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int32 * n)()
    ns = ctypes.c_int32()
    _check(lib().arckv_stage_times(n, names, ms, cnt, ctypes.byref(ns)), "arckv_stage_times")
    return {names[i].decode(): (ms[i], cnt[i]) for i in range(ns.value)}
