"""The C ABI on a machine without a GPU: the library loads, exports every
declared entry point, and rejects bad arguments before touching HIP."""
import ctypes
import os
import re

import pytest

from paper_2609_36835_amd import arckv as A

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "arckv.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(arckv_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 14
    lib = ctypes.CDLL(A.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(A.ENTRY_POINTS)


def test_budget():
    assert A.budget(1024, 0.1) == 102
    assert A.budget(131072, 0.01) == 1311
    assert A.budget(32768, 0.1) == 3277
    assert A.budget(16384, 0.02) == 328
    assert A.budget(10, 0.0) == 1
    assert A.budget(10, 3.0) == 10
    for T, rho in [(0, 0.1), (10, -0.1), (10, float("nan")), (10, float("inf"))]:
        with pytest.raises(A.ArckvError) as e:
            A.budget(T, rho)
        assert e.value.status == A.ERR_INVALID_ARG


def test_budget_matches_oracle():
    import oracle
    for T in (1, 7, 100, 1024, 8191, 32768, 131072):
        for rho in (0.001, 0.01, 0.02, 0.05, 0.1, 0.2, 0.5, 1.0):
            assert A.budget(T, rho) == oracle.budget(T, rho)


def test_status_strings():
    for s in range(5):
        assert A.status_string(s)
    assert A.status_string(99) == "unknown status"


def test_default_params():
    p = A.default_params()
    assert p.lambda_m == pytest.approx(0.25) and p.delta_beta == pytest.approx(1e-6)
    assert p.delta_v == pytest.approx(1e-3) and p.eps_w == pytest.approx(1e-12)
    assert (p.b_min, p.b_max, p.bias_mode, p.max_escalations, p.refine_steps, p.value_refine_steps) == \
        (-30.0, 30.0, 0, 6, 2, 1)
    assert (p.pair_chunk, p.select_chunk, p.nnls_max_iter) == (0, 0, 32)


def ws(prob, t, params=None):
    return A.workspace_size(prob, t, params)


def test_workspace_validation_and_monotonicity():
    p = A.problem_from_dims(8, 8192, 4096)
    full = ws(p, 819)
    half = ws(p, 819, A.default_params(pair_chunk=4))
    one = ws(p, 819, A.default_params(pair_chunk=1))
    assert full > half > one > 0
    assert ws(A.problem_from_dims(8, 8192, 4096, dtype=A.F32), 819) > full   # fp32 profiles are wider
    bad = [
        (A.problem_from_dims(8, 8192, 4096, d=64), 819, A.ERR_UNSUPPORTED),
        (A.problem_from_dims(8, 8192, 4096, dtype=7), 819, A.ERR_UNSUPPORTED),
        (A.problem_from_dims(0, 8192, 4096), 819, A.ERR_INVALID_ARG),
        (A.problem_from_dims(8, 0, 4096), 1, A.ERR_INVALID_ARG),
        (A.problem_from_dims(8, 8192, 0), 819, A.ERR_INVALID_ARG),
        (A.problem_from_dims(8, 8192, 4096), 0, A.ERR_INVALID_ARG),
        (A.problem_from_dims(8, 8192, 4096), 8193, A.ERR_INVALID_ARG),
    ]
    for prob, t, code in bad:
        with pytest.raises(A.ArckvError) as e:
            ws(prob, t)
        assert e.value.status == code


@pytest.mark.parametrize("field,value,code", [
    ("lambda_m", 1.5, A.ERR_INVALID_ARG), ("lambda_m", -0.1, A.ERR_INVALID_ARG),
    ("delta_beta", -1.0, A.ERR_INVALID_ARG), ("delta_v", float("nan"), A.ERR_INVALID_ARG),
    ("eps_w", 0.0, A.ERR_INVALID_ARG), ("b_min", 40.0, A.ERR_INVALID_ARG),
    ("bias_mode", 2, A.ERR_UNSUPPORTED), ("bias_mode", -1, A.ERR_UNSUPPORTED),
    ("nnls_max_iter", 0, A.ERR_INVALID_ARG), ("nnls_max_iter", 257, A.ERR_INVALID_ARG),
    ("max_escalations", 7, A.ERR_INVALID_ARG),
    ("refine_steps", -1, A.ERR_INVALID_ARG), ("value_refine_steps", 5, A.ERR_INVALID_ARG),
    ("pair_chunk", -2, A.ERR_INVALID_ARG),
])
def test_param_validation(field, value, code):
    p = A.problem_from_dims(2, 1024, 256)
    with pytest.raises(A.ArckvError) as e:
        ws(p, 102, A.default_params(**{field: value}))
    assert e.value.status == code


def test_entry_points_reject_bad_arguments_without_gpu():
    """Every error below is returned before any HIP call (no GPU here)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("fake-pointer validation test runs only where no GPU is visible")
    L = A.lib()
    prob = A.Problem(2, 1024, 256, 128, A.BF16, 0.0)
    # Fake device pointers: every case below must fail validation, so nothing is
    # ever launched with them (this test also runs on GPU machines).
    fake = ctypes.c_void_p(0x1000)
    odd = ctypes.c_void_p(0x1001)
    ix = A.Indexer(64, A.BF16, fake, fake, fake, fake)
    bad_ix = A.Indexer(32, A.BF16, fake, fake, fake, fake)
    par = A.default_params()
    t_out = ctypes.c_int32()
    r = ctypes.byref
    cases = [
        (L.arckv_score(None, fake, fake, r(ix), fake, None), A.ERR_INVALID_ARG),
        (L.arckv_score(r(prob), None, fake, r(ix), fake, None), A.ERR_INVALID_ARG),
        (L.arckv_score(r(prob), fake, fake, r(bad_ix), fake, None), A.ERR_UNSUPPORTED),
        (L.arckv_score(r(prob), odd, fake, r(ix), fake, None), A.ERR_INVALID_ARG),
        (L.arckv_select(r(prob), fake, 0, fake, None, 0, None), A.ERR_INVALID_ARG),
        (L.arckv_select(r(prob), fake, 1025, fake, None, 0, None), A.ERR_INVALID_ARG),
        (L.arckv_rowstats(r(prob), fake, fake, None, fake, fake, fake, None), A.ERR_INVALID_ARG),
        (L.arckv_merge(r(prob), fake, fake, fake, fake, 10, 0.25, fake, None, None, ctypes.c_void_p(0x1010),
                       1 << 30, None), A.ERR_WORKSPACE),     # misaligned workspace
        (L.arckv_merge(r(prob), fake, fake, fake, fake, 10, 0.25, fake, None, None, ctypes.c_void_p(0x10000), 16,
                       None), A.ERR_WORKSPACE),              # workspace too small
        (L.arckv_merge(r(prob), fake, fake, fake, fake, 10, 1.5, fake, None, None, fake, 0, None), A.ERR_INVALID_ARG),
        (L.arckv_merge(r(prob), fake, fake, fake, fake, 10, 0.25, odd, None, None, fake, 1 << 40, None),
         A.ERR_INVALID_ARG),                                 # misaligned C_k
        (L.arckv_fit_bias(r(prob), fake, fake, fake, fake, 10, fake, fake, r(A.default_params(bias_mode=2)), fake,
                          fake, None, fake, 0, None), A.ERR_UNSUPPORTED),
        (L.arckv_fit_bias(r(prob), None, fake, fake, fake, 10, None, fake, r(par), fake, fake, None,
                          ctypes.c_void_p(0x10000), 1 << 40, None), A.ERR_INVALID_ARG),  # z recomputed, no K
        (L.arckv_fit_values(r(prob), None, None, fake, fake, fake, 10, None, r(par), fake, fake, None, fake, 0, None),
         A.ERR_INVALID_ARG),                                 # Y recomputed, no K / V
        (L.arckv_fit_values(r(prob), fake, fake, fake, fake, fake, 10, odd, r(par), fake, fake, None,
                            ctypes.c_void_p(0x10000), 1 << 40, None), A.ERR_INVALID_ARG),  # misaligned Y
        (L.arckv_fit_values(r(prob), fake, fake, fake, fake, fake, 10, fake, r(par), None, fake, None,
                            ctypes.c_void_p(0x10000), 1 << 40, None), A.ERR_INVALID_ARG),  # no C_v
        (L.arckv_compact(r(prob), fake, fake, fake, r(ix), float("nan"), r(par), r(t_out), fake, fake, fake, fake,
                         fake, ctypes.c_void_p(0x10000), 1 << 40, None), A.ERR_INVALID_ARG),
        (L.arckv_compact(r(prob), fake, fake, fake, r(ix), 0.1, r(par), r(t_out), fake, fake, fake, fake, fake,
                         ctypes.c_void_p(0x10000), 1024, None), A.ERR_WORKSPACE),
        (L.arckv_compact(r(prob), fake, fake, fake, r(ix), 0.1, r(par), r(t_out), fake, odd, fake, fake, fake,
                         ctypes.c_void_p(0x10000), 1 << 40, None), A.ERR_INVALID_ARG),   # misaligned C_k
    ]
    for i, (got, want) in enumerate(cases):
        assert got == want, (i, got, want)


def test_product_path_has_no_oracle_or_fallback():
    """The binding never imports the oracle and has no CPU path."""
    src = open(os.path.join(os.path.dirname(A.__file__), "arckv.py")).read()
    assert "oracle" not in src.replace("oracle/", "")
    assert "numpy" not in src


def test_attend_workspace_and_validation():
    assert A.attend_workspace_size(512, 4, 6554, 0) > 0
    assert A.attend_workspace_size(512, 4, 6554, 100) >= A.attend_workspace_size(512, 4, 6554, 0)
    for args, st in [((0, 4, 10, 0), A.ERR_INVALID_ARG), ((1, 4, 0, 0), A.ERR_INVALID_ARG),
                     ((1, 4, -1, 5), A.ERR_INVALID_ARG), ((1, 4, 5, -1), A.ERR_INVALID_ARG),
                     ((1, 3, 10, 0), A.ERR_UNSUPPORTED), ((1, 16, 10, 0), A.ERR_UNSUPPORTED)]:
        with pytest.raises(A.ArckvError) as e:
            A.attend_workspace_size(*args)
        assert e.value.status == st, args
    L = A.lib()
    fake = ctypes.c_void_p(0x1000)      # never dereferenced: validation fails first
    nws = A.attend_workspace_size(2, 4, 10, 0)
    # missing pointers, unaligned pointers and a short workspace are rejected before any HIP call
    assert L.arckv_attend(2, 4, 10, 0, 0.0, None, fake, None, fake, None, None, fake, fake, nws, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_attend(2, 4, 10, 0, 0.0, fake, None, None, fake, None, None, fake, fake, nws, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_attend(2, 4, 10, 3, 0.0, fake, fake, None, fake, None, None, fake, fake, nws, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_attend(2, 4, 10, 0, 0.0, ctypes.c_void_p(0x1002), fake, None, fake, None, None, fake, fake, nws,
                          None) == A.ERR_INVALID_ARG
    assert L.arckv_attend(2, 4, 10, 0, float("nan"), fake, fake, None, fake, None, None, fake, fake, nws, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_attend(2, 4, 10, 0, 0.0, fake, fake, None, fake, None, None, fake, fake, nws - 1, None) == \
        A.ERR_WORKSPACE
    assert L.arckv_attend(2, 4, 10, 0, 0.0, fake, fake, None, fake, None, None, fake, ctypes.c_void_p(0x1010), nws,
                          None) == A.ERR_WORKSPACE
    # the no-allocation variant: the same argument checks, and partials beyond its 64 MiB static scratch are
    # rejected before any HIP call
    assert L.arckv_attend_noalloc(2, 4, 10, 0, 0.0, None, fake, None, fake, None, None, fake, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_attend_noalloc(2, 4, 10, 3, 0.0, fake, fake, None, fake, None, None, fake, None) == \
        A.ERR_INVALID_ARG
    assert A.attend_workspace_size(512, 4, 16128, 0) <= 64 << 20 < A.attend_workspace_size(512, 4, 16129, 0)
    assert L.arckv_attend_noalloc(512, 4, 16129, 0, 0.0, fake, fake, None, fake, None, None, fake, None) == \
        A.ERR_WORKSPACE


def test_budgets_and_select_count_match_oracle():
    import numpy as np
    import oracle
    g = np.random.default_rng(0)
    for T in (5000, 10000, 10001, 12000, 20001, 50000, 131072):
        for t in (1, 77, max(1, T // 10), T // 3):
            for L in (0, 4096, 7000, 8192, 200000):
                want = sum(c[2] for c in oracle.chunk_budgets(t, T, L))
                assert A.select_count(T, t, L) == want, (T, t, L)
    for P in (1, 8, 256):
        w = g.uniform(0, 1, P)
        assert A.budgets(list(w), 3277, 32768) == oracle.budgets_per_pair(w, 3277, 32768).tolist()
    assert A.budgets([0, 0.5, 9.5], 10, 20) == [1, 1, 20]
    for a, t, T in (([0, 0], 10, 20), ([-1, 2], 10, 20), ([float("nan")], 5, 10), ([1], 0, 10)):
        with pytest.raises(A.ArckvError):
            A.budgets(a, t, T)
    with pytest.raises(A.ArckvError):
        A.select_count(100, 101, 0)


def test_workspace_covers_chunked_count():
    p = A.problem_from_dims(2, 131072, 512)
    nominal = A.budget(131072, 0.01)
    assert A.select_count(131072, nominal, 8192) > nominal
    assert A.workspace_size(p, nominal, A.default_params(select_chunk=8192)) >= \
        A.workspace_size(p, A.select_count(131072, nominal, 8192))


def test_dsa_validation():
    p = A.problem_from_dims(2, 300, 96)
    assert A.dsa_workspace_size(p) > A.dsa_workspace_size(p, pair_chunk=1) > 0
    L = A.lib()
    fake = ctypes.c_void_p(0x1000)
    ix = A.DSAIndexer(48, 96, 1, 0.0, *([fake] * 10))
    nbytes = A.dsa_workspace_size(p)
    # fp32 inputs are not supported; n must be a multiple of n_pos; a null weight is rejected
    p32 = A.problem_from_dims(2, 300, 96, dtype=A.F32)
    assert L.arckv_score_dsa(ctypes.byref(p32), fake, fake, fake, ctypes.byref(ix), fake, fake, nbytes, None) == \
        A.ERR_UNSUPPORTED
    bad = A.DSAIndexer(50, 96, 1, 0.0, *([fake] * 10))
    assert L.arckv_score_dsa(ctypes.byref(p), fake, fake, fake, ctypes.byref(bad), fake, fake, nbytes, None) == \
        A.ERR_INVALID_ARG
    nul = A.DSAIndexer(48, 96, 1, 0.0, *([fake] * 9 + [None]))
    assert L.arckv_score_dsa(ctypes.byref(p), fake, fake, fake, ctypes.byref(nul), fake, fake, nbytes, None) == \
        A.ERR_INVALID_ARG
    assert L.arckv_score_dsa(ctypes.byref(p), fake, fake, fake, ctypes.byref(ix), fake, ctypes.c_void_p(0x1010),
                             nbytes, None) == A.ERR_WORKSPACE
    assert L.arckv_compact_scored(ctypes.byref(p), fake, fake, fake, None, 0.1, None, ctypes.byref(ctypes.c_int32()),
                                  fake, fake, fake, fake, fake, fake, 1 << 20, None) == A.ERR_INVALID_ARG
