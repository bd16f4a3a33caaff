"""The seeded input generator: determinism, shapes, rounding and RoPE identities."""
import numpy as np

import synth


def test_round_bf16_known_values():
    x = np.array([1.0, 1.00390625, 1.005859375, 1.0078125, -2.5, 3.0e38, 1e-40], dtype=np.float32)
    r = synth.round_bf16(x)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even mantissa (1.0)
    assert r[0] == 1.0 and r[1] == 1.0
    assert r[2] == np.float32(1.0078125)          # above the tie rounds up
    assert r[3] == np.float32(1.0078125)
    assert r[4] == -2.5
    u = r.view(np.uint32)
    assert np.all(u & 0xFFFF == 0)
    # idempotent
    assert np.array_equal(synth.round_bf16(r), r)


def test_pair_inputs_deterministic_and_independent():
    wl = synth.custom("t", T=64, n_pos=16, dtype="bf16", rope=True)
    a = synth.pair_inputs(wl, 0, 0)
    b = synth.pair_inputs(wl, 0, 0)
    c = synth.pair_inputs(wl, 0, 1)
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert not np.array_equal(a["K"], c["K"])
    assert a["K"].shape == (64, 128) and a["Q"].shape == (16, 128) and a["W1"].shape == (64, 256)
    assert np.all(a["K"].view(np.uint32) & 0xFFFF == 0)
    assert np.all(a["W1"].view(np.uint32) & 0xFFFF == 0)


def test_rope_is_a_rotation_with_relative_phase():
    g = np.random.default_rng(0)
    x = g.standard_normal((1, 128)).astype(np.float32)
    y = g.standard_normal((1, 128)).astype(np.float32)
    xr = synth.apply_rope(np.repeat(x, 3, 0), np.array([0, 5, 40]))
    yr = synth.apply_rope(np.repeat(y, 3, 0), np.array([0, 10, 45]))
    np.testing.assert_allclose(np.linalg.norm(xr, axis=1), np.linalg.norm(x), rtol=1e-5)
    assert np.array_equal(xr[0], x[0])                       # position 0 is the identity
    # <R_m x, R_n y> depends only on n - m
    np.testing.assert_allclose(xr[1] @ yr[1], xr[2] @ yr[2], rtol=1e-4)


def test_llama3_frequencies():
    f = synth.llama3_inv_freq()
    base = 1.0 / 500000.0 ** (np.arange(0, 128, 2) / 128)
    assert f[0] == base[0]                                   # high frequencies untouched
    np.testing.assert_allclose(f[-1], base[-1] / 8.0)        # lowest frequency divided by 8
    assert np.all(np.diff(f) < 0)


def test_workload_table():
    w = synth.WORKLOADS["llama8b_bf16_T32768"]
    assert (w.pairs, w.T, w.n) == (256, 32768, 4096)
    assert synth.WORKLOADS["long_bf16_T131072"].n == 8192
    assert synth.WORKLOADS["tiny_f32_T1024"].n == 256
    pos = synth.query_positions(synth.WORKLOADS["layer_bf16_T8192"])
    assert pos.min() == 0 and pos.max() < 8192 and len(pos) == 4096
