"""The seeded input generator: determinism, dtype rounding, fp8 encoding of the stored cache."""

import numpy as np
import torch

import oracle
import synth


def test_bf16_rounding_matches_library_rne():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 3.0e38]  # ties and a large value
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(synth.round_bf16(x), want)


def test_streams_are_keyed_and_reproducible():
    wl = synth.WORKLOADS["tiny_fp32_L40"]
    a = synth.cache_slab(wl, 0, 1, "k")
    b = synth.cache_slab(wl, 0, 1, "k")
    c = synth.cache_slab(wl, 0, 1, "v")
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, c)
    assert a.shape == (40, wl.n_heads, wl.head_dim)


def test_fp8_encoding_picks_a_nearest_code_and_saturates():
    # The encoder (clamp, then round to nearest) must return a code whose decoded value is the
    # nearest E4M3 value to x/scale; checked by brute force over all finite codes.
    rng = np.random.default_rng(1)
    src = synth.round_bf16(rng.standard_normal((300, 2, 16)).astype(np.float32) * 3)
    codes, scale = synth.fp8_encode(src)
    assert codes.dtype == np.uint8 and scale.shape == (2,)
    table = oracle.e4m3fn_decode(np.arange(256, dtype=np.uint8))
    finite = np.where(~np.isnan(table))[0]
    y = src / scale[None, :, None]
    dec = oracle.e4m3fn_decode(codes)
    best = np.abs(table[finite][None, :] - y.reshape(-1, 1)).min(axis=1)
    np.testing.assert_array_equal(np.abs(dec.reshape(-1) - y.reshape(-1)), best)
    # the largest magnitude of each head maps to +-448
    for h in range(2):
        assert np.abs(dec[:, h]).max() == 448.0


def test_ragged_lengths_of_the_fp8_workload():
    wl = synth.WORKLOADS["ragged_fp8_B8"]
    assert len(wl.lengths) == 8 and all(256 <= L <= 16384 for L in wl.lengths)
    assert max(wl.lengths) <= wl.capacity


def test_stress_keys_scale_channels_rows_and_the_sink_row():
    # ones through the transform: channel factor (8 for channels 0-3), row ramp 1 + 3 i / L, sink row 8x more
    L, H, D = 30, 2, 8
    got = synth.stress_keys(np.ones((L, H, D), np.float32))
    ramp = 1.0 + 3.0 * np.arange(L) / L
    for i in range(L):
        sink = 8.0 if i == 20 else 1.0
        np.testing.assert_allclose(got[i, :, 4:], ramp[i] * sink, rtol=1e-6)
        np.testing.assert_allclose(got[i, :, :4], 8.0 * ramp[i] * sink, rtol=1e-6)
    # only the keys of a stress workload change; values and ordinary workloads are untouched
    wl = synth.WORKLOADS["tiny_fp32_L40"]
    ws = wl.replace(stress_keys=True)
    np.testing.assert_array_equal(synth.cache_slab(ws, 0, 0, "v"), synth.cache_slab(wl, 0, 0, "v"))
    np.testing.assert_allclose(synth.cache_slab(ws, 0, 0, "k"), synth.stress_keys(synth.cache_slab(wl, 0, 0, "k")))
