"""The seeded input generator: determinism, coordinates and distribution.

A numpy re-statement of the published generators (SplitMix64's output
function, Box-Muller) checks the C implementation element by element.
"""
import numpy as np

import synth

M64 = np.uint64(0xFFFFFFFFFFFFFFFF)
GOLDEN = np.uint64(0x9E3779B97F4A7C15)


def _mix(z):
    z = z.astype(np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def _normals_np(key, n):
    j = np.arange((n + 1) // 2, dtype=np.uint64)
    with np.errstate(over="ignore"):
        w = _mix(np.uint64(key) + (j + np.uint64(1)) * GOLDEN)
    u1 = ((w >> np.uint64(40)).astype(np.float64) + 0.5) / 16777216.0
    u2 = (((w >> np.uint64(16)) & np.uint64(0xFFFFFF)).astype(np.float64) + 0.5) / 16777216.0
    r = np.sqrt(-2.0 * np.log(u1))
    t = 2 * np.pi * u2
    return np.stack([r * np.cos(t), r * np.sin(t)], axis=1).reshape(-1)[:n]


def test_c_generator_matches_its_definition():
    k = synth.key(0, 1, 2, 3, 4)
    z = _normals_np(k, 100001)
    got = synth.normal_f32(k, (100001,), 0.0, 1.0)
    np.testing.assert_allclose(got, z.astype(np.float32), rtol=1e-6, atol=1e-6)
    bits = synth.normal_bf16(k, (100001,), 0.0, 0.02)
    w = synth.bf16_bits_to_f32(bits).astype(np.float64)
    assert np.max(np.abs(w - 0.02 * z)) <= 0.02 * np.max(np.abs(z)) * 2.0 ** -8


def test_deterministic_and_sliceable_across_threads():
    k = synth.key(0, 2, 0, 8, 6)
    a = synth.normal_bf16(k, (1 << 20,), 0.0, 0.02)
    b = synth.normal_bf16(k, (1 << 20,), 0.0, 0.02)
    assert np.array_equal(a, b)
    small = synth.normal_bf16(k, (1001,), 0.0, 0.02)  # single-threaded path
    assert np.array_equal(small, a[:1001])


def test_coordinates_give_distinct_streams_and_moments():
    a = synth.bf16_bits_to_f32(synth.normal_bf16(synth.key(0, 2, 0, 8, 6), (1 << 20,), 0.0, 0.02))
    b = synth.bf16_bits_to_f32(synth.normal_bf16(synth.key(0, 2, 0, 9, 6), (1 << 20,), 0.0, 0.02))
    assert abs(float(a.mean())) < 1e-4 and abs(float(a.std()) - 0.02) < 2e-4
    assert abs(float(np.corrcoef(a, b)[0, 1])) < 5e-3
    t = synth.uniform_i32(synth.key(0, 3, 3, 0, 0), (200000,), 128256)
    assert t.min() >= 0 and t.max() < 128256 and abs(t.mean() / 128256 - 0.5) < 5e-3


def test_gains_centre_on_one_and_layers_are_global():
    w8 = synth.layer_weights(synth.SHAPE_TINY, 1, 1)
    again = synth.layer_weights(synth.SHAPE_TINY, 1, 1)
    assert all(np.array_equal(w8[k], again[k]) for k in w8)
    g = synth.bf16_bits_to_f32(w8["attn_norm"])
    assert abs(float(g.mean()) - 1.0) < 5e-3 and float(g.std()) > 0.01
    assert w8["wq"].shape == (512, 512) and w8["wk"].shape == (128, 512) and w8["wd"].shape == (512, 1408)


def test_bf16_test_helper_matches_torch_rounding():
    """The tests' float-to-bf16 helper rounds to nearest even exactly as torch does."""
    import torch

    from tests.helpers import f32_to_bf16_bits
    x = np.random.default_rng(0).standard_normal(4096).astype(np.float32) * np.float32(300.0)
    x[:4] = [7e4, -1e-30, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]  # ties round to even
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(f32_to_bf16_bits(x), want)
