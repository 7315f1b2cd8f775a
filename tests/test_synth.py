"""The seeded input generator: determinism, shapes, bf16 rounding, structure."""
import numpy as np
import pytest

import synth


def test_bf16_round_to_nearest_even():
    import torch
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 3.14159, -2.5e-3,
                  65504.0, 1e-30], dtype=np.float32)
    got = synth.round_to_bf16(x)
    assert got[1] == 1.0                          # tie -> even mantissa
    assert got[2] == np.float32(1.015625)         # tie -> even (rounds up)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(got, ref)
    rng = np.random.default_rng(0)
    y = (rng.standard_normal(100000) * 10 ** rng.uniform(-5, 5, 100000)).astype(np.float32)
    np.testing.assert_array_equal(synth.round_to_bf16(y),
                                  torch.from_numpy(y).to(torch.bfloat16).to(torch.float32).numpy())
    bits = synth.bf16_bits(y)
    np.testing.assert_array_equal(synth.bf16_bits_to_float(bits), synth.round_to_bf16(y))


def test_generator_deterministic_and_shaped():
    spec = synth.SPECS["tiny"]
    a = synth.make_layer(spec)
    b = synth.make_layer(spec, threads=1)
    for x, y in ((a.q, b.q), (a.k, b.k), (a.v, b.v)):
        np.testing.assert_array_equal(x, y)
    assert a.q.shape == (2048, 2, 64) and a.k.shape == (2048, 2, 64)
    assert list(a.cu_seqlens) == [0, 2048]
    np.testing.assert_array_equal(synth.round_to_bf16(a.q), a.q)   # bf16-representable


def test_generator_varlen_and_partial_heads():
    spec = synth.SPECS["qwen_varlen"].with_seqlens((300, 129, 1024, 1), name="mini-varlen")
    layer = synth.make_layer(spec, heads=[0, 1])
    assert layer.q.shape == (1454, 28, 128)
    assert list(layer.cu_seqlens) == [0, 300, 429, 1453, 1454]
    assert np.all(layer.q[:, 2:] == 0) and np.any(layer.q[:, :2] != 0)
    for s in range(4):
        for g in range(4):
            vs = layer.verticals[s][g]
            assert np.all((vs >= 1) & (vs < spec.seqlens[s] - 128))


def test_vertical_slash_structure_is_visible():
    """Sink and vertical keys carry the largest logits of the last query block."""
    spec = synth.SPECS["tiny"]
    layer = synth.make_layer(spec)
    q = layer.q[-128:, 0].astype(np.float64)
    k = layer.k[:, 0].astype(np.float64)
    lg = (q @ k.T).mean(axis=0) / 8.0
    top = set(np.argsort(lg)[::-1][:9].tolist())
    assert 0 in top
    assert len(top & set(layer.verticals[0][0].tolist())) >= 6
