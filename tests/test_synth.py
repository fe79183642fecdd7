"""Seeded input generators: determinism, shapes, bf16 rounding (CPU only)."""
import numpy as np
import pytest

import synth


def test_param_counts():
    assert synth.ONE_B.n_params() == 1_235_814_400
    assert synth.TINY.n_params() == 2_499_840


def test_weights_deterministic_and_gain_independent():
    a = synth.make_weights(synth.TINY, 0)
    b = synth.make_weights(synth.TINY, 0)
    c = synth.make_weights(synth.TINY, 0, gain_std=0.1)
    for (name, shp), x, y, z in zip(synth.TINY.tensor_specs(), a, b, c):
        assert x.shape == shp and x.dtype == np.float32
        assert np.array_equal(x, y)
        if len(shp) == 2:
            assert np.array_equal(x, z)
            assert abs(x.std() - 0.02) < 0.002
        else:
            assert np.all(x == 1.0) and not np.all(z == 1.0)


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 0.02,
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8], np.float32)])
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.tensor(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.tensor(x).to(torch.bfloat16).float().numpy())


def test_tokens():
    t = synth.make_tokens(4096, 64, 1)
    assert t.dtype == np.int32 and t.min() >= 0 and t.max() < 4096
    assert np.array_equal(t, synth.make_tokens(4096, 64, 1))
    assert not np.array_equal(t, synth.make_tokens(4096, 64, 2))
