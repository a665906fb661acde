"""Pins of the RMS normalisation oracle (oracle/rmsnorm.py) against what the mathematics and
an independent library routine fix: torch's own rms_norm in float64, exact power-of-two
scale invariance, unit output RMS over the token, the per-token (not per-head) extent of
the statistic, the place of eps, and linearity in the weight."""
import numpy as np
import pytest
import torch

import synth
from oracle import numerics, rmsnorm

C = 1536
H = 12


def _bits(shape, key, scale=1.0):
    return synth.normal_bf16(shape, key, scale)


def test_matches_torch_rms_norm_fp64():
    # independent implementation: torch.nn.functional.rms_norm in float64, then the stated
    # roundings (float64 -> float32 -> bf16, nearest-even) done by torch's own casts
    x = _bits((64, C), (71, 0))
    w = _bits((C,), (71, 1))
    got = rmsnorm.rms_norm_bf16(x, w)
    xt = torch.from_numpy(numerics.bf16_to_f64(x))
    wt = torch.from_numpy(numerics.bf16_to_f64(w))
    ref = torch.nn.functional.rms_norm(xt, (C,), wt, eps=rmsnorm.EPS).to(torch.float32).to(torch.bfloat16)
    assert np.array_equal(got, ref.view(torch.int16).numpy().view(np.uint16))
    ideal = rmsnorm.rms_norm_ideal(numerics.bf16_to_f64(x), numerics.bf16_to_f64(w))
    assert np.allclose(ideal, torch.nn.functional.rms_norm(xt, (C,), wt, eps=rmsnorm.EPS).numpy(), rtol=1e-13,
                       atol=0)


@pytest.mark.parametrize("k", [-8, -1, 3, 7])
def test_power_of_two_scale_invariance_exact(k):
    # with eps = 0, scaling x by 2^k scales the sum of squares by 2^2k and its square root by
    # 2^k exactly, so the normalised output is bit-identical
    x = _bits((16, C), (72, 0))
    w = _bits((C,), (72, 1))
    xs = numerics.f32_to_bf16_bits(numerics.bf16_to_f64(x) * 2.0 ** k)
    assert np.array_equal(numerics.bf16_to_f64(xs), numerics.bf16_to_f64(x) * 2.0 ** k)
    assert np.array_equal(rmsnorm.rms_norm_bf16(xs, w, eps=0.0), rmsnorm.rms_norm_bf16(x, w, eps=0.0))


def test_unit_rms_over_the_token():
    # w = 1, eps = 0: the output's mean square over the token's C channels is exactly 1
    x = numerics.bf16_to_f64(_bits((32, C), (73, 0), scale=3.0))
    y = rmsnorm.rms_norm_ideal(x, np.ones(C), eps=0.0)
    assert np.allclose(np.mean(y * y, axis=-1), 1.0, rtol=0, atol=1e-13)


def test_statistic_spans_all_heads_not_one():
    # head 1 four times as large as head 0: a token-wide statistic keeps the 4:1 ratio of the
    # heads' RMS in the output; a per-head statistic would make both 1
    D = C // H
    x = numerics.bf16_to_f64(_bits((8, C), (74, 0)))
    x[:, D:2 * D] = x[:, 0:D] * 4.0
    y = rmsnorm.split_heads(rmsnorm.rms_norm_ideal(x, np.ones(C), eps=0.0), H)
    rms = np.sqrt(np.mean(y * y, axis=-1))
    assert np.allclose(rms[:, 1] / rms[:, 0], 4.0, rtol=1e-12)


def test_eps_inside_the_square_root():
    # all channels equal to a, w = 1: y = a / sqrt(a^2 + eps); for a^2 << eps the output is
    # linear in x with slope 1/sqrt(eps), for a^2 >> eps it is sign(a)
    for a in (2.0 ** -20, 2.0 ** -16):
        y = rmsnorm.rms_norm_ideal(np.full((1, C), a), np.ones(C))
        assert np.allclose(y, a / np.sqrt(a * a + rmsnorm.EPS), rtol=1e-14)
    tiny = rmsnorm.rms_norm_ideal(np.full((1, C), 2.0 ** -24), np.ones(C))
    assert np.allclose(tiny, 2.0 ** -24 / np.sqrt(rmsnorm.EPS), rtol=1e-9)
    big = rmsnorm.rms_norm_ideal(np.full((1, C), -8.0), np.ones(C))
    assert np.allclose(big, -1.0, rtol=1e-7)


def test_zero_vector_and_weight_linearity():
    w = _bits((C,), (75, 1))
    assert not np.any(numerics.bf16_to_f64(rmsnorm.rms_norm_bf16(np.zeros((2, C), np.uint16), w)))
    x = _bits((8, C), (75, 0))
    w2 = numerics.f32_to_bf16_bits(numerics.bf16_to_f64(w) * 2.0)
    y1 = numerics.bf16_to_f64(rmsnorm.rms_norm_bf16(x, w))
    y2 = numerics.bf16_to_f64(rmsnorm.rms_norm_bf16(x, w2))
    assert np.array_equal(y2, 2.0 * y1)


def test_tokens_independent_and_shape():
    x = _bits((2, 5, C), (76, 0))
    w = _bits((C,), (76, 1))
    y = rmsnorm.rms_norm_bf16(x, w)
    assert y.shape == x.shape and y.dtype == np.uint16
    perm = np.array([3, 0, 4, 1, 2])
    assert np.array_equal(rmsnorm.rms_norm_bf16(x[:, perm], w), y[:, perm])
    with pytest.raises(ValueError):
        rmsnorm.rms_norm_bf16(x, w[:-1])
