"""Pins for the oracle's rotary embedding (paper Appendix A.5 pair arithmetic).

* the rotation equals the complex product (x_2j + i x_2j+1) * exp(i angle),
  the form the paper gives for the original fp64 path;
* the bf16/fp32 rounding contract equals NumPy's own binary32 arithmetic
  followed by torch's bf16 conversion (two implementations independent of the
  oracle's float64 emulation);
* position 0 is the identity, bit for bit;
* norms are preserved, and scores depend only on relative positions.
"""
import numpy as np
import torch

import synth
from oracle import numerics, rope, tables


def _x(shape, key):
    return synth.normal_bf16(shape, key)


def test_rotation_is_complex_multiplication():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 6, 3, 128))
    ang = rng.uniform(-40, 40, size=(6, 64))
    y = rope.rope_ideal(x, ang)
    z = (x[..., 0::2] + 1j * x[..., 1::2]) * np.exp(1j * ang)[None, :, None, :]
    assert np.allclose(y[..., 0::2], z.real, rtol=0, atol=1e-13)
    assert np.allclose(y[..., 1::2], z.imag, rtol=0, atol=1e-13)


def test_contract_matches_numpy_binary32_and_torch_bf16():
    # large enough (2.4M values) that a fused or unrounded intermediate flips some bf16 outputs
    xb = _x((1, 4680, 4, 128), (900, 1))
    c, s = tables.rope_tables(9, 3, 30, 52)
    got = rope.rope_bf16(xb, c, s)
    # independent path: binary32 arithmetic by NumPy (no FMA), bf16 rounding by torch
    x32 = numerics.bf16_to_f64(xb).astype(np.float32)
    xe, xo = x32[..., 0::2], x32[..., 1::2]
    c32, s32 = c[None, :, None, :], s[None, :, None, :]
    ye = (xe * c32) - (xo * s32)
    yo = (xe * s32) + (xo * c32)
    y32 = np.empty_like(x32)
    y32[..., 0::2] = ye
    y32[..., 1::2] = yo
    want = torch.from_numpy(y32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got, want)


def test_contract_close_to_ideal_rotation():
    xb = _x((1, 4680, 2, 128), (901, 1))
    c, s = tables.rope_tables(9, 3, 30, 52)
    got = numerics.bf16_to_f64(rope.rope_bf16(xb, c, s))
    ideal = rope.rope_ideal(numerics.bf16_to_f64(xb), tables.angles_f64(9, 3, 30, 52, 128, 10000.0))
    # bf16 output rounding (2^-9 relative) dominates; fp32 steps add ~2^-23
    err = np.abs(got - ideal)
    assert np.all(err <= 2.0 ** -8 * np.abs(ideal) + 2.0 ** -20)


def test_position_zero_is_bitwise_identity():
    xb = _x((1, 1, 12, 128), (902, 1))
    c, s = tables.rope_tables(0, 1, 1, 1)
    assert np.array_equal(rope.rope_bf16(xb, c, s), xb)


def test_norm_preserved():
    x = numerics.bf16_to_f64(_x((1, 72, 2, 128), (903, 1)))
    ang = tables.angles_f64(6, 3, 4, 6, 128, 10000.0)
    y = rope.rope_ideal(x, ang)
    assert np.allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-13, atol=0)
    # bf16 path: each output element is within 2^-8 relative, so norms are too
    c, s = tables.rope_tables(6, 3, 4, 6)
    yb = numerics.bf16_to_f64(rope.rope_bf16(_x((1, 72, 2, 128), (903, 1)), c, s))
    r = np.linalg.norm(yb, axis=-1) / np.linalg.norm(x, axis=-1)
    assert np.all(np.abs(r - 1.0) < 2.0 ** -8)


def test_scores_invariant_to_common_position_shift():
    # <R(p + d) q, R(p' + d) k> = <R(p) q, R(p') k> for a shift d of every axis position
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 1, 128))
    k = rng.standard_normal((1, 1, 1, 128))

    def ang(frame, row, col):
        out = np.empty((1, 64))
        for j, (axis, kk, d_ax) in enumerate(tables.pair_axes(128)):
            p = (frame, row, col)[axis]
            out[0, j] = p * tables.omega(10000.0, kk, d_ax)
        return out

    base = np.sum(rope.rope_ideal(q, ang(3, 2, 5)) * rope.rope_ideal(k, ang(9, 7, 1)))
    for d in ((4, 0, 0), (0, 11, 0), (0, 0, 13), (17, 3, 8)):
        sh = np.sum(rope.rope_ideal(q, ang(3 + d[0], 2 + d[1], 5 + d[2])) *
                    rope.rope_ideal(k, ang(9 + d[0], 7 + d[1], 1 + d[2])))
        assert abs(sh - base) < 1e-11
    # but not to a shift of one vector only
    moved = np.sum(rope.rope_ideal(q, ang(4, 2, 5)) * rope.rope_ideal(k, ang(9, 7, 1)))
    assert abs(moved - base) > 1e-3


def test_bf16_rounding_ties_to_even():
    # 1 + 2^-8 is halfway between bf16 1.0 and 1.0078125: ties go to the even (1.0)
    x = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8), 1.0 + 2.0 ** -8 + 2.0 ** -20])
    bits = numerics.f32_to_bf16_bits(x)
    assert bits.tolist() == [0x3F80, 0x3F82, 0xBF80, 0x3F81]
