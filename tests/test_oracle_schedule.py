"""Pins of the schedule and clean-cache update oracle (oracle/schedule.py): the paper's printed
schedule table, exact rationals of the shift map, its fixed endpoints, the identities at
sigma = 0 and 1, and the flow-matching consistency of renoise followed by emit."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import numerics, schedule

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_paper_schedule_table():
    g = GOLDEN["shift_five_schedule"]
    u, sigma, t = schedule.shift_schedule(4, g["shift"])
    assert u.tolist() == g["raw_u"]
    assert np.allclose(sigma, g["sigma"], atol=0.5 * 10 ** -g["decimals_printed"]["sigma"], rtol=0)
    assert np.allclose(t, g["t"], atol=0.5 * 10 ** -g["decimals_printed"]["t"], rtol=0)
    # the exact fractions the table prints, to the last float64 bit (correctly rounded division)
    assert [float(Fraction(s)) for s in g["sigma_exact"]] == sigma.tolist()
    assert GOLDEN["clean_cache_noise"]["sigma_unstep"] == schedule.SIGMA_CLEAN_UNSTEP


@pytest.mark.parametrize("n,shift", [(4, 5.0), (8, 3.0), (3, 1.0)])
def test_shift_map_rationals_endpoints_and_order(n, shift):
    u, sigma, t = schedule.shift_schedule(n, shift)
    for ui, si in zip(u, sigma):
        exact = Fraction(shift) * Fraction(ui) / (1000 + (Fraction(shift) - 1) * Fraction(ui))
        assert abs(Fraction(si) - exact) <= Fraction(si) * Fraction(1, 2 ** 50)
    assert sigma[0] == 1.0 and t[0] == 1000.0                      # the map keeps u = 1000
    assert np.all(np.diff(sigma) < 0)
    if shift == 1.0:
        assert np.array_equal(sigma, u / 1000.0)                   # no shift: identity map
    else:
        assert np.all(sigma[1:] > u[1:] / 1000.0)                  # shift > 1 pushes levels up


def test_identities_at_zero_and_one():
    x = synth.normal_bf16((4096,), (91, 0))
    e = synth.normal_bf16((4096,), (91, 1))
    v = synth.normal_bf16((4096,), (91, 2))
    assert np.array_equal(schedule.renoise_bf16(x, e, 0.0), x)      # sigma 0: the original clean pass
    assert np.array_equal(schedule.emit_bf16(x, v, 0.0), x)
    assert np.array_equal(schedule.renoise_bf16(x, e, 1.0), e)      # sigma 1: pure noise
    xv = numerics.bf16_to_f64(x) - numerics.bf16_to_f64(v)
    assert np.array_equal(schedule.emit_bf16(x, v, 1.0), numerics.f32_to_bf16_bits(xv))


def test_renoise_then_emit_with_the_straight_flow_returns_the_input():
    # for the straight path the velocity is v = eps - x, and emit(renoise(x)) = x exactly in
    # real arithmetic; with the float64 steps and one final rounding it returns x's bf16 bits
    x = synth.normal_bf16((8192,), (92, 0))
    e = synth.normal_bf16((8192,), (92, 1))
    xf, ef = numerics.bf16_to_f64(x), numerics.bf16_to_f64(e)
    for sigma in (0.02, 0.625, 5.0 / 6.0):
        xt = (1.0 - sigma) * xf + sigma * ef                         # float64, unrounded
        back = xt - sigma * (ef - xf)
        assert np.max(np.abs(back - xf)) < 1e-15 * 8
        assert np.array_equal(numerics.f32_to_bf16_bits(back), x)


def test_linearity_in_the_inputs():
    x = synth.normal_bf16((2048,), (93, 0))
    e = synth.normal_bf16((2048,), (93, 1))
    x2 = numerics.f32_to_bf16_bits(2.0 * numerics.bf16_to_f64(x))
    e2 = numerics.f32_to_bf16_bits(2.0 * numerics.bf16_to_f64(e))
    r1 = numerics.bf16_to_f64(schedule.renoise_bf16(x, e, 0.02))
    r2 = numerics.bf16_to_f64(schedule.renoise_bf16(x2, e2, 0.02))
    assert np.array_equal(r2, 2.0 * r1)                             # power-of-two scale is exact
