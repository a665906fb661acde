"""Pins for the oracle's rotary tables (paper Appendix A.5).

Each test checks the oracle against something other than itself: the paper's
worked positions, textbook values of cos/sin, closed forms of the frequency
ladder, and trigonometric identities.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import tables

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_axis_split_is_22_21_21_pairs():
    # reading: height and width take 2*(D//6) dims each, time the rest
    assert tables.axis_dims(128) == (44, 42, 42)
    axes = tables.pair_axes(128)
    assert len(axes) == GOLDEN["heads"]["n_pairs"]
    assert [a for a, _, _ in axes].count(tables.TEMPORAL) == 22
    assert [a for a, _, _ in axes].count(tables.HEIGHT) == 21
    assert [a for a, _, _ in axes].count(tables.WIDTH) == 21
    # order: temporal pairs first, then height, then width
    assert axes[0] == (tables.TEMPORAL, 0, 44) and axes[21] == (tables.TEMPORAL, 21, 44)
    assert axes[22] == (tables.HEIGHT, 0, 42) and axes[43] == (tables.WIDTH, 0, 42)
    assert axes[63] == (tables.WIDTH, 20, 42)


def test_frequency_ladder_closed_forms():
    # omega_0 = 1 on every axis; theta^(-1/2) = 0.01 at the middle of the 44-dim ladder
    assert tables.omega(10000.0, 0, 44) == 1.0
    assert tables.omega(10000.0, 0, 42) == 1.0
    assert tables.omega(10000.0, 11, 44) == pytest.approx(0.01, rel=1e-15)
    # 10000^(-2*7/42) = 10000^(-1/3) = 0.0464158883361278
    assert tables.omega(10000.0, 7, 42) == pytest.approx(0.046415888336127795, rel=1e-15)
    # strictly decreasing ladder
    w = [tables.omega(10000.0, k, 42) for k in range(21)]
    assert all(a > b for a, b in zip(w, w[1:]))


def test_paper_worked_positions_chunk_at_6():
    g = GOLDEN["chunk_temporal_positions"]
    pos = tables.token_positions(6, g["chunk_frames"], 2, 3)
    assert sorted(set(pos[:, 0].tolist())) == g["positions_of_start_6"]
    # frame-major, then row, then column
    assert pos[0].tolist() == [6, 0, 0] and pos[1].tolist() == [6, 0, 1] and pos[3].tolist() == [6, 1, 0]
    assert pos[6].tolist() == [7, 0, 0] and pos[-1].tolist() == [8, 1, 2]


def test_position_zero_is_identity():
    c, s = tables.rope_tables(0, 1, 1, 1)
    assert np.all(c[0] == np.float32(1.0)) and np.all(s[0] == np.float32(0.0))


def test_textbook_values_on_unit_frequency_pairs():
    # pair 0 (temporal, omega=1) at frame p has angle p; pair 22 (height, omega=1) has angle = row;
    # pair 43 (width, omega=1) has angle = column.
    cos1, sin1 = 0.5403023058681398, 0.8414709848078965
    cos2, sin2 = -0.4161468365471424, 0.9092974268256817
    c, s = tables.rope_tables(1, 2, 3, 3)          # frames 1, 2; 3x3 grid
    # token 0: (frame 1, row 0, col 0)
    assert c[0, 0] == np.float32(cos1) and s[0, 0] == np.float32(sin1)
    assert c[0, 22] == np.float32(1.0) and s[0, 43] == np.float32(0.0)
    # token 9: (frame 2, row 0, col 0)
    assert c[9, 0] == np.float32(cos2) and s[9, 0] == np.float32(sin2)
    # token 5: (frame 1, row 1, col 2)
    assert c[5, 22] == np.float32(cos1) and s[5, 43] == np.float32(sin2)
    # pair 11 (temporal, omega = 0.01) at frame 2: angle 0.02
    assert c[9, 11] == np.float32(math.cos(0.02)) and s[9, 11] == np.float32(math.sin(0.02))


def test_tables_are_fp32_rounding_of_fp64_angles():
    c, s = tables.rope_tables(9, 3, 30, 52)
    assert c.dtype == np.float32 and c.shape == (4680, 64) and s.shape == (4680, 64)
    ang = tables.angles_f64(9, 3, 30, 52, 128, 10000.0)
    # within half an ulp of binary32 of the float64 values
    assert np.all(np.abs(c.astype(np.float64) - np.cos(ang)) <= 2.0 ** -24 * np.maximum(np.abs(np.cos(ang)), 2.0 ** -126) + 1e-16)
    assert np.all(np.abs(s.astype(np.float64) - np.sin(ang)) <= 2.0 ** -24 * np.maximum(np.abs(np.sin(ang)), 2.0 ** -126) + 1e-16)
    # Pythagoras
    r = c.astype(np.float64) ** 2 + s.astype(np.float64) ** 2
    assert np.max(np.abs(r - 1.0)) < 2.0 ** -22


def test_angle_addition_across_start_frames():
    # cos((p+q) w) = cos(p w) cos(q w) - sin(p w) sin(q w) on the temporal pairs
    ca, sa = tables.rope_tables(4, 1, 1, 1)
    cb, sb = tables.rope_tables(7, 1, 1, 1)
    cc, sc = tables.rope_tables(11, 1, 1, 1)
    ca, sa, cb, sb = (x.astype(np.float64) for x in (ca, sa, cb, sb))
    pred_c = ca * cb - sa * sb
    pred_s = sa * cb + ca * sb
    assert np.max(np.abs(pred_c[:, :22] - cc[:, :22])) < 4e-7
    assert np.max(np.abs(pred_s[:, :22] - sc[:, :22])) < 4e-7


def test_spatial_tables_do_not_depend_on_start_frame():
    c1, s1 = tables.rope_tables(0, 1, 5, 7)
    c2, s2 = tables.rope_tables(41, 1, 5, 7)
    assert np.array_equal(c1[:, 22:], c2[:, 22:]) and np.array_equal(s1[:, 22:], s2[:, 22:])
    assert not np.array_equal(c1[:, :22], c2[:, :22])
