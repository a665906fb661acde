"""Pins of the sampler call sequence and per-layer windows (oracle/sampler.py) against the
paper's stated step counts, schedule table, clip length and window budget, and a brute-force
"first S frames plus the six newest" timeline that shares no formula with the cache oracle."""
import json
import os
from fractions import Fraction

import pytest

from oracle import kvcache, sampler

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))
STEPS = GOLDEN["denoising_steps_per_chunk"]
SIGMA_EXACT = [float(Fraction(s)) for s in GOLDEN["shift_five_schedule"]["sigma_exact"]]


@pytest.mark.parametrize("variant", sampler.VARIANTS)
@pytest.mark.parametrize("n_chunks", [0, 1, 2, 7, 41])
def test_call_counts_follow_the_stated_steps(variant, n_chunks):
    calls = sampler.calls(variant, n_chunks)
    per = STEPS[variant]
    want = 0 if n_chunks == 0 else (per["first_chunk"] + STEPS["clean_calls_per_chunk"]
                                    + (n_chunks - 1) * (per["later_chunks"] + STEPS["clean_calls_per_chunk"]))
    assert len(calls) == want
    # chunks in order, each ending with exactly one clean call at label 0
    assert [c.chunk for c in calls] == sorted(c.chunk for c in calls)
    for ch in range(n_chunks):
        mine = [c for c in calls if c.chunk == ch]
        assert mine[-1].index == sampler.CLEAN and mine[-1].t == 0.0
        assert sum(c.index == sampler.CLEAN for c in mine) == 1
        assert all(c.start_frame == 3 * ch for c in mine)


def test_first_chunk_and_later_chunks_use_the_table():
    for variant in sampler.VARIANTS:
        first = [c for c in sampler.calls(variant, 1) if c.index != sampler.CLEAN]
        assert [c.index for c in first] == STEPS["first_chunk_indices"]
        assert [c.sigma for c in first] == SIGMA_EXACT
        assert [c.t for c in first] == [1000.0 * s for s in SIGMA_EXACT]
    calls = sampler.calls("unstep", 9)
    seconds = []
    for ch in range(1, 9):
        mine = [c for c in calls if c.chunk == ch and c.index != sampler.CLEAN]
        assert mine[0].index == STEPS["later_chunk_first_index"] and mine[0].sigma == 1.0
        seconds.append(mine[1].index)
        assert mine[1].sigma == SIGMA_EXACT[mine[1].index]
    # alternating between the two stated indices: both occur and never twice in a row
    assert set(seconds) == set(STEPS["later_chunk_second_index_alternates"])
    assert all(a != b for a, b in zip(seconds, seconds[1:]))
    one = [c for c in sampler.calls("unstep_one_step", 5) if c.chunk > 0 and c.index != sampler.CLEAN]
    assert {c.index for c in one} == {0}


def test_clean_noise_levels():
    cc = GOLDEN["clean_cache_noise"]
    assert {c.sigma for c in sampler.calls("self_forcing", 3) if c.index == sampler.CLEAN} == {cc["sigma_self_forcing"]}
    for v in ("unstep", "unstep_one_step"):
        assert {c.sigma for c in sampler.calls(v, 3) if c.index == sampler.CLEAN} == {cc["sigma_unstep"]}
    assert {c.sigma for c in sampler.calls("unstep", 2, clean_sigma=0.05) if c.index == sampler.CLEAN} == {0.05}


def test_clip_length():
    g = GOLDEN["latent_frames_per_clip"]
    assert sampler.latent_frames(81) == g["value"]
    assert g["value"] // sampler.CHUNK_FRAMES == g["chunks"]
    last = sampler.calls("unstep", g["chunks"])[-1]
    assert last.start_frame + sampler.CHUNK_FRAMES == g["value"]


def _brute_window(S: int, f0: int, C: int):
    # every frame generated so far, keep the first S and the six newest (chunk included)
    seen = list(range(f0 + C))
    newest = seen[-sampler.RECENT_FRAMES:]
    return sorted(set(seen[:S]) | set(newest))


@pytest.mark.parametrize("budget", [9, 8])
def test_layer_windows_match_the_budget(budget):
    S, W, R = sampler.layer_window(budget)
    g = GOLDEN["windowed_tokens"] if budget == 9 else GOLDEN["eight_frame_layers"]
    assert S == g["sink_frames"] and W + sampler.CHUNK_FRAMES == g["recent_frames_including_chunk"]
    assert R >= W + sampler.CHUNK_FRAMES
    for ch in range(41):
        f0 = 3 * ch
        got = kvcache.retained_frames(f0, 3, S, W)
        assert got == _brute_window(S, f0, 3)
        assert len(got) == min(f0 + 3, budget)
    # full cache: 9 frames = the paper's 14,040 tokens; 8 frames = 12,480
    assert budget * GOLDEN["tokens_per_frame"]["value"] == (14040 if budget == 9 else 12480)
    with pytest.raises(ValueError):
        sampler.layer_window(5)


def test_unknown_variant():
    with pytest.raises(ValueError):
        sampler.calls("nope", 2)


def test_dit_forwards_of_the_five_second_clip():
    g = GOLDEN["dit_forwards_per_clip"]
    assert len(sampler.calls("self_forcing", g["chunks"])) == g["self_forcing"]
    assert len(sampler.calls("unstep", g["chunks"])) == g["unstep"]
