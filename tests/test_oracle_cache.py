"""Pins for the oracle's sink + window KV cache (paper Sections 3.1, 3.3; Appendix A.3, A.5).

* closed forms the paper states: 1560 tokens per frame, 32760 keys for the full
  21-frame context, 14040 keys for 3 sinks + 6 recent frames;
* repeated calls for the same chunk overwrite in place and do not advance;
* the ring's contents for the retained frames equal a plain timeline record
  of every frame ever written (a brute-force model with no slot arithmetic).
"""
import json
import os

import numpy as np
import pytest

import synth
from oracle import kvcache
from oracle.kvcache import KVCacheOracle, OracleError

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _chunk(cache, f0, C, key):
    shape = (cache.B, C * cache.T, cache.H, cache.D)
    return synth.normal_bf16(shape, key + (synth.K,)), synth.normal_bf16(shape, key + (synth.V,))


def test_paper_token_counts():
    g = GOLDEN
    T = g["tokens_per_frame"]["grid_h"] * g["tokens_per_frame"]["grid_w"]
    assert T == g["tokens_per_frame"]["value"]
    # full context: the last chunk of a 21-frame clip with every frame kept
    full = kvcache.retained_frames(18, 3, 0, 10 ** 6)
    assert len(full) * T == g["full_context_tokens"]["value"]
    # UnStep window: 3 sinks + 6 recent frames including the chunk, once the cache is full
    w = g["windowed_tokens"]
    for f0 in (9, 12, 15, 18, 120):
        fr = kvcache.retained_frames(f0, w["chunk_frames"], w["sink_frames"],
                                     w["recent_frames_including_chunk"] - w["chunk_frames"])
        assert len(fr) * T == w["value"]
        assert fr[:3] == [0, 1, 2] and fr[-1] == f0 + 2 and fr[3] == f0 - 3


def test_early_chunks_keep_everything():
    # before the window fills, nothing is evicted and sinks are not duplicated
    assert kvcache.retained_frames(0, 3, 3, 3) == [0, 1, 2]
    assert kvcache.retained_frames(3, 3, 3, 3) == [0, 1, 2, 3, 4, 5]
    assert kvcache.retained_frames(6, 3, 3, 3) == [0, 1, 2, 3, 4, 5, 6, 7, 8]
    assert kvcache.retained_frames(6, 3, 3, 2) == [0, 1, 2, 4, 5, 6, 7, 8]


def test_slot_map_closed_form():
    S, R = 3, 6
    assert [kvcache.slot_of_frame(f, S, R) for f in range(12)] == [0, 1, 2, 3, 4, 5, 6, 7, 8, 3, 4, 5]
    assert [kvcache.slot_of_frame(f, 0, 12) for f in (0, 11, 12, 59)] == [0, 11, 0, 11]


def test_repeated_call_overwrites_without_advancing():
    c = KVCacheOracle(1, 2, 128, 2, 3, 0, 9)
    k0, v0 = _chunk(c, 0, 3, (1, 0))
    c.append(0, 3, k0, v0)
    k1, v1 = _chunk(c, 3, 3, (1, 1))
    c.append(3, 3, k1, v1)
    newest, fmap = c.newest, list(c.frame_of_slot)
    k2, v2 = _chunk(c, 3, 3, (1, 2))
    c.append(3, 3, k2, v2)                     # second denoising call for the same chunk
    assert c.newest == newest and c.frame_of_slot == fmap
    rows = c.key_rows(3, 3, 3)
    assert np.array_equal(c.k[0][:, rows, :], np.transpose(np.concatenate([k0, k2], axis=1)[0], (1, 0, 2)))
    assert np.array_equal(c.v[0][:, rows[-18:], :], np.transpose(v2[0], (1, 0, 2)))


def test_rewriting_an_older_resident_chunk_keeps_newest():
    c = KVCacheOracle(1, 1, 128, 1, 2, 0, 9)
    for f0 in (0, 3, 6):
        k, v = _chunk(c, f0, 3, (6, f0))
        c.append(f0, 3, k, v)
    k, v = _chunk(c, 3, 3, (6, 99))
    c.append(3, 3, k, v)                            # older chunk, still resident
    assert c.newest == 8
    assert c.retained(6, 3, 6) == list(range(9))
    k, v = _chunk(c, 9, 3, (6, 9))
    c.append(9, 3, k, v)                            # continues after frame 8, evicts 0..2
    assert c.frame_of_slot == [9, 10, 11, 3, 4, 5, 6, 7, 8]


def test_ring_matches_timeline_record():
    # stream 1-frame chunks through a small ring with sinks; compare every retained frame's
    # contents with a record {frame: rows} kept without any slot arithmetic
    B, H, D, gh, gw, S, R, W = 1, 2, 128, 2, 2, 2, 4, 3
    c = KVCacheOracle(B, H, D, gh, gw, S, R)
    record = {}
    for f in range(15):
        k, v = _chunk(c, f, 1, (2, f))
        c.append(f, 1, k, v)
        record[f] = (k[0], v[0])                  # [T, H, D]
        if f % 3 == 0 and f > 0:                  # a refine pass re-writes the same frame
            k, v = _chunk(c, f, 1, (3, f))
            c.append(f, 1, k, v)
            record[f] = (k[0], v[0])
        frames = c.retained(f, 1, W)
        rows = c.key_rows(f, 1, W)
        want_k = np.concatenate([record[g][0] for g in frames], axis=0)   # [n, H, D]
        want_v = np.concatenate([record[g][1] for g in frames], axis=0)
        assert np.array_equal(np.transpose(c.k[0][:, rows, :], (1, 0, 2)), want_k)
        assert np.array_equal(np.transpose(c.v[0][:, rows, :], (1, 0, 2)), want_v)
        expect = sorted(set(range(min(S, max(0, f - W)))) | set(range(max(0, f - W), f + 1)))
        assert frames == expect


def test_segments_merge_and_wrap():
    c = KVCacheOracle(1, 1, 128, 1, 2, 3, 6)       # T = 2
    for f0 in range(0, 12, 3):
        k, v = _chunk(c, f0, 3, (4, f0))
        c.append(f0, 3, k, v)
    # frames 0,1,2 sinks (slots 0..2); 6..11 in ring slots 6,7,8,3,4,5
    assert c.segments(9, 3, 3) == [(0, 6), (12, 6), (6, 6)]
    assert c.segments(9, 3, 0) == [(0, 12)]          # sinks and slots 3..5 are adjacent rows


def test_errors():
    c = KVCacheOracle(1, 1, 128, 1, 2, 0, 4)
    k, v = _chunk(c, 0, 2, (5, 0))
    with pytest.raises(OracleError) as e:
        c.append(1, 2, k, v)                        # gap: nothing written yet
    assert e.value.kind == "state"
    c.append(0, 2, k, v)
    with pytest.raises(OracleError) as e:
        c.retained(2, 1, 1)                         # frame 2 never appended
    assert e.value.kind == "state"
    for f0 in (2, 4):
        c.append(f0, 2, k, v)
    with pytest.raises(OracleError) as e:
        c.append(0, 2, k, v)                        # frames 0, 1 were evicted by 4, 5
    assert e.value.kind == "state"
    with pytest.raises(OracleError) as e:
        c.retained(4, 2, 3)                         # 3 prior + 2 chunk frames > 4 ring frames
    assert e.value.kind == "range"
    big = synth.normal_bf16((1, 10, 1, 128), (5, 1))
    with pytest.raises(OracleError) as e:
        c.append(6, 5, big, big)                    # chunk larger than the ring
    assert e.value.kind == "range"
    with pytest.raises(OracleError) as e:
        c.retained(4, 0, 1)
    assert e.value.kind == "shape"
