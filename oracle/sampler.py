"""DiT call sequence of the chunked causal sampler, and the per-layer attention windows
(Section 3.2, Section 3.3, Section 3.4 and Appendix A.2, A.3).

A clip is generated chunk by chunk (chunks of three latent frames; a 5 s clip of 81 video
frames is 21 latent frames, seven chunks).  Every DiT evaluation of a chunk is one call; a
call at noise level sigma renoises the current latent (Equation 1), evaluates the DiT at the
label t and emits the next latent (Equation 3), and every attention layer of the DiT appends
the chunk's keys and values to its cache and attends over its window.

Denoising steps use indices into the four-step shift-five table (sigma = 1, 15/16, 5/6, 5/8):

    self_forcing     every chunk: 0, 1, 2, 3
    unstep           chunk 0: 0, 1, 2, 3; later chunks: 0 then 2 or 3, alternating
    unstep_one_step  chunk 0: 0, 1, 2, 3; later chunks: 0

and every chunk ends with the clean-cache call at label t = 0 and noise level sigma_clean
(0 for Self Forcing, where renoise and emit are identities; 0.02 for UnStep).

Reading where the paper is silent: the alternation starts with index 2 (chunk 1 uses 2,
chunk 2 uses 3, chunk 3 uses 2, ...).

Windows (Appendix A.3): a layer keeps `sinks` sink frames (the first latent frames) and the
six most recent frames including the current chunk, i.e. W = 3 prior frames for three-frame
chunks; nine-frame layers keep three sinks, eight-frame layers two.  The paper does not say
which layers are eight-frame layers; callers name them.

Test infrastructure: nothing in the library imports this module.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List

from .schedule import SIGMA_CLEAN_UNSTEP, shift_schedule

VARIANTS = ("self_forcing", "unstep", "unstep_one_step")
CHUNK_FRAMES = 3
CLEAN = -1                      # schedule index of the clean-cache call


@dataclass(frozen=True)
class Call:
    chunk: int
    start_frame: int
    index: int                  # schedule index 0..3, or CLEAN
    sigma: float
    t: float


def chunk_indices(variant: str, chunk: int) -> List[int]:
    """Denoising schedule indices of one chunk (Section 3.2, Appendix A.2)."""
    if variant not in VARIANTS:
        raise ValueError(f"unknown variant {variant!r}")
    if chunk == 0 or variant == "self_forcing":
        return [0, 1, 2, 3]
    if variant == "unstep":
        return [0, 2 if chunk % 2 == 1 else 3]
    return [0]


def default_clean_sigma(variant: str) -> float:
    return 0.0 if variant == "self_forcing" else SIGMA_CLEAN_UNSTEP


def calls(variant: str, n_chunks: int, chunk_frames: int = CHUNK_FRAMES, clean_sigma=None) -> List[Call]:
    """Every DiT call of a clip of n_chunks chunks, in order."""
    if n_chunks < 0 or chunk_frames < 1:
        raise ValueError("n_chunks >= 0 and chunk_frames >= 1 required")
    cs = default_clean_sigma(variant) if clean_sigma is None else float(clean_sigma)
    _, sigma, t = shift_schedule(4, 5.0)
    out = []
    for c in range(n_chunks):
        f0 = c * chunk_frames
        for i in chunk_indices(variant, c):
            out.append(Call(c, f0, i, float(sigma[i]), float(t[i])))
        out.append(Call(c, f0, CLEAN, cs, 0.0))
    return out


def latent_frames(video_frames: int) -> int:
    """Latent frames of a clip: the first video frame alone, then four per latent frame."""
    return 1 + (video_frames - 1) // 4


RECENT_FRAMES = 6               # the most recent frames kept, the current chunk included


def layer_window(frame_budget: int, chunk_frames: int = CHUNK_FRAMES):
    """(sink frames S, prior window frames W, ring frames R) of a layer that keeps
    frame_budget latent frames: the six most recent (chunk included) plus the sinks.
    Nine-frame layers: (3, 3, 6); eight-frame layers: (2, 3, 6)."""
    S = frame_budget - RECENT_FRAMES
    if S < 0 or chunk_frames > RECENT_FRAMES:
        raise ValueError("frame budget below the recent frames")
    return S, RECENT_FRAMES - chunk_frames, RECENT_FRAMES
