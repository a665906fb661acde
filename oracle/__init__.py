"""Plain, slow CPU oracle of the windowed-attention chunk step (UnStep, arXiv 2609.32518).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything under
``oracle/``; the library itself never does, and the oracle shares no code with
it (only the seeded input generators in ``synth`` serve both).

What it defines, each in fp64 unless the paper fixes a precision:

* ``tables``   -- the per-chunk rotary cos/sin tables (Appendix A.5: cached fp32
                  coefficients keyed by start frame and grid).
* ``rope``     -- the pair rotation of Appendix A.5 under the rounding contract
                  "bf16 in, fp32 math, bf16 out", plus the ideal fp64 rotation.
* ``kvcache``  -- the sink + sliding-window KV cache with host-held indices
                  (Section 3.1, Section 3.3, Appendix A.3, Appendix A.5).
* ``attention`` -- exact softmax attention of the chunk's queries over the
                  retained keys, and a brute-force full-timeline masked version.
* ``rmsnorm``  -- the RMS normalisation of a token's query and key over all heads
                  before the rotation (Appendix A.5).
* ``schedule`` -- the shift-five noise schedule and the renoise/emit updates around
                  one DiT evaluation (Section 3.4, Equations 1 and 3).
* ``sampler``  -- the DiT call sequence of a clip for each sampler and the per-layer
                  attention windows (Sections 3.2-3.4, Appendix A.2 and A.3).
* ``svd``      -- the rank-r truncation of the value and output weights and the
                  projection after attention (Section 3.5, Appendix A.4).
* ``numerics`` -- the bf16 / binary32 rounding helpers the rest build on.

Where the paper is silent, the reading taken is stated in the function that
depends on it.  Parity of attention against the paper itself is unpinned (the
paper prints no tensor values for this path); it is pinned by brute force,
closed forms and invariants in ``tests/test_oracle_*.py``.
"""
from . import numerics, tables, rope, kvcache, attention, rmsnorm, schedule, sampler, svd  # noqa: F401
from .kvcache import OracleError  # noqa: F401
