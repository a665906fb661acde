"""GPU parity of the clean-cache renoise / emit updates (unstep_renoise, unstep_emit) against
the oracle (oracle/schedule.py): bit-exact at the chunk latent shape and on a ragged length,
for the schedule's noise levels and the clean-cache level, in place and out of place.
Inputs from synth only; expected values from oracle only."""
import numpy as np
import pytest
import torch

import synth
from oracle import schedule
from tests.gpu_helpers import dev, host, log

pytestmark = pytest.mark.gpu

u = pytest.importorskip("paper_2609_32518_amd")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

SIGMAS = [0.0, 0.02, 0.625, 5.0 / 6.0, 0.9375, 1.0]


@pytest.mark.parametrize("shape", [(1, 16, 3, 60, 104), (1001,)])
def test_renoise_and_emit_bit_exact(shape):
    log(f"renoise/emit: shape {shape}")
    x = synth.normal_bf16(shape, (95, 0))
    e = synth.normal_bf16(shape, (95, 1))
    v = synth.normal_bf16(shape, (95, 2))
    xd, ed, vd = dev(x), dev(e), dev(v)
    for sigma in SIGMAS:
        xt = u.unstep_renoise(xd, ed, sigma)
        xn = u.unstep_emit(xt, vd, sigma)
        torch.cuda.synchronize()
        want_t = schedule.renoise_bf16(x, e, sigma)
        assert np.array_equal(host(xt), want_t), f"renoise sigma {sigma}"
        assert np.array_equal(host(xn), schedule.emit_bf16(want_t, v, sigma)), f"emit sigma {sigma}"


def test_in_place_and_identity_at_zero():
    x = synth.normal_bf16((4096,), (96, 0))
    e = synth.normal_bf16((4096,), (96, 1))
    xd = dev(x)
    u.unstep_renoise(xd, dev(e), 0.0, out=xd)              # sigma 0: the original clean pass
    torch.cuda.synchronize()
    assert np.array_equal(host(xd), x)
    u.unstep_renoise(xd, dev(e), 0.02, out=xd)             # in place
    torch.cuda.synchronize()
    assert np.array_equal(host(xd), schedule.renoise_bf16(x, e, 0.02))
