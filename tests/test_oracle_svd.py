"""Pins of the V/O truncated-SVD and projection oracle (oracle/svd.py): the paper's rank and
layer range, a matrix of known singular vectors and values built without an SVD, the
Eckart-Young error in the spectral norm by power iteration and in the Frobenius norm, the
orthogonality of kept and discarded parts, optimality against random rank-r matrices, the
rank extremes, and the projection against torch's linear and a brute-force sum."""
import json
import os

import numpy as np
import pytest
import torch

import synth
from oracle import numerics, svd

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))["vo_svd"]


def _orthogonal(n, seed):
    q, r = np.linalg.qr(np.random.default_rng(seed).standard_normal((n, n)))
    return q * np.sign(np.diag(r))


def _known(m, n, seed):
    k = min(m, n)
    u = _orthogonal(m, seed)[:, :k]
    v = _orthogonal(n, seed + 1)[:, :k]
    s = np.sort(np.random.default_rng(seed + 2).uniform(0.05, 3.0, k))[::-1]
    return u, s, v


def test_paper_rank_and_layers():
    assert svd.rank_for(GOLDEN["dim"], GOLDEN["retain"]) == GOLDEN["rank"]
    layers = svd.truncated_layers(GOLDEN["layers"], GOLDEN["first_truncated_layer"])
    assert layers[0] == 8 and layers[-1] == 29 and len(layers) == 22


@pytest.mark.parametrize("m,n,r", [(96, 96, 88), (64, 80, 40), (80, 48, 44)])
def test_known_spectrum_truncation(m, n, r):
    u, s, v = _known(m, n, 11 * m + n)
    w = (u * s) @ v.T
    assert np.allclose(svd.singular_values(w), s, rtol=1e-12, atol=1e-12)
    want = (u[:, :r] * s[:r]) @ v[:, :r].T
    assert np.allclose(svd.truncate(w, r), want, rtol=0, atol=1e-12)


def test_eckart_young_and_orthogonality():
    w = np.random.default_rng(3).standard_normal((160, 160)).astype(np.float32).astype(np.float64) / 13.0
    r = svd.rank_for(160)
    wr = svd.truncate(w, r)
    s = svd.singular_values(w)
    e = w - wr
    # spectral norm of the residual by power iteration on e^T e (no SVD involved)
    x = np.random.default_rng(4).standard_normal(160)
    for _ in range(3000):
        x = e.T @ (e @ x)
        x /= np.linalg.norm(x)
    assert np.isclose(np.linalg.norm(e @ x), s[r], rtol=1e-6)
    assert np.isclose(np.sum(e * e), np.sum(s[r:] ** 2), rtol=1e-10)
    assert np.isclose(np.sum(wr * wr), np.sum(s[:r] ** 2), rtol=1e-10)
    assert np.abs(wr.T @ e).max() < 1e-12 and np.abs(e @ wr.T).max() < 1e-12
    # no random rank-r matrix does better in the Frobenius norm
    rng = np.random.default_rng(5)
    for _ in range(5):
        b = rng.standard_normal((160, r)) @ rng.standard_normal((r, 160)) / 160
        assert np.sum((w - b) ** 2) > np.sum(e * e)
    # rank extremes
    assert np.allclose(svd.truncate(w, 160), w, rtol=0, atol=1e-12)
    assert not np.any(svd.truncate(w, 0))
    with pytest.raises(ValueError):
        svd.truncate(w, 161)


def test_stored_weight_is_the_rounded_reconstruction():
    w = np.random.default_rng(6).standard_normal((64, 64)).astype(np.float32)
    bits = svd.truncate_bf16(w, 50)
    ref = torch.from_numpy(svd.truncate(w, 50)).to(torch.float32).to(torch.bfloat16)
    assert np.array_equal(bits, ref.view(torch.int16).numpy().view(np.uint16))


def test_linear_matches_torch_and_brute_force():
    x = synth.normal_bf16((5, 7, 48), (80, 0))
    w = synth.normal_bf16((33, 48), (80, 1), 0.2)
    b = synth.normal_bf16((33,), (80, 2))
    y = svd.linear(x, w, b)
    xt, wt, bt = (torch.from_numpy(numerics.bf16_to_f64(a)) for a in (x, w, b))
    assert np.allclose(y, torch.nn.functional.linear(xt, wt, bt).numpy(), rtol=1e-14, atol=1e-14)
    xf, wf, bf = (numerics.bf16_to_f64(a) for a in (x, w, b))
    for (i, j, n) in ((0, 0, 0), (4, 6, 32), (2, 3, 17)):
        assert np.isclose(y[i, j, n], sum(xf[i, j, k] * wf[n, k] for k in range(48)) + bf[n], rtol=1e-14)
    assert np.allclose(svd.linear(x, w), y - bf, rtol=1e-13, atol=1e-13)
    with pytest.raises(ValueError):
        svd.linear(x, w[:, :40])
