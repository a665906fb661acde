"""GPU parity of the V/O truncated SVD (unstep_svd_truncate) and the projection after
attention (unstep_linear) against the oracle (oracle/svd.py), through the C ABI.
Inputs from synth only; expected values from oracle only."""
import numpy as np
import pytest
import torch

import synth
from oracle import numerics, svd
from tests.gpu_helpers import dev, host, log

pytestmark = pytest.mark.gpu

u = pytest.importorskip("paper_2609_32518_amd")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)


def _gaussian(m, n, seed):
    # a projection-like weight: N(0, 1/n) entries (Marchenko-Pastur spectrum)
    return synth.normal_f32((m, n), (seed, 500), 1.0 / np.sqrt(n))


def _gapped(m, n, r, seed):
    # random singular vectors (QR of seeded Gaussians) and a spectrum that halves at the cut,
    # so that the rank-r truncation is well conditioned and comparable element by element
    k = min(m, n)
    q1, _ = np.linalg.qr(synth.normal_f32((m, k), (seed, 501)).astype(np.float64))
    q2, _ = np.linalg.qr(synth.normal_f32((n, k), (seed, 502)).astype(np.float64))
    s = 1.5 * 0.999 ** np.arange(k)
    s[r:] *= 0.5
    return ((q1 * s) @ q2.T).astype(np.float32)


def _check_svd(w, r, sig, wr_d, wb_d, elementwise=True):
    m, n = w.shape
    wr = wr_d.cpu().numpy().astype(np.float64)
    s64 = svd.singular_values(w)
    want = svd.truncate(w, r)
    smax = s64[0]
    # float64 Gram matrix and eigendecomposition (backward error ~ sqrt(n) 2^-52 sigma_max^2 in
    # the Gram matrix): singular values within that over 2 sigma, the leading subspace within
    # it over the Gram eigenvalue gap at the cut (sensitivity 1 at rank 0 or the full rank),
    # then one rounding to float32 of each output value
    e64 = 64 * np.sqrt(max(m, n)) * 2.0 ** -52 * smax
    assert np.all(np.abs(sig.astype(np.float64) - s64) <= 2.0 ** -24 * s64 + e64 * smax / np.maximum(s64, 1e-300))
    cond = 1.0 + (2 * smax ** 2 / (s64[r - 1] ** 2 - s64[r] ** 2) if 0 < r < min(m, n) else 0.0)
    err = np.abs(wr - want)
    lim = 2.0 ** -24 * np.abs(want) + e64 * cond
    log(f"  max |W_r - oracle| {err.max():.3g}; worst slack {(err / lim).max():.3f}; cond {cond:.3g}")
    if elementwise:
        assert np.all(err <= lim)
    e32 = 2.0 ** -24 * smax * np.sqrt(min(m, n))
    # Eckart-Young on the library's own result: residual energy and rank
    e = w.astype(np.float64) - wr
    assert np.isclose(np.sum(e * e), np.sum(s64[r:] ** 2), rtol=1e-4, atol=(e32 * min(m, n)) ** 2)
    if r < min(m, n):
        assert svd.singular_values(wr)[r] <= e32
    # the stored bf16 weight is the float32 result rounded to nearest even
    assert np.array_equal(host(wb_d), numerics.f32_to_bf16_bits(wr_d.cpu().numpy()))


@pytest.mark.parametrize("m,n,r", [(1536, 1536, 1413), (96, 160, 88), (160, 96, 40), (160, 96, 0), (64, 64, 64)])
def test_svd_truncation_well_conditioned(m, n, r):
    log(f"svd (gap at the cut): {m}x{n} rank {r}")
    w = _gapped(m, n, r, m + n + r)
    wr_d, wb_d, sig = u.unstep_svd_truncate(torch.from_numpy(w).cuda(), r)
    torch.cuda.synchronize()
    _check_svd(w, r, sig, wr_d, wb_d)


def test_svd_truncation_gaussian_weight_at_the_paper_rank():
    # no gap at the cut: the truncation is less well conditioned, the bound scales with it
    r = svd.rank_for(1536)                        # the paper's rank, 1413
    w = _gaussian(1536, 1536, 7)
    wr_d, wb_d, sig = u.unstep_svd_truncate(torch.from_numpy(w).cuda(), r)
    torch.cuda.synchronize()
    _check_svd(w, r, sig, wr_d, wb_d)


def _linear_bound(x_bits, w_bits, b_bits):
    # fp32 accumulation over K terms (each product exact in fp32) plus the bf16 rounding of y:
    # |err| <= 2^-8 |y| + K 2^-24 (sum_k |x_k w_k| + |b|)
    x = np.abs(numerics.bf16_to_f64(x_bits))
    w = np.abs(numerics.bf16_to_f64(w_bits))
    mag = x @ w.T
    if b_bits is not None:
        mag = mag + np.abs(numerics.bf16_to_f64(b_bits))
    return x.shape[-1] * 2.0 ** -24 * mag


@pytest.mark.parametrize("M,N,K,bias", [(4680, 1536, 1536, True), (72, 1536, 1536, True), (4680, 1536, 1536, False),
                                        (1, 128, 200, True), (300, 256, 8, False), (513, 384, 1032, True),
                                        (1, 40, 48, True), (257, 24, 64, False), (1000, 200, 640, True),
                                        (4680, 1536, 128, True)])
def test_linear(M, N, K, bias):
    log(f"linear: M {M} N {N} K {K} bias {bias}")
    x = synth.normal_bf16((M, K), (M, N, K, 1))
    w = synth.normal_bf16((N, K), (M, N, K, 2), 1.0 / np.sqrt(K))
    b = synth.normal_bf16((N,), (M, N, K, 3)) if bias else None
    y = u.unstep_linear(dev(x), dev(w), dev(b) if bias else None)
    torch.cuda.synchronize()
    got = numerics.bf16_to_f64(host(y))
    want = svd.linear(x, w, b)
    err = np.abs(got - want)
    lim = 2.0 ** -8 * np.abs(want) + _linear_bound(x, w, b)
    log(f"  max err {err.max():.3g}, mean err {err.mean():.3g}; worst slack {(err / lim).max():.3f}")
    assert np.all(err <= lim)


@pytest.mark.parametrize("M,N,K", [(4680, 1536, 1536), (64, 1536, 12288)])
def test_linear_on_two_streams_at_once(M, N, K):
    # calls enqueued on two streams may run at the same time: the kernel keeps no state between
    # calls and uses no scratch, so every result is bit-identical to the call run alone and
    # within the oracle's bound (the deep-K shape runs 192 k steps per tile)
    log(f"linear on two streams: M {M} N {N} K {K}")
    xs = [dev(synth.normal_bf16((M, K), (M, N, K, 10 + i))) for i in range(2)]
    w = dev(synth.normal_bf16((N, K), (M, N, K, 12), 1.0 / np.sqrt(K)))
    b = dev(synth.normal_bf16((N,), (M, N, K, 13)))
    alone = [u.unstep_linear(x, w, b) for x in xs]                # default stream
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for _ in range(4)] for _ in range(2)]
    torch.cuda.synchronize()
    for rep in range(4):
        for i in range(2):
            u.unstep_linear(xs[i], w, b, out=outs[i][rep], stream=streams[i])
    torch.cuda.synchronize()
    for i in range(2):
        want = svd.linear(host(xs[i]), host(w), host(b))
        lim = 2.0 ** -8 * np.abs(want) + _linear_bound(host(xs[i]), host(w), host(b))
        same = 0
        for rep in range(4):
            got = numerics.bf16_to_f64(host(outs[i][rep]))
            assert np.all(np.abs(got - want) <= lim), (i, rep)
            same += bool(torch.equal(outs[i][rep].view(torch.int16), alone[i].view(torch.int16)))
        log(f"  stream {i}: {same} of 4 results bit-identical to the call run alone")
        assert same == 4
