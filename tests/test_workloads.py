"""The shared seeded inputs: determinism, shapes, the bounded Zipf law and bf16 rounding."""

import numpy as np

import workloads as W
from workloads.gen import round_bf16, zipf_cdf


def test_bf16_rounding_is_nearest_even():
    # independent check: pick the nearer of the two neighbouring bf16 grid points, ties to the even one
    x = np.random.default_rng(0).uniform(-3, 3, 200000).astype(np.float32)
    x[:4] = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0], np.float32)   # exact ties
    y = round_bf16(x)
    xb = x.view(np.uint32).astype(np.int64)
    lo = xb & ~0xFFFF
    hi = lo + 0x10000
    flo = lo.astype(np.uint32).view(np.float32).astype(np.float64)
    fhi = hi.astype(np.uint32).view(np.float32).astype(np.float64)
    d0, d1 = np.abs(x - flo), np.abs(fhi - x)
    ref = np.where((d0 < d1) | ((d0 == d1) & (((lo >> 16) & 1) == 0)), flo, fhi).astype(np.float32)
    np.testing.assert_array_equal(y, ref)
    assert y[0] == 1.0 and y[1] == np.float32(1.0 + 2 ** -6)


def test_batches_are_seeded_and_padded():
    w = W.get("default")
    a, la = W.make_batch(w)
    b, lb = W.make_batch(w)
    np.testing.assert_array_equal(a, b)
    assert a.shape == (64, 50) and la.min() >= 10 and la.max() <= 50
    for i in range(64):
        assert (a[i, :la[i]] >= 4).all() and (a[i, la[i]:] == W.PAD_ID).all()


def test_zipf_cdf_bounded_and_exponent():
    c = zipf_cdf(1000, 1.0)
    assert c[-1] == 1.0 and np.all(np.diff(c) > 0)
    p = np.diff(np.concatenate([[0.0], c]))
    assert abs(p[0] / p[1] - 2.0) < 1e-12 and abs(p[0] / p[9] - 10.0) < 1e-9


def test_weights_are_deterministic_and_in_range():
    w = W.get("tiny")
    a = W.make_weights(w)
    b = W.make_weights(w)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
        assert a[k].dtype == np.float32 and np.abs(a[k]).max() <= 0.1
