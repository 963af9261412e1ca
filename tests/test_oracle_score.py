"""Pins for the oracle's binary16 conversions and scores (Sec. 4.3).

The KV-norm sum is checked against exact rational arithmetic in Python
(``fractions.Fraction`` over the exact binary16 values) and against closed
forms; the conversions against numpy's IEEE 754 binary16 casts.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2606_08635_amd import workloads


def test_half_decode_matches_numpy_for_every_pattern():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    want = bits.view(np.float16).astype(np.float64)
    got = np.array([oracle.half_to_double(int(b)) for b in bits])
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    # signs of zeros too
    assert math.copysign(1.0, oracle.half_to_double(0x8000)) == -1.0


def test_float_to_half_matches_numpy_rne():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * np.float32(rng.choice([1e-6, 1e-3, 1, 300, 6e4], 20000)),
        # exact halfway points between adjacent binary16 values (ties to even)
        ((np.arange(1, 4000, dtype=np.float64) + 0.5) * 2.0 ** -24).astype(np.float32),
        ((np.arange(1024, 3000, dtype=np.float64) + 0.5) * 2.0 ** -10).astype(np.float32),
        np.array([0.0, -0.0, 65504, 65519.996, 65520, 7e4, -7e4, np.inf, -np.inf,
                  2.0 ** -24, 2.0 ** -25, 2.0 ** -25 * 1.0000001, 2.0 ** -14, 2.0 ** -14 * (1 - 2 ** -12),
                  6.1e-5, 1.0, -1.0], np.float32),
    ])
    with np.errstate(over="ignore"):
        want = vals.astype(np.float16).view(np.uint16)
    got = np.array([oracle.float_to_half(float(v)) for v in vals], np.uint16)
    assert np.array_equal(got, want), vals[got != want][:10]
    assert oracle.float_to_half(float("nan")) == 0x7E00


def _exact_sumsq(k, v, t):
    """sum over (l, h, i) of k^2 + v^2 for token t, exact, in units of 2^-48."""
    kk = k[:, :, t, :].astype(np.float64).ravel()
    vv = v[:, :, t, :].astype(np.float64).ravel()
    s = Fraction(0)
    for x in np.concatenate([kk, vv]):
        if np.isfinite(x):
            s += Fraction(float(x)) ** 2
    s *= 2 ** 48
    assert s.denominator == 1
    return int(s)


def _rand_half_bits(rng, shape):
    """binary16 patterns spread over every exponent, including subnormals and extremes."""
    bits = rng.integers(0, 0x7C00, size=shape, dtype=np.int64)
    sign = rng.integers(0, 2, size=shape) << 15
    return (bits | sign).astype(np.uint16)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_kvnorm_sum_is_exact(seed):
    rng = np.random.default_rng(seed)
    L, H, n, d = 2, 3, 5, 32
    k = _rand_half_bits(rng, (L, H, n, d))
    v = _rand_half_bits(rng, (L, H, n, d))
    # plant the extremes: largest finite, smallest subnormal, both zeros, inf, NaN
    k[0, 0, 0, :6] = [0x7BFF, 0x0001, 0x0000, 0x8000, 0x7C00, 0x7E01]
    v[1, 2, 3, :3] = [0xFBFF, 0x8001, 0xFC00]
    cfg = oracle.config(L, H, d, n, 0.5)
    for t in range(n):
        assert oracle.sumsq(cfg, k, v, t) == _exact_sumsq(k.view(np.float16), v.view(np.float16), t)


def test_kvnorm_constant_rows_closed_form():
    L, H, n, d = 3, 2, 4, 64
    for c in [1.0, 0.5, 3.25, 2.0 ** -20, 65504.0]:
        k = np.full((L, H, n, d), c, np.float16)
        v = np.full((L, H, n, d), -c, np.float16)
        cfg = oracle.config(L, H, d, n, 0.5)
        S = oracle.sumsq(cfg, k, v, 2)
        assert Fraction(S, 2 ** 48) == 2 * L * H * d * Fraction(float(np.float16(c))) ** 2


def test_kvnorm_key_rounding_and_decay():
    rng = np.random.default_rng(7)
    L, H, n, d = 1, 2, 40, 64
    k = _rand_half_bits(rng, (L, H, n, d))
    v = _rand_half_bits(rng, (L, H, n, d))
    lam = 0.01
    cfg = oracle.config(L, H, d, n, 0.5, decay=lam)
    key = oracle.score(cfg, k, v)
    w2 = oracle.decay_table(lam, 2, n)
    for t in range(n):
        S = oracle.sumsq(cfg, k, v, t)
        # Python's int -> float is correctly rounded; the 2^-48 scaling is exact
        assert key[t] == (float(S) * 2.0 ** -48) * w2[n - 1 - t]


def test_nonfinite_elements_contribute_nothing():
    L, H, n, d = 1, 1, 3, 32
    k = np.ones((L, H, n, d), np.float16)
    v = np.ones((L, H, n, d), np.float16)
    cfg = oracle.config(L, H, d, n, 0.5)
    base = oracle.sumsq(cfg, k, v, 1)
    k[0, 0, 1, 5] = np.inf
    v[0, 0, 1, 7] = np.nan
    assert oracle.sumsq(cfg, k, v, 1) == base - 2 * 2 ** 48


@pytest.mark.parametrize("lam", [0.0, 0.001, 0.005, 0.01])
def test_decay_tables(lam):
    n = 32768
    w1 = oracle.decay_table(lam, 1, n)
    w2 = oracle.decay_table(lam, 2, n)
    assert w1[0] == 1.0 and w2[0] == 1.0
    assert np.all(np.diff(w1) <= 0) and np.all(np.diff(w2) <= 0)
    # e^{-2 lam D} = (e^{-lam D})^2 up to a few rounding errors
    ok = w1 > 1e-300
    assert np.allclose(w2[ok], w1[ok] ** 2, rtol=1e-14, atol=0)
    # e^{-lam D} = (e^{-lam})^D
    D = np.arange(n)
    lam32 = float(np.float32(lam))  # the configuration carries lambda as a binary32
    assert np.allclose(w1, np.exp(-lam32) ** D, rtol=1e-11, atol=1e-300)
    if lam == 0.0:
        assert np.all(w1 == 1.0) and np.all(w2 == 1.0)


def test_recency_mode_is_the_decay_factor():
    n = 100
    cfg = oracle.config(1, 1, 32, n, 0.5, decay=0.01, score_mode=oracle.RECENCY)
    k = np.zeros((1, 1, n, 32), np.uint16)
    key = oracle.score(cfg, k, k)
    assert np.allclose(key, np.exp(-float(np.float32(0.01)) * (n - 1 - np.arange(n))), rtol=1e-12)
    assert np.all(np.diff(key) > 0)


def test_generated_workload_shapes_and_outliers():
    k, v = workloads.make_kv(2, 3, 100, 64, seed=0)
    assert k.shape == (2, 3, 100, 64) and k.dtype == torch.float16
    # 4 outlier channels per (layer, head): their RMS is about 8x the others'
    rms = k.float().pow(2).mean(dim=2).sqrt()  # [L, H, d]
    top = rms.topk(4, dim=-1).values.mean()
    rest = rms.sort(dim=-1).values[..., :-4].mean()
    assert 5 < float(top / rest) < 11
    k2, _ = workloads.make_kv(2, 3, 100, 64, seed=0)
    assert torch.equal(k, k2)
