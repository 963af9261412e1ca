"""Pins for the oracle's tier assignment.

Proposition 1 (Sec. 2.3, exchange argument): for fixed tier counts an
optimal assignment never gives a lower-precision tier to a more important
token than to a less important one.  Sinks are pinned to FP16 before ranking
(Sec. 4.4; Algorithm 1, scoring).  Checked by brute force over every placement
on tiny inputs, by the monotonicity property on large ones, and by the closed
form of the recency-only score.
"""
import itertools
import struct

import numpy as np
import pytest

import oracle

PREC = {oracle.FP16: 3, oracle.INT8: 2, oracle.INT4: 1, oracle.DROP: 0}


def _cfg(n, b, tiers=3, sink=0, mode=oracle.KVNORM, decay=0.0):
    return oracle.config(1, 1, 32, n, b, num_sink=sink, num_tiers=tiers, score_mode=mode, decay=decay)


def _counts(tier):
    return [int(np.sum(tier == t)) for t in range(4)]


@pytest.mark.parametrize("seed", range(6))
def test_brute_force_optimal_and_unique(seed):
    rng = np.random.default_rng(seed)
    for trial in range(12):
        n = int(rng.integers(2, 9))
        tiers = int(rng.integers(2, 4))
        b = float(np.float32(rng.uniform(0.2, 1.0)))
        sink = int(rng.integers(0, 2))
        cfg = _cfg(n, b, tiers, sink)
        try:
            p = oracle.plan(cfg)
        except oracle.OracleError:
            continue
        key = rng.permutation(np.arange(1, n + 1)).astype(np.float64) * rng.uniform(0.5, 2.0)
        tier = oracle.assign(cfg, key)
        s = p["n_sink"]
        assert np.all(tier[:s] == oracle.FP16)
        multiset = [oracle.FP16] * p["n_fp16"] + [oracle.INT8] * p["n_int8"] + \
                   [oracle.INT4] * p["n_int4"] + [oracle.DROP] * p["n_drop"]
        for _ in range(3):
            delta = np.sort(rng.uniform(0, 10, 4))  # strictly increasing error per tier
            delta_of = {oracle.FP16: delta[0], oracle.INT8: delta[1], oracle.INT4: delta[2], oracle.DROP: delta[3]}
            best, best_maps = None, set()
            for perm in set(itertools.permutations(multiset)):
                obj = sum(key[s + i] * delta_of[perm[i]] for i in range(len(perm)))
                if best is None or obj < best - 1e-9:
                    best, best_maps = obj, {perm}
                elif abs(obj - best) <= 1e-9:
                    best_maps.add(perm)
            assert best_maps == {tuple(int(x) for x in tier[s:])}, (key, tier, best_maps)


@pytest.mark.parametrize("seed", range(3))
def test_monotone_in_score_and_counts(seed):
    rng = np.random.default_rng(seed)
    n = 20000
    cfg = oracle.config(1, 1, 32, n, 0.37, first_ratio=0.02, num_tiers=3, decay=0.0)
    p = oracle.plan(cfg)
    key = rng.lognormal(0, 2, n)
    key[rng.integers(0, n, 500)] = key[0]  # many exact ties
    tier = oracle.assign(cfg, key)
    assert _counts(tier) == [p["n_sink"] + p["n_fp16"], p["n_int8"], p["n_int4"], p["n_drop"]]
    s = p["n_sink"]
    assert np.all(tier[:s] == oracle.FP16)
    comp = np.array([oracle.composite(key[t], t) for t in range(s, n)], dtype=np.uint64)
    prec = np.array([PREC[int(x)] for x in tier[s:]])
    order = np.argsort(comp)[::-1]
    # precision never increases along decreasing composite key
    assert np.all(np.diff(prec[order]) <= 0)


def test_ties_go_to_the_more_recent_token():
    n = 10
    cfg = _cfg(n, 0.375, 3)  # B = 15 over 10 tokens: 5 int8, 5 int4
    tier = oracle.assign(cfg, np.ones(n))
    assert list(tier) == [oracle.INT4] * 5 + [oracle.INT8] * 5


def test_composite_key_layout():
    # 32 fraction bits of the binary64 score, then the index in 21 bits
    x = 1.2345678901234567
    bits = struct.unpack("<Q", struct.pack("<d", x))[0]
    assert oracle.composite(x, 77) == ((bits >> 20) << 21) | 77
    # scores that are not positive, or NaN, rank as +0
    for bad in [0.0, -0.0, -3.0, float("nan"), -float("inf")]:
        assert oracle.composite(bad, 5) == 5
    assert oracle.composite(float("inf"), 5) == ((0x7FF0000000000000 >> 20) << 21) | 5
    # scores that differ only below the 32nd fraction bit tie and fall back to the index
    y = struct.unpack("<d", struct.pack("<Q", bits + 1))[0]
    assert oracle.composite(y, 3) < oracle.composite(x, 4)


@pytest.mark.parametrize("tiers,b", [(3, 0.5), (3, 0.3), (2, 0.3), (3, 0.2), (3, 0.8)])
@pytest.mark.parametrize("lam", [0.0, 0.01])
def test_recency_closed_form(tiers, b, lam):
    n = 1000
    cfg = oracle.config(1, 1, 32, n, b, first_ratio=0.02, num_tiers=tiers,
                        score_mode=oracle.RECENCY, decay=lam)
    p = oracle.plan(cfg)
    z = np.zeros((1, 1, n, 32), np.uint16)
    tier = oracle.assign(cfg, oracle.score(cfg, z, z))
    s = p["n_sink"]
    # newest tokens get the highest tiers, oldest non-sink tokens the lowest
    want = []
    for t, c in zip((oracle.FP16, oracle.INT8, oracle.INT4, oracle.DROP),
                    (p["n_fp16"], p["n_int8"], p["n_int4"], p["n_drop"])):
        want += [t] * c
    want = [oracle.FP16] * s + list(reversed(want))
    assert list(tier) == want
