"""Pins for the oracle's plan (tier counts) against what the paper fixes.

Sources: eq. "budget" (Sec. 2.1), the budget-to-tier mapping (Sec. 4.4), the
2-tier drop rule (Sec. 7.4.3), sink reservation charged to the budget
(Sec. 4.4, Algorithm 1, scoring) and the fractions the paper prints
(tests/golden/paper_tier_fractions.txt).
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_tier_fractions.txt")


def _golden_rows():
    rows = []
    for line in open(GOLDEN):
        body = line.split("#", 1)[0].split()
        if body:
            tiers, b, f16, f8, f4, fd = body
            rows.append((int(tiers), float(b), float(f16), float(f8), float(f4), float(fd)))
    return rows


def _cfg(n, b, tiers=3, sink=0, rho=0.0):
    return oracle.config(1, 1, 64, n, b, first_ratio=rho, num_sink=sink, num_tiers=tiers, decay=0.0)


@pytest.mark.parametrize("row", _golden_rows())
@pytest.mark.parametrize("n", [4096, 8192, 32768, 1000, 777])
def test_paper_printed_fractions(row, n):
    tiers, b, f16, f8, f4, fd = row
    p = oracle.plan(_cfg(n, b, tiers))
    got = np.array([p["n_fp16"], p["n_int8"], p["n_int4"], p["n_drop"]]) / n
    # the plan rounds the budget down to whole quarter-units, so each count
    # may sit one or two tokens away from the exact fraction
    assert np.all(np.abs(got - np.array([f16, f8, f4, fd])) <= 2.0 / n + 1e-12), (row, n, p)


def test_headline_counts_match_printed_special_cases():
    # 2-tier at b=0.3, n=4096: 60% sent at INT8, 40% dropped (Sec. 7.4.3)
    p = oracle.plan(_cfg(4096, 0.3, 2))
    assert (p["n_int8"], p["n_drop"]) == (2457, 1639)
    # b = 0.5 without sinks: every token INT8 (Sec. 2.1)
    p = oracle.plan(_cfg(4096, 0.5, 3))
    assert (p["n_fp16"], p["n_int8"], p["n_int4"], p["n_drop"]) == (0, 4096, 0, 0)
    # b = 0.25: every token INT4 (Sec. 7.5)
    p = oracle.plan(_cfg(8192, 0.25, 3))
    assert (p["n_int8"], p["n_int4"]) == (0, 8192)
    # b = 1: every token FP16
    p = oracle.plan(_cfg(999, 1.0, 3))
    assert p["n_fp16"] == 999


@pytest.mark.parametrize("tiers", [2, 3])
def test_mapping_formulas_over_budget_grid(tiers):
    """Sec. 4.4 fractions, b in [0.25, 1], no sinks."""
    n = 100000
    for b in np.linspace(0.25, 1.0, 61):
        b32 = float(np.float32(b))
        p = oracle.plan(_cfg(n, b32, tiers))
        f16, f8, f4, fd = (p["n_fp16"] / n, p["n_int8"] / n, p["n_int4"] / n, p["n_drop"] / n)
        if b32 >= 0.5:
            want = (2 * b32 - 1, 2 - 2 * b32, 0.0, 0.0)
        elif tiers == 3:
            want = (0.0, 4 * b32 - 1, 2 - 4 * b32, 0.0)
        else:  # 2-tier below b=0.5: int8 at cost 1/2, the rest dropped
            want = (0.0, 2 * b32, 0.0, 1 - 2 * b32)
        assert np.allclose((f16, f8, f4, fd), want, atol=2.0 / n), (b32, p)


def _cost(p):
    return 4 * (p["n_sink"] + p["n_fp16"]) + 2 * p["n_int8"] + p["n_int4"]


@pytest.mark.parametrize("seed", range(5))
def test_budget_never_exceeded_and_tight(seed):
    rng = np.random.default_rng(seed)
    for _ in range(400):
        n = int(rng.integers(1, 5000))
        b = float(np.float32(rng.uniform(0.01, 1.0)))
        rho = float(np.float32(rng.uniform(0, 0.1)))
        tiers = int(rng.integers(2, 4))
        cfg = oracle.config(2, 2, 32, n, b, first_ratio=rho, num_tiers=tiers)
        B = math.floor(4 * b * n)  # exact: b is a binary32, n < 2^24
        s = min(n, math.ceil(rho * n))
        if 4 * s > B:
            with pytest.raises(oracle.OracleError) as e:
                oracle.plan(cfg)
            assert e.value.status == oracle.ERR_BUDGET
            continue
        p = oracle.plan(cfg)
        assert p["n_sink"] == s
        assert p["n_sink"] + p["n_fp16"] + p["n_int8"] + p["n_int4"] + p["n_drop"] == n
        assert p["budget_units"] == B
        assert _cost(p) == p["used_units"] <= B
        # bytes of the element payload never exceed b * F (eq. "budget", "fullbytes")
        assert p["used_units"] / (4 * n) <= b
        assert B - p["used_units"] <= 1 or (p["n_drop"] == 0 and p["n_int4"] == 0 and p["n_int8"] == 0)
        if tiers == 2:
            assert p["n_int4"] == 0
        # at most two adjacent tiers among the ranked (non-sink) tokens
        used = [i for i, key in enumerate(("n_fp16", "n_int8", "n_int4", "n_drop")) if p[key] > 0]
        if tiers == 2:
            used = [{0: 0, 1: 1, 3: 2}[u] for u in used]
        assert len(used) <= 2 and (len(used) < 2 or used[1] == used[0] + 1), p


def test_sinks_charged_to_budget():
    # ceil(0.02 * n) sinks on the stated workloads (first-ratio 0.02)
    for n, s in [(512, 11), (4096, 82), (8192, 164), (32768, 656)]:
        p = oracle.plan(oracle.config(1, 1, 64, n, 0.5, first_ratio=0.02, num_tiers=3))
        assert p["n_sink"] == s
        # remaining budget 2n - 4s over m = n - s tokens: int8 + int4 mix
        m, R = n - s, 2 * n - 4 * s
        assert (p["n_int8"], p["n_int4"]) == (R - m, 2 * m - R)
    # 2-tier at b = 0.5 with sinks must drop s tokens
    p = oracle.plan(oracle.config(1, 1, 64, 4096, 0.5, first_ratio=0.02, num_tiers=2))
    assert p["n_drop"] == 82 and p["n_int8"] == 4096 - 2 * 82


def test_explicit_sink_count_and_budget_error():
    p = oracle.plan(oracle.config(1, 1, 64, 100, 0.5, num_sink=7))
    assert p["n_sink"] == 7
    with pytest.raises(oracle.OracleError) as e:
        oracle.plan(oracle.config(1, 1, 64, 100, 0.1, num_sink=11))  # 44 > floor(40)
    assert e.value.status == oracle.ERR_BUDGET


@pytest.mark.parametrize("field,value", [
    ("head_dim", 48), ("head_dim", 512), ("num_tokens", 0), ("num_tokens", (1 << 21) + 1),
    ("budget", 0.0), ("budget", 1.5), ("budget", float("nan")), ("first_ratio", -0.1),
    ("num_tiers", 4), ("score_mode", 3), ("decay", -1.0), ("decay", 1.0), ("num_sink", -2),
    ("num_layers", 0), ("num_kv_heads", 0)])
def test_invalid_configs(field, value):
    cfg = oracle.config(2, 2, 64, 1000, 0.5)
    setattr(cfg, field, value)
    assert oracle.validate(cfg) == oracle.ERR_INVALID_ARG


def test_attention_mode_requires_grouping():
    cfg = oracle.config(1, 2, 64, 16, 0.5, score_mode=oracle.ATTN, num_q_heads=3, obs_window=4)
    assert oracle.validate(cfg) == oracle.ERR_INVALID_ARG
    cfg.num_q_heads = 4
    assert oracle.validate(cfg) == oracle.OK
