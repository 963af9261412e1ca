"""Property tests over random shapes and settings (hypothesis, derandomized so
every run draws the same cases).

CPU: the library's host-side plan and payload size equal the oracle's for any
configuration, and the plan obeys its invariants (counts add up, the budget
is never exceeded and at most one quarter-unit is left unused, more budget
never drops more tokens).  The oracle's round trip keeps FP16 rows verbatim,
zeroes DROP rows and reconstructs quantized rows within half a step.

GPU: for random shapes, budgets, tier policies, score modes and quantizer
descriptors the GPU scores, tier map, payload bytes and decoded caches are
bit-identical to the oracle's.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from paper_2606_08635_amd import skv, workloads

PROFILE = dict(deadline=None, derandomize=True, database=None,
               suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large])

budgets = st.floats(min_value=0.0, max_value=1.0, exclude_min=True, allow_nan=False, width=32)
QUANTS = [0, 0, 0, 1, 2, 4, 8, 13, 14, 16, 20, 28, 26]


def _both(L, H, d, n, b, **kw):
    return skv.config(L, H, d, n, b, **kw), oracle.config(L, H, d, n, b, **kw)


@settings(max_examples=300, **PROFILE)
@given(n=st.integers(1, 1 << 21), b=budgets, rho=st.sampled_from([0.0, 0.001, 0.02, 0.1, 0.5, 1.0]),
       tiers=st.sampled_from([2, 3]), sink=st.sampled_from([-1, -1, 0, 1, 7]), d=st.sampled_from([32, 64, 128, 256]),
       q8=st.sampled_from(QUANTS), q4=st.sampled_from(QUANTS))
def test_plan_and_size_match_oracle_and_invariants(n, b, rho, tiers, sink, d, q8, q4):
    c, o = _both(2, 3, d, n, b, first_ratio=rho, num_sink=sink, num_tiers=tiers, quant_int8=q8, quant_int4=q4)
    try:
        want = oracle.plan(o)
    except oracle.OracleError as e:
        with pytest.raises(skv.SkvError) as got:
            skv.plan_tiers(c)
        assert got.value.status == e.status
        return
    assert skv.plan_tiers(c) == want
    assert skv.payload_size(c) == oracle.payload_size(o)
    s, n16, n8, n4, nd = want["n_sink"], want["n_fp16"], want["n_int8"], want["n_int4"], want["n_drop"]
    assert s + n16 + n8 + n4 + nd == n and min(s, n16, n8, n4, nd) >= 0
    used = 4 * (s + n16) + 2 * n8 + n4
    assert used == want["used_units"] <= want["budget_units"] <= used + 1
    if tiers == 2:
        assert n4 == 0
    # more budget never drops more tokens nor buys fewer units
    b2 = min(1.0, float(np.float32(b) * np.float32(1.25)))
    o2 = oracle.config(2, 3, d, n, b2, first_ratio=rho, num_sink=sink, num_tiers=tiers)
    p2 = oracle.plan(o2)
    assert p2["n_drop"] <= nd and p2["budget_units"] >= want["budget_units"]


@settings(max_examples=25, **PROFILE)
@given(d=st.sampled_from([32, 64, 128, 256]), n=st.integers(1, 700), b=budgets, tiers=st.sampled_from([2, 3]),
       seed=st.integers(0, 1000))
def test_oracle_round_trip_properties(d, n, b, tiers, seed):
    cfg = oracle.config(1, 2, d, n, b, num_tiers=tiers)
    try:
        oracle.plan(cfg)
    except oracle.OracleError:
        return
    k, v = workloads.make_kv(1, 2, n, d, seed=seed)
    k, v = k.numpy().view(np.uint16), v.numpy().view(np.uint16)
    tier = oracle.assign(cfg, oracle.score(cfg, k, v))
    pay = oracle.pack(cfg, k, v, tier)
    nb = workloads.blocks_for(n)
    bt = workloads.make_block_table(n, 16, nb, seed=seed).numpy()
    kc, vc = (np.full((1, nb, 16, 2, d), 0xABCD, np.uint16) for _ in range(2))
    assert oracle.unpack(cfg, pay, kc, vc, bt, 16) == oracle.OK
    for src, cache in ((k, kc), (v, vc)):
        got = cache[0, bt[np.arange(n) // 16], np.arange(n) % 16].transpose(1, 0, 2)  # [H][n][d]
        x = src[0].view(np.float16).astype(np.float64)
        y = got.view(np.float16).astype(np.float64)
        fp16, drop = tier == oracle.FP16, tier == oracle.DROP
        assert np.array_equal(got[:, fp16], src[0][:, fp16])
        assert (got[:, drop] == 0).all()
        for tr, Q in ((oracle.INT8, 127), (oracle.INT4, 7)):
            rows = tier == tr
            if not rows.any():
                continue
            a = np.abs(x[:, rows]).max(axis=2, keepdims=True)
            s = (a.astype(np.float32) / np.float32(Q)).astype(np.float64)
            ulp = np.spacing(np.abs(y[:, rows]).astype(np.float16)).astype(np.float64)
            assert (np.abs(y[:, rows] - x[:, rows]) <= s / 2 * (1 + 2.0 ** -20) + ulp).all()


@pytest.mark.gpu
@settings(max_examples=30, **PROFILE)
@given(d=st.sampled_from([32, 64, 128, 256]), L=st.integers(1, 2), H=st.integers(1, 3), n=st.integers(1, 2100),
       b=budgets, tiers=st.sampled_from([2, 3]), rho=st.sampled_from([0.0, 0.02, 0.2]),
       lam=st.sampled_from([0.0, 0.005, 0.05]), mode=st.sampled_from([oracle.KVNORM, oracle.KVNORM, oracle.RECENCY]),
       q8=st.sampled_from(QUANTS), q4=st.sampled_from(QUANTS), seed=st.integers(0, 10_000))
def test_random_shapes_bit_exact(d, L, H, n, b, tiers, rho, lam, mode, q8, q4, seed):
    from gpu_helpers import gpu_decode, gpu_encode, oracle_decode, say, u16

    if 2.0 * lam * (n - 1) > 700.0:
        lam = 0.0
    kw = dict(first_ratio=rho, decay=lam, num_tiers=tiers, score_mode=mode, quant_int8=q8, quant_int4=q4)
    cfg, ocfg = _both(L, H, d, n, b, **kw)
    try:
        oracle.plan(ocfg)
    except oracle.OracleError:
        return
    say(f"props d={d} L={L} H={H} n={n} b={b} tiers={tiers} rho={rho} lam={lam} mode={mode} q={q8},{q4} seed={seed}")
    k, v = workloads.make_kv(L, H, n, d, seed=seed)
    okey = oracle.score(ocfg, u16(k), u16(v))
    otier = oracle.assign(ocfg, okey)
    want = oracle.pack(ocfg, u16(k), u16(v), otier)
    codec = gpu_encode(cfg, k.cuda(), v.cuda())
    assert np.array_equal(codec.scores.cpu().numpy().view(np.uint64), okey.view(np.uint64))
    assert np.array_equal(codec.tier.cpu().numpy(), otier)
    assert int(codec.status[0].item()) == 0
    assert np.array_equal(codec.payload.cpu().numpy(), want)
    bs = 16
    nb = workloads.blocks_for(n, bs) + 2
    bt = workloads.make_block_table(n, bs, nb, seed=seed)
    okc, ovc, ost = oracle_decode(ocfg, want, L, H, d, bs, nb, bt.numpy())
    kc, vc, gst = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)
