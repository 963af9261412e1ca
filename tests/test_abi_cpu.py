"""C-ABI checks that need no GPU: the library loads, exports every function
include/skv.h declares, and its host-only entry points (plan, sizes, argument
checks) agree with the oracle.  No device work is enqueued here: every call
either is host-only or fails its argument check before any HIP call."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_08635_amd import skv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "skv.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(skv.LIB_PATH):
        from paper_2606_08635_amd import build
        build.build()
    return skv.lib()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(skv_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
    assert sorted(skv.EXPORTED) == names
    assert lib.skv_abi_version() == skv.ABI_VERSION == 2


def _pair(L, H, d, n, b, **kw):
    return skv.config(L, H, d, n, b, **kw), oracle.config(L, H, d, n, b, **kw)


@pytest.mark.parametrize("seed", range(4))
def test_plan_and_payload_size_match_oracle(lib, seed):
    rng = np.random.default_rng(seed)
    for _ in range(300):
        L, H = int(rng.integers(1, 6)), int(rng.integers(1, 9))
        d = int(rng.choice([32, 64, 128, 256]))
        n = int(rng.integers(1, 70000))
        b = float(np.float32(rng.uniform(0.01, 1.0)))
        kw = dict(first_ratio=float(np.float32(rng.uniform(0, 0.1))), num_tiers=int(rng.integers(2, 4)),
                  decay=0.0, num_sink=int(rng.choice([-1, -1, 0, 5])),
                  quant_int8=int(rng.choice([0, 0, 1, 2, 4, 8, 13, 14, 16, 28])), quant_int4=int(rng.choice([0, 0, 5, 10, 12, 17, 22])))
        c, o = _pair(L, H, d, n, b, **kw)
        try:
            want = oracle.plan(o)
        except oracle.OracleError as e:
            with pytest.raises(skv.SkvError) as got:
                skv.plan_tiers(c)
            assert got.value.status == e.status
            continue
        assert skv.plan_tiers(c) == want
        assert skv.payload_size(c) == oracle.payload_size(o)


def test_invalid_configs_rejected_like_the_oracle(lib):
    base = dict(num_layers=2, num_kv_heads=2, head_dim=64, num_tokens=1000, budget=0.5)
    for field, value in [("head_dim", 48), ("head_dim", 512), ("num_tokens", 0), ("num_tokens", (1 << 21) + 1),
                         ("budget", 0.0), ("budget", 1.5), ("budget", float("nan")), ("first_ratio", -0.1),
                         ("num_tiers", 4), ("score_mode", 3), ("decay", -1.0), ("decay", float("inf")),
                         ("decay", 1.0), ("num_sink", -2), ("num_layers", 0), ("num_kv_heads", 0),
                         ("quant_int8", 3), ("quant_int4", 32), ("quant_int8", 19), ("quant_int4", -1)]:
        c = skv.config(**base)
        setattr(c, field, value)
        o = oracle.config(**base)
        setattr(o, field, value)
        assert oracle.validate(o) == oracle.ERR_INVALID_ARG
        with pytest.raises(skv.SkvError) as e:
            skv.payload_size(c)
        assert e.value.status == skv.ERR_INVALID_ARG
    with pytest.raises(skv.SkvError) as e:
        skv.plan_tiers(skv.config(1, 1, 64, 100, 0.1, num_sink=11))
    assert e.value.status == skv.ERR_BUDGET


def test_workspace_size(lib):
    c = skv.config(32, 8, 128, 32768, 0.5)
    ws = skv.workspace_size(c)
    assert ws >= 8 * 32768 and ws % 256 == 0
    c.score_mode = skv.RECENCY
    assert skv.workspace_size(c) == 8 * 32768
    # past 32768 tokens the split tier cut needs its scratch after the decay
    # table: two histograms of 3 x 2048 counts plus the cuts' state, 256-aligned
    for n in (32769, 1 << 21):
        c = skv.config(1, 1, 32, n, 0.5, score_mode=skv.RECENCY, decay=1e-4)
        assert skv.workspace_size(c) == (8 * n + 255) // 256 * 256 + 49408


def test_host_side_argument_errors(lib):
    """Bad pointers, capacities and sizes are refused before any device work."""
    cfg = skv.config(2, 2, 64, 300, 0.5)
    P = ctypes.c_void_p
    fake = P(1 << 20)        # aligned, never dereferenced: the calls must fail first
    odd = P((1 << 20) + 8)   # misaligned
    total = skv.payload_size(cfg)
    L = lib
    by = ctypes.byref(cfg)
    assert L.skv_pack(by, fake, fake, fake, fake, total - 1, None, None) == skv.ERR_CAPACITY
    assert L.skv_pack(by, None, fake, fake, fake, total, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack(by, odd, fake, fake, fake, total, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack(by, fake, total - 1, fake, fake, fake, 20, 16, fake, None) == skv.ERR_FORMAT
    assert L.skv_unpack(by, fake, total, fake, fake, fake, 20, 16, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack(by, fake, total, fake, fake, fake, 0, 16, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack(by, fake, total, fake, fake, fake, 1 << 30, 16, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_score(by, fake, fake, None, odd, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_score(None, fake, fake, None, fake, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_assign_tiers(by, None, fake, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_prepare(by, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_link(None, fake, 16, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_link(fake, fake, 0, None, None) == skv.OK
    attn = skv.config(2, 2, 64, 300, 0.5, score_mode=skv.ATTN, num_q_heads=4, obs_window=8)
    assert L.skv_score(ctypes.byref(attn), fake, fake, None, fake, fake, None) == skv.ERR_INVALID_ARG
    for s in range(6):
        assert skv.status_string(s)


def test_batch_argument_errors(lib):
    cfg = skv.config(2, 2, 64, 300, 0.5)
    fake = 1 << 20
    reqs = (skv.Request * 2)()
    for i, n in enumerate((300, 77)):
        c = skv.config(2, 2, 64, n, 0.5)
        reqs[i].num_tokens, reqs[i].k, reqs[i].v, reqs[i].tier, reqs[i].payload = n, fake, fake, fake, fake
        reqs[i].payload_bytes = skv.payload_size(c)
        reqs[i].block_table, reqs[i].dev_status = fake, fake
    by = ctypes.byref(cfg)
    L = lib
    # every check happens before any device work: the first failing request decides
    reqs[1].payload_bytes -= 1
    assert L.skv_pack_batch(by, reqs, 2, 0, 2, None) == skv.ERR_CAPACITY
    assert L.skv_unpack_batch(by, reqs, 2, fake, fake, 100, 16, 0, 2, None) == skv.ERR_FORMAT
    reqs[1].payload_bytes += 1
    assert L.skv_pack_batch(by, reqs, 0, 0, 2, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_batch(by, reqs, 2, 1, 2, None) == skv.ERR_INVALID_ARG   # layers past L
    assert L.skv_pack_batch(by, reqs, 2, 0, 0, None) == skv.ERR_INVALID_ARG
    reqs[0].reserved = 1
    assert L.skv_pack_batch(by, reqs, 2, 0, 2, None) == skv.ERR_INVALID_ARG
    reqs[0].reserved = 0
    reqs[1].num_tokens = 0
    assert L.skv_pack_batch(by, reqs, 2, 0, 2, None) == skv.ERR_INVALID_ARG
    reqs[1].num_tokens = 77
    reqs[1].dev_status = None
    assert L.skv_unpack_batch(by, reqs, 2, fake, fake, 100, 16, 0, 2, None) == skv.ERR_INVALID_ARG


def test_upgrade_size_and_argument_errors(lib):
    rng = np.random.default_rng(7)
    for _ in range(200):
        L, H = int(rng.integers(1, 5)), int(rng.integers(1, 9))
        d = int(rng.choice([32, 64, 128, 256]))
        n = int(rng.integers(1, 40000))
        m = int(rng.integers(0, n + 2))
        mode = int(rng.integers(0, 3))
        c, o = _pair(L, H, d, n, 0.5, decay=0.0)
        try:
            want = oracle.upgrade_size(o, m, mode)
        except oracle.OracleError as e:
            with pytest.raises(skv.SkvError) as got:
                skv.upgrade_size(c, m, mode)
            assert got.value.status == e.status == skv.ERR_INVALID_ARG
            continue
        assert skv.upgrade_size(c, m, mode) == want
    cfg = skv.config(2, 2, 64, 300, 0.5)
    by = ctypes.byref(cfg)
    P = ctypes.c_void_p
    fake, odd = P(1 << 20), P((1 << 20) + 8)
    size = skv.upgrade_size(cfg, 10, skv.UPGRADE_RESIDUAL8)
    L = lib
    assert L.skv_pack_upgrade(by, fake, fake, fake, fake, 10, 1, fake, size - 1, None, None) == skv.ERR_CAPACITY
    assert L.skv_pack_upgrade(by, fake, fake, fake, None, 10, 1, fake, size, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_upgrade(by, fake, fake, fake, fake, 0, 1, fake, size, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_upgrade(by, fake, fake, fake, fake, 301, 1, fake, size, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_upgrade(by, fake, odd, fake, fake, 10, 1, fake, size, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_upgrade(by, fake, fake, fake, fake, 10, 2, fake, size, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_upgrade(by, fake, size - 1, 10, 1, fake, fake, fake, 20, 16, fake, None) == skv.ERR_FORMAT
    assert L.skv_unpack_upgrade(by, fake, size, 10, 1, fake, fake, fake, 20, 16, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_upgrade(by, fake, size, 10, 1, fake, fake, None, 20, 16, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_upgrade(by, fake, size, 10, 1, fake, fake, fake, 0, 16, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_upgrade(by, odd, size, 10, 1, fake, fake, fake, 20, 16, fake, None) == skv.ERR_INVALID_ARG


def test_grouped_workspace_holds_the_split_tier_cut(lib):
    """Past 32768 tokens the grouped tier cut keeps one row of split-form
    scratch per group (two 3 x 2048 count histograms and the cuts' state,
    49192 bytes) after the tables; the recency score needs no other scratch,
    so the workspace grows by exactly that, 256-aligned."""
    for n in (32768, 32769, 100_000):
        for gran, G in ((skv.GROUP_LAYER, 3), (skv.GROUP_HEAD, 6)):
            c = skv.config(3, 2, 32, n, 0.5, score_mode=skv.RECENCY, decay=1e-3)
            size = skv.group_workspace_size(c, skv.Groups(gran, None))
            # decay table, group table (32 B per group), segment table (32 B per (layer, head))
            tables = (8 * n + 255) // 256 * 256 + (32 * G + 255) // 256 * 256 + (32 * 6 + 255) // 256 * 256
            extra = 0 if n <= 32768 else (G * 49192 + 255) // 256 * 256
            assert size == tables + extra, (n, gran)


@pytest.mark.parametrize("seed", range(3))
def test_grouped_plans_and_sizes_match_oracle(lib, seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(120):
        L, H = int(rng.integers(1, 6)), int(rng.integers(1, 9))
        d = int(rng.choice([32, 64, 128, 256]))
        n = int(rng.integers(1, 40000))
        gran = int(rng.integers(0, 3))
        kw = dict(num_tiers=int(rng.integers(2, 4)), decay=0.0, num_sink=int(rng.choice([-1, -1, 0, 3])))
        c, o = _pair(L, H, d, n, float(np.float32(rng.uniform(0.05, 1.0))), **kw)
        G = oracle.group_count(o, gran)
        budgets = None if rng.random() < 0.3 else np.float32(rng.uniform(0.02, 1.0, G))
        groups = skv.Groups(gran, budgets)
        assert skv.group_count(c, groups) == G
        try:
            want = oracle.grouped_size(o, gran, budgets)
        except oracle.OracleError as e:
            with pytest.raises(skv.SkvError) as got:
                skv.grouped_payload_size(c, groups)
            assert got.value.status == e.status
            continue
        assert skv.grouped_payload_size(c, groups) == want
        assert skv.plan_groups(c, groups) == [oracle.plan_group(o, gran, budgets, g) for g in range(G)]
        assert skv.group_workspace_size(c, groups) % 256 == 0


def test_grouped_argument_errors(lib):
    cfg = skv.config(2, 2, 64, 300, 0.5)
    by = ctypes.byref(cfg)
    P = ctypes.c_void_p
    fake, odd = P(1 << 20), P((1 << 20) + 8)
    for gran, budgets in ((3, None), (-1, None), (skv.GROUP_LAYER, [0.5, 0.0]), (skv.GROUP_LAYER, [0.5, 1.5]),
                          (skv.GROUP_HEAD, [0.5, 0.5, float("nan"), 0.5])):
        with pytest.raises(skv.SkvError) as e:
            skv.grouped_payload_size(cfg, skv.Groups(gran, budgets))
        assert e.value.status == skv.ERR_INVALID_ARG
    for q8, q4 in ((skv.QUANT_FP16, 0), (0, skv.QUANT_CHANNEL)):  # grouped maps use the default quantizer
        with pytest.raises(skv.SkvError) as e:
            skv.grouped_payload_size(skv.config(2, 2, 64, 300, 0.5, quant_int8=q8, quant_int4=q4),
                                     skv.Groups(skv.GROUP_LAYER))
        assert e.value.status == skv.ERR_INVALID_ARG
    g = skv.Groups(skv.GROUP_LAYER, [0.9, 0.1])
    g.spec.reserved = 1
    with pytest.raises(skv.SkvError):
        skv.group_count(cfg, g)
    with pytest.raises(skv.SkvError) as e:  # sinks alone exceed a group's budget
        skv.plan_groups(skv.config(2, 1, 64, 100, 0.5, num_sink=20), skv.Groups(skv.GROUP_LAYER, [0.5, 0.04]))
    assert e.value.status == skv.ERR_BUDGET
    with pytest.raises(skv.SkvError):  # too many (layer, head) pairs for one grid dimension
        skv.grouped_payload_size(skv.config(256, 256, 32, 10, 0.5), skv.Groups(skv.GROUP_HEAD))
    g = skv.Groups(skv.GROUP_HEAD)
    total = skv.grouped_payload_size(cfg, g)
    L = lib
    assert L.skv_pack_groups(by, g.ref, fake, fake, fake, fake, fake, total - 1, None, None) == skv.ERR_CAPACITY
    assert L.skv_pack_groups(by, g.ref, fake, odd, fake, fake, fake, total, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_pack_groups(by, g.ref, fake, fake, fake, None, fake, total, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_groups(by, g.ref, fake, fake, total - 1, fake, fake, fake, 20, 16, fake, None) == skv.ERR_FORMAT
    assert L.skv_unpack_groups(by, g.ref, fake, fake, total, fake, fake, fake, 20, 16, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_unpack_groups(by, g.ref, fake, fake, total, fake, fake, fake, 0, 16, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_score_groups(by, g.ref, fake, fake, None, odd, fake, None) == skv.ERR_INVALID_ARG
    assert L.skv_assign_groups(by, g.ref, fake, fake, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_prepare_groups(by, g.ref, None, None) == skv.ERR_INVALID_ARG
    assert L.skv_score_groups(by, None, fake, fake, None, fake, fake, None) == skv.ERR_INVALID_ARG


def _score_reqs(lengths, ptr=256):
    reqs = (skv.ScoreRequest * len(lengths))()
    for i, n in enumerate(lengths):
        reqs[i].num_tokens = n
        reqs[i].k = reqs[i].v = reqs[i].score = reqs[i].tier = ptr
    return reqs


def test_batched_score_host_checks(lib):
    """Argument errors of the batched score / assign are caught on the host
    (placeholder aligned addresses are never dereferenced)."""
    import ctypes
    cfg = skv.config(2, 2, 64, 1000, 0.5)
    out = ctypes.c_uint64()
    reqs = _score_reqs([1000, 10, 999])
    assert lib.skv_batch_workspace_size(ctypes.byref(cfg), reqs, 3, ctypes.byref(out)) == skv.OK
    table = 8 * 1000
    assert out.value >= -(-table // 256) * 256 + 16 * (1000 + 10 + 999)
    one = ctypes.c_uint64()
    assert lib.skv_batch_workspace_size(ctypes.byref(cfg), _score_reqs([10]), 1, ctypes.byref(one)) == skv.OK
    assert one.value < out.value
    assert lib.skv_batch_workspace_size(ctypes.byref(cfg), reqs, 0, ctypes.byref(one)) == skv.OK
    # a request longer than the configured table
    assert lib.skv_batch_workspace_size(ctypes.byref(cfg), _score_reqs([1001]), 1, ctypes.byref(out)) \
        == skv.ERR_INVALID_ARG
    bad = _score_reqs([10])
    bad[0].reserved = 1
    assert lib.skv_score_batch(ctypes.byref(cfg), bad, 1, ctypes.c_void_p(256), None) == skv.ERR_INVALID_ARG
    # attention mode has no batched form
    acfg = skv.config(2, 2, 64, 1000, 0.5, score_mode=skv.ATTN, num_q_heads=4, obs_window=8)
    assert lib.skv_score_batch(ctypes.byref(acfg), _score_reqs([10]), 1, ctypes.c_void_p(256), None) \
        == skv.ERR_INVALID_ARG
    # misaligned score pointer
    assert lib.skv_assign_batch(ctypes.byref(cfg), _score_reqs([10], ptr=258), 1, None, None) == skv.ERR_INVALID_ARG
    # misaligned workspace
    assert lib.skv_assign_batch(ctypes.byref(cfg), _score_reqs([10]), 1, ctypes.c_void_p(264), None) \
        == skv.ERR_INVALID_ARG
    # a request whose sinks exceed its own budget: one token, one sink, b = 0.5
    assert lib.skv_assign_batch(ctypes.byref(cfg), _score_reqs([10, 1]), 2, None, None) == skv.ERR_BUDGET


def test_batched_workspace_holds_the_split_tier_cut(lib):
    """The batch workspace holds, after the decay table, either the KV-norm
    partial sums or the split tier cut's select state (49192 bytes per request
    past 32768 tokens, at most 48 per launch), whichever is larger."""
    import ctypes
    state = 49192
    for mode in (skv.KVNORM, skv.RECENCY):
        cfg = skv.config(2, 2, 64, 200_000, 0.5, score_mode=mode, decay=1e-4)
        table = -(-8 * 200_000 // 256) * 256
        for lengths, longs in (([100], 0), ([32768, 20_000], 0), ([32769], 1), ([200_000, 5, 40_000], 2),
                               ([40_000] * 50, 48)):
            out = ctypes.c_uint64()
            assert lib.skv_batch_workspace_size(ctypes.byref(cfg), _score_reqs(lengths), len(lengths),
                                                ctypes.byref(out)) == skv.OK
            select = -(-longs * state // 256) * 256
            if mode == skv.KVNORM:
                assert out.value >= table + max(16 * sum(lengths), select), (mode, lengths)
            else:  # no partial sums: the select state alone
                assert out.value == table + select, (mode, lengths)
