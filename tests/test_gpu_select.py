"""Tier assignment on both sides of its kernel forms vs the oracle.

Rows with at most 32 * 1024 non-sink tokens keep the high words of their
ranking keys resident in LDS; longer rows recompute the keys from the scores on
every pass, on one workgroup (no workspace) or split over the GPU (the
request's workspace given: one counting launch per pass; grouped maps always
take the split form past 32768 tokens, one row per group).  Each side of that
boundary, and both forms past it, are checked bit for bit against the
oracle's tier map, for one map and for per-layer grouped maps, with score sets
that spread over many binades, that tie in the keys' high 32 bits and differ
only below them, and that hold exact ties, non-positive scores and NaN.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

RESIDENT_MAX = 32 * 1024  # non-sink tokens per row of the resident form


def _scores(kind, shape, seed):
    rng = np.random.default_rng(seed)
    if kind == "binades":
        return np.ldexp(1.0 + rng.random(shape), rng.integers(-40, 40, shape))
    if kind == "low_word":
        # equal exponent and top 21 mantissa bits: keys tie in their high word
        # and differ in mantissa bits 30..20 (and then in the token index)
        return 1.0 + rng.integers(0, 2048, shape) * 2.0 ** -32
    s = np.round(rng.random(shape) * 4) / 4
    s[rng.random(shape) < 0.1] = -1.0
    s[rng.random(shape) < 0.01] = np.nan
    return s


@pytest.mark.parametrize("kind,b", [("binades", 0.7), ("low_word", 0.4), ("ties", 0.15)])
@pytest.mark.parametrize("extra", [0, 1], ids=["resident", "past_resident"])
def test_single_map_at_the_form_boundary(kind, b, extra):
    n_sink = 100
    n = n_sink + RESIDENT_MAX + extra
    say(f"assign n={n} sinks={n_sink} b={b} scores={kind}")
    cfg, ocfg = configs(1, 1, 32, n, b, 3, num_sink=n_sink)
    key = _scores(kind, n, seed=n + len(kind))
    want = oracle.assign(ocfg, key)
    dkey = torch.from_numpy(key).cuda()
    ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    for w in (None, ws):
        tier = torch.empty(n, dtype=torch.uint8, device="cuda")
        skv.assign_tiers(cfg, dkey, tier, ws=w)
        torch.cuda.synchronize()
        assert np.array_equal(tier.cpu().numpy(), want), "workspace given" if w is not None else "no workspace"


# plans whose cuts coincide or vanish: no FP16 cut (b = 0.15, 3-tier: INT4 +
# DROP), INT8 + INT4 only, FP16 + INT8 (the INT4 cut equals the INT8 one), all
# FP16 (every cut at the last rank), 2-tier with and without DROP
@pytest.mark.parametrize("b,tiers", [(0.15, 3), (0.4, 3), (0.7, 3), (1.0, 3), (0.3, 2), (0.6, 2)])
@pytest.mark.parametrize("kind", ["binades", "low_word", "ties"])
def test_split_form_long_rows(kind, b, tiers):
    n_sink = 37
    n = (1 << 18) + 12345
    say(f"split assign n={n} sinks={n_sink} b={b} tiers={tiers} scores={kind}")
    # decay 1e-3: 2 lambda (n - 1) = 549 stays inside the decay table's range (<= 700)
    cfg, ocfg = configs(1, 1, 32, n, b, tiers, num_sink=n_sink, decay=1e-3)
    key = _scores(kind, n, seed=n + 31 * len(kind) + tiers)
    want = oracle.assign(ocfg, key)
    ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    tier = torch.empty(n, dtype=torch.uint8, device="cuda")
    skv.assign_tiers(cfg, torch.from_numpy(key).cuda(), tier, ws=ws)
    torch.cuda.synchronize()
    assert np.array_equal(tier.cpu().numpy(), want)


def test_split_form_decayed_kvnorm_scores_twice():
    """Realistic keys (KV-norm times decay: exponents ordered by position),
    two requests in a row through one workspace, the second shorter."""
    for n, b in ((200_003, 0.5), (70_001, 0.3)):
        say(f"split assign, decayed scores, n={n} b={b}")
        cfg, ocfg = configs(1, 2, 64, n, b, 3, decay=0.0015)
        k, v = workloads.make_kv(1, 2, n, 64, seed=n)
        key = oracle.score(ocfg, u16(k), u16(v))
        want = oracle.assign(ocfg, key)
        ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
        tier = torch.empty(n, dtype=torch.uint8, device="cuda")
        skv.assign_tiers(cfg, torch.from_numpy(key).cuda(), tier, ws=ws)
        torch.cuda.synchronize()
        assert np.array_equal(tier.cpu().numpy(), want)


@pytest.mark.parametrize("kind", ["binades", "low_word", "ties"])
@pytest.mark.parametrize("n", [RESIDENT_MAX, RESIDENT_MAX + 1], ids=["resident", "past_resident"])
def test_grouped_maps_at_the_form_boundary(kind, n):
    L = 3
    say(f"grouped assign L={L} n={n} scores={kind}")
    cfg, ocfg = configs(L, 1, 32, n, 0.4, 3)
    gran = oracle.GRAN_LAYER
    budgets = np.float32([0.7, 0.3, 0.05])
    groups = skv.Groups(gran, budgets)
    key = _scores(kind, (L, n), seed=7 * n + len(kind))
    want = oracle.assign_groups(ocfg, gran, key, budgets)
    ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
    skv.prepare_groups(cfg, groups, ws)
    tier = torch.empty(L * n, dtype=torch.uint8, device="cuda")
    skv.assign_groups(cfg, groups, torch.from_numpy(key.ravel()).cuda(), tier, ws)
    torch.cuda.synchronize()
    assert np.array_equal(tier.cpu().numpy().reshape(L, n), want)


@pytest.mark.parametrize("kind", ["binades", "low_word", "ties"])
def test_split_form_per_head_maps(kind):
    """Per-head maps (one group per (layer, KV head)) past the resident form:
    eight rows cut together by the split form, budgets from all-FP16 down to
    INT4 + DROP, each row's map equal to the oracle's."""
    L, H, n = 2, 4, 70_001
    say(f"grouped split assign L={L} H={H} n={n} scores={kind}")
    cfg, ocfg = configs(L, H, 32, n, 0.4, 3, decay=1e-3)
    gran = oracle.GRAN_HEAD
    budgets = np.float32([1.0, 0.9, 0.6, 0.5, 0.4, 0.3, 0.2, 0.1])
    groups = skv.Groups(gran, budgets)
    key = _scores(kind, (L * H, n), seed=11 * n + len(kind))
    want = oracle.assign_groups(ocfg, gran, key, budgets)
    ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
    skv.prepare_groups(cfg, groups, ws)
    tier = torch.empty(L * H * n, dtype=torch.uint8, device="cuda")
    skv.assign_groups(cfg, groups, torch.from_numpy(key.ravel()).cuda(), tier, ws)
    torch.cuda.synchronize()
    got = tier.cpu().numpy().reshape(L * H, n)
    for g in range(L * H):
        assert np.array_equal(got[g], want[g]), f"group {g} (b = {budgets[g]})"


@pytest.mark.parametrize("tiers", [2, 3])
@pytest.mark.parametrize("extra", [0, 200_000], ids=["resident", "split"])
def test_budget_of_the_sinks_only_drops_every_other_token(tiers, extra):
    """A budget that pays for the sinks alone: every cut has rank 0, so both
    forms must leave the sinks FP16 and drop every other token."""
    n_sink = 37
    n = n_sink + 30_000 + extra
    b = float(np.float32((4 * n_sink + 0.5) / (4 * n)))  # floor(4 b n) = 4 * n_sink: nothing left after the sinks
    say(f"sinks-only budget n={n} b={b} tiers={tiers}")
    cfg, ocfg = configs(1, 1, 32, n, b, tiers, num_sink=n_sink, decay=1e-3)
    plan = skv.plan_tiers(cfg)
    assert plan["n_fp16"] == plan["n_int8"] == plan["n_int4"] == 0 and plan["n_drop"] == n - n_sink
    key = _scores("binades", n, seed=n)
    want = oracle.assign(ocfg, key)
    ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    tier = torch.empty(n, dtype=torch.uint8, device="cuda")
    skv.assign_tiers(cfg, torch.from_numpy(key).cuda(), tier, ws=ws)
    torch.cuda.synchronize()
    got = tier.cpu().numpy()
    assert np.array_equal(got, want)
    assert (got[:n_sink] == oracle.FP16).all() and (got[n_sink:] == oracle.DROP).all()


def _random_case(rng):
    """A random long row: length past the resident form, sinks, budget, tier
    policy and score distribution (with heavy ties in some)."""
    n = int(rng.integers(32_769, 400_000))
    n_sink = int(rng.choice([0, 1, 37, int(rng.integers(0, 5_000))]))
    tiers = int(rng.choice([2, 3]))
    kind = str(rng.choice(["binades", "low_word", "ties", "few_values", "decayed"]))
    if kind == "few_values":  # exact ties across the whole row
        key = rng.choice(np.array([0.0, 1e-300, 0.5, 1.0, 2.0, np.inf]), n)
    elif kind == "decayed":  # magnitudes times an exponential decay by position
        key = rng.random(n) * np.exp(-float(rng.uniform(0, 1e-3)) * (n - 1 - np.arange(n)))
    else:
        key = _scores(kind, n, seed=int(rng.integers(1 << 30)))
    return n, n_sink, tiers, kind, key


def test_split_form_random_rows():
    """Forty seeded random long rows through the split form (each with the
    budget drawn until the sinks fit), every map equal to the oracle's."""
    rng = np.random.default_rng(2606)
    done = 0
    while done < 40:
        n, n_sink, tiers, kind, key = _random_case(rng)
        b = float(np.float32(rng.uniform(0.0, 1.0)))
        if not (0.0 < b <= 1.0) or 4 * n_sink > int(4 * np.float64(np.float32(b)) * n):
            continue
        say(f"random split assign #{done} n={n} sinks={n_sink} b={b} tiers={tiers} scores={kind}")
        # decay 1e-4: 2 lambda (n - 1) < 80, inside the decay table's range (<= 700)
        cfg, ocfg = configs(1, 1, 32, n, b, tiers, num_sink=n_sink, decay=1e-4)
        want = oracle.assign(ocfg, key)
        ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
        tier = torch.empty(n, dtype=torch.uint8, device="cuda")
        skv.assign_tiers(cfg, torch.from_numpy(key).cuda(), tier, ws=ws)
        torch.cuda.synchronize()
        got = tier.cpu().numpy()
        assert np.array_equal(got, want), f"case {done}: {int((got != want).sum())} tokens differ"
        done += 1


def test_split_form_random_grouped_rows():
    """Twelve seeded random grouped cuts past the resident form (per layer or
    per head, random budgets per group), every group's map equal to the
    oracle's."""
    rng = np.random.default_rng(9)
    for case in range(12):
        L, H = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        gran = int(rng.choice([oracle.GRAN_LAYER, oracle.GRAN_HEAD]))
        n = int(rng.integers(32_769, 120_000))
        tiers = int(rng.choice([2, 3]))
        cfg, ocfg = configs(L, H, 32, n, 0.5, tiers, decay=1e-4)
        G = oracle.group_count(ocfg, gran)
        budgets = np.float32(rng.uniform(0.03, 1.0, G))
        kind = str(rng.choice(["binades", "low_word", "ties"]))
        key = _scores(kind, (G, n), seed=int(rng.integers(1 << 30)))
        say(f"random grouped split assign #{case} L={L} H={H} gran={gran} n={n} tiers={tiers} scores={kind}")
        want = oracle.assign_groups(ocfg, gran, key, budgets)
        groups = skv.Groups(gran, budgets)
        ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
        skv.prepare_groups(cfg, groups, ws)
        tier = torch.empty(G * n, dtype=torch.uint8, device="cuda")
        skv.assign_groups(cfg, groups, torch.from_numpy(key.ravel()).cuda(), tier, ws)
        torch.cuda.synchronize()
        assert np.array_equal(tier.cpu().numpy().reshape(G, n), want), f"case {case}"


@pytest.mark.parametrize("tiers,b", [(3, 0.4), (2, 0.7)])
def test_batched_split_form_matches_oracle(tiers, b):
    """skv_assign_batch with requests on both sides of the resident form
    (4 sinks: 32772 tokens fit it, 32773 do not) and up to 250k tokens: with
    the workspace (split form) and without (one workgroup per request) every
    request's map equals the oracle's for that request alone; a second call on
    the same workspace with other scores and fewer requests starts clean."""
    lengths = [32_772, 32_773, 100_003, 40, 250_000, 40_000, 2048, 65_536]
    kinds = ["binades", "low_word", "ties"]
    cfg, _ = configs(1, 1, 32, max(lengths), b, tiers, num_sink=4, decay=1e-4)

    def case(lens, seed):
        keys = [_scores(kinds[i % 3], n, seed=seed + i) for i, n in enumerate(lens)]
        want = [oracle.assign(configs(1, 1, 32, n, b, tiers, num_sink=4, decay=1e-4)[1], k)
                for n, k in zip(lens, keys)]
        return [torch.from_numpy(k).cuda() for k in keys], want

    scores, want = case(lengths, 500)
    ws = torch.empty(skv.batch_workspace_size(cfg, scores), dtype=torch.uint8, device="cuda")
    for w in (ws, None):
        say(f"batched assign {len(lengths)} requests tiers={tiers} b={b} ws={w is not None}")
        out = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in lengths]
        skv.assign_batch(cfg, scores, out, ws=w)
        torch.cuda.synchronize()
        for i, (t, wt) in enumerate(zip(out, want)):
            assert np.array_equal(t.cpu().numpy(), wt), f"request {i} (n={lengths[i]}), ws={w is not None}"
    sub = [100_003, 32_773, 70_001]
    scores, want = case(sub, 900)
    say(f"batched assign, second call {sub}")
    out = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in sub]
    skv.assign_batch(cfg, scores, out, ws=ws)
    torch.cuda.synchronize()
    for i, (t, wt) in enumerate(zip(out, want)):
        assert np.array_equal(t.cpu().numpy(), wt), f"second call, request {i} (n={sub[i]})"


def test_batched_split_form_more_than_one_launch():
    """Fifty long requests (two split launch sequences of at most 48 sharing
    one select state area) with seeded random lengths, score kinds and sink
    counts under one budget: every map equals the oracle's."""
    rng = np.random.default_rng(31)
    lengths = [int(x) for x in rng.integers(32_769, 60_000, 50)]
    b, tiers, n_sink = 0.35, 3, 16
    cfg, _ = configs(1, 1, 32, max(lengths), b, tiers, num_sink=n_sink, decay=1e-4)
    kinds = ["binades", "low_word", "ties"]
    keys = [_scores(kinds[int(rng.integers(3))], n, seed=int(rng.integers(1 << 30))) for n in lengths]
    scores = [torch.from_numpy(k).cuda() for k in keys]
    out = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in lengths]
    ws = torch.empty(skv.batch_workspace_size(cfg, scores), dtype=torch.uint8, device="cuda")
    say("batched assign, 50 long requests")
    skv.assign_batch(cfg, scores, out, ws=ws)
    torch.cuda.synchronize()
    for i, n in enumerate(lengths):
        want = oracle.assign(configs(1, 1, 32, n, b, tiers, num_sink=n_sink, decay=1e-4)[1], keys[i])
        assert np.array_equal(out[i].cpu().numpy(), want), f"request {i} (n={n})"
