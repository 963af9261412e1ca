"""Batched, variable-length pack/unpack and layer-range calls vs the oracle.

A batch of requests with different lengths packs to the same bytes as each
request on its own (checked against the oracle's payloads), unpacks into one
shared paged cache exactly as the oracle unpacks each request, batches larger
than one launch's 16 requests are split transparently, a payload that fails
its check only disables its own request, and packing or unpacking layer by
layer in several calls gives the same bytes as one call.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

L, H, d, B, TIERS = 2, 2, 64, 0.4, 3


def _requests(lengths, seed0=0, q8=0, q4=0):
    out = []
    for i, n in enumerate(lengths):
        cfg, ocfg = configs(L, H, d, n, B, TIERS, q8=q8, q4=q4)
        k, v = workloads.make_kv(L, H, n, d, seed=seed0 + 16 * i)
        key = oracle.score(ocfg, u16(k), u16(v))
        tier = oracle.assign(ocfg, key)
        out.append(dict(n=n, cfg=cfg, ocfg=ocfg, k=k, v=v, tier=tier, payload=oracle.pack(ocfg, u16(k), u16(v), tier)))
    return out


def _pool_tables(lengths, bs, seed):
    nbs = [workloads.blocks_for(n, bs) for n in lengths]
    pool = sum(nbs) + 3
    perm = workloads.make_block_table(pool * bs, bs, pool, seed=seed)
    tables, start = [], 0
    for nb in nbs:
        tables.append(perm[start:start + nb].contiguous())
        start += nb
    return pool, tables


def _gpu_pack(reqs, layer_ranges=None):
    cfg = reqs[0]["cfg"]
    ks = [r["k"].cuda() for r in reqs]
    vs = [r["v"].cuda() for r in reqs]
    tiers = [torch.from_numpy(r["tier"]).cuda() for r in reqs]
    pays = [torch.empty(r["payload"].size, dtype=torch.uint8, device="cuda") for r in reqs]
    sts = [torch.full((1,), -1, dtype=torch.int32, device="cuda") for _ in reqs]
    for lb, lc in (layer_ranges or [(0, L)]):
        skv.pack_batch(cfg, ks, vs, tiers, pays, sts, layer_begin=lb, layer_count=lc)
    torch.cuda.synchronize()
    return pays, [int(s.item()) for s in sts]


def _gpu_unpack(reqs, pays, tables, pool, bs, layer_ranges=None):
    cfg = reqs[0]["cfg"]
    kc, vc = caches(L, pool, bs, H, d, "cuda")
    sts = [torch.full((1,), -1, dtype=torch.int32, device="cuda") for _ in reqs]
    for lb, lc in (layer_ranges or [(0, L)]):
        skv.unpack_batch(cfg, pays, [r["n"] for r in reqs], [t.cuda() for t in tables], kc, vc, bs, sts,
                         layer_begin=lb, layer_count=lc)
    torch.cuda.synchronize()
    return kc, vc, [int(s.item()) for s in sts]


def _oracle_unpack(reqs, payloads, tables, pool, bs):
    okc = np.full((L, pool, bs, H, d), 0xABCD, np.uint16)
    ovc = okc.copy()
    sts = [oracle.unpack(r["ocfg"], p, okc, ovc, t.numpy(), bs) for r, p, t in zip(reqs, payloads, tables)]
    return okc, ovc, sts


@pytest.mark.parametrize("lengths", [[5, 17, 300, 777, 4099], [256, 256, 512], [33] * 20])
def test_batch_matches_oracle(lengths):
    say(f"batch {lengths[:6]}{'...' if len(lengths) > 6 else ''} ({len(lengths)} requests)")
    reqs = _requests(lengths)
    pays, sts = _gpu_pack(reqs)
    assert sts == [0] * len(reqs)
    for r, p in zip(reqs, pays):
        assert np.array_equal(p.cpu().numpy(), r["payload"]), r["n"]
    bs = 16
    pool, tables = _pool_tables(lengths, bs, seed=3)
    kc, vc, gst = _gpu_unpack(reqs, pays, tables, pool, bs)
    okc, ovc, ost = _oracle_unpack(reqs, [r["payload"] for r in reqs], tables, pool, bs)
    assert gst == [0] * len(reqs) and ost == [oracle.OK] * len(reqs)
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


VARIANTS = [(0, 0), (skv.QUANT_GROUP64, skv.QUANT_GROUP32 | skv.QUANT_ASYM),
            (skv.QUANT_CHANNEL | skv.QUANT_ASYM, skv.QUANT_GROUP32 | skv.QUANT_FP16),
            (skv.QUANT_FP16, skv.QUANT_CHANNEL)]


@pytest.mark.parametrize("q8,q4", VARIANTS, ids=lambda x: f"{x}")
def test_layer_ranges_equal_one_call(q8, q4):
    global L
    L_saved, L = L, 4
    try:
        say(f"layer ranges, quantizer descriptors int8={q8} int4={q4}")
        lengths = [700, 129]
        reqs = _requests(lengths, seed0=5, q8=q8, q4=q4)
        full, _ = _gpu_pack(reqs)
        parts, sts = _gpu_pack(reqs, layer_ranges=[(0, 1), (1, 2), (3, 1)])
        assert sts == [0, 0]
        for a, b, r in zip(full, parts, reqs):
            assert torch.equal(a, b) and np.array_equal(a.cpu().numpy(), r["payload"])
        bs = 16
        pool, tables = _pool_tables(lengths, bs, seed=4)
        kc1, vc1, _ = _gpu_unpack(reqs, full, tables, pool, bs)
        kc2, vc2, st2 = _gpu_unpack(reqs, full, tables, pool, bs, layer_ranges=[(0, 2), (2, 1), (3, 1)])
        assert st2 == [0, 0] and torch.equal(kc1.view(torch.int16), kc2.view(torch.int16))
        assert torch.equal(vc1.view(torch.int16), vc2.view(torch.int16))
        okc, ovc, ost = _oracle_unpack(reqs, [r["payload"] for r in reqs], tables, pool, bs)
        assert ost == [oracle.OK] * 2 and np.array_equal(u16(kc2), okc) and np.array_equal(u16(vc2), ovc)
    finally:
        L = L_saved


def test_bad_payload_only_disables_its_request():
    lengths = [300, 500, 260]
    reqs = _requests(lengths, seed0=9)
    pays, _ = _gpu_pack(reqs)
    pays[1][20] ^= 1  # token count in the header of request 1
    bs = 16
    pool, tables = _pool_tables(lengths, bs, seed=5)
    kc, vc, sts = _gpu_unpack(reqs, pays, tables, pool, bs)
    assert sts == [0, skv.ERR_FORMAT, 0]
    okc, ovc, ost = _oracle_unpack([reqs[0], reqs[2]], [reqs[0]["payload"], reqs[2]["payload"]],
                                   [tables[0], tables[2]], pool, bs)
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)  # request 1's blocks untouched


SCORE_CASES = [
    # L, H, d, lengths, budget, tiers, mode
    (2, 2, 64, [3, 5, 255, 256, 257, 1000, 4099, 4], 0.4, 3, oracle.KVNORM),
    # 50 requests: two launches of the 48-request descriptor table
    (1, 2, 32, [30 + 11 * i for i in range(50)], 0.3, 2, oracle.KVNORM),
    # more than 32768 non-sink tokens (the general form of the select) next to
    # short ones (the resident form) in one call
    (1, 1, 32, [33000, 100, 40000], 0.5, 3, oracle.KVNORM),
    (1, 2, 256, [2048, 777], 0.7, 3, oracle.KVNORM),
    (2, 1, 128, [7, 3000, 512], 0.5, 3, oracle.RECENCY),
]


@pytest.mark.parametrize("case", SCORE_CASES, ids=[f"L{c[0]}H{c[1]}d{c[2]}x{len(c[3])}m{c[6]}" for c in SCORE_CASES])
def test_batched_score_and_assign_match_oracle(case):
    """skv_score_batch and skv_assign_batch give every request exactly the
    oracle's scores and tier map for that request alone."""
    Lb, Hb, db, lengths, b, tiers, mode = case
    say(f"batched score/assign {case[:3]} {len(lengths)} requests mode {mode}")
    cfg, _ = configs(Lb, Hb, db, max(lengths), b, tiers, mode=mode)
    ks, vs, want_key, want_tier = [], [], [], []
    for i, n in enumerate(lengths):
        _, ocfg = configs(Lb, Hb, db, n, b, tiers, mode=mode)
        k, v = workloads.make_kv(Lb, Hb, n, db, seed=100 + 16 * i)
        key = oracle.score(ocfg, u16(k), u16(v))
        want_key.append(key)
        want_tier.append(oracle.assign(ocfg, key))
        ks.append(k.cuda())
        vs.append(v.cuda())
    scores = [torch.full((n,), float("nan"), dtype=torch.float64, device="cuda") for n in lengths]
    tier_out = [torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda") for n in lengths]
    ws = torch.empty(max(skv.batch_workspace_size(cfg, scores), skv.workspace_size(cfg)), dtype=torch.uint8,
                     device="cuda")
    skv.prepare(cfg, ws)
    skv.score_batch(cfg, ks, vs, scores, ws)
    skv.assign_batch(cfg, scores, tier_out)
    torch.cuda.synchronize()
    for i, n in enumerate(lengths):
        assert np.array_equal(bits64(scores[i].cpu().numpy()), bits64(want_key[i])), f"scores of request {i} (n={n})"
        assert np.array_equal(tier_out[i].cpu().numpy(), want_tier[i]), f"tier map of request {i} (n={n})"


def test_batched_assign_of_foreign_scores():
    """The batched assignment takes any scores, like skv_assign_tiers: ties,
    zeros, negatives and NaN rank as the oracle ranks them."""
    lengths = [600, 3, 2500]
    cfg, _ = configs(1, 1, 32, max(lengths), 0.45, 3)
    rng = np.random.default_rng(7)
    scores, want = [], []
    for n in lengths:
        _, ocfg = configs(1, 1, 32, n, 0.45, 3)
        s = rng.choice(np.array([0.0, -1.0, np.nan, 1.0, 2.0, 2.0, 3.5]), size=n)
        scores.append(torch.from_numpy(s).cuda())
        want.append(oracle.assign(ocfg, s))
    tiers = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in lengths]
    skv.assign_batch(cfg, scores, tiers)
    torch.cuda.synchronize()
    for t, w in zip(tiers, want):
        assert np.array_equal(t.cpu().numpy(), w)


def test_batched_score_and_assign_full_size():
    """The 64 x 2048-token batch the benchmark times (32 layers x 8 KV heads x
    128): every request's batched scores and tier map equal the per-request
    calls' (bit for bit), and four requests spread over both launches of the
    batch are recomputed by the oracle."""
    w = workloads.WORKLOADS["short_batch"]
    L_, H_, d_ = w.layers, w.kv_heads, w.head_dim
    lens = list(w.batch_tokens)
    kw = dict(first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    bcfg = skv.config(L_, H_, d_, max(lens), w.budget, **kw)
    ks, vs, scores, tiers = [], [], [], []
    for r, n in enumerate(lens):
        k, v = workloads.make_kv(L_, H_, n, d_, seed=16 * r, outliers=w.outliers, device="cuda")
        ks.append(k)
        vs.append(v)
        scores.append(torch.full((n,), float("nan"), dtype=torch.float64, device="cuda"))
        tiers.append(torch.full((n,), 0xEE, dtype=torch.uint8, device="cuda"))
    ws = torch.empty(max(skv.batch_workspace_size(bcfg, scores), skv.workspace_size(bcfg)), dtype=torch.uint8,
                     device="cuda")
    skv.prepare(bcfg, ws)
    say("short_batch: batched score and assign")
    skv.score_batch(bcfg, ks, vs, scores, ws)
    skv.assign_batch(bcfg, scores, tiers)
    torch.cuda.synchronize()
    for r, n in enumerate(lens):
        c = skv.Codec(skv.config(L_, H_, d_, n, w.budget, **kw))
        skv.score(c.cfg, ks[r], vs[r], None, c.scores, c.ws)
        skv.assign_tiers(c.cfg, c.scores, c.tier)
        torch.cuda.synchronize()
        assert torch.equal(c.scores.view(torch.int64), scores[r].view(torch.int64)), f"scores of request {r}"
        assert torch.equal(c.tier, tiers[r]), f"tier map of request {r}"
    for r in (0, 17, 47, 63):
        say(f"short_batch: oracle request {r}")
        ocfg = oracle.config(L_, H_, d_, lens[r], w.budget, **kw)
        okey = oracle.score(ocfg, u16(ks[r]), u16(vs[r]))
        assert np.array_equal(bits64(scores[r].cpu().numpy()), bits64(okey)), f"oracle scores of request {r}"
        assert np.array_equal(tiers[r].cpu().numpy(), oracle.assign(ocfg, okey)), f"oracle tier map of request {r}"
