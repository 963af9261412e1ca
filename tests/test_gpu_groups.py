"""Per-layer and per-head tier maps on the GPU vs the oracle, through the C ABI.

Bar: grouped KV-norm and recency scores, every group's tier map, the grouped
payload and the decoded caches are bit-identical to the oracle; attention
scores match within the attention mode's tolerance (tier maps then compared
on the oracle's scores).  Off-plan maps and malformed payloads are refused
through the status words; at full size the benchmark's launch is checked on
all scores and maps, the whole metadata and sampled rows.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

ATTN_RTOL = 1e-4


def _setup(cfg, groups, device="cuda"):
    ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device=device)
    skv.prepare_groups(cfg, groups, ws)
    return ws


def _gpu_codec(cfg, groups, k, v, q=None, scores=None):
    """score -> assign -> pack on the GPU; scores (numpy [G][n]) replace the
    GPU scores before the assignment when given."""
    G = skv.group_count(cfg, groups)
    n = cfg.num_tokens
    ws = _setup(cfg, groups)
    sc = torch.empty(G * n, dtype=torch.float64, device="cuda")
    skv.score_groups(cfg, groups, k, v, q, sc, ws)
    gscore = sc.cpu().numpy().reshape(G, n).copy()
    if scores is not None:
        sc.copy_(torch.from_numpy(np.ascontiguousarray(scores).ravel()).cuda())
    tier = torch.empty(G * n, dtype=torch.uint8, device="cuda")
    skv.assign_groups(cfg, groups, sc, tier, ws)
    pay = torch.full((skv.grouped_payload_size(cfg, groups),), 0xA5, dtype=torch.uint8, device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.pack_groups(cfg, groups, k, v, tier, ws, pay, st)
    torch.cuda.synchronize()
    return ws, gscore, tier.cpu().numpy().reshape(G, n), pay, int(st.item())


def _gpu_decode(cfg, groups, ws, pay, L, H, d, n, bs, nb, bt, fill=0xABCD):
    kc, vc = caches(L, nb, bs, H, d, "cuda", fill)
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.unpack_groups(cfg, groups, ws, pay, kc, vc, bt, bs, st)
    torch.cuda.synchronize()
    return kc, vc, int(st.item())


CASES = [
    # L, H, d, n, gran, budgets (None: uniform), extra
    (2, 2, 64, 700, oracle.GRAN_TOKEN, None, {}),
    (3, 2, 128, 1000, oracle.GRAN_LAYER, [0.8, 0.5, 0.2], {}),
    (2, 3, 32, 777, oracle.GRAN_HEAD, "ramp", {}),
    (4, 1, 256, 300, oracle.GRAN_LAYER, [1.0, 0.6, 0.3, 0.1], {}),
    (2, 2, 64, 257, oracle.GRAN_HEAD, None, {"tiers": 2}),
    (2, 2, 128, 1, oracle.GRAN_LAYER, [1.0, 1.0], {}),
    (2, 2, 64, 600, oracle.GRAN_HEAD, "ramp", {"mode": oracle.RECENCY}),
    (1, 4, 64, 1031, oracle.GRAN_HEAD, "ramp", {"specials": True}),
    # more than 512 KV heads: a layer's partial sums are taken one pair at a
    # time (the per-pair kernel's partial form) and added by the finish
    (2, 520, 32, 90, oracle.GRAN_LAYER, None, {"specials": True}),
]


def _budgets(spec, G):
    if spec is None:
        return None
    if spec == "ramp":
        return np.float32(np.linspace(0.9, 0.15, G))
    return np.float32(spec)


@pytest.mark.parametrize("case", CASES, ids=[f"L{c[0]}H{c[1]}d{c[2]}n{c[3]}g{c[4]}-{i}" for i, c in enumerate(CASES)])
def test_grouped_stages_bit_exact(case):
    L, H, d, n, gran, bspec, extra = case
    mode = extra.get("mode", oracle.KVNORM)
    cfg, ocfg = configs(L, H, d, n, 0.5, extra.get("tiers", 3), mode=mode)
    G = oracle.group_count(ocfg, gran)
    budgets = _budgets(bspec, G)
    groups = skv.Groups(gran, budgets)
    say(f"grouped L={L} H={H} d={d} n={n} gran={gran} mode={mode}")
    k, v = workloads.make_kv(L, H, n, d, seed=n)
    if extra.get("specials"):
        plant_specials(k, v, seed=n)
    okey = oracle.score_groups(ocfg, gran, u16(k), u16(v))
    otier = oracle.assign_groups(ocfg, gran, okey, budgets)
    ws, gkey, gtier, pay, st = _gpu_codec(cfg, groups, k.cuda(), v.cuda())
    assert np.array_equal(bits64(gkey), bits64(okey)), "scores"
    assert np.array_equal(gtier, otier), "tier maps"
    assert st == 0
    want = oracle.pack_groups(ocfg, gran, u16(k), u16(v), otier, budgets)
    got = pay.cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert got.size == want.size and bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"
    bs = 16
    nb = workloads.blocks_for(n, bs) + 3
    bt = workloads.make_block_table(n, bs, nb, seed=7)
    okc, ovc = (np.full((L, nb, bs, H, d), 0xABCD, np.uint16) for _ in range(2))
    assert oracle.unpack_groups(ocfg, gran, want, okc, ovc, bt.numpy(), bs, budgets) == 0
    kc, vc, gst = _gpu_decode(cfg, groups, ws, pay, L, H, d, n, bs, nb, bt.cuda())
    assert gst == 0
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


@pytest.mark.parametrize("gran", [oracle.GRAN_LAYER, oracle.GRAN_HEAD])
def test_grouped_attention_scores(gran):
    L, H, Hq, W, d, n = 2, 2, 4, 8, 64, 600
    cfg, ocfg = configs(L, H, d, n, 0.4, 3, mode=oracle.ATTN, Hq=Hq, W=W)
    G = oracle.group_count(ocfg, gran)
    budgets = np.float32(np.linspace(0.7, 0.3, G))
    groups = skv.Groups(gran, budgets)
    k, v = workloads.make_kv(L, H, n, d, seed=4)
    q = workloads.make_qobs(L, Hq, W, d, seed=4)
    say(f"grouped attention gran={gran}")
    okey = oracle.score_groups(ocfg, gran, u16(k), None, u16(q))
    otier = oracle.assign_groups(ocfg, gran, okey, budgets)
    ws, gkey, gtier, pay, st = _gpu_codec(cfg, groups, k.cuda(), v.cuda(), q.cuda(), scores=okey)
    np.testing.assert_allclose(gkey, okey, rtol=ATTN_RTOL, atol=0)
    assert np.array_equal(gtier, otier) and st == 0
    want = oracle.pack_groups(ocfg, gran, u16(k), u16(v), otier, budgets)
    assert np.array_equal(pay.cpu().numpy(), want)


def test_token_granularity_decodes_like_the_per_token_codec():
    L, H, d, n = 2, 2, 128, 900
    cfg, ocfg = configs(L, H, d, n, 0.35, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=21)
    k, v = k.cuda(), v.cuda()
    groups = skv.Groups(skv.GROUP_TOKEN)
    ws, _, gtier, gpay, st = _gpu_codec(cfg, groups, k, v)
    codec = gpu_encode(cfg, k, v)
    assert st == 0 and np.array_equal(gtier[0], codec.tier.cpu().numpy())
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=5).cuda()
    kc, vc, s1 = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt)
    gkc, gvc, s2 = _gpu_decode(cfg, groups, ws, gpay, L, H, d, n, bs, nb, bt)
    assert s1 == 0 and s2 == 0
    assert torch.equal(kc.view(torch.int16), gkc.view(torch.int16))
    assert torch.equal(vc.view(torch.int16), gvc.view(torch.int16))


def test_off_plan_group_map_is_flagged():
    L, H, d, n = 2, 2, 64, 500
    cfg, ocfg = configs(L, H, d, n, 0.5, 3)
    groups = skv.Groups(skv.GROUP_HEAD)
    k, v = workloads.make_kv(L, H, n, d, seed=2)
    tier = oracle.assign_groups(ocfg, oracle.GRAN_HEAD, oracle.score_groups(ocfg, oracle.GRAN_HEAD, u16(k), u16(v)))
    for g, value in ((1, oracle.FP16), (3, 7)):
        bad = tier.copy()
        t = int(np.flatnonzero(bad[g] == oracle.INT8)[0])
        bad[g, t] = value
        ws = _setup(cfg, groups)
        pay = torch.zeros(skv.grouped_payload_size(cfg, groups), dtype=torch.uint8, device="cuda")
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        skv.pack_groups(cfg, groups, k.cuda(), v.cuda(), torch.from_numpy(bad).cuda(), ws, pay, st)
        torch.cuda.synchronize()
        assert int(st.item()) == skv.ERR_INVALID_ARG
        assert pay[132:136].cpu().numpy().view(np.uint32)[0] == skv.ERR_INVALID_ARG
        lo = int(pay[112:120].cpu().numpy().view(np.uint64)[0])
        assert not bool(pay[lo:].any()), "no row written"


def test_malformed_grouped_payloads_are_refused():
    L, H, d, n = 2, 2, 64, 400
    cfg, ocfg = configs(L, H, d, n, 0.5, 3)
    gran = oracle.GRAN_HEAD
    budgets = np.float32([0.9, 0.6, 0.4, 0.2])
    groups = skv.Groups(gran, budgets)
    k, v = workloads.make_kv(L, H, n, d, seed=8)
    tier = oracle.assign_groups(ocfg, gran, oracle.score_groups(ocfg, gran, u16(k), u16(v)), budgets)
    good = oracle.pack_groups(ocfg, gran, u16(k), u16(v), tier, budgets)
    hdr64 = good[64:128].view(np.uint64)
    tiermaps_off, stride, chunkidx_off, cstride, segtab_off = (int(x) for x in hdr64[1:6])
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=3)
    ws = _setup(cfg, groups)
    cases = [(off, bt) for off in (0, 20, 24, 40, 120, 132, 200, 256 + 4, 256 + 32 * 2 + 20,
                                   tiermaps_off + n // 4 + 1, tiermaps_off + stride + 5,
                                   chunkidx_off + cstride + 8, chunkidx_off + 8 * 2 + 4, segtab_off + 40)]
    bt_bad = bt.clone()
    bt_bad[2] = -1
    cases.append((None, bt_bad))
    for i, (off, table) in enumerate(cases):
        pay = good.copy()
        if off is not None:
            pay[off] ^= 0x10
        okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
        assert oracle.unpack_groups(ocfg, gran, pay, okc, okc.copy(), table.numpy(), bs, budgets) == oracle.ERR_FORMAT, i
        say(f"malformed grouped payload case {i}")
        kc, vc, st = _gpu_decode(cfg, groups, ws, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, table.cuda())
        assert st == skv.ERR_FORMAT, (i, off)
        assert bool((kc.view(torch.int16) == -21555).all()) and bool((vc.view(torch.int16) == -21555).all()), i
    pay = good.copy()
    pay[128] ^= 1  # the non-finite count is data, not checked
    kc, vc, st = _gpu_decode(cfg, groups, ws, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert st == 0


SAMPLES = 1500


@pytest.mark.parametrize("gran", [oracle.GRAN_LAYER, oracle.GRAN_HEAD])
def test_full_size_grouped(gran):
    """Mistral-7B shape, 32768 tokens: per-layer budgets falling from 0.7 to 0.3
    (mean 0.5; early layers favoured, Sec. 2.6), or per-head maps at b = 0.5."""
    w = workloads.WORKLOADS["mistral7b_32k"]
    L, H, d, n = w.layers, w.kv_heads, w.head_dim, w.tokens
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    ocfg = oracle.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    G = oracle.group_count(ocfg, gran)
    budgets = np.float32(np.linspace(0.7, 0.3, G)) if gran == oracle.GRAN_LAYER else None
    groups = skv.Groups(gran, budgets)
    say(f"full-size grouped gran={gran}: GPU")
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    ws, gkey, gtier, pay, st = _gpu_codec(cfg, groups, k, v)
    assert st == 0
    kh, vh = u16(k), u16(v)
    rng = np.random.default_rng(gran)
    if gran == oracle.GRAN_LAYER:
        say("full-size grouped: oracle scores and maps")
        okey = oracle.score_groups(ocfg, gran, kh, vh)
        assert np.array_equal(bits64(gkey), bits64(okey)), "scores"
    else:
        # per-head scores: every group on sampled tokens (exact sums), maps from the GPU scores
        w2 = oracle.decay_table(w.decay, 2, n)
        for t in rng.choice(n, 64, replace=False):
            for g in range(G):
                s = oracle.sumsq_group(ocfg, gran, kh, vh, g, int(t))
                assert gkey[g, t] == float(s) * 2.0 ** -48 * w2[n - 1 - t], (g, int(t))
        okey = gkey
    otier = oracle.assign_groups(ocfg, gran, okey, budgets)
    assert np.array_equal(gtier, otier), "tier maps"
    meta = oracle.pack_groups_meta(ocfg, gran, otier, budgets)
    gmeta = pay[:meta.size].cpu().numpy().copy()
    gmeta[128:132] = 0
    assert np.array_equal(gmeta, meta), "metadata"
    segtab = meta[int(meta[104:112].view(np.uint64)[0]):][:32 * L * H].view(np.uint64).reshape(L, 2, H, 2)
    offs = [oracle.offsets(otier[g]) for g in range(G)]
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc, vc, gst = _gpu_decode(cfg, groups, ws, pay, L, H, d, n, bs, nb, bt)
    assert gst == 0
    btn = bt.cpu().numpy()
    say(f"full-size grouped: {SAMPLES} sampled rows")
    for (l, kv, h, t) in sample_rows(rng, L, H, n, SAMPLES):
        g = 0 if gran == oracle.GRAN_TOKEN else l if gran == oracle.GRAN_LAYER else l * H + h
        tr = otier[g, t]
        src = (kh if kv == 0 else vh)[l, h, t]
        want, scale, _ = oracle.encode_row(tr, src)
        units, qrank = offs[g]
        row_off = int(segtab[l, kv, h, 1]) + int(units[t]) * (d // 2)
        assert np.array_equal(pay[row_off:row_off + want.size].cpu().numpy(), want), (l, kv, h, t, int(tr))
        if tr in (oracle.INT8, oracle.INT4):
            so = int(segtab[l, kv, h, 0]) + 4 * int(qrank[t])
            assert pay[so:so + 4].cpu().numpy().view(np.uint32)[0] == np.float32(scale).view(np.uint32)
        cache = kc if kv == 0 else vc
        grow = cache[l, int(btn[t // bs]), t % bs, h].cpu().numpy().view(np.uint16)
        assert np.array_equal(grow, oracle.decode_row(tr, d, want, scale)), ("cache", l, kv, h, t)
