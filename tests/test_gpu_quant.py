"""Per-tier quantizer variants on the GPU vs the oracle, through the C ABI.

Bar: with any pair of descriptors (scale groups of 64/32, asymmetric codes,
binary16 metadata, per-channel key scales) the payload (codes, per-group and
per-channel metadata, 16-byte chunk index) and the decoded caches are
bit-identical to the oracle's, including rows with inf/NaN, zero rows,
constant groups and subnormals; malformed variant chunk indexes and channel
prefixes are refused; at full size the launch the benchmark times is checked
on the whole metadata and sampled rows (per-channel K rows against the
oracle's groups of their chunk).
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

Q = skv
ALL = [g | a | f for g in (0, Q.QUANT_GROUP64, Q.QUANT_GROUP32) for a in (0, Q.QUANT_ASYM) for f in (0, Q.QUANT_FP16)]


def _pair(L, H, d, n, b, q8, q4, tiers=3):
    kw = dict(num_tiers=tiers, quant_int8=q8, quant_int4=q4)
    return skv.config(L, H, d, n, b, **kw), oracle.config(L, H, d, n, b, **kw)


def _run(L, H, d, n, b, q8, q4, seed, specials=True, tiers=3):
    cfg, ocfg = _pair(L, H, d, n, b, q8, q4, tiers)
    k, v = workloads.make_kv(L, H, n, d, seed=seed)
    if specials:
        plant_specials(k, v, seed)
        k[0, 0, n // 2, :] = 1.5  # a constant row: zero range for asymmetric groups
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    want = oracle.pack(ocfg, u16(k), u16(v), tier)
    codec = gpu_encode(cfg, k.cuda(), v.cuda(), tier=tier)
    got = codec.payload.cpu().numpy()
    assert int(codec.status[0].item()) == 0
    bad = np.flatnonzero(got != want)
    assert got.size == want.size and bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"
    bs = 16
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=seed)
    okc, ovc, ost = oracle_decode(ocfg, want, L, H, d, bs, nb, bt.numpy())
    kc, vc, gst = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


@pytest.mark.parametrize("q", ALL)
def test_every_descriptor_on_both_tiers(q):
    say(f"quantizer variant q8=q4={q}")
    _run(2, 2, 64, 777, 0.35, q, q, seed=q + 1)


@pytest.mark.parametrize("d,n,b,q8,q4", [
    (32, 300, 0.4, Q.QUANT_GROUP32 | Q.QUANT_FP16, Q.QUANT_ASYM),
    (128, 1030, 0.3, 0, Q.QUANT_ASYM | Q.QUANT_GROUP32),          # INT8 default, INT4 KIVI-style
    (256, 513, 0.45, Q.QUANT_GROUP64 | Q.QUANT_ASYM | Q.QUANT_FP16, Q.QUANT_FP16),
    (128, 257, 0.2, Q.QUANT_ASYM, Q.QUANT_GROUP64 | Q.QUANT_FP16),  # INT4 + DROP regime
    (64, 5, 0.5, Q.QUANT_GROUP32, Q.QUANT_GROUP32),                # tiny request: 2 INT8 + 2 INT4 rows
])
def test_mixed_descriptors(d, n, b, q8, q4):
    say(f"mixed descriptors d={d} n={n} q8={q8} q4={q4}")
    _run(2, 3, d, n, b, q8, q4, seed=d + n)


def test_two_tier_variant():
    _run(2, 2, 128, 900, 0.3, Q.QUANT_GROUP32 | Q.QUANT_ASYM, 0, seed=5, tiers=2)


CHAN = [Q.QUANT_CHANNEL | a | f for a in (0, Q.QUANT_ASYM) for f in (0, Q.QUANT_FP16)]


@pytest.mark.parametrize("q", CHAN)
def test_per_channel_keys_on_both_tiers(q):
    say(f"per-channel keys q8=q4={q}")
    _run(2, 2, 64, 777, 0.35, q, q, seed=q + 3)


@pytest.mark.parametrize("d,n,b,q8,q4,tiers", [
    (32, 300, 0.4, Q.QUANT_CHANNEL | Q.QUANT_GROUP32, Q.QUANT_ASYM, 3),               # per-channel INT8 only
    (128, 1030, 0.3, Q.QUANT_GROUP64, Q.QUANT_CHANNEL | Q.QUANT_ASYM | Q.QUANT_GROUP32, 3),  # INT4 KIVI-style
    (256, 513, 0.45, Q.QUANT_CHANNEL | Q.QUANT_FP16, Q.QUANT_CHANNEL | Q.QUANT_ASYM, 3),
    (128, 257, 0.2, Q.QUANT_CHANNEL, Q.QUANT_CHANNEL | Q.QUANT_FP16, 3),               # INT4 + DROP regime
    (64, 5, 0.5, Q.QUANT_CHANNEL, Q.QUANT_CHANNEL, 3),                                 # one partial chunk
    (128, 900, 0.3, Q.QUANT_CHANNEL | Q.QUANT_ASYM, Q.QUANT_CHANNEL, 2),               # 2-tier, INT4 blocks unused
])
def test_per_channel_mixed(d, n, b, q8, q4, tiers):
    say(f"per-channel mixed d={d} n={n} q8={q8} q4={q4} tiers={tiers}")
    _run(2, 3, d, n, b, q8, q4, seed=d + n + 1, tiers=tiers)


def test_malformed_channel_prefix_is_refused():
    L, H, d, n = 1, 2, 64, 700
    cfg, ocfg = _pair(L, H, d, n, 0.35, Q.QUANT_GROUP32, Q.QUANT_CHANNEL | Q.QUANT_ASYM)
    k, v = workloads.make_kv(L, H, n, d, seed=6)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    good = oracle.pack(ocfg, u16(k), u16(v), tier)
    geo = oracle.geometry(ocfg)
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=6)
    for off in (geo["chunkidx_off"] + 16 + 12, geo["chunkidx_off"] + 32 + 12, 168):
        pay = good.copy()
        pay[off] ^= 0x01
        okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
        assert oracle.unpack(ocfg, pay, okc, okc.copy(), bt.numpy(), bs) == oracle.ERR_FORMAT
        kc, vc, st = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
        assert st == skv.ERR_FORMAT, off
        assert bool((kc.view(torch.int16) == -21555).all())


def test_malformed_variant_chunk_index_is_refused():
    L, H, d, n = 2, 2, 64, 700
    cfg, ocfg = _pair(L, H, d, n, 0.35, Q.QUANT_GROUP32, Q.QUANT_ASYM | Q.QUANT_FP16)
    k, v = workloads.make_kv(L, H, n, d, seed=3)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    good = oracle.pack(ocfg, u16(k), u16(v), tier)
    geo = oracle.geometry(ocfg)
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=3)
    for off in (geo["chunkidx_off"] + 16 + 8, geo["chunkidx_off"] + 32 + 12, 156, 160):
        pay = good.copy()
        pay[off] ^= 0x01
        okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
        assert oracle.unpack(ocfg, pay, okc, okc.copy(), bt.numpy(), bs) == oracle.ERR_FORMAT
        kc, vc, st = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
        assert st == skv.ERR_FORMAT, off
        assert bool((kc.view(torch.int16) == -21555).all())


SAMPLES = 1500


@pytest.mark.parametrize("q8,q4", [(Q.QUANT_GROUP32 | Q.QUANT_FP16, Q.QUANT_ASYM | Q.QUANT_GROUP32),
                                   (Q.QUANT_FP16, Q.QUANT_FP16),
                                   (Q.QUANT_CHANNEL | Q.QUANT_FP16, Q.QUANT_CHANNEL | Q.QUANT_ASYM | Q.QUANT_FP16)])
def test_full_size_variant(q8, q4):
    w = workloads.WORKLOADS["mistral7b_32k"]
    L, H, d, n = w.layers, w.kv_heads, w.head_dim, w.tokens
    kw = dict(first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers, quant_int8=q8, quant_int4=q4)
    cfg, ocfg = skv.config(L, H, d, n, w.budget, **kw), oracle.config(L, H, d, n, w.budget, **kw)
    say(f"full-size variant q8={q8} q4={q4}")
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    codec = skv.Codec(cfg)
    codec.encode(k, v)
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    codec.decode(codec.payload, kc, vc, bt, bs)
    torch.cuda.synchronize()
    assert codec.status.cpu().tolist() == [0, 0]
    tier = codec.tier.cpu().numpy()
    geo = oracle.geometry(ocfg)
    meta = oracle.pack_meta(ocfg, tier)
    gmeta = codec.payload[:geo["layers_off"]].cpu().numpy().copy()
    gmeta[144:148] = 0
    assert np.array_equal(gmeta, meta), "header / tier map / chunk index"
    units, _ = oracle.offsets(tier)
    CH = Q.QUANT_CHANNEL
    e8, e4 = oracle.meta_bytes(q8, d), oracle.meta_bytes(q4, d)
    sb = oracle.scale_offsets(tier, e8, e4)
    sbk = oracle.scale_offsets(tier, 0 if q8 & CH else e8, 0 if q4 & CH else e4)
    cb8 = d * oracle.channel_entry_bytes(q8) if q8 & CH else 0
    cb4 = d * oracle.channel_entry_bytes(q4) if q4 & CH else 0
    nch = -(-n // 256)
    kh, vh = u16(k), u16(v)
    btn = bt.cpu().numpy()
    pay = codec.payload
    rng = np.random.default_rng(q8 * 16 + q4)
    groups = {}
    for (l, kv, h, t) in sample_rows(rng, L, H, n, SAMPLES):
        tr = tier[t]
        q = q8 if tr == oracle.INT8 else q4
        lay = geo["layers_off"] + l * geo["layer_stride"]
        off = lay + geo["scales_bytes"] + geo["channel_bytes"] + (kv * H + h) * geo["seg_stride"] + int(units[t]) * (d // 2)
        cache = kc if kv == 0 else vc
        grow = cache[l, int(btn[t // bs]), t % bs, h].cpu().numpy().view(np.uint16)
        if kv == 0 and tr in (oracle.INT8, oracle.INT4) and q & CH:
            # per-channel K row: the oracle's groups of its chunk, channel by channel
            c = t // 256
            key = (l, h, c, int(tr))
            if key not in groups:
                rows = [u for u in range(c * 256, min(n, (c + 1) * 256)) if tier[u] == tr]
                ent, codes = [], np.zeros((len(rows), d), np.int32)
                for i in range(d):
                    cc, m, _ = oracle.quant_group(tr, q, kh[l, h, rows, i])
                    codes[:, i] = cc
                    ent.append(m)
                groups[key] = (rows, codes, np.concatenate(ent))
            rows, codes, block = groups[key]
            boff = lay + geo["scales_bytes"] + (h * nch + c) * (cb8 + cb4) + (cb8 if tr == oracle.INT4 else 0)
            assert np.array_equal(pay[boff:boff + block.size].cpu().numpy(), block), ("channel block", key)
            cj = codes[rows.index(t)]
            want = (cj & 0xFF).astype(np.uint8) if tr == oracle.INT8 else \
                ((cj[0::2] & 0xF) | ((cj[1::2] & 0xF) << 4)).astype(np.uint8)
            data = pay[off:off + want.size].cpu().numpy()
            assert np.array_equal(data, want), ("channel row", l, h, t)
            assert np.array_equal(grow, oracle.decode_row_channel(tr, q, d, data, block)), ("cache", l, kv, h, t)
            continue
        data, mb, _ = oracle.encode_row_q(tr, q, (kh if kv == 0 else vh)[l, h, t])
        assert np.array_equal(pay[off:off + data.size].cpu().numpy(), data), (l, kv, h, t, int(tr))
        if mb.size:
            base = h * geo["seg_scale_bytes_k"] if kv == 0 else H * geo["seg_scale_bytes_k"] + h * geo["seg_scale_bytes"]
            mo = lay + base + int((sbk if kv == 0 else sb)[t])
            assert np.array_equal(pay[mo:mo + mb.size].cpu().numpy(), mb), ("meta", l, kv, h, t)
        assert np.array_equal(grow, oracle.decode_row_q(tr, q, d, data, mb)), ("cache", l, kv, h, t)


DESCRIPTORS = [g | a | f | c for g in (0, Q.QUANT_GROUP64, Q.QUANT_GROUP32) for a in (0, Q.QUANT_ASYM)
               for f in (0, Q.QUANT_FP16) for c in (0, Q.QUANT_CHANNEL)]


def _random_pair_case(rng):
    """A seeded random shape, budget, tier policy and descriptor pair (every
    group size, asymmetric codes, binary16 metadata and per-channel keys, so
    metadata entries of different widths interleave at 2-byte offsets)."""
    d = int(rng.choice([32, 64, 128, 256]))
    n = int(rng.integers(64, 1500))
    b = float(np.float32(rng.uniform(0.1, 1.0)))
    tiers = int(rng.choice([2, 3]))
    q8, q4 = (int(x) for x in rng.choice(DESCRIPTORS, 2))
    return int(rng.integers(1, 3)), int(rng.integers(1, 4)), d, n, b, q8, q4, tiers


def test_random_descriptor_pairs():
    """Twenty-four seeded random descriptor pairs on random shapes: payload and
    decoded caches bit-identical to the oracle's."""
    rng = np.random.default_rng(4242)
    for case in range(24):
        L, H, d, n, b, q8, q4, tiers = _random_pair_case(rng)
        say(f"random descriptor pair #{case}: L={L} H={H} d={d} n={n} b={b} q8={q8} q4={q4} tiers={tiers}")
        _run(L, H, d, n, b, q8, q4, seed=1000 + case, tiers=tiers)
