"""Corrupted payloads: the GPU decoder agrees with the oracle on every one.

Seeded single-bit corruptions anywhere in a payload (header, tier map,
chunk index, per-row metadata, per-channel entries, codes) for the default
and a variant layout, and in upgrade payloads (both modes) and grouped
payloads.  For each, the oracle's unpack either refuses the
payload (format error) or decodes it; the GPU must return the same status,
leave the caches untouched when it refuses, and otherwise write exactly the
oracle's bytes (corrupted scales included: NaN, infinities and overflow
follow IEEE arithmetic on both sides).  Every offset the GPU decoder follows
comes from the header, chunk index and 2-bit map it has validated, so no
corruption can move a read outside the payload.

A directed case replaces every scale with one the quantizer never produces,
where rounding the product once to binary16 and rounding it to binary32
first disagree: the decoder must take the oracle's two roundings.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

TRIALS = 120


def same(got, want, what):
    """Equality of two uint16 arrays, reporting the first differing elements."""
    bad = np.argwhere(got != want)
    assert bad.size == 0, (f"{what}: {len(bad)} elements differ; first {bad[:4].tolist()} "
                           f"got {[hex(got[tuple(i)]) for i in bad[:4]]} want {[hex(want[tuple(i)]) for i in bad[:4]]}")


@pytest.mark.parametrize("q8,q4", [(0, 0), (skv.QUANT_CHANNEL | skv.QUANT_FP16, skv.QUANT_GROUP32 | skv.QUANT_ASYM)])
def test_random_corruptions_match_oracle(q8, q4):
    L, H, d, n, bs = 2, 2, 64, 700, 16
    say(f"fuzz q8={q8} q4={q4}")
    kw = dict(quant_int8=q8, quant_int4=q4)
    cfg, ocfg = skv.config(L, H, d, n, 0.35, **kw), oracle.config(L, H, d, n, 0.35, **kw)
    k, v = workloads.make_kv(L, H, n, d, seed=21)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    good = oracle.pack(ocfg, u16(k), u16(v), tier)
    geo = oracle.geometry(ocfg)
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=21)
    btn, btd = bt.numpy(), bt.cuda()
    rng = np.random.default_rng(1234 + q8 + q4)
    # half the trials in the metadata before layer 0, half anywhere in the layers
    offsets = np.concatenate([rng.integers(0, geo["layers_off"], TRIALS // 2),
                              rng.integers(geo["layers_off"], good.size, TRIALS - TRIALS // 2)])
    refused = 0
    for i, off in enumerate(offsets):
        pay = good.copy()
        pay[off] ^= np.uint8(1 << int(rng.integers(0, 8)))
        okc, ovc, ost = oracle_decode(ocfg, pay, L, H, d, bs, nb, btn)
        kc, vc, gst = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, btd)
        assert gst == ost, (i, int(off), gst, ost)
        same(u16(kc), okc, f"trial {i} offset {int(off)} K")
        same(u16(vc), ovc, f"trial {i} offset {int(off)} V")
        refused += ost != 0
    # the metadata corruptions are nearly all caught (the non-finite counter and padding are not checked)
    assert refused >= TRIALS // 4, refused


@pytest.mark.parametrize("mode", [skv.UPGRADE_FP16, skv.UPGRADE_RESIDUAL8])
def test_random_upgrade_corruptions_match_oracle(mode):
    """Upgrade payloads: the decoder applies or refuses exactly as the oracle."""
    L, H, d, n, bs = 2, 2, 64, 700, 16
    say(f"fuzz upgrade mode={mode}")
    cfg, ocfg = configs(L, H, d, n, 0.3, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=31)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    rng = np.random.default_rng(77 + mode)
    tokens = np.sort(rng.choice(n, size=300, replace=False)).astype(np.int32)
    good = oracle.pack_upgrade(ocfg, u16(k), u16(v), tier, tokens, mode)
    payload = oracle.pack(ocfg, u16(k), u16(v), tier)
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=31)
    base_k, base_v, st = oracle_decode(ocfg, payload, L, H, d, bs, nb, bt.numpy())
    assert st == 0
    for i in range(60):
        pay = good.copy()
        off = int(rng.integers(0, pay.size)) if i % 2 else int(rng.integers(0, min(pay.size, 4096)))
        pay[off] ^= np.uint8(1 << int(rng.integers(0, 8)))
        okc, ovc = base_k.copy(), base_v.copy()
        ost = oracle.unpack_upgrade(ocfg, pay, okc, ovc, bt.numpy(), bs)
        kc = torch.from_numpy(base_k.view(np.int16)).cuda().view(torch.float16)
        vc = torch.from_numpy(base_v.view(np.int16)).cuda().view(torch.float16)
        ust = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        skv.unpack_upgrade(cfg, torch.from_numpy(pay).cuda(), tokens.size, mode, kc, vc, bt.cuda(), bs, ust)
        torch.cuda.synchronize()
        assert int(ust.item()) == (0 if ost == 0 else skv.ERR_FORMAT), (i, off, int(ust.item()), ost)
        same(u16(kc), okc, f"trial {i} offset {off} K")
        same(u16(vc), ovc, f"trial {i} offset {off} V")


def test_random_grouped_corruptions_match_oracle():
    """Grouped payloads (one map per layer): refused or decoded exactly as the oracle."""
    L, H, d, n, bs = 3, 2, 64, 700, 16
    say("fuzz grouped")
    gran = oracle.GRAN_LAYER
    budgets = np.float32([0.8, 0.45, 0.2])
    cfg, ocfg = configs(L, H, d, n, 0.5, 3)
    groups = skv.Groups(gran, budgets)
    ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
    skv.prepare_groups(cfg, groups, ws)
    k, v = workloads.make_kv(L, H, n, d, seed=41)
    otier = oracle.assign_groups(ocfg, gran, oracle.score_groups(ocfg, gran, u16(k), u16(v)), budgets)
    good = oracle.pack_groups(ocfg, gran, u16(k), u16(v), otier, budgets)
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=41)
    rng = np.random.default_rng(4141)
    for i in range(80):
        pay = good.copy()
        off = int(rng.integers(0, pay.size)) if i % 2 else int(rng.integers(0, min(pay.size, 8192)))
        pay[off] ^= np.uint8(1 << int(rng.integers(0, 8)))
        okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
        ovc = okc.copy()
        ost = oracle.unpack_groups(ocfg, gran, pay, okc, ovc, bt.numpy(), bs, budgets)
        kc, vc = caches(L, nb, bs, H, d, "cuda")
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        skv.unpack_groups(cfg, groups, ws, torch.from_numpy(pay).cuda(), kc, vc, bt.cuda(), bs, st)
        torch.cuda.synchronize()
        assert int(st.item()) == (0 if ost == 0 else skv.ERR_FORMAT), (i, off, int(st.item()), ost)
        same(u16(kc), okc, f"trial {i} offset {off} K")
        same(u16(vc), ovc, f"trial {i} offset {off} V")


# Scales the quantizer never produces (it writes RN32(amax / Q)), chosen so
# that code * scale rounded once to binary16 differs from rounding it to
# binary32 first at the codes +-Q, which every quantized row holds.
FOREIGN_SCALES = {oracle.INT8: 0x3D92F5EC, oracle.INT4: 0x3EFFA492}


@pytest.mark.parametrize("grouped", [False, True])
def test_foreign_scales_decode_like_the_oracle(grouped):
    """Every INT8 / INT4 scale replaced by a foreign one: the decoder rounds the
    product to binary32 before the binary16 conversion, as the oracle does."""
    L, H, d, n, bs = 2, 2, 64, 700, 16
    say(f"foreign scales grouped={grouped}")
    cfg, ocfg = configs(L, H, d, n, 0.35, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=5)
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=5)
    if grouped:
        gran, budgets = oracle.GRAN_LAYER, np.float32([0.6, 0.3])
        tiers = oracle.assign_groups(ocfg, gran, oracle.score_groups(ocfg, gran, u16(k), u16(v)), budgets)
        pay = oracle.pack_groups(ocfg, gran, u16(k), u16(v), tiers, budgets)
        segtab_off = int(pay[104:112].view(np.uint64)[0])
        segtab = pay[segtab_off:segtab_off + 32 * L * H].view(np.uint64)
        base = lambda l, kv, h: int(segtab[2 * ((l * 2 + kv) * H + h)])  # noqa: E731
    else:
        tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
        tiers = np.stack([tier] * L)
        pay = oracle.pack(ocfg, u16(k), u16(v), tier)
        geo = oracle.geometry(ocfg)
        base = lambda l, kv, h: geo["layers_off"] + l * geo["layer_stride"] + (kv * H + h) * geo["nq"] * 4  # noqa: E731
    words = pay.view(np.uint32)
    replaced = 0
    for l in range(L):
        _, qrank = oracle.offsets(tiers[l])
        for kv in range(2):
            for h in range(H):
                b4 = base(l, kv, h) // 4
                for tr, bits in FOREIGN_SCALES.items():
                    sel = tiers[l] == tr
                    words[b4 + qrank[sel].astype(np.int64)] = bits
                    replaced += int(sel.sum())
    assert replaced > 0
    okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
    ovc = okc.copy()
    if grouped:
        ost = oracle.unpack_groups(ocfg, gran, pay, okc, ovc, bt.numpy(), bs, budgets)
        groups = skv.Groups(gran, budgets)
        ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
        skv.prepare_groups(cfg, groups, ws)
        kc, vc = caches(L, nb, bs, H, d, "cuda")
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        skv.unpack_groups(cfg, groups, ws, torch.from_numpy(pay).cuda(), kc, vc, bt.cuda(), bs, st)
        torch.cuda.synchronize()
        gst = int(st.item())
    else:
        ost = oracle.unpack(ocfg, pay, okc, ovc, bt.numpy(), bs)
        kc, vc, gst = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    same(u16(kc), okc, "K")
    same(u16(vc), ovc, "V")


@pytest.mark.parametrize("q8,q4", [(skv.QUANT_GROUP64, skv.QUANT_GROUP32 | skv.QUANT_ASYM),
                                   (skv.QUANT_CHANNEL, skv.QUANT_CHANNEL | skv.QUANT_ASYM)])
def test_foreign_variant_scales_decode_like_the_oracle(q8, q4):
    """Variant layouts with binary32 metadata: every group scale and every
    per-channel scale replaced by a seeded random binary32 value (minimums
    kept).  Some products then round differently once than through binary32
    (4 of the 121 344 INT8 elements of the group-64 case alone); the decoder
    must match the oracle bit for bit."""
    L, H, d, n, bs = 2, 2, 64, 700, 16
    say(f"foreign variant scales q8={q8} q4={q4}")
    CH = skv.QUANT_CHANNEL
    kw = dict(num_tiers=3, quant_int8=q8, quant_int4=q4)
    cfg, ocfg = skv.config(L, H, d, n, 0.35, **kw), oracle.config(L, H, d, n, 0.35, **kw)
    k, v = workloads.make_kv(L, H, n, d, seed=9)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    pay = oracle.pack(ocfg, u16(k), u16(v), tier)
    geo = oracle.geometry(ocfg)
    e8, e4 = oracle.meta_bytes(q8, d), oracle.meta_bytes(q4, d)
    sb = oracle.scale_offsets(tier, e8, e4)
    sbk = oracle.scale_offsets(tier, 0 if q8 & CH else e8, 0 if q4 & CH else e4)
    eb = {oracle.INT8: oracle.channel_entry_bytes(q8), oracle.INT4: oracle.channel_entry_bytes(q4)}
    cb8 = d * eb[oracle.INT8] if q8 & CH else 0
    cb4 = d * eb[oracle.INT4] if q4 & CH else 0
    nch = -(-n // 256)
    rng = np.random.default_rng(q8 * 32 + q4)

    def foreign(count):
        return rng.uniform(2.0 ** -9, 2.0 ** -2, count).astype(np.float32).view(np.uint8).reshape(count, 4)

    replaced = 0
    quantized = np.flatnonzero((tier == oracle.INT8) | (tier == oracle.INT4))
    for l in range(L):
        lay = geo["layers_off"] + l * geo["layer_stride"]
        for kv in range(2):
            for h in range(H):
                base = h * geo["seg_scale_bytes_k"] if kv == 0 else H * geo["seg_scale_bytes_k"] + h * geo["seg_scale_bytes"]
                for t in quantized:
                    q = q8 if tier[t] == oracle.INT8 else q4
                    if kv == 0 and q & CH:
                        continue  # per-channel K rows carry no per-row metadata
                    mo = lay + base + int((sbk if kv == 0 else sb)[t])
                    for e in range(oracle.meta_bytes(q, d) // eb[tier[t]]):
                        pay[mo + e * eb[tier[t]]:mo + e * eb[tier[t]] + 4] = foreign(1)[0]
                        replaced += 1
        for h in range(H):
            for c in range(nch):
                for tr, q, off in ((oracle.INT8, q8, 0), (oracle.INT4, q4, cb8)):
                    if not q & CH:
                        continue
                    boff = lay + geo["scales_bytes"] + (h * nch + c) * (cb8 + cb4) + off
                    for ch in range(d):
                        pay[boff + ch * eb[tr]:boff + ch * eb[tr] + 4] = foreign(1)[0]
                        replaced += 1
    assert replaced > 0
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=9)
    okc, ovc, ost = oracle_decode(ocfg, pay, L, H, d, bs, nb, bt.numpy())
    kc, vc, gst = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    same(u16(kc), okc, "K")
    same(u16(vc), ovc, "V")


def test_infinite_scales_decode_like_the_oracle():
    """Rows whose scale is +inf or -inf: code 0 gives a NaN product (written
    as 0x7E00), other codes an infinity; the decoder matches the oracle."""
    L, H, d, n, bs = 1, 2, 64, 600, 16
    say("infinite scales")
    cfg, ocfg = configs(L, H, d, n, 0.4, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=13)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    pay = oracle.pack(ocfg, u16(k), u16(v), tier)
    geo = oracle.geometry(ocfg)
    _, qrank = oracle.offsets(tier)
    words = pay.view(np.uint32)
    quantized = np.flatnonzero((tier == oracle.INT8) | (tier == oracle.INT4))
    for kv in range(2):
        for h in range(H):
            base = (geo["layers_off"] + ((kv * H + h) * geo["nq"]) * 4) // 4
            for i, t in enumerate(quantized[:120]):
                words[base + int(qrank[t])] = 0x7F800000 if i % 2 else 0xFF800000
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=13)
    okc, ovc, ost = oracle_decode(ocfg, pay, L, H, d, bs, nb, bt.numpy())
    kc, vc, gst = gpu_decode(cfg, torch.from_numpy(pay).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    assert (okc == 0x7E00).any() and ((okc & 0x7FFF) == 0x7C00).any()  # the case has both outcomes
    same(u16(kc), okc, "K")
    same(u16(vc), ovc, "V")


def test_infinite_residual_scales_apply_like_the_oracle():
    """RESIDUAL8 upgrade rows whose scale is +inf or -inf: held + code * scale
    is an infinity or, for code 0, a NaN written as 0x7E00, as in the oracle."""
    L, H, d, n, bs = 1, 2, 64, 600, 16
    say("infinite residual scales")
    cfg, ocfg = configs(L, H, d, n, 0.3, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=17)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    tokens = np.flatnonzero(tier != oracle.FP16).astype(np.int32)[:200]
    mode = skv.UPGRADE_RESIDUAL8
    up = oracle.pack_upgrade(ocfg, u16(k), u16(v), tier, tokens, mode)
    m = tokens.size
    scales_off = int(up[48:56].view(np.uint64)[0])  # header: u64 scales_off at byte 48
    sc = up[scales_off:scales_off + 8 * L * H * m].view(np.uint32)
    sc[0::3] = 0x7F800000
    sc[1::3] = 0xFF800000
    payload = oracle.pack(ocfg, u16(k), u16(v), tier)
    nb = workloads.blocks_for(n, bs) + 1
    bt = workloads.make_block_table(n, bs, nb, seed=17)
    bk, bv, st = oracle_decode(ocfg, payload, L, H, d, bs, nb, bt.numpy())
    assert st == 0
    okc, ovc = bk.copy(), bv.copy()
    assert oracle.unpack_upgrade(ocfg, up, okc, ovc, bt.numpy(), bs) == 0
    assert (okc == 0x7E00).any() or (ovc == 0x7E00).any()
    kc = torch.from_numpy(bk.view(np.int16)).cuda().view(torch.float16)
    vc = torch.from_numpy(bv.view(np.int16)).cuda().view(torch.float16)
    ust = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.unpack_upgrade(cfg, torch.from_numpy(up).cuda(), m, mode, kc, vc, bt.cuda(), bs, ust)
    torch.cuda.synchronize()
    assert int(ust.item()) == 0
    same(u16(kc), okc, "K")
    same(u16(vc), ovc, "V")
