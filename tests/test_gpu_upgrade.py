"""Cold-tier precision upgrade (Sec. 4.2, Sec. 8 cold-tier fetch) on the GPU
vs the oracle, through the C ABI.

The upgrade payload must equal the oracle's byte for byte (both modes, every
head size, token lists spanning several 256-token chunks with a ragged tail,
rows with non-finite and zero elements), and applying it to the cache that
unpack filled must give the oracle's cache bit for bit.  At full size the
launch the benchmark times is checked on sampled tokens.  Bad token lists
and mismatched payloads are refused through the status words.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

MODES = (skv.UPGRADE_FP16, skv.UPGRADE_RESIDUAL8)


def _setup(L, H, d, n, b, seed, specials=False):
    cfg, ocfg = configs(L, H, d, n, b, 3)
    k, v = workloads.make_kv(L, H, n, d, seed=seed)
    if specials:
        plant_specials(k, v, seed)
    tier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    return cfg, ocfg, k, v, tier


def _tokens(rng, n, m):
    return np.sort(rng.choice(n, size=m, replace=False)).astype(np.int32)


def _gpu_upgrade(cfg, k, v, tier, tokens, mode):
    up = torch.full((skv.upgrade_size(cfg, tokens.size, mode),), 0xA5, dtype=torch.uint8, device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.pack_upgrade(cfg, k.cuda(), v.cuda(), torch.from_numpy(tier).cuda(), torch.from_numpy(tokens).cuda(),
                     mode, up, st)
    torch.cuda.synchronize()
    return up, int(st.item())


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("L,H,d,n,b,m", [(2, 2, 64, 700, 0.3, 555), (1, 3, 32, 300, 0.2, 300),
                                         (2, 1, 128, 1000, 0.6, 257), (1, 2, 256, 520, 0.4, 1),
                                         (3, 2, 128, 2000, 0.15, 1300)])
def test_upgrade_payload_and_apply_match_oracle(mode, L, H, d, n, b, m):
    say(f"upgrade mode={mode} L={L} H={H} d={d} n={n} b={b} m={m}")
    rng = np.random.default_rng(n + m)
    cfg, ocfg, k, v, tier = _setup(L, H, d, n, b, seed=n, specials=True)
    tokens = _tokens(rng, n, m)
    want = oracle.pack_upgrade(ocfg, u16(k), u16(v), tier, tokens, mode)
    up, st = _gpu_upgrade(cfg, k, v, tier, tokens, mode)
    assert st == 0
    got = up.cpu().numpy()
    assert got.size == want.size
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} bytes differ, first at {bad[:8]}"

    # apply on top of the unpacked cache: GPU unpack + GPU upgrade vs the oracle chain
    bs = 16
    nb = workloads.blocks_for(n, bs) + 2
    bt = workloads.make_block_table(n, bs, nb, seed=m)
    payload = oracle.pack(ocfg, u16(k), u16(v), tier)
    okc, ovc, ost = oracle_decode(ocfg, payload, L, H, d, bs, nb, bt.numpy())
    assert ost == 0
    assert oracle.unpack_upgrade(ocfg, want, okc, ovc, bt.numpy(), bs) == 0
    kc, vc, gst = gpu_decode(cfg, torch.from_numpy(payload).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert gst == 0
    ust = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.unpack_upgrade(cfg, up, m, mode, kc, vc, bt.cuda(), bs, ust)
    torch.cuda.synchronize()
    assert int(ust.item()) == 0
    assert np.array_equal(u16(kc), okc), "K cache"
    assert np.array_equal(u16(vc), ovc), "V cache"


def test_fp16_upgrade_restores_exact_rows():
    L, H, d, n = 2, 2, 64, 600
    cfg, ocfg, k, v, tier = _setup(L, H, d, n, 0.25, seed=3)
    tokens = np.flatnonzero(tier != oracle.FP16).astype(np.int32)
    up, st = _gpu_upgrade(cfg, k, v, tier, tokens, skv.UPGRADE_FP16)
    assert st == 0
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=1).cuda()
    kc, vc, gst = gpu_decode(cfg, torch.from_numpy(oracle.pack(ocfg, u16(k), u16(v), tier)).cuda(),
                             L, H, d, n, bs, nb, bt)
    ust = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.unpack_upgrade(cfg, up, tokens.size, skv.UPGRADE_FP16, kc, vc, bt, bs, ust)
    torch.cuda.synchronize()
    assert gst == 0 and int(ust.item()) == 0
    pos = bt.cpu().numpy()[np.arange(n) // bs] * bs + np.arange(n) % bs
    for cache, src in ((kc, k), (vc, v)):
        flat = u16(cache).reshape(L, -1, H, d)[:, pos]  # [L][n][H][d]
        assert np.array_equal(flat.transpose(0, 2, 1, 3), u16(src)), "every row exact after the upgrade"


def test_bad_token_lists_are_refused():
    L, H, d, n = 1, 2, 64, 300
    cfg, ocfg, k, v, tier = _setup(L, H, d, n, 0.3, seed=5)
    for tokens in ([5, 5, 9], [9, 5], [0, n], [-1, 3]):
        t = np.asarray(tokens, np.int32)
        with pytest.raises(oracle.OracleError) as e:
            oracle.pack_upgrade(ocfg, u16(k), u16(v), tier, t, skv.UPGRADE_RESIDUAL8)
        assert e.value.status == oracle.ERR_INVALID_ARG
        up, st = _gpu_upgrade(cfg, k, v, tier, t, skv.UPGRADE_RESIDUAL8)
        assert st == skv.ERR_INVALID_ARG
        assert up[72:76].cpu().numpy().view(np.uint32)[0] == skv.ERR_INVALID_ARG
    bad_tier = tier.copy()
    bad_tier[7] = 9
    up, st = _gpu_upgrade(cfg, k, v, bad_tier, np.asarray([3, 7], np.int32), skv.UPGRADE_FP16)
    assert st == skv.ERR_INVALID_ARG


def test_mismatched_upgrade_is_refused_and_writes_nothing():
    L, H, d, n = 2, 2, 64, 400
    cfg, ocfg, k, v, tier = _setup(L, H, d, n, 0.3, seed=8)
    tokens = np.arange(10, 300, 3, dtype=np.int32)
    good = oracle.pack_upgrade(ocfg, u16(k), u16(v), tier, tokens, skv.UPGRADE_RESIDUAL8)
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=2)
    cases = []
    for off, val in ((0, 0x12345678), (20, n + 1), (24, tokens.size + 1), (28, 0), (72, 1)):
        bad = good.copy()
        bad[off:off + 4] = np.asarray([val], np.uint32).view(np.uint8)
        cases.append((bad, bt))
    unsorted = good.copy()
    unsorted[256:264] = np.asarray([tokens[1], tokens[0]], np.int32).view(np.uint8)
    cases.append((unsorted, bt))
    bt_bad = bt.clone()
    bt_bad[3] = nb
    cases.append((good, bt_bad))
    for i, (pay, table) in enumerate(cases):
        say(f"mismatch case {i}")
        kc, vc = caches(L, nb, bs, H, d, "cuda")
        st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
        skv.unpack_upgrade(cfg, torch.from_numpy(pay).cuda(), tokens.size, skv.UPGRADE_RESIDUAL8, kc, vc,
                           table.cuda(), bs, st)
        torch.cuda.synchronize()
        assert int(st.item()) == skv.ERR_FORMAT, i
        assert bool((kc.view(torch.int16) == -21555).all()) and bool((vc.view(torch.int16) == -21555).all()), i
        okc = np.full((L, nb, bs, H, d), 0xABCD, np.uint16)
        assert oracle.unpack_upgrade(ocfg, pay, okc, okc.copy(), table.numpy(), bs) == oracle.ERR_FORMAT, i


@pytest.mark.parametrize("mode", MODES)
def test_full_size_upgrade_sampled(mode):
    """Mistral-7B shape, 32768 tokens at b = 0.3: every INT4 and DROP token
    is upgraded in one launch; sampled tokens are rebuilt by the oracle one at
    a time and compared with their rows and scales in the GPU payload."""
    w = workloads.WORKLOADS["mistral7b_32k"]
    L, H, d, n = w.layers, w.kv_heads, w.head_dim, w.tokens
    say(f"full-size upgrade mode={mode}")
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    codec = skv.Codec(cfg)
    codec.encode(k, v)
    tier = codec.tier.cpu().numpy()
    tokens = np.flatnonzero((tier == oracle.INT4) | (tier == oracle.DROP)).astype(np.int32)
    assert tokens.size > 256
    m = tokens.size
    up = torch.empty(skv.upgrade_size(cfg, m, mode), dtype=torch.uint8, device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.pack_upgrade(cfg, k, v, codec.tier, torch.from_numpy(tokens).cuda(), mode, up, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    ocfg = oracle.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    hdr = up[:256].cpu().numpy()
    offs = hdr[32:72].view(np.uint64)
    assert hdr[:32].view(np.uint32).tolist() == [0x55564B53, 1, L, H, d, n, m, mode]
    assert int(offs[4]) == up.numel() == oracle.upgrade_size(ocfg, m, mode)
    assert np.array_equal(up[int(offs[0]):int(offs[0]) + 4 * m].cpu().numpy().view(np.int32), tokens)
    assert np.array_equal(up[int(offs[1]):int(offs[1]) + m].cpu().numpy(), tier[tokens])
    rng = np.random.default_rng(mode)
    picks = np.concatenate([[0, m - 1], rng.choice(m, size=40, replace=False)])
    kh_rows = k.view(torch.int16)
    vh_rows = v.view(torch.int16)
    row_bytes = 2 * d if mode == skv.UPGRADE_FP16 else d
    segs = 2 * L * H
    for i in picks:
        t = int(tokens[i])
        kt = kh_rows[:, :, t:t + 1].cpu().numpy().view(np.uint16)
        vt = vh_rows[:, :, t:t + 1].cpu().numpy().view(np.uint16)
        one = oracle.pack_upgrade(oracle.config(L, H, d, 1, 1.0, first_ratio=0.0, decay=0.0), kt, vt,
                                  tier[t:t + 1], np.zeros(1, np.int32), mode)
        o_offs = one[32:72].view(np.uint64)
        want_rows = one[int(o_offs[3]):].reshape(segs, row_bytes)
        idx = int(offs[3]) + (np.arange(segs, dtype=np.int64) * m + int(i)) * row_bytes
        got = up[torch.from_numpy(idx[:, None] + np.arange(row_bytes)).cuda()].cpu().numpy()
        assert np.array_equal(got, want_rows), ("rows", int(i), t)
        if mode == skv.UPGRADE_RESIDUAL8:
            want_s = one[int(o_offs[2]):int(o_offs[2]) + 4 * segs].view(np.uint32)
            sidx = int(offs[2]) + (np.arange(segs, dtype=np.int64) * m + int(i)) * 4
            got_s = up[torch.from_numpy(sidx[:, None] + np.arange(4)).cuda()].cpu().numpy().view(np.uint32)
            assert np.array_equal(got_s.ravel(), want_s), ("scales", int(i), t)
