"""GPU path vs the CPU oracle, stage by stage, through the C ABI.

Bar: scores (KV-norm and recency modes), tier maps, payload bytes and
dequantized caches are bit-identical to the oracle (the fp16 reconstruction
tolerance of one ulp is therefore met with zero slack).  Sizes span several
256-token chunks with ragged tails, every head dim, 2- and 3-tier policies,
the drop regimes, n = 1, all-FP16 and all-INT4 budgets, and inputs holding
NaN, infinities, subnormals and zero rows.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

CASES = [
    # L, H, d, n, b, tiers, extra
    (1, 2, 64, 512, 0.5, 3, {}),                       # the paper's tiny setting
    (2, 3, 32, 777, 0.3, 3, {}),
    (2, 2, 128, 1000, 0.3, 2, {}),                     # 2-tier drop regime
    (1, 4, 256, 300, 0.7, 3, {}),
    (3, 2, 64, 257, 0.2, 3, {}),                       # 3-tier below b'=1/4: INT4 + DROP
    (2, 2, 128, 1, 1.0, 3, {}),                        # a single token
    (1, 1, 32, 17, 0.5, 3, {}),
    (2, 2, 64, 4099, 0.45, 3, {}),
    (1, 2, 128, 600, 1.0, 3, {}),                      # all FP16: lossless
    (2, 1, 64, 513, 0.25, 3, {"rho": 0.0}),            # all INT4
    (2, 2, 128, 700, 0.6, 3, {"mode": oracle.RECENCY}),
    (1, 2, 64, 100, 1.0, 3, {"num_sink": 100}),        # every token a sink
    (2, 2, 256, 1031, 0.5, 2, {"decay": 0.01}),
    (4, 2, 128, 2048, 0.35, 3, {"outliers": "student_t"}),
]


def _ids(c):
    L, H, d, n, b, tiers, extra = c
    return f"L{L}H{H}d{d}n{n}b{b}t{tiers}" + "".join(f"-{k}{v}" for k, v in extra.items())


@pytest.mark.parametrize("case", CASES, ids=[_ids(c) for c in CASES])
def test_stages_bit_exact(case):
    L, H, d, n, b, tiers, extra = case
    extra = dict(extra)
    outliers = extra.pop("outliers", "x8")
    say(f"stages {_ids(case)}")
    cfg, ocfg = configs(L, H, d, n, b, tiers, **extra)
    k, v = workloads.make_kv(L, H, n, d, seed=n, outliers=outliers)
    kh, vh = u16(k), u16(v)
    kd, vd = k.cuda(), v.cuda()
    okey = oracle.score(ocfg, kh, vh)
    otier = oracle.assign(ocfg, okey)
    opay = oracle.pack(ocfg, kh, vh, otier)

    # end to end on the GPU
    codec = gpu_encode(cfg, kd, vd)
    assert np.array_equal(bits64(codec.scores.cpu().numpy()), bits64(okey)), "scores"
    assert np.array_equal(codec.tier.cpu().numpy(), otier), "tier map"
    assert codec.status[0].item() == 0
    gpay = codec.payload.cpu().numpy()
    assert gpay.size == opay.size
    diff = np.nonzero(gpay != opay)[0]
    assert diff.size == 0, f"payload differs at {diff.size} bytes, first {diff[:8]}"

    # each later stage fed the oracle's own intermediate
    c2 = gpu_encode(cfg, kd, vd, scores=okey)
    assert np.array_equal(c2.tier.cpu().numpy(), otier)
    c3 = gpu_encode(cfg, kd, vd, tier=otier)
    assert np.array_equal(c3.payload.cpu().numpy(), opay)

    bs = 16
    nb = workloads.blocks_for(n, bs) + 3
    bt = workloads.make_block_table(n, bs, nb, seed=n)
    kc, vc, st = gpu_decode(cfg, torch.from_numpy(opay).cuda(), L, H, d, n, bs, nb, bt.cuda())
    okc, ovc, ost = oracle_decode(ocfg, opay, L, H, d, bs, nb, bt.numpy())
    assert st == 0 and ost == oracle.OK
    assert np.array_equal(u16(kc), okc), "K cache"
    assert np.array_equal(u16(vc), ovc), "V cache"


@pytest.mark.parametrize("d", [32, 64, 128, 256])
@pytest.mark.parametrize("b,tiers", [(0.5, 3), (0.3, 2), (0.3, 3)])
def test_special_values(d, b, tiers):
    L, H, n = 2, 2, 530
    say(f"specials d{d} b{b} t{tiers}")
    cfg, ocfg = configs(L, H, d, n, b, tiers)
    k, v = workloads.make_kv(L, H, n, d, seed=d)
    k, v = plant_specials(k, v, seed=d)
    kh, vh = u16(k), u16(v)
    okey = oracle.score(ocfg, kh, vh)
    otier = oracle.assign(ocfg, okey)
    opay = oracle.pack(ocfg, kh, vh, otier)
    codec = gpu_encode(cfg, k.cuda(), v.cuda())
    assert np.array_equal(bits64(codec.scores.cpu().numpy()), bits64(okey))
    assert np.array_equal(codec.tier.cpu().numpy(), otier)
    assert np.array_equal(codec.payload.cpu().numpy(), opay)
    # non-finite quantized rows are counted in the header
    kf, vf = k.float().numpy(), v.float().numpy()
    quant = (otier == 1) | (otier == 2)
    bad_rows = (~np.isfinite(kf[:, :, quant]).all(-1)).sum() + (~np.isfinite(vf[:, :, quant]).all(-1)).sum()
    assert opay[:256].view(np.uint32)[36] == bad_rows
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=1)
    kc, vc, st = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt.cuda())
    okc, ovc, _ = oracle_decode(ocfg, opay, L, H, d, bs, nb, bt.numpy())
    assert st == 0
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


def test_block_sizes_and_pool():
    L, H, d, n, b = 2, 2, 64, 301, 0.5
    cfg, ocfg = configs(L, H, d, n, b)
    k, v = workloads.make_kv(L, H, n, d, seed=5)
    opay = oracle.pack(ocfg, u16(k), u16(v), oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v))))
    pay = torch.from_numpy(opay).cuda()
    for bs in (1, 7, 16, 64, 512):
        say(f"block size {bs}")
        nb = workloads.blocks_for(n, bs) + 5
        bt = workloads.make_block_table(n, bs, nb, seed=bs)
        kc, vc, st = gpu_decode(cfg, pay, L, H, d, n, bs, nb, bt.cuda())
        okc, ovc, _ = oracle_decode(ocfg, opay, L, H, d, bs, nb, bt.numpy())
        assert st == 0 and np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


def test_rejects_corrupted_payloads_without_writing():
    L, H, d, n, b = 2, 2, 64, 700, 0.5
    cfg, ocfg = configs(L, H, d, n, b)
    k, v = workloads.make_kv(L, H, n, d, seed=9)
    opay = oracle.pack(ocfg, u16(k), u16(v), oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v))))
    bs = 16
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=2)
    cidx = int(opay[:256].view(np.uint64)[11])
    tmap = int(opay[:256].view(np.uint64)[10])
    corruptions = {"magic": (0, 1), "version": (4, 1), "tokens": (20, 1), "count": (52, 1),
                   "status": (148, 1), "chunk-index": (cidx + 8, 1), "tier-map": (tmap + 70, 0x0F)}
    for name, (off, flip) in corruptions.items():
        say(f"corrupt {name}")
        bad = opay.copy()
        bad[off] ^= flip
        assert oracle_decode(ocfg, bad, L, H, d, bs, nb, bt.numpy())[2] == oracle.ERR_FORMAT
        kc, vc, st = gpu_decode(cfg, torch.from_numpy(bad).cuda(), L, H, d, n, bs, nb, bt.cuda(), fill=0x1234)
        assert st == skv.ERR_FORMAT, name
        assert np.all(u16(kc) == 0x1234) and np.all(u16(vc) == 0x1234), name
    say("corrupt block table")
    bad_bt = bt.clone()
    bad_bt[5] = nb
    kc, vc, st = gpu_decode(cfg, torch.from_numpy(opay).cuda(), L, H, d, n, bs, nb, bad_bt.cuda(), fill=0x1234)
    assert st == skv.ERR_FORMAT and np.all(u16(kc) == 0x1234)
    with pytest.raises(skv.SkvError) as e:
        gpu_decode(cfg, torch.from_numpy(opay[:-1].copy()).cuda(), L, H, d, n, bs, nb, bt.cuda())
    assert e.value.status == skv.ERR_FORMAT


def test_pack_flags_tier_maps_off_plan():
    L, H, d, n, b = 1, 2, 64, 300, 0.5
    cfg, ocfg = configs(L, H, d, n, b)
    k, v = workloads.make_kv(L, H, n, d, seed=3)
    otier = oracle.assign(ocfg, oracle.score(ocfg, u16(k), u16(v)))
    for name, mutate in [("count", lambda t: t.__setitem__(200, 0 if t[200] else 1)),
                         ("code", lambda t: t.__setitem__(17, 9))]:
        say(f"off-plan tier map: {name}")
        bad = otier.copy()
        mutate(bad)
        codec = gpu_encode(cfg, k.cuda(), v.cuda(), tier=bad)
        assert codec.status[0].item() == skv.ERR_INVALID_ARG
        assert codec.payload[:256].cpu().numpy().view(np.uint32)[37] == skv.ERR_INVALID_ARG
        with pytest.raises(oracle.OracleError):
            oracle.pack(ocfg, u16(k), u16(v), bad)


def test_deterministic_and_stream_ordered():
    L, H, d, n, b = 4, 4, 128, 3000, 0.4
    cfg, _ = configs(L, H, d, n, b)
    k, v = workloads.make_kv(L, H, n, d, seed=7, device="cuda")
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    outs = []
    for stream in (None, s):
        say(f"determinism stream={stream}")
        with torch.cuda.stream(s if stream is not None else torch.cuda.current_stream()):
            codec = skv.Codec(cfg)
            codec.encode(k, v, stream=stream)
        torch.cuda.synchronize()
        outs.append((codec.scores.cpu().numpy().copy(), codec.payload.cpu().numpy().copy()))
    assert np.array_equal(bits64(outs[0][0]), bits64(outs[1][0]))
    assert np.array_equal(outs[0][1], outs[1][1])


def test_host_link_pieces_overlap_in_order():
    """Several 32 MiB pieces and a ragged tail through one pinned buffer, twice
    in a row with different data; the copies made right after each call on the
    same stream, with no synchronization, must see the whole payload."""
    n = 3 * (32 << 20) + 12345
    host = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    x1 = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    x2 = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    z1, z2 = torch.zeros_like(x1), torch.zeros_like(x2)
    stream = torch.cuda.current_stream()
    skv.link(z1, x1, n, host_staging=host, stream=stream)
    w1 = z1.clone()
    skv.link(z2, x2, n, host_staging=host, stream=stream)
    w2 = z2.clone()
    torch.cuda.synchronize()
    assert torch.equal(w1, x1) and torch.equal(w2, x2)


def test_link_emulation_round_trip():
    x = torch.randint(0, 255, (1 << 20,), dtype=torch.uint8, device="cuda")
    y = torch.zeros_like(x)
    z = torch.zeros_like(x)
    skv.link(y, x, x.numel())
    host = torch.empty(x.numel(), dtype=torch.uint8, pin_memory=True)
    skv.link(z, x, x.numel(), host_staging=host)
    torch.cuda.synchronize()
    assert torch.equal(x, y) and torch.equal(x, z)


def test_link_device_copy_sizes_and_alignment():
    """The device-to-device link: the library's copy kernel (aligned, whole
    16-byte units: one unit, one workgroup's 4096 units and one more, a ragged
    last workgroup) and the runtime copy it hands other cases to (odd sizes,
    pointers off 16-byte alignment) move exactly nbytes and nothing past them."""
    say("link device copy")
    total = (1 << 20) + 4096
    src = torch.randint(0, 255, (total,), dtype=torch.uint8, device="cuda")
    for off, nbytes in [(0, 16), (0, 65536), (0, 65536 + 16), (0, 65536 * 3 + 16 * 7), (0, 1 << 20),
                        (0, 100003), (4, 4096), (16, (1 << 19) + 5), (8, 65536 * 2)]:
        dst = torch.full((total,), 0x5A, dtype=torch.uint8, device="cuda")
        skv.link(dst[off:], src[off:], nbytes)
        torch.cuda.synchronize()
        assert torch.equal(dst[off:off + nbytes], src[off:off + nbytes]), (off, nbytes)
        assert bool((dst[:off] == 0x5A).all()) and bool((dst[off + nbytes:] == 0x5A).all()), (off, nbytes)


@pytest.mark.parametrize("d", [32, 128])
def test_every_binary16_row_maximum(d):
    """Rows whose absmax runs over every positive finite binary16 value, once
    as an INT8 and once as an INT4 row (the quantizer's quotients and code
    range for all row maxima), with every other element a random pattern of
    magnitude at most the row's maximum; payload and cache vs the oracle."""
    L, H, n = 1, 1, 65536
    cfg, ocfg = configs(L, H, d, n, 0.375, 3, num_sink=0)
    plan = skv.plan_tiers(cfg)
    assert (plan["n_int8"], plan["n_int4"]) == (32768, 32768)
    rng = np.random.default_rng(d)
    maxima = np.arange(1, 0x7C00, dtype=np.int64)
    tier = np.full(n, oracle.INT4, np.uint8)
    tier[rng.permutation(n)[:32768]] = oracle.INT8
    planes = []
    for plane in range(2):
        amax = np.empty(n, np.int64)
        for tr in (oracle.INT8, oracle.INT4):
            rows = np.flatnonzero(tier == tr)
            amax[rows] = np.resize(rng.permutation(maxima), rows.size)
        mag = (rng.random((n, d)) * (amax[:, None] + 1)).astype(np.int64)
        mag[np.arange(n), rng.integers(0, d, n)] = amax
        sign = rng.integers(0, 2, (n, d)) << 15
        planes.append(torch.from_numpy((mag | sign).astype(np.uint16).view(np.int16)).view(torch.float16)
                      .reshape(L, H, n, d))
    k, v = planes
    say(f"every-maximum rows d={d}")
    want = oracle.pack(ocfg, u16(k), u16(v), tier)
    pay = torch.empty(want.size, dtype=torch.uint8, device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    skv.pack(cfg, k.cuda(), v.cuda(), torch.from_numpy(tier).cuda(), pay, st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    got = pay.cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} payload bytes differ, first at {bad[:8]}"
    bs, nb = 16, n // 16
    bt = workloads.make_block_table(n, bs, nb, seed=d)
    okc, ovc, ost = oracle_decode(ocfg, want, L, H, d, bs, nb, bt.numpy())
    kc, vc, gst = gpu_decode(cfg, pay, L, H, d, n, bs, nb, bt.cuda())
    assert ost == 0 and gst == 0
    assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc)


def _random_request(rng):
    """A seeded random request: shape, budget, tier policy, sinks, decay,
    score mode, input distribution and paged block size, redrawn until the
    oracle's plan accepts it (sinks within the budget, decay table in range)."""
    while True:
        L, H = int(rng.integers(1, 4)), int(rng.integers(1, 5))
        d = int(rng.choice([32, 64, 128, 256]))
        n = int(np.exp(rng.uniform(0.0, np.log(6000.0))))
        b = float(np.float32(rng.uniform(0.02, 1.0)))
        tiers = int(rng.choice([2, 3]))
        rho = float(rng.choice([0.0, 0.02, 0.1]))
        num_sink = int(rng.choice([-1, -1, int(rng.integers(0, min(n, 64) + 1))]))
        decay = float(rng.choice([1e-4, 1e-3, 5e-3, 1e-2]))
        mode = int(rng.choice([oracle.KVNORM, oracle.RECENCY]))
        cfg, ocfg = configs(L, H, d, n, b, tiers, rho=rho, num_sink=num_sink, decay=decay, mode=mode)
        if oracle.validate(ocfg) != oracle.OK:
            continue
        try:
            oracle.plan(ocfg)
        except oracle.OracleError:
            continue
        extra = dict(outliers=str(rng.choice(["x8", "student_t", "none"])), specials=bool(rng.integers(0, 2)),
                     bs=int(rng.choice([1, 8, 16, 32])))
        return (L, H, d, n, b, tiers, rho, num_sink, decay, mode), cfg, ocfg, extra


def test_random_requests_bit_exact():
    """Thirty seeded random requests end to end (score, assign, pack, unpack
    into a paged cache with a random block size): every stage bit-identical to
    the oracle."""
    rng = np.random.default_rng(8635)
    for case in range(30):
        shape, cfg, ocfg, extra = _random_request(rng)
        L, H, d, n = shape[:4]
        say(f"random request #{case}: {shape} {extra}")
        k, v = workloads.make_kv(L, H, n, d, seed=case, outliers=extra["outliers"])
        if extra["specials"]:
            plant_specials(k, v, case)
        kh, vh = u16(k), u16(v)
        okey = oracle.score(ocfg, kh, vh)
        otier = oracle.assign(ocfg, okey)
        opay = oracle.pack(ocfg, kh, vh, otier)
        codec = gpu_encode(cfg, k.cuda(), v.cuda())
        assert np.array_equal(bits64(codec.scores.cpu().numpy()), bits64(okey)), f"case {case}: scores"
        assert np.array_equal(codec.tier.cpu().numpy(), otier), f"case {case}: tier map"
        assert codec.status[0].item() == 0
        assert np.array_equal(codec.payload.cpu().numpy(), opay), f"case {case}: payload"
        bs = extra["bs"]
        nb = workloads.blocks_for(n, bs) + 2
        bt = workloads.make_block_table(n, bs, nb, seed=case)
        kc, vc, st = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt.cuda())
        okc, ovc, ost = oracle_decode(ocfg, opay, L, H, d, bs, nb, bt.numpy())
        assert st == 0 and ost == oracle.OK, f"case {case}: status {st} / {ost}"
        assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc), f"case {case}: caches"
