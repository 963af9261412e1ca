"""The hot path under HIP graph capture.

score -> assign -> pack -> unpack are kernel launches only (no memsets, no
allocations, no host synchronization), so a caller can capture one request's
step into a HIP graph and replay it.  The graph is replayed three times with
new K/V contents copied into the captured buffers and eager library calls in
between; after every replay the scores, tier map, payload and decoded caches
equal an eager run on the same inputs, byte for byte.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("q8,q4", [(0, 0), (skv.QUANT_CHANNEL | skv.QUANT_FP16, skv.QUANT_GROUP32 | skv.QUANT_ASYM)])
def test_captured_step_replays_match_eager(q8, q4):
    L, H, d, n, bs = 2, 2, 128, 3000, 16
    say(f"graph capture q8={q8} q4={q4}")
    cfg = skv.config(L, H, d, n, 0.4, quant_int8=q8, quant_int4=q4)
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=1, device="cuda")
    k = torch.empty(L, H, n, d, dtype=torch.float16, device="cuda")
    v = torch.empty_like(k)
    codec = skv.Codec(cfg)
    # slots no token maps to (the tail of the last block) keep this fill in every buffer
    kc, vc = caches(L, nb, bs, H, d, "cuda")

    def step(c, kc_, vc_):
        skv.score(cfg, k, v, None, c.scores, c.ws)
        skv.assign_tiers(cfg, c.scores, c.tier)
        skv.pack(cfg, k, v, c.tier, c.payload, c.status[0:1])
        skv.unpack(cfg, c.payload, kc_, vc_, bt, bs, c.status[1:2])

    def load(seed):
        k0, v0 = workloads.make_kv(L, H, n, d, seed=seed)
        k.copy_(k0.cuda())
        v.copy_(v0.cuda())

    load(100)
    step(codec, kc, vc)  # warm-up outside capture
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        step(codec, kc, vc)
    torch.cuda.synchronize()

    ref = skv.Codec(cfg)
    rkc, rvc = caches(L, nb, bs, H, d, "cuda")
    for seed in (11, 12, 13):
        load(seed)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        step(ref, rkc, rvc)  # eager, same inputs
        torch.cuda.synchronize()
        assert codec.status.cpu().tolist() == [0, 0] and ref.status.cpu().tolist() == [0, 0]
        assert torch.equal(codec.scores.view(torch.int64), ref.scores.view(torch.int64)), seed
        assert torch.equal(codec.tier, ref.tier), seed
        assert torch.equal(codec.payload, ref.payload), seed
        assert torch.equal(kc.view(torch.int16), rkc.view(torch.int16)), seed
        assert torch.equal(vc.view(torch.int16), rvc.view(torch.int16)), seed


def test_captured_split_tier_cut_replays_match_oracle():
    """The split tier cut (a row past 32768 non-sink tokens, workspace given:
    14 launches that clear their histograms with kernels, not memsets) under
    capture: every replay on new scores equals the oracle's map."""
    n = 100_003
    say(f"graph capture, split tier cut n={n}")
    cfg, ocfg = configs(1, 1, 32, n, 0.4, 3, decay=1e-3)
    ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device="cuda")
    scores = torch.empty(n, dtype=torch.float64, device="cuda")
    tier = torch.empty(n, dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(5)
    scores.copy_(torch.from_numpy(rng.random(n)))
    skv.assign_tiers(cfg, scores, tier, ws=ws)  # warm-up outside capture
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        skv.assign_tiers(cfg, scores, tier, ws=ws)
    torch.cuda.synchronize()
    for seed in (21, 22, 23):
        key = np.ldexp(1.0 + np.random.default_rng(seed).random(n), np.random.default_rng(seed + 1).integers(-30, 30, n))
        scores.copy_(torch.from_numpy(key))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(tier.cpu().numpy(), oracle.assign(ocfg, key)), seed
        # eager work between replays on the same buffers
        skv.assign_tiers(cfg, scores, tier, ws=ws)
        torch.cuda.synchronize()


def test_captured_batched_split_tier_cut_replays_match_oracle():
    """skv_assign_batch with its workspace under capture: three requests past
    the resident form and one inside it; every replay on new scores equals the
    oracle's maps."""
    lengths = [100_003, 1000, 40_000, 33_000]
    cfg, _ = configs(1, 1, 32, max(lengths), 0.45, 3, decay=1e-3)
    ocfgs = [configs(1, 1, 32, n, 0.45, 3, decay=1e-3)[1] for n in lengths]
    say(f"graph capture, batched split tier cut {lengths}")
    scores = [torch.rand(n, dtype=torch.float64, device="cuda") for n in lengths]
    tiers = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in lengths]
    ws = torch.empty(skv.batch_workspace_size(cfg, scores), dtype=torch.uint8, device="cuda")
    skv.assign_batch(cfg, scores, tiers, ws=ws)  # warm-up outside capture
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        skv.assign_batch(cfg, scores, tiers, ws=ws)
    torch.cuda.synchronize()
    for seed in (31, 32, 33):
        rng = np.random.default_rng(seed)
        keys = [np.ldexp(1.0 + rng.random(n), rng.integers(-30, 30, n)) for n in lengths]
        for s, k in zip(scores, keys):
            s.copy_(torch.from_numpy(k))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (t, k) in enumerate(zip(tiers, keys)):
            assert np.array_equal(t.cpu().numpy(), oracle.assign(ocfgs[i], k)), (seed, i)
        skv.assign_batch(cfg, scores, tiers, ws=ws)  # eager work between replays
        torch.cuda.synchronize()
