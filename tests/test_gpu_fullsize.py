"""GPU vs oracle at the workloads' full sizes, in the launch configuration the
benchmark times (one Codec per request: score -> assign -> pack, then unpack
into a paged cache).

The oracle recomputes every score and the whole tier map (compared bit for
bit), the header / tier map / chunk index section (byte for byte), and a
random sample of rows: payload bytes and scale of the sampled (layer, K/V,
head, token) rows, and the dequantized cache rows.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

SAMPLES = 1500


def _check_request(w, n, k, v, codec, kc, vc, bt, bs, seed):
    cfg = codec.cfg
    ocfg = oracle.config(w.layers, w.kv_heads, w.head_dim, n, w.budget, first_ratio=w.first_ratio,
                         decay=w.decay, num_tiers=w.num_tiers)
    L, H, d = w.layers, w.kv_heads, w.head_dim
    kh, vh = u16(k), u16(v)
    say(f"{w.name} n={n}: oracle scores")
    okey = oracle.score(ocfg, kh, vh)
    assert np.array_equal(bits64(codec.scores.cpu().numpy()), bits64(okey)), "scores"
    otier = oracle.assign(ocfg, okey)
    gtier = codec.tier.cpu().numpy()
    assert np.array_equal(gtier, otier), f"tier maps differ at {np.count_nonzero(gtier != otier)} tokens"
    geo = oracle.geometry(ocfg)
    assert codec.payload.numel() == geo["total"] and codec.status[0].item() == 0
    meta = oracle.pack_meta(ocfg, otier)
    gmeta = codec.payload[:geo["layers_off"]].cpu().numpy().copy()
    gmeta[144:148] = 0  # the non-finite row count is data-dependent; checked below
    assert np.array_equal(gmeta, meta), "header / tier map / chunk index"
    units, qrank = oracle.offsets(otier)
    rng = np.random.default_rng(seed)
    rows = sample_rows(rng, L, H, n, SAMPLES)
    say(f"{w.name} n={n}: {len(rows)} sampled rows")
    pay = codec.payload
    for (l, kv, h, t) in rows:
        src = (kh if kv == 0 else vh)[l, h, t]
        want, scale, _ = oracle.encode_row(otier[t], src)
        off = oracle.row_offset(ocfg, geo, units, l, kv, h, t)
        got = pay[off:off + want.size].cpu().numpy()
        assert np.array_equal(got, want), (l, kv, h, t, int(otier[t]))
        if otier[t] in (oracle.INT8, oracle.INT4):
            so = oracle.scale_offset(ocfg, geo, qrank, l, kv, h, t)
            gs = pay[so:so + 4].cpu().numpy().view(np.uint32)[0]
            assert gs == np.float32(scale).view(np.uint32), (l, kv, h, t)
        rec = oracle.decode_row(otier[t], d, want, scale)
        cache = kc if kv == 0 else vc
        grow = cache[l, int(bt[t // bs]), t % bs, h].cpu().numpy().view(np.uint16)
        assert np.array_equal(grow, rec), ("cache", l, kv, h, t)
    return otier


@pytest.mark.parametrize("name", ["qwen7b_b0.3", "qwen7b_b0.5", "mistral7b_8k", "gemma9b_b0.3",
                                  "gemma9b_b0.5", "gemma9b_b0.7", "mistral7b_32k"])
def test_full_size_workload(name):
    w = workloads.WORKLOADS[name]
    n, bs = w.tokens, 16
    say(f"{name}: generate and run on the GPU")
    k, v = workloads.make_kv(w.layers, w.kv_heads, n, w.head_dim, seed=0, outliers=w.outliers, device="cuda")
    cfg = skv.config(w.layers, w.kv_heads, w.head_dim, n, w.budget, first_ratio=w.first_ratio, decay=w.decay,
                     num_tiers=w.num_tiers)
    codec = skv.Codec(cfg)
    codec.encode(k, v)
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(w.layers, nb, bs, w.kv_heads, w.head_dim, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    codec.decode(codec.payload, kc, vc, bt, bs)
    torch.cuda.synchronize()
    assert codec.status.cpu().tolist() == [0, 0]
    _check_request(w, n, k, v, codec, kc, vc, bt.cpu().numpy(), bs, seed=1)


def test_long_context_batch():
    w = workloads.WORKLOADS["long_batch"]
    bs = 16
    lens = w.batch_tokens
    nbs = [workloads.blocks_for(n, bs) for n in lens]
    pool = sum(nbs)
    perm = workloads.make_block_table(pool * bs, bs, pool, seed=0)  # shared pool, shuffled
    kc = torch.empty(w.layers, pool, bs, w.kv_heads, w.head_dim, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    start = 0
    for r, n in enumerate(lens):
        say(f"long batch request {r}: n={n}")
        bt = perm[start:start + nbs[r]].contiguous()
        start += nbs[r]
        k, v = workloads.make_kv(w.layers, w.kv_heads, n, w.head_dim, seed=16 * r, device="cuda")
        cfg = skv.config(w.layers, w.kv_heads, w.head_dim, n, w.budget, first_ratio=w.first_ratio,
                         decay=w.decay, num_tiers=w.num_tiers)
        codec = skv.Codec(cfg)
        codec.encode(k, v)
        codec.decode(codec.payload, kc, vc, bt.cuda(), bs)
        torch.cuda.synchronize()
        assert codec.status.cpu().tolist() == [0, 0]
        _check_request(w, n, k, v, codec, kc, vc, bt.numpy(), bs, seed=100 + r)
        del k, v, codec
