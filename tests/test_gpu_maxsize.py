"""The largest request the codec accepts: n = 2^21 tokens (8192 chunks, the
capacity of the per-request prep and check kernels' shared arrays), at the
smallest row (one layer, one KV head, d = 32) so the oracle finishes in
seconds.  Scores, tier map, payload and decoded caches must equal the
oracle's bit for bit, for the default quantizer at n = 2^21 and for a 2-tier
per-channel/asymmetric variant at n = 2^21 - 1 (a ragged last chunk).
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

N_MAX = 1 << 21


@pytest.mark.parametrize("n,b,tiers,q8,q4", [
    (N_MAX, 0.5, 3, 0, 0),
    (N_MAX - 1, 0.3, 2, skv.QUANT_CHANNEL | skv.QUANT_ASYM, 0),
])
def test_largest_request_bit_exact(n, b, tiers, q8, q4):
    L, H, d, bs = 1, 1, 32, 16
    say(f"max size n={n} b={b} tiers={tiers} q8={q8}")
    # decay 1e-4: 2 lambda (n - 1) = 419 stays inside the decay table's range (<= 700)
    kw = dict(num_tiers=tiers, quant_int8=q8, quant_int4=q4, decay=1e-4)
    cfg, ocfg = skv.config(L, H, d, n, b, **kw), oracle.config(L, H, d, n, b, **kw)
    k, v = workloads.make_kv(L, H, n, d, seed=7)
    kh, vh = u16(k), u16(v)
    okey = oracle.score(ocfg, kh, vh)
    otier = oracle.assign(ocfg, okey)
    opay = oracle.pack(ocfg, kh, vh, otier)
    codec = gpu_encode(cfg, k.cuda(), v.cuda())
    assert np.array_equal(bits64(codec.scores.cpu().numpy()), bits64(okey)), "scores"
    assert np.array_equal(codec.tier.cpu().numpy(), otier), "tier map"
    assert int(codec.status[0].item()) == 0
    gpay = codec.payload.cpu().numpy()
    diff = np.flatnonzero(gpay != opay)
    assert gpay.size == opay.size and diff.size == 0, f"{diff.size} bytes differ, first {diff[:8]}"
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=7)
    kc, vc, st = gpu_decode(cfg, codec.payload, L, H, d, n, bs, nb, bt.cuda())
    okc, ovc, ost = oracle_decode(ocfg, opay, L, H, d, bs, nb, bt.numpy())
    assert st == 0 and ost == oracle.OK
    assert np.array_equal(u16(kc), okc), "K cache"
    assert np.array_equal(u16(vc), ovc), "V cache"


def test_one_token_past_the_maximum_is_refused():
    cfg = skv.config(1, 1, 32, N_MAX + 1, 0.5)
    with pytest.raises(skv.SkvError) as e:
        skv.payload_size(cfg)
    assert e.value.status == skv.ERR_INVALID_ARG
