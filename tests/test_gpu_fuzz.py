"""Corrupted payloads: the GPU decoder agrees with the oracle on every one.

Seeded single-byte corruptions anywhere in a payload (header, tier map,
chunk index, per-row metadata, per-channel entries, codes) for the default
and a variant layout.  For each, the oracle's unpack either refuses the
payload (format error) or decodes it; the GPU must return the same status,
leave the caches untouched when it refuses, and otherwise write exactly the
oracle's bytes (corrupted scales included: NaN, infinities and overflow
follow IEEE arithmetic on both sides).  Every offset the GPU decoder follows
comes from the header, chunk index and 2-bit map it has validated, so no
corruption can move a read outside the payload.
"""
import pytest

from gpu_helpers import *  # noqa: F401,F403

pytestmark = pytest.mark.gpu

TRIALS = 120


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
        assert np.array_equal(u16(kc), okc) and np.array_equal(u16(vc), ovc), (i, int(off))
        refused += ost != 0
    # the metadata corruptions are nearly all caught (the non-finite counter and padding are not checked)
    assert refused >= TRIALS // 4, refused
