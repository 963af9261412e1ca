"""Pins for the oracle's cold-tier precision upgrade (Sec. 4.2, Fig.
"sysarch": on-demand upgrade of tokens already held at low precision).

FP16 mode restores the listed rows bit for bit whatever their tier (a dropped
token becomes present); residual mode leaves FP16 rows unchanged and shrinks
the error of INT8/INT4/DROP rows to the residual quantizer's half step; rows
not listed are untouched; bad token lists and headers are refused.
"""
import numpy as np
import pytest

import oracle
from paper_2606_08635_amd import workloads


def _setup(L=2, H=2, d=64, n=600, b=0.35, tiers=3, seed=0):
    cfg = oracle.config(L, H, d, n, b, num_tiers=tiers)
    k, v = workloads.make_kv(L, H, n, d, seed=seed)
    k, v = k.numpy().view(np.uint16), v.numpy().view(np.uint16)
    tier = oracle.assign(cfg, oracle.score(cfg, k, v))
    payload = oracle.pack(cfg, k, v, tier)
    nb = workloads.blocks_for(n)
    bt = workloads.make_block_table(n, 16, nb, seed=seed).numpy()
    kc = np.zeros((L, nb, 16, H, d), np.uint16)
    vc = np.zeros_like(kc)
    assert oracle.unpack(cfg, payload, kc, vc, bt, 16) == oracle.OK
    return cfg, k, v, tier, bt, kc, vc


def _rows(cache, bt, t, l, h):
    return cache[l, bt[t // 16], t % 16, h]


def _pick(tier, rng, m):
    # a mix of every tier present
    toks = []
    for tr in range(4):
        idx = np.nonzero(tier == tr)[0]
        if idx.size:
            toks += list(rng.choice(idx, size=min(m, idx.size), replace=False))
    return np.array(sorted(set(toks)), np.int32)


def test_fp16_upgrade_restores_rows_exactly():
    cfg, k, v, tier, bt, kc, vc = _setup()
    toks = _pick(tier, np.random.default_rng(0), 10)
    before_k, before_v = kc.copy(), vc.copy()
    up = oracle.pack_upgrade(cfg, k, v, tier, toks, oracle.UPGRADE_FP16)
    assert up.size == oracle.upgrade_size(cfg, toks.size, oracle.UPGRADE_FP16)
    assert oracle.unpack_upgrade(cfg, up, kc, vc, bt) == oracle.OK
    L, H = cfg.num_layers, cfg.num_kv_heads
    listed = np.zeros(cfg.num_tokens, bool)
    listed[toks] = True
    for t in range(cfg.num_tokens):
        for l in range(L):
            for h in range(H):
                if listed[t]:
                    assert np.array_equal(_rows(kc, bt, t, l, h), k[l, h, t])
                    assert np.array_equal(_rows(vc, bt, t, l, h), v[l, h, t])
                else:
                    assert np.array_equal(_rows(kc, bt, t, l, h), _rows(before_k, bt, t, l, h))


@pytest.mark.parametrize("tiers,b", [(3, 0.35), (2, 0.3), (3, 0.2)])
def test_residual_upgrade_shrinks_error_to_half_step(tiers, b):
    cfg, k, v, tier, bt, kc, vc = _setup(b=b, tiers=tiers, seed=3)
    toks = _pick(tier, np.random.default_rng(1), 12)
    before = kc.copy()
    up = oracle.pack_upgrade(cfg, k, v, tier, toks, oracle.UPGRADE_RESIDUAL8)
    assert oracle.unpack_upgrade(cfg, up, kc, vc, bt) == oracle.OK
    L, H, d, m = cfg.num_layers, cfg.num_kv_heads, cfg.head_dim, toks.size
    data_off = int(up[56:64].view(np.uint64)[0])
    scales_off = int(up[48:56].view(np.uint64)[0])
    for i, t in enumerate(toks):
        for l in range(L):
            for h in range(H):
                x = k[l, h, t].view(np.float16).astype(np.float64)
                old = _rows(before, bt, t, l, h).view(np.float16).astype(np.float64)
                new = _rows(kc, bt, t, l, h).view(np.float16).astype(np.float64)
                seg = (l * 2 + 0) * H + h
                scale = float(up[scales_off + 4 * (seg * m + i):][:4].view(np.float32)[0])
                if tier[t] == oracle.FP16:
                    assert scale == 0.0 and np.array_equal(new, x)
                    continue
                # residual quantizer: half a step, slack for the rounded
                # reciprocal and the two roundings of the sum
                ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -14))) - 10)
                bound = scale * (0.5 + 2.0 ** -14) + ulp
                assert np.all(np.abs(new - x) <= bound), (t, l, h)
                assert np.abs(new - x).max() <= np.abs(old - x).max()
                codes = up[data_off + (seg * m + i) * d:][:d].view(np.int8)
                assert np.abs(codes).max() == 127 or scale == 0.0


def test_upgrade_layout_and_errors():
    cfg, k, v, tier, bt, kc, vc = _setup()
    L, H, d, n = cfg.num_layers, cfg.num_kv_heads, cfg.head_dim, cfg.num_tokens
    toks = np.array([3, 50, 51, 599], np.int32)
    up = oracle.pack_upgrade(cfg, k, v, tier, toks, oracle.UPGRADE_RESIDUAL8)
    hdr = up[:256].view(np.uint32)
    assert hdr[0] == 0x55564B53 and hdr[1] == 1 and list(hdr[2:8]) == [L, H, d, n, 4, 1]
    up256 = lambda x: (x + 255) // 256 * 256
    total = 256 + up256(16) + up256(4) + up256(L * 2 * H * 4 * 4) + L * 2 * H * 4 * d
    assert up.size == total == int(up[64:72].view(np.uint64)[0])
    assert np.array_equal(up[256:272].view(np.int32), toks)
    assert np.array_equal(up[512:516], tier[toks])
    for bad in ([3, 3, 9], [5, 2], [-1, 4], [n]):
        with pytest.raises(oracle.OracleError):
            oracle.pack_upgrade(cfg, k, v, tier, np.array(bad, np.int32), oracle.UPGRADE_FP16)
    for off in (0, 4, 20, 24, 72):
        bad = up.copy()
        bad[off] ^= 1
        assert oracle.unpack_upgrade(cfg, bad, kc.copy(), vc.copy(), bt) == oracle.ERR_FORMAT
    bad = up.copy()
    bad[260:264] = np.frombuffer(np.int32(n + 5).tobytes(), np.uint8)  # token out of range
    assert oracle.unpack_upgrade(cfg, bad, kc.copy(), vc.copy(), bt) == oracle.ERR_FORMAT
