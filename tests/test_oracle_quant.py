"""Pins for the oracle's per-tier quantizer variants (Sec. 6.10 and Sec. 8:
any per-tier scheme applies within a tier, e.g. KIVI-style asymmetric
quantization; Sec. 10 on KIVI and KVQuant): scale groups of 64 or 32
elements, asymmetric min/max codes, binary16 metadata.

Checked against definitions that do not go through the oracle's code: every
code is the nearest point of its group's lattice (brute force over all codes
in exact rational arithmetic, up to the rounding of the reciprocal), the
reconstruction error stays within half a step, the stored minimum is the
group's minimum, binary16 metadata is numpy's correctly rounded conversion,
a symmetric group quantizes exactly like the row quantizer on that sub-row,
descriptor 0 is the row quantizer, and the payload layout (per-row metadata
offsets, 16-byte chunk-index entries) follows its definition.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2606_08635_amd import workloads

GROUP = {0: None, oracle.QUANT_GROUP64: 64, oracle.QUANT_GROUP32: 32}
DESCRIPTORS = [g | a | f for g in (0, oracle.QUANT_GROUP64, oracle.QUANT_GROUP32)
               for a in (0, oracle.QUANT_ASYM) for f in (0, oracle.QUANT_FP16)]


def _rows(d, count, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((count, d)) * rng.choice([0.01, 1.0, 300.0], (count, 1))).astype(np.float16)
    x[0, :] = 0
    x[1, :] = np.float16(3.5)                   # a constant group
    x[2, ::3] = np.float16(-0.0)
    x[3, 5] = np.float16(60000.0)               # an outlier channel
    x[4, :] = np.float16(2.0 ** -24) * rng.integers(-3, 4, d)  # subnormals
    return x.view(np.uint16)


def _meta(q, meta, groups):
    dt = np.float16 if q & oracle.QUANT_FP16 else np.float32
    vals = meta.view(dt).astype(np.float64)
    per = 2 if q & oracle.QUANT_ASYM else 1
    return vals.reshape(groups, per)


def _codes(tr, q, d, data):
    if tr == oracle.INT8:
        c = data.view(np.uint8).astype(np.int64)
        return c if q & oracle.QUANT_ASYM else np.where(c >= 128, c - 256, c)
    nib = np.stack([data & 0xF, data >> 4], axis=1).reshape(-1).astype(np.int64)
    return nib if q & oracle.QUANT_ASYM else np.where(nib >= 8, nib - 16, nib)


@pytest.mark.parametrize("q", DESCRIPTORS)
@pytest.mark.parametrize("tr", [oracle.INT8, oracle.INT4])
@pytest.mark.parametrize("d", [32, 128])
def test_codes_are_nearest_lattice_points(q, tr, d):
    gs = min(GROUP[q & 3] or d, d)
    asym = bool(q & oracle.QUANT_ASYM)
    Q, M = (127, 255) if tr == oracle.INT8 else (7, 15)
    for x in _rows(d, 8, seed=q * 7 + tr + d):
        data, meta, bad = oracle.encode_row_q(tr, q, x)
        assert not bad
        assert meta.size == oracle.meta_bytes(q, d)
        m = _meta(q, meta, d // gs)
        codes = _codes(tr, q, d, data)
        xf = x.view(np.float16).astype(np.float64)
        y = oracle.decode_row_q(tr, q, d, data, meta).view(np.float16).astype(np.float64)
        for j in range(d // gs):
            sl = slice(j * gs, (j + 1) * gs)
            s = m[j, 0]
            lo = m[j, 1] if asym else 0.0
            xs = xf[sl]
            if asym:
                assert lo == xs.min()                           # the stored minimum is the group's minimum
                assert codes[sl].min() >= 0 and codes[sl].max() <= M
            else:
                assert np.abs(codes[sl]).max() <= Q
            if s == 0.0:
                assert (codes[sl] == 0).all()
                continue
            if q & oracle.QUANT_FP16:
                raw = (np.float32(xs.max() - xs.min()) / np.float32(M)) if asym else \
                    (np.float32(np.abs(xs).max()) / np.float32(Q))
                assert np.float16(raw) == np.float16(s)          # RN16 of the fp32 quotient
            lattice = range(0, M + 1) if asym else range(-Q, Q + 1)
            S, LO = Fraction(s), Fraction(lo)
            for i, xi in enumerate(xs):
                X = Fraction(float(xi))
                best = min(abs(X - (c * S + LO)) for c in lattice)
                got = abs(X - (int(codes[sl][i]) * S + LO))
                # nearest, up to the rounding of the reciprocal and of x r (relative 2^-22 of a code <= M + 1)
                assert got <= best + S * Fraction(M + 1, 1 << 21), (j, i)
            # reconstruction within half a step plus the binary16 rounding of the result
            ulp = np.spacing(np.abs(y[sl]).astype(np.float16)).astype(np.float64)
            assert (np.abs(y[sl] - xs) <= s / 2 * (1 + 2.0 ** -20) + ulp + 1e-300).all()


@pytest.mark.parametrize("tr", [oracle.INT8, oracle.INT4])
def test_symmetric_groups_are_row_quantizers_on_sub_rows(tr):
    d = 128
    for q, gs in ((oracle.QUANT_GROUP64, 64), (oracle.QUANT_GROUP32, 32)):
        for x in _rows(d, 8, seed=gs + tr):
            data, meta, _ = oracle.encode_row_q(tr, q, x)
            scales = meta.view(np.float32)
            for j in range(d // gs):
                sub, sc, _ = oracle.encode_row(tr, x[j * gs:(j + 1) * gs])
                w = sub.size
                assert np.array_equal(data[j * w:(j + 1) * w], sub)
                assert scales[j].view(np.uint32) == np.float32(sc).view(np.uint32)


@pytest.mark.parametrize("tr", [oracle.INT8, oracle.INT4])
def test_descriptor_zero_is_the_row_quantizer(tr):
    for x in _rows(64, 10, seed=tr):
        data, meta, bad = oracle.encode_row_q(tr, 0, x)
        want, sc, wbad = oracle.encode_row(tr, x)
        assert np.array_equal(data, want) and bad == wbad
        assert meta.view(np.float32)[0].view(np.uint32) == np.float32(sc).view(np.uint32)
        assert np.array_equal(oracle.decode_row_q(tr, 0, 64, data, meta), oracle.decode_row(tr, 64, want, sc))


@pytest.mark.parametrize("q", [oracle.QUANT_ASYM, oracle.QUANT_GROUP32 | oracle.QUANT_FP16,
                               oracle.QUANT_GROUP64 | oracle.QUANT_ASYM | oracle.QUANT_FP16])
def test_non_finite_and_constant_groups(q):
    d = 64
    gs = min(GROUP[q & 3] or d, d)
    x = np.full(d, np.float16(1.25)).view(np.uint16).copy()
    x[gs + 3 if gs < d else 3] = 0x7C00  # +inf in the second group (or the only one)
    for tr in (oracle.INT8, oracle.INT4):
        data, meta, bad = oracle.encode_row_q(tr, q, x)
        assert bad
        y = oracle.decode_row_q(tr, q, d, data, meta)
        bad_group = slice(gs, 2 * gs) if gs < d else slice(0, d)
        assert (y[bad_group] == 0x7E00).all()
        if gs < d:
            # the constant group is reproduced exactly (asymmetric: lo itself; symmetric: 1.25 = Q/Q*1.25)
            np.testing.assert_array_equal(y[:gs].view(np.float16), np.float16(1.25))


@pytest.mark.parametrize("q8,q4", [(oracle.QUANT_GROUP32, oracle.QUANT_ASYM | oracle.QUANT_FP16),
                                   (oracle.QUANT_ASYM, oracle.QUANT_GROUP64 | oracle.QUANT_ASYM),
                                   (oracle.QUANT_FP16, 0)])
def test_variant_payload_layout_and_round_trip(q8, q4):
    L, H, d, n = 2, 2, 64, 600
    cfg = oracle.config(L, H, d, n, 0.35, quant_int8=q8, quant_int4=q4)
    k, v = workloads.make_kv(L, H, n, d, seed=9)
    k, v = k.numpy().view(np.uint16), v.numpy().view(np.uint16)
    k[1, 0, 50, 3] = 0x7E00
    tier = oracle.assign(cfg, oracle.score(cfg, k, v))
    pay = oracle.pack(cfg, k, v, tier)
    geo = oracle.geometry(cfg)
    plan = oracle.plan(cfg)
    e8, e4 = oracle.meta_bytes(q8, d), oracle.meta_bytes(q4, d)
    assert geo["seg_scale_bytes"] == plan["n_int8"] * e8 + plan["n_int4"] * e4
    assert geo["scales_bytes"] == -(-2 * H * geo["seg_scale_bytes"] // 256) * 256
    nch = -(-n // 256)
    assert geo["layers_off"] == geo["chunkidx_off"] + -(-16 * nch // 256) * 256
    hdr = pay[:256].view(np.uint32)
    assert (hdr[39], hdr[40]) == (q8, q4)
    units, qrank = oracle.offsets(tier)
    sb = oracle.scale_offsets(tier, e8, e4)
    ci = pay[geo["chunkidx_off"]:geo["chunkidx_off"] + 16 * nch].view(np.uint32).reshape(nch, 4)
    assert (ci[:, 0] == units[::256]).all() and (ci[:, 1] == qrank[::256]).all()
    assert (ci[:, 2] == sb[::256]).all() and (ci[:, 3] == 0).all()
    width = {oracle.FP16: 2 * d, oracle.INT8: d, oracle.INT4: d // 2, oracle.DROP: 0}
    nb = workloads.blocks_for(n)
    bt = workloads.make_block_table(n, 16, nb, seed=1).numpy()
    kc, vc = (np.zeros((L, nb, 16, H, d), np.uint16) for _ in range(2))
    assert oracle.unpack(cfg, pay, kc, vc, bt, 16) == 0
    for l in range(L):
        lay = geo["layers_off"] + l * geo["layer_stride"]
        for kv in range(2):
            for h in range(H):
                seg = lay + geo["scales_bytes"] + (kv * H + h) * geo["seg_stride"]
                sc = lay + (kv * H + h) * geo["seg_scale_bytes"]
                for t in range(n):
                    tr = tier[t]
                    q = q8 if tr == oracle.INT8 else q4
                    data, meta, _ = oracle.encode_row_q(tr, q, (k if kv == 0 else v)[l, h, t])
                    off = seg + int(units[t]) * (d // 2)
                    assert np.array_equal(pay[off:off + width[tr]], data)
                    assert np.array_equal(pay[sc + int(sb[t]):sc + int(sb[t]) + meta.size], meta)
                    cache = kc if kv == 0 else vc
                    assert np.array_equal(cache[l, bt[t // 16], t % 16, h], oracle.decode_row_q(tr, q, d, data, meta))
    bad = pay.copy()
    bad[geo["chunkidx_off"] + 16 + 8] ^= 1  # a chunk's metadata offset
    assert oracle.unpack(cfg, bad, kc, vc, bt, 16) == oracle.ERR_FORMAT


def test_invalid_descriptors_and_unsupported_paths():
    for q in (3, 32, -1, 0x13, 0x30):
        assert oracle.validate(oracle.config(1, 1, 64, 100, 0.5, quant_int8=q)) == oracle.ERR_INVALID_ARG
    cfg = oracle.config(1, 1, 64, 100, 0.5, quant_int4=oracle.QUANT_ASYM)
    with pytest.raises(oracle.OracleError):
        oracle.upgrade_size(cfg, 4, 0)
    with pytest.raises(oracle.OracleError):
        oracle.grouped_size(cfg, oracle.GRAN_LAYER)
