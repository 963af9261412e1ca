"""CPU oracle for the SpectrumKV per-token mixed-precision KV transfer codec.

TEST INFRASTRUCTURE ONLY: only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  The GPU library
never reads, links or calls anything here.

This is a thin ctypes wrapper over ``skv_oracle.c`` (plain, single-threaded C);
every function passes numpy arrays through unchanged and raises
``OracleError`` on a nonzero status.  Arrays of binary16 values travel as
``uint16`` bit patterns so that no conversion happens on the way in or out.
"""
import ctypes
import os

import numpy as np

from . import build as _build

OK, ERR_INVALID_ARG, ERR_BUDGET, ERR_CAPACITY, ERR_FORMAT = 0, 1, 2, 3, 4
FP16, INT8, INT4, DROP = 0, 1, 2, 3
KVNORM, ATTN, RECENCY = 0, 1, 2
# quantizer variant descriptor bits: group size (0 row, 1: 64, 2: 32), asymmetric, binary16 metadata
QUANT_GROUP64, QUANT_GROUP32, QUANT_ASYM, QUANT_FP16, QUANT_CHANNEL = 1, 2, 4, 8, 16
GRAN_TOKEN, GRAN_LAYER, GRAN_HEAD = 0, 1, 2
CHUNK_TOKENS = 256


class OracleError(RuntimeError):
    def __init__(self, status, what):
        super().__init__(f"oracle {what} failed with status {status}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("budget", ctypes.c_float), ("first_ratio", ctypes.c_float),
                ("num_sink", ctypes.c_int32), ("decay", ctypes.c_float),
                ("num_tiers", ctypes.c_int32), ("score_mode", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("obs_window", ctypes.c_int32),
                ("quant_int8", ctypes.c_int32), ("quant_int4", ctypes.c_int32)]


class Plan(ctypes.Structure):
    _fields_ = [("n_sink", ctypes.c_int32), ("n_fp16", ctypes.c_int32),
                ("n_int8", ctypes.c_int32), ("n_int4", ctypes.c_int32),
                ("n_drop", ctypes.c_int32), ("budget_units", ctypes.c_int64),
                ("used_units", ctypes.c_int64)]


def _load():
    if not os.path.exists(_build.LIB) or os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    P = ctypes.POINTER
    cfgp = P(Config)
    vp = ctypes.c_void_p
    sig = {
        "ora_validate": (ctypes.c_int, [cfgp]),
        "ora_plan": (ctypes.c_int, [cfgp, P(Plan)]),
        "ora_payload_size": (ctypes.c_int, [cfgp, P(ctypes.c_uint64)]),
        "ora_decay_table": (None, [ctypes.c_float, ctypes.c_int, ctypes.c_int32, vp]),
        "ora_sumsq": (ctypes.c_int, [cfgp, vp, vp, ctypes.c_int32, P(ctypes.c_uint64), P(ctypes.c_uint64)]),
        "ora_score": (ctypes.c_int, [cfgp, vp, vp, vp, vp]),
        "ora_composite": (ctypes.c_uint64, [ctypes.c_double, ctypes.c_int32]),
        "ora_assign": (ctypes.c_int, [cfgp, vp, vp]),
        "ora_offsets": (None, [ctypes.c_int32, vp, vp, vp]),
        "ora_encode_row": (ctypes.c_int, [ctypes.c_int, ctypes.c_int32, vp, vp, P(ctypes.c_float)]),
        "ora_decode_row": (None, [ctypes.c_int, ctypes.c_int32, vp, ctypes.c_float, vp]),
        "ora_encode_row_q": (ctypes.c_int, [ctypes.c_int, ctypes.c_int32, ctypes.c_int32, vp, vp, vp]),
        "ora_decode_row_q": (None, [ctypes.c_int, ctypes.c_int32, ctypes.c_int32, vp, vp, vp]),
        "ora_scale_offsets": (None, [ctypes.c_int32, vp, ctypes.c_uint64, ctypes.c_uint64, vp]),
        "ora_quant_group": (ctypes.c_int, [ctypes.c_int, ctypes.c_int32, ctypes.c_int64, vp, vp, vp]),
        "ora_decode_row_channel": (None, [ctypes.c_int, ctypes.c_int32, ctypes.c_int32, vp, vp, vp]),
        "ora_pack": (ctypes.c_int, [cfgp, vp, vp, vp, vp, ctypes.c_uint64]),
        "ora_check_header": (ctypes.c_int, [cfgp, vp, ctypes.c_uint64]),
        "ora_geometry": (ctypes.c_int, [cfgp, vp]),
        "ora_pack_meta": (ctypes.c_int, [cfgp, vp, vp, ctypes.c_uint64]),
        "ora_unpack": (ctypes.c_int, [cfgp, vp, ctypes.c_uint64, vp, vp, vp, ctypes.c_int32, ctypes.c_int32]),
        "ora_upgrade_size": (ctypes.c_int, [cfgp, ctypes.c_int32, ctypes.c_int32, P(ctypes.c_uint64)]),
        "ora_pack_upgrade": (ctypes.c_int, [cfgp, vp, vp, vp, vp, ctypes.c_int32, ctypes.c_int32, vp, ctypes.c_uint64]),
        "ora_unpack_upgrade": (ctypes.c_int, [cfgp, vp, ctypes.c_uint64, vp, vp, vp, ctypes.c_int32, ctypes.c_int32]),
        "ora_group_count": (ctypes.c_int32, [cfgp, ctypes.c_int32]),
        "ora_plan_group": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, ctypes.c_int32, P(Plan)]),
        "ora_grouped_size": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, P(ctypes.c_uint64)]),
        "ora_sumsq_group": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, ctypes.c_int32, ctypes.c_int32,
                                           P(ctypes.c_uint64), P(ctypes.c_uint64)]),
        "ora_score_groups": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, vp, vp]),
        "ora_assign_groups": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, vp]),
        "ora_pack_groups": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, vp, vp, vp, ctypes.c_uint64]),
        "ora_unpack_groups": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, ctypes.c_uint64, vp, vp, vp,
                                             ctypes.c_int32, ctypes.c_int32]),
        "ora_pack_groups_meta": (ctypes.c_int, [cfgp, ctypes.c_int32, vp, vp, vp, ctypes.c_uint64,
                                                P(ctypes.c_uint64)]),
        "ora_half_to_double": (ctypes.c_double, [ctypes.c_uint16]),
        "ora_float_to_half": (ctypes.c_uint16, [ctypes.c_float]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def _ptr(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.float16:
        a = a.view(np.uint16)
    if a.dtype != np.uint16:
        raise TypeError(f"expected float16/uint16 array, got {a.dtype}")
    return a


def config(num_layers, num_kv_heads, head_dim, num_tokens, budget, first_ratio=0.02, num_sink=-1,
           decay=0.005, num_tiers=3, score_mode=KVNORM, num_q_heads=0, obs_window=0, quant_int8=0, quant_int4=0):
    return Config(num_layers, num_kv_heads, head_dim, num_tokens, budget, first_ratio, num_sink,
                  decay, num_tiers, score_mode, num_q_heads, obs_window, quant_int8, quant_int4)


def validate(cfg):
    return _lib.ora_validate(ctypes.byref(cfg))


def plan(cfg):
    p = Plan()
    st = _lib.ora_plan(ctypes.byref(cfg), ctypes.byref(p))
    if st:
        raise OracleError(st, "plan")
    return {f: getattr(p, f) for f, _ in Plan._fields_}


def payload_size(cfg):
    out = ctypes.c_uint64()
    st = _lib.ora_payload_size(ctypes.byref(cfg), ctypes.byref(out))
    if st:
        raise OracleError(st, "payload_size")
    return out.value


def decay_table(decay, which, count):
    out = np.empty(count, np.float64)
    _lib.ora_decay_table(ctypes.c_float(decay), which, count, _ptr(out))
    return out


def sumsq(cfg, k, v, t):
    """Exact sum of squares of token t over all layers/heads/K/V, in units of 2^-48."""
    k, v = _u16(k), _u16(v)
    hi, lo = ctypes.c_uint64(), ctypes.c_uint64()
    _lib.ora_sumsq(ctypes.byref(cfg), _ptr(k), _ptr(v), t, ctypes.byref(hi), ctypes.byref(lo))
    return (hi.value << 64) | lo.value


def score(cfg, k, v, q=None):
    k, v = _u16(k), _u16(v)
    q = None if q is None else _u16(q)
    out = np.empty(cfg.num_tokens, np.float64)
    st = _lib.ora_score(ctypes.byref(cfg), _ptr(k), _ptr(v), _ptr(q), _ptr(out))
    if st:
        raise OracleError(st, "score")
    return out


def composite(key, t):
    return _lib.ora_composite(float(key), int(t))


def assign(cfg, key):
    key = np.ascontiguousarray(key, np.float64)
    out = np.empty(cfg.num_tokens, np.uint8)
    st = _lib.ora_assign(ctypes.byref(cfg), _ptr(key), _ptr(out))
    if st:
        raise OracleError(st, "assign")
    return out


def offsets(tier):
    tier = np.ascontiguousarray(tier, np.uint8)
    n = tier.shape[0]
    units = np.empty(n, np.uint32)
    qrank = np.empty(n, np.uint32)
    _lib.ora_offsets(n, _ptr(tier), _ptr(units), _ptr(qrank))
    return units, qrank


def encode_row(tier, row):
    """Returns (payload bytes of the row, scale as float32, non-finite flag)."""
    row = _u16(row)
    d = row.shape[0]
    width = {FP16: 2 * d, INT8: d, INT4: d // 2, DROP: 0}[int(tier)]
    out = np.zeros(max(width, 1), np.uint8)
    sc = ctypes.c_float(0.0)
    bad = _lib.ora_encode_row(int(tier), d, _ptr(row), _ptr(out), ctypes.byref(sc))
    return out[:width], np.float32(sc.value), bool(bad)


def meta_bytes(q, d):
    """Metadata bytes of one quantized row under variant descriptor q."""
    g = d if q & 3 == 0 else (64 if q & 3 == 1 else 32)
    g = min(g, d)
    return (d // g) * (2 if q & QUANT_ASYM else 1) * (2 if q & QUANT_FP16 else 4)


def channel_entry_bytes(q):
    """Bytes of one per-channel (or group) entry under descriptor q: s, then lo."""
    return (2 if q & QUANT_ASYM else 1) * (2 if q & QUANT_FP16 else 4)


def quant_group(tier, q, values):
    """One quantization group of binary16 values under descriptor q's bits 2-3:
    returns (codes int32[cnt], metadata entry bytes, non-finite flag)."""
    x = _u16(values)
    codes = np.zeros(x.shape[0], np.int32)
    meta = np.zeros(channel_entry_bytes(q), np.uint8)
    bad = _lib.ora_quant_group(int(tier), int(q), int(x.shape[0]), _ptr(x), _ptr(codes), _ptr(meta))
    return codes, meta, bool(bad)


def decode_row_channel(tier, q, d, data, block):
    """A per-channel K row decoded with its chunk's d channel entries."""
    y = np.zeros(d, np.uint16)
    data = np.ascontiguousarray(data, np.uint8)
    block = np.ascontiguousarray(block, np.uint8)
    _lib.ora_decode_row_channel(int(tier), int(q), int(d), _ptr(data), _ptr(block), _ptr(y))
    return y


def encode_row_q(tier, q, row):
    """Returns (payload bytes of the row, its metadata bytes, non-finite flag)."""
    row = _u16(row)
    d = row.shape[0]
    width = {FP16: 2 * d, INT8: d, INT4: d // 2, DROP: 0}[int(tier)]
    out = np.zeros(max(width, 1), np.uint8)
    mb = meta_bytes(q, d) if int(tier) in (INT8, INT4) else 0
    meta = np.zeros(max(mb, 1), np.uint8)
    bad = _lib.ora_encode_row_q(int(tier), q, d, _ptr(row), _ptr(out), _ptr(meta))
    return out[:width], meta[:mb], bool(bad)


def decode_row_q(tier, q, d, data, meta):
    data = np.ascontiguousarray(data, np.uint8)
    meta = np.ascontiguousarray(meta, np.uint8)
    if data.size == 0:
        data = np.zeros(1, np.uint8)
    if meta.size == 0:
        meta = np.zeros(1, np.uint8)
    out = np.empty(d, np.uint16)
    _lib.ora_decode_row_q(int(tier), q, d, _ptr(data), _ptr(meta), _ptr(out))
    return out


def scale_offsets(tier, e8, e4):
    tier = np.ascontiguousarray(tier, np.uint8)
    out = np.empty(tier.size, np.uint32)
    _lib.ora_scale_offsets(tier.size, _ptr(tier), e8, e4, _ptr(out))
    return out


def decode_row(tier, d, data, scale):
    data = np.ascontiguousarray(data, np.uint8)
    if data.size == 0:
        data = np.zeros(1, np.uint8)
    out = np.empty(d, np.uint16)
    _lib.ora_decode_row(int(tier), d, _ptr(data), ctypes.c_float(scale), _ptr(out))
    return out


def pack(cfg, k, v, tier):
    k, v = _u16(k), _u16(v)
    tier = np.ascontiguousarray(tier, np.uint8)
    size = payload_size(cfg)
    out = np.empty(size, np.uint8)
    st = _lib.ora_pack(ctypes.byref(cfg), _ptr(k), _ptr(v), _ptr(tier), _ptr(out), size)
    if st:
        raise OracleError(st, "pack")
    return out


GEOMETRY_FIELDS = ("tiermap_off", "chunkidx_off", "layers_off", "seg_bytes", "seg_stride",
                   "scales_bytes", "layer_stride", "total", "nq", "seg_scale_bytes",
                   "seg_scale_bytes_k", "chan_block", "channel_bytes")


def geometry(cfg):
    out = np.zeros(len(GEOMETRY_FIELDS), np.uint64)
    st = _lib.ora_geometry(ctypes.byref(cfg), _ptr(out))
    if st:
        raise OracleError(st, "geometry")
    return {f: int(x) for f, x in zip(GEOMETRY_FIELDS, out)}


def pack_meta(cfg, tier):
    """Header, tier map and chunk index: the payload bytes before layer 0."""
    tier = np.ascontiguousarray(tier, np.uint8)
    size = geometry(cfg)["layers_off"]
    out = np.empty(size, np.uint8)
    st = _lib.ora_pack_meta(ctypes.byref(cfg), _ptr(tier), _ptr(out), size)
    if st:
        raise OracleError(st, "pack_meta")
    return out


def row_offset(cfg, geo, units, l, kv, h, t):
    """Byte offset of row (layer l, K/V kv, head h, token t) in the payload."""
    H, d = cfg.num_kv_heads, cfg.head_dim
    return (geo["layers_off"] + l * geo["layer_stride"] + geo["scales_bytes"] + (kv * H + h) * geo["seg_stride"]
            + int(units[t]) * (d // 2))


def scale_offset(cfg, geo, qrank, l, kv, h, t):
    H = cfg.num_kv_heads
    return geo["layers_off"] + l * geo["layer_stride"] + ((kv * H + h) * geo["nq"] + int(qrank[t])) * 4


def check_header(cfg, payload):
    payload = np.ascontiguousarray(payload, np.uint8)
    return _lib.ora_check_header(ctypes.byref(cfg), _ptr(payload), payload.size)


def unpack(cfg, payload, k_cache, v_cache, block_table, block_size=16):
    """Dequantizes into k_cache/v_cache (uint16 [L][num_blocks][block_size][H][d]) in place."""
    payload = np.ascontiguousarray(payload, np.uint8)
    block_table = np.ascontiguousarray(block_table, np.int32)
    for c in (k_cache, v_cache):
        if c.dtype != np.uint16 or not c.flags.c_contiguous:
            raise TypeError("caches must be C-contiguous uint16 arrays")
    num_blocks = k_cache.shape[1]
    st = _lib.ora_unpack(ctypes.byref(cfg), _ptr(payload), payload.size, _ptr(k_cache),
                         _ptr(v_cache), _ptr(block_table), num_blocks, block_size)
    return st


UPGRADE_FP16, UPGRADE_RESIDUAL8 = 0, 1


def upgrade_size(cfg, m, mode):
    out = ctypes.c_uint64()
    st = _lib.ora_upgrade_size(ctypes.byref(cfg), m, mode, ctypes.byref(out))
    if st:
        raise OracleError(st, "upgrade_size")
    return out.value


def pack_upgrade(cfg, k, v, tier, tokens, mode):
    """Upgrade payload for the listed tokens (ascending int32 indices)."""
    k, v = _u16(k), _u16(v)
    tier = np.ascontiguousarray(tier, np.uint8)
    tokens = np.ascontiguousarray(tokens, np.int32)
    size = upgrade_size(cfg, tokens.size, mode)
    out = np.empty(size, np.uint8)
    st = _lib.ora_pack_upgrade(ctypes.byref(cfg), _ptr(k), _ptr(v), _ptr(tier), _ptr(tokens), tokens.size, mode,
                               _ptr(out), size)
    if st:
        raise OracleError(st, "pack_upgrade")
    return out


def unpack_upgrade(cfg, upgrade, k_cache, v_cache, block_table, block_size=16):
    """Applies an upgrade payload to the caches in place; returns the status."""
    upgrade = np.ascontiguousarray(upgrade, np.uint8)
    block_table = np.ascontiguousarray(block_table, np.int32)
    return _lib.ora_unpack_upgrade(ctypes.byref(cfg), _ptr(upgrade), upgrade.size, _ptr(k_cache), _ptr(v_cache),
                                   _ptr(block_table), k_cache.shape[1], block_size)


def group_count(cfg, gran):
    return _lib.ora_group_count(ctypes.byref(cfg), gran)


def _budgets(budgets):
    return None if budgets is None else np.ascontiguousarray(budgets, np.float32)


def plan_group(cfg, gran, budgets, g):
    p = Plan()
    b = _budgets(budgets)
    st = _lib.ora_plan_group(ctypes.byref(cfg), gran, _ptr(b), g, ctypes.byref(p))
    if st:
        raise OracleError(st, "plan_group")
    return {f: getattr(p, f) for f, _ in Plan._fields_}


def grouped_size(cfg, gran, budgets=None):
    out = ctypes.c_uint64()
    b = _budgets(budgets)
    st = _lib.ora_grouped_size(ctypes.byref(cfg), gran, _ptr(b), ctypes.byref(out))
    if st:
        raise OracleError(st, "grouped_size")
    return out.value


def sumsq_group(cfg, gran, k, v, g, t):
    """Exact sum of squares of token t over group g, in units of 2^-48 (int)."""
    k, v = _u16(k), _u16(v)
    hi, lo = ctypes.c_uint64(), ctypes.c_uint64()
    _lib.ora_sumsq_group(ctypes.byref(cfg), gran, _ptr(k), _ptr(v), g, t, ctypes.byref(hi), ctypes.byref(lo))
    return (hi.value << 64) | lo.value


def score_groups(cfg, gran, k, v=None, q=None):
    """float64 [G][n]: every group's score of every token."""
    k = _u16(k)
    v = None if v is None else _u16(v)
    q = None if q is None else _u16(q)
    G = group_count(cfg, gran)
    out = np.empty((G, cfg.num_tokens), np.float64)
    st = _lib.ora_score_groups(ctypes.byref(cfg), gran, _ptr(k), _ptr(v), _ptr(q), _ptr(out))
    if st:
        raise OracleError(st, "score_groups")
    return out


def assign_groups(cfg, gran, key, budgets=None):
    """uint8 [G][n] tier maps."""
    key = np.ascontiguousarray(key, np.float64)
    b = _budgets(budgets)
    tier = np.empty(key.shape, np.uint8)
    st = _lib.ora_assign_groups(ctypes.byref(cfg), gran, _ptr(b), _ptr(key), _ptr(tier))
    if st:
        raise OracleError(st, "assign_groups")
    return tier


def pack_groups(cfg, gran, k, v, tier, budgets=None):
    k, v = _u16(k), _u16(v)
    tier = np.ascontiguousarray(tier, np.uint8)
    b = _budgets(budgets)
    size = grouped_size(cfg, gran, b)
    out = np.empty(size, np.uint8)
    st = _lib.ora_pack_groups(ctypes.byref(cfg), gran, _ptr(b), _ptr(k), _ptr(v), _ptr(tier), _ptr(out), size)
    if st:
        raise OracleError(st, "pack_groups")
    return out


def pack_groups_meta(cfg, gran, tier, budgets=None):
    """The grouped payload's bytes before the layers (header, group table, tier
    maps, chunk indexes, segment table) for on-plan tier maps."""
    tier = np.ascontiguousarray(tier, np.uint8)
    b = _budgets(budgets)
    size = grouped_size(cfg, gran, b)
    out = np.empty(size, np.uint8)
    lo = ctypes.c_uint64()
    st = _lib.ora_pack_groups_meta(ctypes.byref(cfg), gran, _ptr(b), _ptr(tier), _ptr(out), size, ctypes.byref(lo))
    if st:
        raise OracleError(st, "pack_groups_meta")
    return out[:lo.value].copy()


def unpack_groups(cfg, gran, payload, k_cache, v_cache, block_table, block_size=16, budgets=None):
    """Decodes a grouped payload into the caches in place; returns the status."""
    payload = np.ascontiguousarray(payload, np.uint8)
    block_table = np.ascontiguousarray(block_table, np.int32)
    b = _budgets(budgets)
    return _lib.ora_unpack_groups(ctypes.byref(cfg), gran, _ptr(b), _ptr(payload), payload.size, _ptr(k_cache),
                                  _ptr(v_cache), _ptr(block_table), k_cache.shape[1], block_size)


def half_to_double(h):
    return _lib.ora_half_to_double(int(h))


def float_to_half(f):
    return _lib.ora_float_to_half(ctypes.c_float(f))
