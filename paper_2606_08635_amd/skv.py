"""ctypes binding over ``libskv.so`` (the C ABI of ``include/skv.h``).

Argument marshalling only: every function checks that the torch tensors it is
given have the dtype, device and size the configuration implies (the C library
cannot see device buffer sizes), passes their ``data_ptr()`` and the current
HIP stream, and raises ``SkvError`` on a nonzero status.  All codec work runs
in the library's HIP kernels; there is no fallback.  If ``libskv.so`` has not
been built, the first call raises.
"""
import ctypes
import os
from typing import Optional

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libskv.so")

OK, ERR_INVALID_ARG, ERR_BUDGET, ERR_CAPACITY, ERR_FORMAT, ERR_DEVICE = range(6)
FP16, INT8, INT4, DROP = 0, 1, 2, 3
KVNORM, ATTN, RECENCY = 0, 1, 2
UPGRADE_FP16, UPGRADE_RESIDUAL8 = 0, 1
GROUP_TOKEN, GROUP_LAYER, GROUP_HEAD = 0, 1, 2
QUANT_GROUP64, QUANT_GROUP32, QUANT_ASYM, QUANT_FP16, QUANT_CHANNEL = 1, 2, 4, 8, 16
ABI_VERSION = 2
STATIC_SCRATCH_BYTES = 48 << 20  # SKV_STATIC_SCRATCH_BYTES

EXPORTED = ("skv_abi_version", "skv_status_string", "skv_plan_tiers", "skv_payload_size",
            "skv_workspace_size", "skv_prepare", "skv_score", "skv_score_static", "skv_assign_tiers", "skv_pack",
            "skv_unpack", "skv_pack_batch", "skv_unpack_batch", "skv_link", "skv_upgrade_size",
            "skv_pack_upgrade", "skv_unpack_upgrade", "skv_group_count", "skv_plan_groups",
            "skv_grouped_payload_size", "skv_group_workspace_size", "skv_prepare_groups", "skv_score_groups",
            "skv_assign_groups", "skv_pack_groups", "skv_unpack_groups", "skv_batch_workspace_size",
            "skv_score_batch", "skv_assign_batch")


class SkvError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} (status {status})")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("num_layers", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_tokens", ctypes.c_int32),
                ("budget", ctypes.c_float), ("first_ratio", ctypes.c_float),
                ("num_sink", ctypes.c_int32), ("decay", ctypes.c_float),
                ("num_tiers", ctypes.c_int32), ("score_mode", ctypes.c_int32),
                ("num_q_heads", ctypes.c_int32), ("obs_window", ctypes.c_int32),
                ("quant_int8", ctypes.c_int32), ("quant_int4", ctypes.c_int32)]


class Request(ctypes.Structure):
    _fields_ = [("num_tokens", ctypes.c_int32), ("reserved", ctypes.c_int32), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("tier", ctypes.c_void_p), ("payload", ctypes.c_void_p),
                ("payload_bytes", ctypes.c_uint64), ("block_table", ctypes.c_void_p),
                ("dev_status", ctypes.c_void_p)]


class ScoreRequest(ctypes.Structure):
    _fields_ = [("num_tokens", ctypes.c_int32), ("reserved", ctypes.c_int32), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("score", ctypes.c_void_p), ("tier", ctypes.c_void_p)]


class GroupSpec(ctypes.Structure):
    _fields_ = [("granularity", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("budgets", ctypes.POINTER(ctypes.c_float))]


class Plan(ctypes.Structure):
    _fields_ = [("n_sink", ctypes.c_int32), ("n_fp16", ctypes.c_int32),
                ("n_int8", ctypes.c_int32), ("n_int4", ctypes.c_int32),
                ("n_drop", ctypes.c_int32), ("budget_units", ctypes.c_int64),
                ("used_units", ctypes.c_int64)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(the codec has no non-HIP fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P, vp, u64, i32 = ctypes.POINTER, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int32
        cfgp = P(Config)
        sigs = {
            "skv_abi_version": (i32, []),
            "skv_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "skv_plan_tiers": (ctypes.c_int, [cfgp, P(Plan)]),
            "skv_payload_size": (ctypes.c_int, [cfgp, P(u64)]),
            "skv_workspace_size": (ctypes.c_int, [cfgp, P(u64)]),
            "skv_prepare": (ctypes.c_int, [cfgp, vp, vp]),
            "skv_score": (ctypes.c_int, [cfgp, vp, vp, vp, vp, vp, vp]),
            "skv_score_static": (ctypes.c_int, [cfgp, vp, vp, vp, vp, vp]),
            "skv_assign_tiers": (ctypes.c_int, [cfgp, vp, vp, vp, vp]),
            "skv_pack": (ctypes.c_int, [cfgp, vp, vp, vp, vp, u64, vp, vp]),
            "skv_unpack": (ctypes.c_int, [cfgp, vp, u64, vp, vp, vp, i32, i32, vp, vp]),
            "skv_link": (ctypes.c_int, [vp, vp, u64, vp, vp]),
            "skv_pack_batch": (ctypes.c_int, [cfgp, P(Request), i32, i32, i32, vp]),
            "skv_unpack_batch": (ctypes.c_int, [cfgp, P(Request), i32, vp, vp, i32, i32, i32, i32, vp]),
            "skv_upgrade_size": (ctypes.c_int, [cfgp, i32, i32, P(u64)]),
            "skv_group_count": (ctypes.c_int, [cfgp, P(GroupSpec), P(i32)]),
            "skv_plan_groups": (ctypes.c_int, [cfgp, P(GroupSpec), P(Plan)]),
            "skv_grouped_payload_size": (ctypes.c_int, [cfgp, P(GroupSpec), P(u64)]),
            "skv_group_workspace_size": (ctypes.c_int, [cfgp, P(GroupSpec), P(u64)]),
            "skv_prepare_groups": (ctypes.c_int, [cfgp, P(GroupSpec), vp, vp]),
            "skv_score_groups": (ctypes.c_int, [cfgp, P(GroupSpec), vp, vp, vp, vp, vp, vp]),
            "skv_assign_groups": (ctypes.c_int, [cfgp, P(GroupSpec), vp, vp, vp, vp]),
            "skv_pack_groups": (ctypes.c_int, [cfgp, P(GroupSpec), vp, vp, vp, vp, vp, u64, vp, vp]),
            "skv_unpack_groups": (ctypes.c_int, [cfgp, P(GroupSpec), vp, vp, u64, vp, vp, vp, i32, i32, vp, vp]),
            "skv_pack_upgrade": (ctypes.c_int, [cfgp, vp, vp, vp, vp, i32, i32, vp, u64, vp, vp]),
            "skv_unpack_upgrade": (ctypes.c_int, [cfgp, vp, u64, i32, i32, vp, vp, vp, i32, i32, vp, vp]),
            "skv_batch_workspace_size": (ctypes.c_int, [cfgp, P(ScoreRequest), i32, P(u64)]),
            "skv_score_batch": (ctypes.c_int, [cfgp, P(ScoreRequest), i32, vp, vp]),
            "skv_assign_batch": (ctypes.c_int, [cfgp, P(ScoreRequest), i32, vp, vp]),
        }
        for name, (res, args) in sigs.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().skv_status_string(int(status)).decode()


def config(num_layers, num_kv_heads, head_dim, num_tokens, budget, first_ratio=0.02, num_sink=-1,
           decay=0.005, num_tiers=3, score_mode=KVNORM, num_q_heads=0, obs_window=0, quant_int8=0,
           quant_int4=0) -> Config:
    return Config(num_layers, num_kv_heads, head_dim, num_tokens, budget, first_ratio, num_sink,
                  decay, num_tiers, score_mode, num_q_heads, obs_window, quant_int8, quant_int4)


def _check(status: int, what: str):
    if status != OK:
        raise SkvError(status, what)


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: Optional[torch.Tensor], dtype, numel: int, name: str) -> ctypes.c_void_p:
    """Device pointer of a contiguous tensor holding at least `numel` elements of `dtype`."""
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def plan_tiers(cfg: Config) -> dict:
    p = Plan()
    _check(lib().skv_plan_tiers(ctypes.byref(cfg), ctypes.byref(p)), "skv_plan_tiers")
    return {f: getattr(p, f) for f, _ in Plan._fields_}


def payload_size(cfg: Config) -> int:
    out = ctypes.c_uint64()
    _check(lib().skv_payload_size(ctypes.byref(cfg), ctypes.byref(out)), "skv_payload_size")
    return out.value


def workspace_size(cfg: Config) -> int:
    out = ctypes.c_uint64()
    _check(lib().skv_workspace_size(ctypes.byref(cfg), ctypes.byref(out)), "skv_workspace_size")
    return out.value


def _kv_numel(cfg: Config) -> int:
    return cfg.num_layers * cfg.num_kv_heads * cfg.num_tokens * cfg.head_dim


def prepare(cfg: Config, ws: torch.Tensor, stream=None):
    _check(lib().skv_prepare(ctypes.byref(cfg), _dev(ws, torch.uint8, workspace_size(cfg), "ws"),
                             _stream(stream)), "skv_prepare")


def score(cfg: Config, k: torch.Tensor, v: torch.Tensor, q_obs: Optional[torch.Tensor],
          out: torch.Tensor, ws: torch.Tensor, stream=None):
    n = _kv_numel(cfg)
    kp = _dev(k, torch.float16, n, "k")
    vp = _dev(v, torch.float16, n, "v") if cfg.score_mode != ATTN else ctypes.c_void_p(None)
    qp = ctypes.c_void_p(None)
    if cfg.score_mode == ATTN:
        qn = cfg.num_layers * cfg.num_q_heads * cfg.obs_window * cfg.head_dim
        qp = _dev(q_obs, torch.float16, qn, "q_obs")
    _check(lib().skv_score(ctypes.byref(cfg), kp, vp, qp, _dev(out, torch.float64, cfg.num_tokens, "score"),
                           _dev(ws, torch.uint8, workspace_size(cfg), "ws"), _stream(stream)), "skv_score")


def score_static(cfg: Config, k: torch.Tensor, v: torch.Tensor, q_obs: Optional[torch.Tensor],
                 out: torch.Tensor, stream=None):
    """skv_score_static: skv_score with the library's own scratch (no workspace)."""
    n = _kv_numel(cfg)
    kp = _dev(k, torch.float16, n, "k") if cfg.score_mode != RECENCY else ctypes.c_void_p(None)
    vp = _dev(v, torch.float16, n, "v") if cfg.score_mode == KVNORM else ctypes.c_void_p(None)
    qp = ctypes.c_void_p(None)
    if cfg.score_mode == ATTN:
        qn = cfg.num_layers * cfg.num_q_heads * cfg.obs_window * cfg.head_dim
        qp = _dev(q_obs, torch.float16, qn, "q_obs")
    _check(lib().skv_score_static(ctypes.byref(cfg), kp, vp, qp, _dev(out, torch.float64, cfg.num_tokens, "score"),
                                  _stream(stream)), "skv_score_static")


def assign_tiers(cfg: Config, scores: torch.Tensor, tier: torch.Tensor, stream=None,
                 ws: Optional[torch.Tensor] = None):
    """ws: the request's workspace (workspace_size bytes), or None; with it,
    rows past 32768 non-sink tokens are cut by the split form."""
    wsp = ctypes.c_void_p(None) if ws is None else _dev(ws, torch.uint8, workspace_size(cfg), "ws")
    _check(lib().skv_assign_tiers(ctypes.byref(cfg), _dev(scores, torch.float64, cfg.num_tokens, "score"),
                                  _dev(tier, torch.uint8, cfg.num_tokens, "tier"), wsp,
                                  _stream(stream)), "skv_assign_tiers")


def pack(cfg: Config, k: torch.Tensor, v: torch.Tensor, tier: torch.Tensor, payload: torch.Tensor,
         dev_status: Optional[torch.Tensor] = None, stream=None):
    n = _kv_numel(cfg)
    st = ctypes.c_void_p(None) if dev_status is None else _dev(dev_status, torch.int32, 1, "dev_status")
    _check(lib().skv_pack(ctypes.byref(cfg), _dev(k, torch.float16, n, "k"), _dev(v, torch.float16, n, "v"),
                          _dev(tier, torch.uint8, cfg.num_tokens, "tier"),
                          _dev(payload, torch.uint8, 0, "payload"), payload.numel(), st,
                          _stream(stream)), "skv_pack")


def unpack(cfg: Config, payload: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
           block_table: torch.Tensor, block_size: int, dev_status: torch.Tensor, stream=None):
    """k_cache/v_cache: float16 [L][num_blocks][block_size][H][d]."""
    if k_cache.dim() != 5 or k_cache.shape[2] != block_size or tuple(k_cache.shape) != tuple(v_cache.shape):
        raise ValueError("caches must be [L][num_blocks][block_size][H][d] and alike")
    L, nb, _, H, d = k_cache.shape
    if (L, H, d) != (cfg.num_layers, cfg.num_kv_heads, cfg.head_dim):
        raise ValueError("cache shape does not match the configuration")
    nbt = -(-cfg.num_tokens // block_size)
    _check(lib().skv_unpack(ctypes.byref(cfg), _dev(payload, torch.uint8, 0, "payload"), payload.numel(),
                            _dev(k_cache, torch.float16, k_cache.numel(), "k_cache"),
                            _dev(v_cache, torch.float16, v_cache.numel(), "v_cache"),
                            _dev(block_table, torch.int32, nbt, "block_table"), nb, block_size,
                            _dev(dev_status, torch.int32, 1, "dev_status"), _stream(stream)), "skv_unpack")


def upgrade_size(cfg: Config, m: int, mode: int) -> int:
    out = ctypes.c_uint64()
    _check(lib().skv_upgrade_size(ctypes.byref(cfg), m, mode, ctypes.byref(out)), "skv_upgrade_size")
    return out.value


def pack_upgrade(cfg: Config, k: torch.Tensor, v: torch.Tensor, tier: torch.Tensor, tokens: torch.Tensor,
                 mode: int, out: torch.Tensor, dev_status: Optional[torch.Tensor] = None, stream=None):
    """Upgrade payload for the listed tokens (int32, strictly ascending)."""
    n = _kv_numel(cfg)
    m = tokens.numel()
    st = ctypes.c_void_p(None) if dev_status is None else _dev(dev_status, torch.int32, 1, "dev_status")
    _check(lib().skv_pack_upgrade(ctypes.byref(cfg), _dev(k, torch.float16, n, "k"), _dev(v, torch.float16, n, "v"),
                                  _dev(tier, torch.uint8, cfg.num_tokens, "tier"),
                                  _dev(tokens, torch.int32, m, "tokens"), m, mode,
                                  _dev(out, torch.uint8, 0, "out"), out.numel(), st, _stream(stream)),
           "skv_pack_upgrade")


def unpack_upgrade(cfg: Config, upgrade: torch.Tensor, m: int, mode: int, k_cache: torch.Tensor,
                   v_cache: torch.Tensor, block_table: torch.Tensor, block_size: int, dev_status: torch.Tensor,
                   stream=None):
    """Applies an upgrade payload in place to caches filled by unpack."""
    if k_cache.dim() != 5 or k_cache.shape[2] != block_size or tuple(k_cache.shape) != tuple(v_cache.shape):
        raise ValueError("caches must be [L][num_blocks][block_size][H][d] and alike")
    L, nb, _, H, d = k_cache.shape
    if (L, H, d) != (cfg.num_layers, cfg.num_kv_heads, cfg.head_dim):
        raise ValueError("cache shape does not match the configuration")
    nbt = -(-cfg.num_tokens // block_size)
    _check(lib().skv_unpack_upgrade(ctypes.byref(cfg), _dev(upgrade, torch.uint8, 0, "upgrade"), upgrade.numel(),
                                    m, mode, _dev(k_cache, torch.float16, k_cache.numel(), "k_cache"),
                                    _dev(v_cache, torch.float16, v_cache.numel(), "v_cache"),
                                    _dev(block_table, torch.int32, nbt, "block_table"), nb, block_size,
                                    _dev(dev_status, torch.int32, 1, "dev_status"), _stream(stream)),
           "skv_unpack_upgrade")


class Groups:
    """A granularity and optional per-group budgets (host float32 array of G
    entries in (0, 1]) for the grouped calls; keeps the budget array alive."""

    def __init__(self, granularity: int, budgets=None):
        import numpy as np

        self.budgets = None if budgets is None else np.ascontiguousarray(budgets, np.float32)
        ptr = None if self.budgets is None else self.budgets.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        self.spec = GroupSpec(granularity, 0, ptr)

    @property
    def ref(self):
        return ctypes.byref(self.spec)


def group_count(cfg: Config, groups: Groups) -> int:
    out = ctypes.c_int32()
    _check(lib().skv_group_count(ctypes.byref(cfg), groups.ref, ctypes.byref(out)), "skv_group_count")
    return out.value


def plan_groups(cfg: Config, groups: Groups) -> list:
    G = group_count(cfg, groups)
    plans = (Plan * G)()
    _check(lib().skv_plan_groups(ctypes.byref(cfg), groups.ref, plans), "skv_plan_groups")
    return [{f: getattr(p, f) for f, _ in Plan._fields_} for p in plans]


def grouped_payload_size(cfg: Config, groups: Groups) -> int:
    out = ctypes.c_uint64()
    _check(lib().skv_grouped_payload_size(ctypes.byref(cfg), groups.ref, ctypes.byref(out)),
           "skv_grouped_payload_size")
    return out.value


def group_workspace_size(cfg: Config, groups: Groups) -> int:
    out = ctypes.c_uint64()
    _check(lib().skv_group_workspace_size(ctypes.byref(cfg), groups.ref, ctypes.byref(out)),
           "skv_group_workspace_size")
    return out.value


def prepare_groups(cfg: Config, groups: Groups, ws: torch.Tensor, stream=None):
    _check(lib().skv_prepare_groups(ctypes.byref(cfg), groups.ref,
                                    _dev(ws, torch.uint8, group_workspace_size(cfg, groups), "ws"),
                                    _stream(stream)), "skv_prepare_groups")


def score_groups(cfg: Config, groups: Groups, k: torch.Tensor, v: Optional[torch.Tensor],
                 q_obs: Optional[torch.Tensor], out: torch.Tensor, ws: torch.Tensor, stream=None):
    n = _kv_numel(cfg)
    G = group_count(cfg, groups)
    kp = _dev(k, torch.float16, n, "k")
    vp = _dev(v, torch.float16, n, "v") if cfg.score_mode != ATTN else ctypes.c_void_p(None)
    qp = ctypes.c_void_p(None)
    if cfg.score_mode == ATTN:
        qp = _dev(q_obs, torch.float16, cfg.num_layers * cfg.num_q_heads * cfg.obs_window * cfg.head_dim, "q_obs")
    _check(lib().skv_score_groups(ctypes.byref(cfg), groups.ref, kp, vp, qp,
                                  _dev(out, torch.float64, G * cfg.num_tokens, "score"),
                                  _dev(ws, torch.uint8, group_workspace_size(cfg, groups), "ws"), _stream(stream)),
           "skv_score_groups")


def assign_groups(cfg: Config, groups: Groups, scores: torch.Tensor, tier: torch.Tensor, ws: torch.Tensor,
                  stream=None):
    G = group_count(cfg, groups)
    _check(lib().skv_assign_groups(ctypes.byref(cfg), groups.ref,
                                   _dev(scores, torch.float64, G * cfg.num_tokens, "score"),
                                   _dev(tier, torch.uint8, G * cfg.num_tokens, "tier"),
                                   _dev(ws, torch.uint8, group_workspace_size(cfg, groups), "ws"),
                                   _stream(stream)), "skv_assign_groups")


def pack_groups(cfg: Config, groups: Groups, k: torch.Tensor, v: torch.Tensor, tier: torch.Tensor,
                ws: torch.Tensor, payload: torch.Tensor, dev_status: Optional[torch.Tensor] = None, stream=None):
    n = _kv_numel(cfg)
    G = group_count(cfg, groups)
    st = ctypes.c_void_p(None) if dev_status is None else _dev(dev_status, torch.int32, 1, "dev_status")
    _check(lib().skv_pack_groups(ctypes.byref(cfg), groups.ref, _dev(k, torch.float16, n, "k"),
                                 _dev(v, torch.float16, n, "v"), _dev(tier, torch.uint8, G * cfg.num_tokens, "tier"),
                                 _dev(ws, torch.uint8, group_workspace_size(cfg, groups), "ws"),
                                 _dev(payload, torch.uint8, 0, "payload"), payload.numel(), st, _stream(stream)),
           "skv_pack_groups")


def unpack_groups(cfg: Config, groups: Groups, ws: torch.Tensor, payload: torch.Tensor, k_cache: torch.Tensor,
                  v_cache: torch.Tensor, block_table: torch.Tensor, block_size: int, dev_status: torch.Tensor,
                  stream=None):
    if k_cache.dim() != 5 or k_cache.shape[2] != block_size or tuple(k_cache.shape) != tuple(v_cache.shape):
        raise ValueError("caches must be [L][num_blocks][block_size][H][d] and alike")
    L, nb, _, H, d = k_cache.shape
    if (L, H, d) != (cfg.num_layers, cfg.num_kv_heads, cfg.head_dim):
        raise ValueError("cache shape does not match the configuration")
    nbt = -(-cfg.num_tokens // block_size)
    _check(lib().skv_unpack_groups(ctypes.byref(cfg), groups.ref,
                                   _dev(ws, torch.uint8, group_workspace_size(cfg, groups), "ws"),
                                   _dev(payload, torch.uint8, 0, "payload"), payload.numel(),
                                   _dev(k_cache, torch.float16, k_cache.numel(), "k_cache"),
                                   _dev(v_cache, torch.float16, v_cache.numel(), "v_cache"),
                                   _dev(block_table, torch.int32, nbt, "block_table"), nb, block_size,
                                   _dev(dev_status, torch.int32, 1, "dev_status"), _stream(stream)),
           "skv_unpack_groups")


def _with_tokens(cfg: Config, n: int) -> Config:
    c = Config.from_buffer_copy(cfg)
    c.num_tokens = n
    return c


def pack_batch(cfg: Config, ks, vs, tiers, payloads, statuses=None, layer_begin=0, layer_count=None,
               stream=None):
    """Packs len(ks) requests (n taken from each tier map's length) in batched launches."""
    count = len(ks)
    reqs = (Request * count)()
    for i in range(count):
        n = tiers[i].numel()
        c = _with_tokens(cfg, n)
        kv_n = _kv_numel(c)
        reqs[i].num_tokens = n
        reqs[i].k = _dev(ks[i], torch.float16, kv_n, "k").value
        reqs[i].v = _dev(vs[i], torch.float16, kv_n, "v").value
        reqs[i].tier = _dev(tiers[i], torch.uint8, n, "tier").value
        reqs[i].payload = _dev(payloads[i], torch.uint8, 0, "payload").value
        reqs[i].payload_bytes = payloads[i].numel()
        if statuses is not None:
            reqs[i].dev_status = _dev(statuses[i], torch.int32, 1, "dev_status").value
    lc = cfg.num_layers - layer_begin if layer_count is None else layer_count
    _check(lib().skv_pack_batch(ctypes.byref(cfg), reqs, count, layer_begin, lc, _stream(stream)),
           "skv_pack_batch")


def _score_requests(cfg: Config, scores, ks=None, vs=None, tiers=None):
    count = len(scores)
    reqs = (ScoreRequest * count)()
    for i in range(count):
        n = scores[i].numel()
        reqs[i].num_tokens = n
        reqs[i].score = _dev(scores[i], torch.float64, n, "score").value
        if ks is not None and cfg.score_mode == KVNORM:
            kv_n = _kv_numel(_with_tokens(cfg, n))
            reqs[i].k = _dev(ks[i], torch.float16, kv_n, "k").value
            reqs[i].v = _dev(vs[i], torch.float16, kv_n, "v").value
        if tiers is not None:
            reqs[i].tier = _dev(tiers[i], torch.uint8, n, "tier").value
    return reqs, count


def batch_workspace_size(cfg: Config, scores) -> int:
    """Workspace bytes of score_batch and assign_batch for requests of these
    lengths (cfg.num_tokens >= every n)."""
    count = len(scores)
    reqs = (ScoreRequest * count)()
    for i in range(count):
        reqs[i].num_tokens = scores[i].numel()
        reqs[i].score = 256  # sizes only: the pointers are not dereferenced
        reqs[i].k = reqs[i].v = 256
    out = ctypes.c_uint64()
    _check(lib().skv_batch_workspace_size(ctypes.byref(cfg), reqs, count, ctypes.byref(out)),
           "skv_batch_workspace_size")
    return out.value


def score_batch(cfg: Config, ks, vs, scores, ws: torch.Tensor, stream=None):
    """Scores len(scores) requests (n = each score buffer's length) in batched
    launches; ws prepared by prepare(cfg, ws) with cfg.num_tokens >= every n."""
    reqs, count = _score_requests(cfg, scores, ks, vs)
    _check(lib().skv_score_batch(ctypes.byref(cfg), reqs, count,
                                 _dev(ws, torch.uint8, batch_workspace_size(cfg, scores), "ws"), _stream(stream)),
           "skv_score_batch")


def assign_batch(cfg: Config, scores, tiers, stream=None, ws=None):
    """Assigns the tiers of len(scores) requests: one workgroup per request of
    at most 32768 non-sink tokens; longer requests split over the GPU when ws
    (batch_workspace_size bytes) is given, else one workgroup each."""
    reqs, count = _score_requests(cfg, scores, tiers=tiers)
    w = ctypes.c_void_p(None) if ws is None else _dev(ws, torch.uint8, batch_workspace_size(cfg, scores), "ws")
    _check(lib().skv_assign_batch(ctypes.byref(cfg), reqs, count, w, _stream(stream)), "skv_assign_batch")


def unpack_batch(cfg: Config, payloads, token_counts, block_tables, k_cache: torch.Tensor,
                 v_cache: torch.Tensor, block_size: int, statuses, layer_begin=0, layer_count=None,
                 stream=None):
    """Unpacks len(payloads) requests into one shared paged cache in batched launches."""
    if k_cache.dim() != 5 or k_cache.shape[2] != block_size or tuple(k_cache.shape) != tuple(v_cache.shape):
        raise ValueError("caches must be [L][num_blocks][block_size][H][d] and alike")
    L, nb, _, H, d = k_cache.shape
    if (L, H, d) != (cfg.num_layers, cfg.num_kv_heads, cfg.head_dim):
        raise ValueError("cache shape does not match the configuration")
    count = len(payloads)
    reqs = (Request * count)()
    for i in range(count):
        n = int(token_counts[i])
        reqs[i].num_tokens = n
        reqs[i].payload = _dev(payloads[i], torch.uint8, 0, "payload").value
        reqs[i].payload_bytes = payloads[i].numel()
        reqs[i].block_table = _dev(block_tables[i], torch.int32, -(-n // block_size), "block_table").value
        reqs[i].dev_status = _dev(statuses[i], torch.int32, 1, "dev_status").value
    lc = cfg.num_layers - layer_begin if layer_count is None else layer_count
    _check(lib().skv_unpack_batch(ctypes.byref(cfg), reqs, count,
                                  _dev(k_cache, torch.float16, k_cache.numel(), "k_cache"),
                                  _dev(v_cache, torch.float16, v_cache.numel(), "v_cache"), nb, block_size,
                                  layer_begin, lc, _stream(stream)), "skv_unpack_batch")


def link(dst: torch.Tensor, src: torch.Tensor, nbytes: int, host_staging: Optional[torch.Tensor] = None,
         stream=None):
    """Emulated transfer of nbytes (device to device, or through pinned host memory)."""
    if dst.numel() * dst.element_size() < nbytes or src.numel() * src.element_size() < nbytes:
        raise ValueError("link buffers smaller than nbytes")
    hs = ctypes.c_void_p(None)
    if host_staging is not None:
        if host_staging.is_cuda or not host_staging.is_pinned() or host_staging.numel() * host_staging.element_size() < nbytes:
            raise ValueError("host_staging must be pinned host memory of at least nbytes")
        hs = ctypes.c_void_p(host_staging.data_ptr())
    _check(lib().skv_link(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), nbytes, hs,
                          _stream(stream)), "skv_link")


class Codec:
    """Device buffers for one request shape: workspace (prepared), scores,
    tier map, payload and status words, plus the encode/decode sequence."""

    def __init__(self, cfg: Config, device="cuda"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.plan = plan_tiers(cfg)
        self.payload_bytes = payload_size(cfg)
        self.ws = torch.empty(workspace_size(cfg), dtype=torch.uint8, device=self.device)
        self.scores = torch.empty(cfg.num_tokens, dtype=torch.float64, device=self.device)
        self.tier = torch.empty(cfg.num_tokens, dtype=torch.uint8, device=self.device)
        self.payload = torch.empty(self.payload_bytes, dtype=torch.uint8, device=self.device)
        self.status = torch.zeros(2, dtype=torch.int32, device=self.device)
        prepare(cfg, self.ws)

    def encode(self, k, v, q_obs=None, stream=None):
        score(self.cfg, k, v, q_obs, self.scores, self.ws, stream)
        assign_tiers(self.cfg, self.scores, self.tier, stream, ws=self.ws)
        pack(self.cfg, k, v, self.tier, self.payload, self.status[0:1], stream)
        return self.payload

    def decode(self, payload, k_cache, v_cache, block_table, block_size=16, stream=None):
        unpack(self.cfg, payload, k_cache, v_cache, block_table, block_size, self.status[1:2], stream)
