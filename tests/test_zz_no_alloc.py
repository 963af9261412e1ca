"""skv_score_static, the scoring call that allocates nothing, against skv_score.

Both run the same kernels, so the scores must agree bit for bit in every mode
(KV-norm and recency are exact; attention mode is deterministic).  Each case
calls the static entry point several times in a row on one device, the later
calls smaller, and with decay rates that force the resident decay table to be
reused, extended and rewritten; every call is compared with skv_score on a
freshly prepared workspace.
"""
import ctypes

import pytest
import torch

from paper_2606_08635_amd import skv, workloads


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _ws_scores(cfg, k, v, q):
    dev = torch.device("cuda:0")
    ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device=dev)
    skv.prepare(cfg, ws)
    out = torch.full((cfg.num_tokens,), float("nan"), dtype=torch.float64, device=dev)
    skv.score(cfg, k, v, q, out, ws)
    return out


def _static_scores(cfg, k, v, q):
    out = torch.full((cfg.num_tokens,), float("nan"), dtype=torch.float64, device=torch.device("cuda:0"))
    skv.score_static(cfg, k, v, q, out)
    return out


def _check(cfg, k, v, q, what):
    say(f"skv_score_static {what}: L={cfg.num_layers} H={cfg.num_kv_heads} d={cfg.head_dim} "
        f"n={cfg.num_tokens} mode={cfg.score_mode} decay={cfg.decay}")
    assert skv.workspace_size(cfg) <= skv.STATIC_SCRATCH_BYTES
    got = _static_scores(cfg, k, v, q)
    want = _ws_scores(cfg, k, v, q)
    torch.cuda.synchronize()
    g, w = got.cpu().view(torch.int64), want.cpu().view(torch.int64)
    bad = (g != w).nonzero().flatten()
    assert bad.numel() == 0, f"{what}: {bad.numel()} scores differ, first at token {int(bad[0])}"


def _kv(L, H, d, n, seed):
    return workloads.make_kv(L, H, n, d, seed=seed, device=torch.device("cuda:0"))


@pytest.mark.gpu
def test_static_kvnorm_headline_then_smaller():
    torch.cuda.set_device(0)
    # the full 32-layer x 8-head x 128-dim x 32768-token request, as the benchmark scores it
    w = workloads.WORKLOADS["mistral7b_32k"]
    cfg = skv.config(w.layers, w.kv_heads, w.head_dim, w.tokens, w.budget, decay=w.decay)
    k, v = _kv(w.layers, w.kv_heads, w.head_dim, w.tokens, 0)
    _check(cfg, k, v, None, "headline")
    del k, v
    # smaller, same decay rate: the resident table is reused, the scratch overwritten
    cfg = skv.config(2, 2, 64, 3001, 0.5, decay=w.decay)
    k, v = _kv(2, 2, 64, 3001, 7)
    _check(cfg, k, v, None, "smaller, same rate")
    # longer than the table the last call left resident: the table is extended
    cfg = skv.config(3, 4, 256, 5000, 0.5, decay=w.decay)
    k, v = _kv(3, 4, 256, 5000, 8)
    _check(cfg, k, v, None, "longer, same rate")
    # another rate: the table is rewritten
    cfg = skv.config(1, 1, 32, 777, 0.5, decay=0.01)
    k, v = _kv(1, 1, 32, 777, 9)
    _check(cfg, k, v, None, "new rate")


@pytest.mark.gpu
def test_static_attention_then_smaller():
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    L, H, Hq, W, d, n = 1, 8, 32, 32, 128, 32768
    cfg = skv.config(L, H, d, n, 0.5, decay=0.005, score_mode=skv.ATTN, num_q_heads=Hq, obs_window=W)
    k, v = _kv(L, H, d, n, 0)
    q = workloads.make_qobs(L, Hq, W, d, seed=0, device=dev)
    _check(cfg, k, None, q, "attention, 32 query heads")
    L, H, Hq, W, d, n = 2, 2, 4, 16, 64, 1000
    cfg = skv.config(L, H, d, n, 0.5, decay=0.002, score_mode=skv.ATTN, num_q_heads=Hq, obs_window=W)
    k, v = _kv(L, H, d, n, 3)
    q = workloads.make_qobs(L, Hq, W, d, seed=3, device=dev)
    _check(cfg, k, None, q, "attention, smaller")


@pytest.mark.gpu
def test_static_recency_then_smaller():
    torch.cuda.set_device(0)
    for n, decay in ((20000, 0.003), (100, 0.003), (4099, 0.0)):
        cfg = skv.config(1, 1, 32, n, 0.5, decay=decay, score_mode=skv.RECENCY)
        k, v = _kv(1, 1, 32, n, 1)  # not read in recency mode
        _check(cfg, k, v, None, f"recency n={n}")


def test_static_rejects_oversized_request_before_any_device_call():
    # 2^21 tokens over 64 layers x 16 heads need two 32 MiB sets of KV-norm
    # partials plus a 16 MiB table: above the static array, refused on the host
    # (pointers are never dereferenced, so placeholder aligned addresses suffice)
    cfg = skv.config(64, 16, 128, 1 << 21, 0.5, decay=1e-4)
    assert skv.workspace_size(cfg) > skv.STATIC_SCRATCH_BYTES
    fake = ctypes.c_void_p(1 << 20)
    st = skv.lib().skv_score_static(ctypes.byref(cfg), fake, fake, None, fake, None)
    assert st == skv.ERR_CAPACITY
    assert "static scratch" in skv.status_string(st)


def test_headline_requests_fit_the_static_array():
    w = workloads.WORKLOADS["mistral7b_32k"]
    for mode, hq, win in ((skv.KVNORM, 0, 0), (skv.ATTN, w.q_heads, 32), (skv.RECENCY, 0, 0)):
        cfg = skv.config(w.layers, w.kv_heads, w.head_dim, w.tokens, w.budget, score_mode=mode,
                         num_q_heads=hq, obs_window=win)
        assert skv.workspace_size(cfg) <= skv.STATIC_SCRATCH_BYTES
