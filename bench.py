"""Benchmark of the KV transfer codec on one MI355X.

One step = the whole hot path on one request: score (KV-norm x decay) ->
assign tiers -> pack -> emulated link (device-to-device copy of the payload)
-> unpack into the paged fp16 cache.  Inputs are resident in HBM before the
timed region.  The reported metric is the paper-shaped codec throughput:
fp16-equivalent bytes F = 4 L H d n per (pack + unpack) second.  Per-stage
times come from HIP events recorded on the stream the library launches on;
before each stage a 1 GiB write evicts the 256 MB Infinity Cache and the L2s,
then a 1 GiB read evicts the write's own dirty lines, so a stage neither reads
what the previous one left in cache nor pays for writing the flush back
(outside the events; --no-flush skips it).  The line also carries the p10/p50/p90 of the
per-step pack + unpack time, the same pack and unpack timed back to back
with no eviction (each paying the previous one's write-backs), a
same-process device copy of F bytes as the
achievable-bandwidth reference, and the oracle's host rate on one thread and
on every host thread (cpu_baseline).

Prints one JSON line (see the keys below); with --gpus N > 1 it exits with a
message, since the codec is measured on one GPU.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "KV codec GB/s (fp16-equivalent in, pack+unpack) and % of HBM peak, 7B-shape 32k"
HBM_PEAK_GBS = 8000.0
CSRC = os.path.join(ROOT, "paper_2606_08635_amd", "csrc")

# HBM bytes per dispatch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs (scaled by
# a plain-copy calibration; see profiles/traffic_*.md), valid only for the
# kernel sources they were taken on: the first 16 hex digits of SHA-256 over
# the kernel's .hip file and every header of the library (source_digest).
MEASURED_TRAFFIC = {
    ("mistral7b_32k", "pack"): (6.5085e9, "pack.hip", "0502305a78d59ddf"),
    ("mistral7b_32k", "unpack"): (6.5127e9, "unpack.hip", "1a37b814f06ffd0e"),
    ("gemma9b_b0.3", "pack"): (3.6863e9, "pack.hip", "0502305a78d59ddf"),
    ("gemma9b_b0.3", "unpack"): (3.6886e9, "unpack.hip", "1a37b814f06ffd0e"),
    ("gemma9b_b0.5", "pack"): (4.2500e9, "pack.hip", "0502305a78d59ddf"),
    ("gemma9b_b0.5", "unpack"): (4.2524e9, "unpack.hip", "1a37b814f06ffd0e"),
    ("gemma9b_b0.7", "pack"): (4.8051e9, "pack.hip", "0502305a78d59ddf"),
    ("gemma9b_b0.7", "unpack"): (4.8079e9, "unpack.hip", "1a37b814f06ffd0e"),
}


def source_digest(kernel_file):
    """Hash of a kernel's source and every header it may include, with
    comments and blank space removed (so that a comment edit does not retire
    the counter figures taken on that code)."""
    import glob
    import hashlib
    import re

    h = hashlib.sha256()
    for path in [os.path.join(CSRC, kernel_file)] + sorted(glob.glob(os.path.join(CSRC, "*.h"))):
        with open(path, encoding="utf-8") as f:
            code = f.read()
        code = re.sub(r"/\*.*?\*/", " ", code, flags=re.S)
        code = re.sub(r"//[^\n]*", " ", code)
        code = " ".join(code.split())
        h.update(os.path.basename(path).encode())
        h.update(code.encode())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    entry = MEASURED_TRAFFIC.get((workload, kernel))
    if entry is None:
        return None
    nbytes, kernel_file, digest = entry
    if source_digest(kernel_file) != digest:
        return None  # the kernel changed since the counters were taken
    return nbytes


def algorithmic_bytes(w, plan, payload_bytes, block_size):
    """Bytes the method must move per launch of pack and of unpack."""
    L, H, d, n = w.layers, w.kv_heads, w.head_dim, w.tokens
    row = 2 * d  # bytes of one fp16 row
    kept = n - plan["n_drop"]
    pack = 2 * L * H * kept * row + n + payload_bytes  # read kept K/V rows + tier map, write payload
    unpack = payload_bytes + 4 * (-(-n // block_size)) + 2 * L * H * n * row  # read payload + table, write cache
    return pack, unpack


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def _host_threads(cap=16):
    """Host cores this process may use, capped at the per-GPU share of the box."""
    try:
        return max(1, min(cap, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(cap, os.cpu_count() or 1))


def cpu_baseline(w, layers: int):
    """The oracle's pack + unpack on the host, as it stands: single-threaded on
    the first `layers` layers of the same request shape, then one oracle call
    per layer on every host thread at once (one layer each; the C oracle runs
    without the GIL).  GB/s of fp16-equivalent input like the metric; `value`
    is the all-thread rate, `cores` the threads it used."""
    import concurrent.futures

    import numpy as np

    import oracle
    from paper_2606_08635_amd import workloads

    n, H, d, bs = w.tokens, w.kv_heads, w.head_dim, 16
    threads = _host_threads()
    nl = max(layers, threads)
    k, v = workloads.make_kv(nl, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    kh, vh = k.cpu().numpy().view(np.uint16), v.cpu().numpy().view(np.uint16)
    del k, v
    kw = dict(first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    ocfg = oracle.config(layers, H, d, n, w.budget, **kw)
    tier = oracle.assign(ocfg, oracle.score(ocfg, kh[:layers], vh[:layers]))
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0).numpy()
    kc = np.zeros((layers, nb, bs, H, d), np.uint16)
    vc = np.zeros_like(kc)
    t0 = time.perf_counter()
    payload = oracle.pack(ocfg, kh[:layers], vh[:layers], tier)
    t1 = time.perf_counter()
    st = oracle.unpack(ocfg, payload, kc, vc, bt, bs)
    t2 = time.perf_counter()
    assert st == oracle.OK
    single = 4 * layers * H * d * n / (t2 - t0) / 1e9
    del payload, kc, vc

    cfg1 = oracle.config(1, H, d, n, w.budget, **kw)

    def one_layer(l):
        kc1 = np.zeros((1, nb, bs, H, d), np.uint16)
        vc1 = np.zeros_like(kc1)
        pay = oracle.pack(cfg1, kh[l:l + 1], vh[l:l + 1], tier)
        return oracle.unpack(cfg1, pay, kc1, vc1, bt, bs)

    with concurrent.futures.ThreadPoolExecutor(threads) as ex:
        t3 = time.perf_counter()
        codes = list(ex.map(one_layer, range(threads)))
        t4 = time.perf_counter()
    assert all(c == oracle.OK for c in codes)
    multi = 4 * threads * H * d * n / (t4 - t3) / 1e9
    return {"value": round(multi, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "single_thread_value": round(single, 4),
            "sample": f"{w.name} request shape ({H} KV heads x {d} dim x {n} tokens per layer) on {_cpu_model()}: "
                      f"{layers} layers on one thread (pack {t1 - t0:.2f} s, unpack {t2 - t1:.2f} s), then "
                      f"{threads} layers, one per thread on {threads} threads ({t4 - t3:.2f} s)"}


def input_digest(k, v, seed):
    """Identifies the seeded synthetic inputs: the generator, its seed and the
    SHA-256 of layer 0 of K and of V as stored (binary16 bytes)."""
    import hashlib

    out = {"generator": "paper_2606_08635_amd.workloads.make_kv", "seed": seed}
    for name, t in (("k", k), ("v", v)):
        out[f"sha256_layer0_{name}"] = hashlib.sha256(t[0].contiguous().cpu().numpy().tobytes()).hexdigest()
    return out


def _events(count):
    import torch
    return [torch.cuda.Event(enable_timing=True) for _ in range(count)]


def run_batch(args, w):
    """Per-request calls vs batched launches (score, assign, pack, unpack) over
    the workload's requests (NEXT-1).  Returns a JSON-able dict."""
    import torch

    from paper_2606_08635_amd import skv, workloads

    L, H, d, bs = w.layers, w.kv_heads, w.head_dim, 16
    lens = list(w.batch_tokens)
    base = skv.config(L, H, d, lens[0], w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    nbs = [workloads.blocks_for(n, bs) for n in lens]
    perm = workloads.make_block_table(sum(nbs) * bs, bs, sum(nbs), seed=0, device="cuda")
    tables, start = [], 0
    for nb in nbs:
        tables.append(perm[start:start + nb].contiguous())
        start += nb
    kc = torch.empty(L, sum(nbs), bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    codecs, ks, vs = [], [], []
    for r, n in enumerate(lens):
        k, v = workloads.make_kv(L, H, n, d, seed=16 * r, outliers=w.outliers, device="cuda")
        c = skv.Codec(skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay,
                                 num_tiers=w.num_tiers))
        c.encode(k, v)
        codecs.append(c)
        ks.append(k)
        vs.append(v)
    torch.cuda.synchronize()
    pays = [c.payload for c in codecs]
    tiers = [c.tier for c in codecs]
    pst = [c.status[0:1] for c in codecs]
    ust = [c.status[1:2] for c in codecs]

    bcfg = skv.config(L, H, d, max(lens), w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    bscores = [torch.empty(n, dtype=torch.float64, device="cuda") for n in lens]
    btiers = [torch.empty(n, dtype=torch.uint8, device="cuda") for n in lens]
    bws = torch.empty(max(skv.batch_workspace_size(bcfg, bscores), skv.workspace_size(bcfg)), dtype=torch.uint8,
                      device="cuda")
    skv.prepare(bcfg, bws)

    def single_score():
        for c, k, v in zip(codecs, ks, vs):
            skv.score(c.cfg, k, v, None, c.scores, c.ws)

    def single_assign():
        for c in codecs:
            skv.assign_tiers(c.cfg, c.scores, c.tier)

    def single():
        for c, k, v in zip(codecs, ks, vs):
            skv.pack(c.cfg, k, v, c.tier, c.payload, c.status[0:1])

    def single_unpack():
        for c, t in zip(codecs, tables):
            skv.unpack(c.cfg, c.payload, kc, vc, t, bs, c.status[1:2])

    def batched_score():
        skv.score_batch(bcfg, ks, vs, bscores, bws)

    def batched_assign():
        skv.assign_batch(bcfg, bscores, btiers, ws=bws)

    def batched():
        skv.pack_batch(base, ks, vs, btiers, pays, pst)

    def batched_unpack():
        skv.unpack_batch(base, pays, lens, tables, kc, vc, bs, ust)

    out = {}
    F = sum(4 * L * H * d * n for n in lens)
    for name, stages in (("per_request", (single_score, single_assign, single, single_unpack)),
                         ("batched", (batched_score, batched_assign, batched, batched_unpack))):
        for _ in range(args.warmup):
            for f in stages:
                f()
        ev = [_events(5) for _ in range(args.steps)]
        for e in ev:
            e[0].record()
            for i, f in enumerate(stages):
                f()
                e[i + 1].record()
        torch.cuda.synchronize()
        t = [sum(e[i].elapsed_time(e[i + 1]) for e in ev) / args.steps for i in range(4)]
        ts, ta, tp, tu = t
        out[name] = {"score_ms": round(ts, 4), "assign_ms": round(ta, 4), "pack_ms": round(tp, 4),
                     "unpack_ms": round(tu, 4), "encode_ms": round(ts + ta + tp, 4),
                     "fp16eq_gbps": round(F / ((tp + tu) / 1e3) / 1e9, 2),
                     "tokens_per_s": round(sum(lens) / ((tp + tu) / 1e3), 1),
                     "encode_tokens_per_s": round(sum(lens) / ((ts + ta + tp) / 1e3), 1),
                     "handoff_tokens_per_s": round(sum(lens) / ((ts + ta + tp + tu) / 1e3), 1)}
        if any(int(c.status[0].item()) != 0 or int(c.status[1].item()) != 0 for c in codecs):
            raise RuntimeError("codec reported a nonzero status")
    # the batched maps and payloads are the per-request ones
    for c, bt in zip(codecs, btiers):
        if not torch.equal(c.tier, bt):
            raise RuntimeError("batched tier map differs from the per-request one")
    return {"requests": len(lens), "tokens": sum(lens), **out}


def run_pipeline(args, w, group):
    """Prefill->decode handoff latency of one request: pack, link and unpack in
    sequence vs layer groups pipelined over three streams (NEXT-1).  With
    --link host the link goes through pinned host memory (PCIe and the copy
    engines), which the pack and unpack of other layer groups can overlap."""
    import torch

    from paper_2606_08635_amd import skv, workloads

    L, H, d, n, bs = w.layers, w.kv_heads, w.head_dim, w.tokens, 16
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    codec = skv.Codec(cfg)
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    codec.encode(k, v)
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    rx = torch.empty_like(codec.payload)
    staging = torch.empty(codec.payload_bytes, dtype=torch.uint8, pin_memory=True) if args.link == "host" else None
    geo = codec.payload[:256].cpu().numpy().view("<u8")
    layers_off, layer_stride = int(geo[12]), int(geo[16])
    torch.cuda.synchronize()
    s_pack, s_link, s_unpack = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    rst = torch.zeros(1, dtype=torch.int32, device="cuda")

    def sequential():
        skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1])
        skv.link(rx, codec.payload, codec.payload_bytes, staging)
        skv.unpack(cfg, rx, kc, vc, bt, bs, codec.status[1:2])

    def pipelined():
        for g0 in range(0, L, group):
            gc = min(group, L - g0)
            with torch.cuda.stream(s_pack):
                skv.pack_batch(cfg, [k], [v], [codec.tier], [codec.payload], [codec.status[0:1]], g0, gc)
                e1 = torch.cuda.Event()
                e1.record()
            lo = 0 if g0 == 0 else layers_off + g0 * layer_stride
            hi = layers_off + (g0 + gc) * layer_stride
            with torch.cuda.stream(s_link):
                s_link.wait_event(e1)
                skv.link(rx[lo:hi], codec.payload[lo:hi], hi - lo, None if staging is None else staging[lo:hi],
                         stream=s_link)
                e2 = torch.cuda.Event()
                e2.record()
            with torch.cuda.stream(s_unpack):
                s_unpack.wait_event(e2)
                skv.unpack_batch(cfg, [rx], [n], [bt], kc, vc, bs, [rst], g0, gc)
        torch.cuda.current_stream().wait_stream(s_unpack)

    out = {"group_layers": group, "link": args.link}
    for name, fn in (("sequential", sequential), ("pipelined", pipelined)):
        for _ in range(args.warmup):
            fn()
            torch.cuda.synchronize()
        times = []
        for _ in range(args.steps):
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            times.append((time.perf_counter() - t0) * 1e3)
        times.sort()
        out[name + "_ms"] = round(times[len(times) // 2], 4)
    if int(rst.item()) != 0 or codec.status.cpu().tolist() != [0, 0]:
        raise RuntimeError("codec reported a nonzero status")
    return out


def run_upgrade(args, w):
    """Cold-tier precision upgrade (NEXT-2) after the workload's codec step:
    an upgrade payload for a token set is packed on the prefill side and
    applied to the decoder's cache, in both modes.  Token sets: the lowest
    tier present (INT4 and DROP tokens; the paper's INT4 -> FP16 case) and
    every quantized or dropped token.  Returns a JSON-able dict."""
    import numpy as np
    import torch

    from paper_2606_08635_amd import skv, workloads

    L, H, d, n, bs = w.layers, w.kv_heads, w.head_dim, w.tokens, 16
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    codec = skv.Codec(cfg)
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    codec.encode(k, v)
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    codec.decode(codec.payload, kc, vc, bt, bs)
    tier = codec.tier.cpu().numpy()
    sets = {"int4_drop": np.flatnonzero(tier >= skv.INT4), "below_fp16": np.flatnonzero(tier != skv.FP16)}
    st = torch.zeros(2, dtype=torch.int32, device="cuda")
    rows_per_token = 2 * L * H
    out = {"workload": w.name, "tokens": n}
    for set_name, toks in sets.items():
        m = int(toks.size)
        if m == 0:
            continue
        tok = torch.from_numpy(toks.astype(np.int32)).cuda()
        res = {"m": m}
        for mode, mname in ((skv.UPGRADE_FP16, "fp16"), (skv.UPGRADE_RESIDUAL8, "residual8")):
            up = torch.empty(skv.upgrade_size(cfg, m, mode), dtype=torch.uint8, device="cuda")
            kw, vw = kc.clone(), vc.clone()  # the decoder's cache, refreshed before every apply
            for _ in range(args.warmup):
                skv.pack_upgrade(cfg, k, v, codec.tier, tok, mode, up, st[0:1])
                skv.unpack_upgrade(cfg, up, m, mode, kw, vw, bt, bs, st[1:2])
            ev = [_events(3) for _ in range(args.steps)]
            for e in ev:
                kw.copy_(kc)
                vw.copy_(vc)
                e[0].record()
                skv.pack_upgrade(cfg, k, v, codec.tier, tok, mode, up, st[0:1])
                e[1].record()
                skv.unpack_upgrade(cfg, up, m, mode, kw, vw, bt, bs, st[1:2])
                e[2].record()
            torch.cuda.synchronize()
            if st.cpu().tolist() != [0, 0]:
                raise RuntimeError(f"upgrade reported status {st.cpu().tolist()}")
            tp = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
            ta = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
            rows = rows_per_token * m
            row_out = 2 * d if mode == skv.UPGRADE_FP16 else d + 4
            pack_b = rows * (2 * d + row_out)          # read fp16 rows, write upgrade rows (+ scales)
            apply_b = rows * (row_out + 2 * d) + (0 if mode == skv.UPGRADE_FP16 else rows * 2 * d)
            res[mname] = {"bytes": up.numel(), "bytes_per_elem": round(up.numel() / (rows * d), 4),
                          "pack_ms": round(tp, 4), "apply_ms": round(ta, 4),
                          "pack_gbps": round(pack_b / (tp / 1e3) / 1e9, 1),
                          "apply_gbps": round(apply_b / (ta / 1e3) / 1e9, 1)}
        out[set_name] = res
    if codec.status.cpu().tolist() != [0, 0]:
        raise RuntimeError("codec reported a nonzero status")
    return out


def run_groups(args, w):
    """Per-layer and per-head tier maps (NEXT-3) on the workload's request:
    score -> assign -> pack -> unpack with one map per layer (budgets falling
    linearly from 0.7 to 0.3, mean 0.5) and with one map per (layer, head) at
    the workload's budget.  Returns a JSON-able dict."""
    import numpy as np
    import torch

    from paper_2606_08635_amd import skv, workloads

    L, H, d, n, bs = w.layers, w.kv_heads, w.head_dim, w.tokens, 16
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers)
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    out = {"workload": w.name}
    for name, gran, budgets in (("per_layer", skv.GROUP_LAYER, np.float32(np.linspace(0.7, 0.3, L))),
                                ("per_head", skv.GROUP_HEAD, None)):
        groups = skv.Groups(gran, budgets)
        G = skv.group_count(cfg, groups)
        ws = torch.empty(skv.group_workspace_size(cfg, groups), dtype=torch.uint8, device="cuda")
        skv.prepare_groups(cfg, groups, ws)
        sc = torch.empty(G * n, dtype=torch.float64, device="cuda")
        tier = torch.empty(G * n, dtype=torch.uint8, device="cuda")
        pay = torch.empty(skv.grouped_payload_size(cfg, groups), dtype=torch.uint8, device="cuda")
        st = torch.zeros(2, dtype=torch.int32, device="cuda")

        def step(ev=None):
            if ev: ev[0].record()
            skv.score_groups(cfg, groups, k, v, None, sc, ws)
            if ev: ev[1].record()
            skv.assign_groups(cfg, groups, sc, tier, ws)
            if ev: ev[2].record()
            skv.pack_groups(cfg, groups, k, v, tier, ws, pay, st[0:1])
            if ev: ev[3].record()
            skv.unpack_groups(cfg, groups, ws, pay, kc, vc, bt, bs, st[1:2])
            if ev: ev[4].record()

        for _ in range(args.warmup):
            step()
        evs = [_events(5) for _ in range(args.steps)]
        for e in evs:
            step(e)
        torch.cuda.synchronize()
        if st.cpu().tolist() != [0, 0]:
            raise RuntimeError(f"grouped codec reported status {st.cpu().tolist()}")
        ms = {nm: sum(e[i].elapsed_time(e[i + 1]) for e in evs) / args.steps
              for i, nm in enumerate(("score", "assign", "pack", "unpack"))}
        t = (ms["pack"] + ms["unpack"]) / 1e3
        out[name] = {"groups": G, "payload_bytes": pay.numel(), "stages_ms": {a: round(b, 4) for a, b in ms.items()},
                     "fp16eq_gbps": round(w.fp16_bytes / t / 1e9, 2)}
    return out


def run_quant(args, w):
    """Per-tier quantizer variants (NEXT-4) on the workload's request: pack
    and unpack times and payload/metadata sizes for a few descriptor pairs
    (INT8 tier, INT4 tier).  Returns a JSON-able dict."""
    import torch

    from paper_2606_08635_amd import skv, workloads

    L, H, d, n, bs = w.layers, w.kv_heads, w.head_dim, w.tokens, 16
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device="cuda")
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device="cuda")
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device="cuda")
    vc = torch.empty_like(kc)
    variants = {
        "row_sym_fp32": (0, 0),
        "row_sym_fp16": (skv.QUANT_FP16, skv.QUANT_FP16),
        "g32_sym_fp16": (skv.QUANT_GROUP32 | skv.QUANT_FP16, skv.QUANT_GROUP32 | skv.QUANT_FP16),
        "int4_g32_asym_fp16": (0, skv.QUANT_GROUP32 | skv.QUANT_ASYM | skv.QUANT_FP16),
        "g64_asym_fp32": (skv.QUANT_GROUP64 | skv.QUANT_ASYM, skv.QUANT_GROUP64 | skv.QUANT_ASYM),
        # KIVI-style: keys per channel over each chunk's rows of the tier, values per row
        "kchan_asym_fp16": (skv.QUANT_CHANNEL | skv.QUANT_ASYM | skv.QUANT_FP16,
                            skv.QUANT_CHANNEL | skv.QUANT_ASYM | skv.QUANT_FP16),
        "kchan_sym_fp32": (skv.QUANT_CHANNEL, skv.QUANT_CHANNEL),
    }
    out = {"workload": w.name}
    for name, (q8, q4) in variants.items():
        cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers,
                         quant_int8=q8, quant_int4=q4)
        codec = skv.Codec(cfg)
        codec.encode(k, v)
        for _ in range(args.warmup):
            skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1])
            skv.unpack(cfg, codec.payload, kc, vc, bt, bs, codec.status[1:2])
        evs = [_events(3) for _ in range(args.steps)]
        for e in evs:
            e[0].record()
            skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1])
            e[1].record()
            skv.unpack(cfg, codec.payload, kc, vc, bt, bs, codec.status[1:2])
            e[2].record()
        torch.cuda.synchronize()
        if codec.status.cpu().tolist() != [0, 0]:
            raise RuntimeError(f"codec reported status {codec.status.cpu().tolist()}")
        tp = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
        tu = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
        hdr = codec.payload[:256].cpu().numpy().view("<u8")  # u64 words: 15 per-row metadata, 21 per-channel area
        out[name] = {"quant_int8": q8, "quant_int4": q4, "payload_bytes": codec.payload_bytes,
                     "metadata_bytes_per_layer": int(hdr[15] + hdr[21]), "pack_ms": round(tp, 4), "unpack_ms": round(tu, 4),
                     "fp16eq_gbps": round(w.fp16_bytes / ((tp + tu) / 1e3) / 1e9, 2)}
        del codec
        torch.cuda.empty_cache()
    return out


def run_select(args):
    """The tier cut alone (skv_assign_tiers / skv_assign_batch) on seeded
    random scores: the resident form at 32768 tokens; past it, the split form
    (workspace given) and the one-workgroup form (no workspace) at 65536 and
    2^21 tokens; 32 per-layer maps of 2^21 tokens (split form); 64
    requests of 2048 tokens per request vs batched; and 8 batched requests of
    2^18 tokens in both forms.  HIP events, mean over the timed launches."""
    import torch

    from paper_2606_08635_amd import skv

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    g = torch.Generator(device=dev)
    g.manual_seed(0)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        ev = _events(2 * args.steps)
        for i in range(args.steps):
            ev[2 * i].record()
            fn()
            ev[2 * i + 1].record()
        torch.cuda.synchronize()
        return sum(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)) / args.steps

    out = {}
    for n in (32768, 65536, 1 << 21):
        cfg = skv.config(32, 8, 128, n, 0.5, decay=1e-4)
        sc = torch.rand(n, generator=g, device=dev, dtype=torch.float64)
        tier = torch.empty(n, dtype=torch.uint8, device=dev)
        ws = torch.empty(skv.workspace_size(cfg), dtype=torch.uint8, device=dev)
        forms = [("single", None)] if n <= 32768 else [("split", ws), ("one_workgroup", None)]
        for name, w in forms:
            ms = timed(lambda: skv.assign_tiers(cfg, sc, tier, ws=w))
            out[f"{name}_n{n}"] = {"ms": round(ms, 4), "tokens_per_s": round(n / (ms / 1e3), 1)}
    # grouped maps past the resident form: 32 per-layer rows of 2^21 tokens,
    # cut together by the split form
    import numpy as np
    n = 1 << 21
    gcfg = skv.config(32, 8, 128, n, 0.5, decay=1e-4)
    groups = skv.Groups(skv.GROUP_LAYER, np.linspace(0.7, 0.3, 32).astype(np.float32))
    gws = torch.empty(skv.group_workspace_size(gcfg, groups), dtype=torch.uint8, device=dev)
    skv.prepare_groups(gcfg, groups, gws)
    gsc = torch.rand(32 * n, generator=g, device=dev, dtype=torch.float64)
    gtier = torch.empty(32 * n, dtype=torch.uint8, device=dev)
    ms = timed(lambda: skv.assign_groups(gcfg, groups, gsc, gtier, gws))
    out["groups_layer_32x2097152_split"] = {"ms": round(ms, 4), "tokens_per_s": round(32 * n / (ms / 1e3), 1)}
    del gws, gsc, gtier
    lens = [2048] * 64
    cfgs = [skv.config(32, 8, 128, n, 0.5) for n in lens]
    bcfg = skv.config(32, 8, 128, max(lens), 0.5)
    scores = [torch.rand(n, generator=g, device=dev, dtype=torch.float64) for n in lens]
    tiers = [torch.empty(n, dtype=torch.uint8, device=dev) for n in lens]

    def per_request():
        for c, s_, t_ in zip(cfgs, scores, tiers):
            skv.assign_tiers(c, s_, t_)

    out["per_request_64x2048"] = {"ms": round(timed(per_request), 4)}
    out["batched_64x2048"] = {"ms": round(timed(lambda: skv.assign_batch(bcfg, scores, tiers)), 4)}
    # eight requests of 2^18 tokens: split form (workspace given) vs one
    # workgroup per request
    lens = [1 << 18] * 8
    lcfg = skv.config(32, 8, 128, max(lens), 0.5, decay=1e-4)
    scores = [torch.rand(n, generator=g, device=dev, dtype=torch.float64) for n in lens]
    tiers = [torch.empty(n, dtype=torch.uint8, device=dev) for n in lens]
    lws = torch.empty(skv.batch_workspace_size(lcfg, scores), dtype=torch.uint8, device=dev)
    for name, w in (("split", lws), ("one_workgroup", None)):
        ms = timed(lambda: skv.assign_batch(lcfg, scores, tiers, ws=w))
        out[f"batched_8x262144_{name}"] = {"ms": round(ms, 4), "tokens_per_s": round(sum(lens) / (ms / 1e3), 1)}
    return out


CEILING_PATTERNS = ["read", "write_nt", "write_default", "copy", "read2_write1", "read1_write2_8b",
                    "read1_write2_16b", "nhd_scatter", "read1_write4", "stage_direct",
                    "stage_regs", "stage_direct_cached",
                    "write_cpol_default", "write_cpol_sc0", "write_cpol_nt", "write_cpol_sc0_nt", "write_cpol_sc1",
                    "write_cpol_sc0_sc1", "write_cpol_nt_sc1", "write_cpol_sc0_nt_sc1"]  # skv_ceiling.h, in enum order


def run_ceiling(args):
    """Streaming reference kernels (libskv_ceiling.so): the HBM rate of plain
    read/write mixes at `--ceiling-gib` GiB and 4, 8 or 16 loads in flight per
    thread (the best of the three is the pattern's reference), each launch
    timed with HIP events on the stream it runs on, back to back (buffers far
    larger than the caches)."""
    import ctypes

    import torch

    path = os.path.join(ROOT, "paper_2606_08635_amd", "libskv_ceiling.so")
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    lib.skv_ceiling_run.restype = ctypes.c_int
    lib.skv_ceiling_run.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
    lib.skv_ceiling_bytes.restype = ctypes.c_uint64
    lib.skv_ceiling_bytes.argtypes = [ctypes.c_int32, ctypes.c_uint64, ctypes.c_int32]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    nbytes = int(args.ceiling_gib * (1 << 30))
    nbytes -= nbytes % (128 << 10)
    src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    sink = torch.zeros(1024, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    out = {}
    for pat, name in enumerate(CEILING_PATTERNS):
        rd, wr = lib.skv_ceiling_bytes(pat, nbytes, 0), lib.skv_ceiling_bytes(pat, nbytes, 1)
        depths = (4,) if name.startswith("write") else (4, 8, 16)
        res = {}
        for depth in depths:
            def launch():
                rc = lib.skv_ceiling_run(pat, depth, ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()),
                                         nbytes, ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
                if rc != 0:
                    raise RuntimeError(f"skv_ceiling_run({name}, {depth}) returned {rc}")
            for _ in range(args.warmup):
                launch()
            ev = _events(2 * args.steps)
            for i in range(args.steps):
                ev[2 * i].record(stream)
                launch()
                ev[2 * i + 1].record(stream)
            torch.cuda.synchronize()
            mean = sum(ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(args.steps)) / args.steps
            res[depth] = {"ms_mean": round(mean, 4), "gbps": round((rd + wr) / (mean / 1e3) / 1e9, 1)}
        best = max(res, key=lambda k: res[k]["gbps"])
        out[name] = {"read_bytes": rd, "write_bytes": wr, "best_gbps": res[best]["gbps"], "best_inflight": best,
                     "by_inflight": res}
        if name.startswith("write"):
            # the write followed by a read of the other buffer (16 in flight),
            # pairs back to back: what the write leaves in the caches is paid
            # for inside the pair
            def pair():
                for p_, b_ in ((pat, 4), (0, 16)):
                    if lib.skv_ceiling_run(p_, b_, ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()),
                                           nbytes, ctypes.c_void_p(sink.data_ptr()),
                                           ctypes.c_void_p(stream.cuda_stream)) != 0:
                        raise RuntimeError(f"skv_ceiling_run({p_}) failed")
            for _ in range(args.warmup):
                pair()
            ev = _events(2 * args.steps)
            for i in range(args.steps):
                ev[2 * i].record(stream)
                pair()
                ev[2 * i + 1].record(stream)
            torch.cuda.synchronize()
            out[name]["then_read_ms"] = round(sum(ev[2 * i].elapsed_time(ev[2 * i + 1])
                                                  for i in range(args.steps)) / args.steps, 4)
        print(f"[ceiling] {name}: {out[name]['best_gbps']} GB/s ({best} in flight)", file=sys.stderr, flush=True)
    return {"bytes": nbytes, "steps": args.steps, "warmup": args.warmup, "patterns": out}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mistral7b_32k")
    ap.add_argument("--cpu-layers", type=int, default=4, help="layers in the CPU-baseline sample (0: skip)")
    ap.add_argument("--link", choices=["d2d", "host"], default="d2d")
    ap.add_argument("--score", choices=["kvnorm", "attn"], default="kvnorm",
                    help="importance statistic; attn uses a W-query observation window per query head")
    ap.add_argument("--obs-window", type=int, default=32)
    ap.add_argument("--no-flush", dest="flush_cache", action="store_false",
                    help="do not evict the caches (1 GiB write, then 1 GiB read) before each stage")
    ap.add_argument("--mode", choices=["step", "batch", "pipeline", "upgrade", "groups", "quant", "ceiling", "select"],
                    default="step",
                    help="step: the headline codec step; batch: per-request vs batched launches over "
                         "a multi-request workload; pipeline: layer-pipelined handoff latency; "
                         "upgrade: cold-tier precision upgrade after the step; "
                         "groups: per-layer and per-head tier maps; quant: per-tier quantizer variants; "
                         "ceiling: streaming reference kernels (achievable HBM rate of the codec's read/write mixes); "
                         "select: the tier cut alone at 32768 and 2^21 tokens and over 64 short requests")
    ap.add_argument("--ceiling-gib", type=float, default=4.0, help="buffer size of --mode ceiling")
    ap.add_argument("--group-layers", type=int, default=4, help="layers per pipeline stage (--mode pipeline)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-sized buffer with the runtime's device copy (reference for byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures the codec on one GPU; --gpus {args.gpus} is not supported "
              "(the codec has no multi-GPU path to time)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_08635_amd import skv, workloads

    if args.calibrate_copy:
        nbytes = args.calibrate_copy << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.warmup + args.steps):
            dst.copy_(src)  # the runtime's device copy: a fixed reference kernel
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": nbytes, "copies": args.warmup + args.steps}), flush=True)
        return

    if args.mode == "ceiling":
        print(json.dumps({"mode": "ceiling", **run_ceiling(args)}), flush=True)
        return
    if args.mode == "select":
        print(json.dumps({"mode": "select", **run_select(args)}), flush=True)
        return
    w = workloads.WORKLOADS[args.workload]
    if args.mode == "batch":
        if not w.batch_tokens:
            w = workloads.WORKLOADS["long_batch"]
        print(json.dumps({"mode": "batch", "workload": w.name, **run_batch(args, w)}), flush=True)
        return
    if args.mode == "pipeline":
        print(json.dumps({"mode": "pipeline", "workload": w.name, **run_pipeline(args, w, args.group_layers)}),
              flush=True)
        return
    if args.mode == "upgrade":
        print(json.dumps({"mode": "upgrade", **run_upgrade(args, w)}), flush=True)
        return
    if args.mode == "groups":
        print(json.dumps({"mode": "groups", **run_groups(args, w)}), flush=True)
        return
    if args.mode == "quant":
        print(json.dumps({"mode": "quant", **run_quant(args, w)}), flush=True)
        return
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    L, H, d, n, bs = w.layers, w.kv_heads, w.head_dim, w.tokens, 16
    attn = args.score == "attn"
    cfg = skv.config(L, H, d, n, w.budget, first_ratio=w.first_ratio, decay=w.decay, num_tiers=w.num_tiers,
                     score_mode=skv.ATTN if attn else skv.KVNORM, num_q_heads=w.q_heads if attn else 0,
                     obs_window=args.obs_window if attn else 0)
    codec = skv.Codec(cfg, dev)
    k, v = workloads.make_kv(L, H, n, d, seed=0, outliers=w.outliers, device=dev)
    q_obs = workloads.make_qobs(L, w.q_heads, args.obs_window, d, seed=0, device=dev) if attn else None
    nb = workloads.blocks_for(n, bs)
    bt = workloads.make_block_table(n, bs, nb, seed=0, device=dev)
    kc = torch.empty(L, nb, bs, H, d, dtype=torch.float16, device=dev)
    vc = torch.empty_like(kc)
    rx = torch.empty_like(codec.payload)
    staging = torch.empty(codec.payload_bytes, dtype=torch.uint8, pin_memory=True) if args.link == "host" else None
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    # Between stages, outside the stage events: a 1 GiB write evicts the 256 MB
    # Infinity Cache and the L2s, so no stage reads what the previous one left
    # there; a 1 GiB read then evicts the write's dirty lines, so no stage pays
    # for writing the flush back.
    flush_buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev) if args.flush_cache else None
    flush_read = torch.ones(1 << 28, dtype=torch.float32, device=dev) if args.flush_cache else None
    names = ["score", "assign", "pack", "link", "unpack"]

    def step(ev=None):
        calls = [lambda: skv.score(cfg, k, v, q_obs, codec.scores, codec.ws),
                 lambda: skv.assign_tiers(cfg, codec.scores, codec.tier, ws=codec.ws),
                 lambda: skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1]),
                 lambda: skv.link(rx, codec.payload, codec.payload_bytes, staging),
                 lambda: skv.unpack(cfg, rx, kc, vc, bt, bs, codec.status[1:2])]
        for i, call in enumerate(calls):
            if flush_buf is not None:
                flush_buf.fill_(i)
                flush_read.sum()
            if ev: ev[2 * i].record(stream)
            call()
            if ev: ev[2 * i + 1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * len(names))] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    status = codec.status.cpu().tolist()
    if status != [0, 0]:
        raise RuntimeError(f"codec reported status {status}")

    per_step = [{nm: e[2 * i].elapsed_time(e[2 * i + 1]) for i, nm in enumerate(names)} for e in events]
    codec_ms = sorted(p["pack"] + p["unpack"] for p in per_step)

    def pct(q):
        return codec_ms[min(len(codec_ms) - 1, int(q * (len(codec_ms) - 1) + 0.5))]

    # achievable-bandwidth reference in the same process: a runtime copy of the
    # F bytes of K and V into the cache buffers (F read + F written)
    ce = _events(2)
    ce[0].record(stream)
    for _ in range(3):
        skv.link(kc, k, k.numel() * 2)
        skv.link(vc, v, v.numel() * 2)
    ce[1].record(stream)
    torch.cuda.synchronize()
    copy_gbs = 3 * 2 * w.fp16_bytes / (ce[0].elapsed_time(ce[1]) / 1e3) / 1e9

    # the same pack and unpack back to back with no eviction between them: each
    # one pays for writing back what the one before left dirty in the caches,
    # so a store policy that defers its write-back past its own end event
    # cannot look faster here than in the evicted steps
    bb = [_events(3) for _ in range(args.steps)]
    for e in bb:
        e[0].record(stream)
        skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1])
        e[1].record(stream)
        skv.unpack(cfg, rx, kc, vc, bt, bs, codec.status[1:2])
        e[2].record(stream)
    torch.cuda.synchronize()
    if codec.status.cpu().tolist() != [0, 0]:
        raise RuntimeError(f"codec reported status {codec.status.cpu().tolist()}")
    bb_pack = sum(e[0].elapsed_time(e[1]) for e in bb) / args.steps
    bb_unpack = sum(e[1].elapsed_time(e[2]) for e in bb) / args.steps

    stage_ms = {nm: sum(p[nm] for p in per_step) / args.steps for nm in names}
    F = w.fp16_bytes
    t_codec = (stage_ms["pack"] + stage_ms["unpack"]) / 1e3
    pack_b, unpack_b = algorithmic_bytes(w, codec.plan, codec.payload_bytes, bs)
    pack_gbs = pack_b / (stage_ms["pack"] / 1e3) / 1e9
    unpack_gbs = unpack_b / (stage_ms["unpack"] / 1e3) / 1e9
    dominant = "pack" if stage_ms["pack"] >= stage_ms["unpack"] else "unpack"
    dom_bytes, dom_gbs = (pack_b, pack_gbs) if dominant == "pack" else (unpack_b, unpack_gbs)
    alg_gbs = (pack_b + unpack_b) / t_codec / 1e9
    out = {
        "metric": METRIC,
        "value": round(F / t_codec / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "layers": L, "kv_heads": H, "head_dim": d, "tokens": n,
                   "budget": w.budget, "num_tiers": w.num_tiers, "first_ratio": w.first_ratio, "decay": w.decay,
                   "score": args.score, "block_size": bs, "link": args.link, "fp16_bytes": F,
                   "payload_bytes": codec.payload_bytes},
        "inputs": input_digest(k, v, seed=0),
        "tokens_per_s": round(n / t_codec, 1),
        "alg_gbps": round(alg_gbs, 2),
        "pct_hbm_peak": round(100 * alg_gbs / HBM_PEAK_GBS, 2),
        "stages_ms": {kk: round(vv, 4) for kk, vv in stage_ms.items()},
        "codec_ms": {"mean": round(t_codec * 1e3, 4), "p10": round(pct(0.1), 4), "p50": round(pct(0.5), 4),
                     "p90": round(pct(0.9), 4)},
        "hot_path_ms_per_step": round(sum(stage_ms.values()), 4),
        "cache_flushed": bool(args.flush_cache),
        "copy_ref_gbps": round(copy_gbs, 2),
        "back_to_back_ms": {"pack": round(bb_pack, 4), "unpack": round(bb_unpack, 4),
                            "fp16eq_gbps": round(w.fp16_bytes / ((bb_pack + bb_unpack) / 1e3) / 1e9, 2)},
        "pack_gbps": round(pack_gbs, 2),
        "unpack_gbps": round(unpack_gbs, 2),
        "roofline": {"bound": "hbm", "kernel": f"skv_{dominant}", "achieved": round(dom_gbs, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dom_gbs / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(w.name, dominant), "bytes_per_launch": dom_bytes},
    }
    if attn:
        # two passes of Q.K^T over the observation rows: 2 * 2 * L * H * M * n * d flops, K read twice
        rows = (w.q_heads // H) * args.obs_window
        flops = 4.0 * L * H * rows * n * d
        out["config"]["obs_window"] = args.obs_window
        out["score_attn"] = {"ms": round(stage_ms["score"], 4), "tflops": round(flops / (stage_ms["score"] / 1e3) / 1e12, 2),
                             "mfma_peak_tflops": 2500.0, "k_read_gbps": round(F / (stage_ms["score"] / 1e3) / 1e9, 2)}
    else:
        out["score_kvnorm"] = {"ms": round(stage_ms["score"], 4),
                               "read_gbps": round(F / (stage_ms["score"] / 1e3) / 1e9, 2)}
    if args.cpu_layers > 0:
        del kc, vc, rx, flush_buf, flush_read
        torch.cuda.empty_cache()
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_layers)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
