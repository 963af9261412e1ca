"""Shared helpers for the GPU parity tests: run each codec stage through the
C ABI and the same stage in the CPU oracle on identical inputs."""
import numpy as np
import torch

import oracle
from paper_2606_08635_amd import skv, workloads


def say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def configs(L, H, d, n, b, tiers=3, rho=0.02, num_sink=-1, decay=0.005, mode=oracle.KVNORM, Hq=0, W=0, q8=0, q4=0):
    kw = dict(first_ratio=rho, num_sink=num_sink, decay=decay, num_tiers=tiers, score_mode=mode,
              num_q_heads=Hq, obs_window=W, quant_int8=q8, quant_int4=q4)
    return skv.config(L, H, d, n, b, **kw), oracle.config(L, H, d, n, b, **kw)


def gpu_encode(cfg, k, v, q=None, scores=None, tier=None):
    """Runs score -> assign -> pack on the GPU; optional overrides feed the
    oracle's scores or tier map into the later stages instead."""
    codec = skv.Codec(cfg, k.device)
    skv.score(cfg, k, v, q, codec.scores, codec.ws)
    if scores is not None:
        codec.scores.copy_(torch.from_numpy(scores).to(k.device))
    skv.assign_tiers(cfg, codec.scores, codec.tier, ws=codec.ws)
    if tier is not None:
        codec.tier.copy_(torch.from_numpy(tier).to(k.device))
    skv.pack(cfg, k, v, codec.tier, codec.payload, codec.status[0:1])
    torch.cuda.synchronize()
    return codec


def caches(L, nb, bs, H, d, device, fill=0xABCD):
    signed = fill - 65536 if fill >= 32768 else fill
    kc = torch.full((L, nb, bs, H, d), signed, dtype=torch.int16, device=device).view(torch.float16)
    return kc, kc.clone()


def gpu_decode(cfg, payload, L, H, d, n, bs, nb, bt, fill=0xABCD):
    kc, vc = caches(L, nb, bs, H, d, payload.device, fill)
    status = torch.full((1,), -1, dtype=torch.int32, device=payload.device)
    skv.unpack(cfg, payload, kc, vc, bt, bs, status)
    torch.cuda.synchronize()
    return kc, vc, int(status.item())


def oracle_decode(ocfg, payload, L, H, d, bs, nb, bt, fill=0xABCD):
    okc = np.full((L, nb, bs, H, d), fill, np.uint16)
    ovc = okc.copy()
    st = oracle.unpack(ocfg, payload, okc, ovc, bt, bs)
    return okc, ovc, st


def bits64(a) -> np.ndarray:
    return np.ascontiguousarray(a, np.float64).view(np.uint64)


def plant_specials(k: torch.Tensor, v: torch.Tensor, seed: int):
    """Puts NaN, infinities, subnormals, signed zeros, extremes and all-zero
    rows into CPU tensors k, v (binary16, [L][H][n][d])."""
    L, H, n, d = k.shape
    rng = np.random.default_rng(seed)
    kb, vb = k.view(torch.int16), v.view(torch.int16)
    specials = [0x7E00, 0x7C00, -1024, 0x0001, -32767, 0x7BFF, -1025, 0x8000 - 65536, 0x03FF]
    # -1024 = 0xFC00 (-inf), -32767 = 0x8001 (tiny negative), -1025 = 0xFBFF (-65504)
    for i in range(max(4, n // 50)):
        l, h, t, c = (int(rng.integers(0, L)), int(rng.integers(0, H)), int(rng.integers(0, n)),
                      int(rng.integers(0, d)))
        (kb if i % 2 else vb)[l, h, t, c] = specials[i % len(specials)]
    for i in range(max(2, n // 100)):
        l, h, t = int(rng.integers(0, L)), int(rng.integers(0, H)), int(rng.integers(0, n))
        (kb if i % 2 else vb)[l, h, t, :] = 0
    t = int(rng.integers(0, n))
    kb[0, 0, t, :] = 0x0001  # a row of the smallest subnormal
    return k, v


def sample_rows(rng, L, H, n, count):
    return [(int(rng.integers(0, L)), int(rng.integers(0, 2)), int(rng.integers(0, H)), int(rng.integers(0, n)))
            for _ in range(count)]


__all__ = ["say", "u16", "configs", "gpu_encode", "gpu_decode", "oracle_decode", "bits64", "plant_specials",
           "caches", "sample_rows", "workloads", "skv", "oracle", "np", "torch"]
