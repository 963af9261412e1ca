"""Seeded synthetic inputs for the KV transfer codec.

This module holds no codec arithmetic: it only draws random K/V caches,
observation queries and block tables with the shapes of the paper's models
(Qwen2.5-7B, Mistral-7B, Gemma-2-9B; Sec. 5) and the value structure stated
below.  Both the GPU path and the CPU oracle are fed from here.

Recipe (every tensor is drawn with ``torch.Generator`` on the requested device):
  * K and V: float32 N(0, 1) rounded to binary16 (round-to-nearest-even),
    layout [L][H][n][d]; K uses ``seed``, V uses ``seed + 1``.
  * Outlier channels: for every (layer, head) and each of K and V, 4 channels
    drawn without replacement (generator ``seed + 3``).  ``outliers="x8"``
    multiplies them by 8; ``outliers="student_t"`` replaces them by
    8 * Student-t(nu=4) samples (generator ``seed + 5``), the heavy-tailed
    variant.
  * Observation queries (attention-mode scoring): N(0, 1) binary16,
    [L][Hq][W][d], generator ``seed + 2``.
  * Block table: a random permutation of the physical blocks (generator
    ``seed + 4``), its first ceil(n / block_size) entries used.
  * Request r of a multi-request batch uses ``seed + 16 r``.
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple

import torch

OUTLIER_CHANNELS = 4
OUTLIER_SCALE = 8.0


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _outlier_channels(L: int, H: int, d: int, g: torch.Generator, device) -> torch.Tensor:
    """[L, H, 4] channel indices, drawn without replacement per (layer, head)."""
    r = torch.rand(L, H, d, generator=g, device=device)
    return torch.argsort(r, dim=-1)[..., :OUTLIER_CHANNELS]


def _student_t(shape, nu: int, g: torch.Generator, device) -> torch.Tensor:
    z = torch.randn(shape, generator=g, device=device)
    chi2 = torch.zeros(shape, device=device)
    for _ in range(nu):
        chi2 += torch.randn(shape, generator=g, device=device) ** 2
    return z / torch.sqrt(chi2 / nu)


def make_kv(L: int, H: int, n: int, d: int, seed: int = 0, outliers: str = "x8",
            device="cpu") -> Tuple[torch.Tensor, torch.Tensor]:
    """K and V caches, binary16 [L][H][n][d], generated one layer at a time."""
    if outliers not in ("x8", "student_t", "none"):
        raise ValueError(outliers)
    out = []
    g_ch = _gen(seed + 3, device)
    g_t = _gen(seed + 5, device)
    for which in range(2):
        g = _gen(seed + which, device)
        t = torch.empty(L, H, n, d, dtype=torch.float16, device=device)
        ch = _outlier_channels(L, H, d, g_ch, device)
        for l in range(L):
            x = torch.randn(H, n, d, generator=g, device=device)
            if outliers != "none":
                idx = ch[l].unsqueeze(1).expand(H, n, OUTLIER_CHANNELS)
                if outliers == "x8":
                    x.scatter_(2, idx, torch.gather(x, 2, idx) * OUTLIER_SCALE)
                else:
                    x.scatter_(2, idx, OUTLIER_SCALE * _student_t((H, n, OUTLIER_CHANNELS), 4, g_t, device))
            t[l] = x.to(torch.float16)
        out.append(t)
    return out[0], out[1]


def make_qobs(L: int, Hq: int, W: int, d: int, seed: int = 0, device="cpu") -> torch.Tensor:
    g = _gen(seed + 2, device)
    return torch.randn(L, Hq, W, d, generator=g, device=device).to(torch.float16)


def make_block_table(n: int, block_size: int = 16, num_blocks: Optional[int] = None,
                     seed: int = 0, device="cpu") -> torch.Tensor:
    need = (n + block_size - 1) // block_size
    num_blocks = need if num_blocks is None else num_blocks
    if num_blocks < need:
        raise ValueError("num_blocks too small for the request")
    g = _gen(seed + 4, "cpu")
    perm = torch.randperm(num_blocks, generator=g)[:need].to(torch.int32)
    return perm.to(device)


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: a model's KV-cache shape plus codec settings."""
    name: str
    layers: int
    kv_heads: int
    head_dim: int
    tokens: int
    budget: float
    num_tiers: int
    q_heads: int
    outliers: str = "x8"
    first_ratio: float = 0.02
    decay: float = 0.005
    obs_window: int = 0
    batch_tokens: Tuple[int, ...] = field(default_factory=tuple)

    @property
    def fp16_bytes(self) -> int:
        """Full-precision K+V bytes, 2 * L * H * d * n * 2 (Sec. 2.1, eq. "fullbytes")."""
        return 4 * self.layers * self.kv_heads * self.head_dim * self.tokens


# Shapes of the paper's models (Sec. 5) and the stress case; budgets and tier
# policies as evaluated in the paper (Sec. 6.2, Sec. 7.4.3).
WORKLOADS = {
    "tiny": Workload("tiny", 1, 2, 64, 512, 0.5, 3, 4, obs_window=32),
    "qwen7b_b0.3": Workload("qwen7b_b0.3", 28, 4, 128, 4096, 0.3, 2, 28),
    "qwen7b_b0.5": Workload("qwen7b_b0.5", 28, 4, 128, 4096, 0.5, 2, 28),
    "mistral7b_8k": Workload("mistral7b_8k", 32, 8, 128, 8192, 0.5, 3, 32, outliers="student_t"),
    "gemma9b_b0.3": Workload("gemma9b_b0.3", 42, 8, 256, 8192, 0.3, 3, 16),
    "gemma9b_b0.5": Workload("gemma9b_b0.5", 42, 8, 256, 8192, 0.5, 3, 16),
    "gemma9b_b0.7": Workload("gemma9b_b0.7", 42, 8, 256, 8192, 0.7, 3, 16),
    "mistral7b_32k": Workload("mistral7b_32k", 32, 8, 128, 32768, 0.5, 3, 32),
    "long_batch": Workload("long_batch", 32, 8, 128, 32768, 0.5, 3, 32,
                           batch_tokens=(32768, 24581, 16395, 8189)),
    # many short prompts of one model: the case batching is for
    "short_batch": Workload("short_batch", 32, 8, 128, 2048, 0.5, 3, 32, batch_tokens=(2048,) * 64),
}


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def blocks_for(n: int, block_size: int = 16) -> int:
    return ceil_div(n, block_size)


__all__ = ["make_kv", "make_qobs", "make_block_table", "Workload", "WORKLOADS", "blocks_for",
           "ceil_div"]
