"""Pins for the oracle's attention-mode score: A_j is the mean softmax mass a
token receives from the observation queries of every layer and query head
(Sec. 3: aggregated over layers, heads and decode observations; Sec. 4.3:
I_j = A_j exp(-lambda Delta_j)).
"""
import numpy as np
import pytest
from scipy.special import softmax

import oracle


def _cfg(L, H, Hq, W, n, d, lam=0.0):
    return oracle.config(L, H, d, n, 0.5, decay=lam, score_mode=oracle.ATTN, num_q_heads=Hq, obs_window=W)


def _inputs(L, H, Hq, W, n, d, seed):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((L, H, n, d)).astype(np.float16)
    q = rng.standard_normal((L, Hq, W, d)).astype(np.float16)
    return k, q


def test_masses_sum_to_one_and_match_scipy():
    L, H, Hq, W, n, d = 2, 2, 4, 3, 50, 32
    k, q = _inputs(L, H, Hq, W, n, d, 0)
    A = oracle.score(_cfg(L, H, Hq, W, n, d), k.view(np.uint16), k.view(np.uint16), q.view(np.uint16))
    assert abs(A.sum() - 1.0) < 1e-12
    # the same statistic through scipy's softmax and numpy's matmul
    want = np.zeros(n)
    kf, qf = k.astype(np.float64), q.astype(np.float64)
    for l in range(L):
        for hq in range(Hq):
            z = qf[l, hq] @ kf[l, hq // (Hq // H)].T / np.sqrt(d)  # [W, n]
            want += softmax(z, axis=1).sum(0)
    want /= L * Hq * W
    assert np.allclose(A, want, rtol=1e-12, atol=1e-15)


def test_identical_keys_share_mass_equally():
    L, H, Hq, W, n, d = 1, 2, 2, 4, 37, 64
    _, q = _inputs(L, H, Hq, W, n, d, 1)
    row = np.random.default_rng(2).standard_normal(d).astype(np.float16)
    k = np.broadcast_to(row, (L, H, n, d)).copy()
    A = oracle.score(_cfg(L, H, Hq, W, n, d), k.view(np.uint16), k.view(np.uint16), q.view(np.uint16))
    assert np.allclose(A, 1.0 / n, rtol=1e-13)


def test_aligned_key_takes_all_mass():
    L, H, Hq, W, n, d = 1, 1, 2, 3, 20, 32
    k = np.zeros((L, H, n, d), np.float16)
    q = np.zeros((L, Hq, W, d), np.float16)
    q[..., 0] = 8.0
    k[0, 0, 13, 0] = 8.0  # logit 64/sqrt(32) ~ 11.3 above every other key
    A = oracle.score(_cfg(L, H, Hq, W, n, d), k.view(np.uint16), k.view(np.uint16), q.view(np.uint16))
    assert A[13] > 0.999 and np.argmax(A) == 13


@pytest.mark.parametrize("lam", [0.001, 0.01])
def test_decay_multiplies_mass(lam):
    L, H, Hq, W, n, d = 1, 1, 1, 2, 30, 32
    k, q = _inputs(L, H, Hq, W, n, d, 3)
    A = oracle.score(_cfg(L, H, Hq, W, n, d), k.view(np.uint16), k.view(np.uint16), q.view(np.uint16))
    key = oracle.score(_cfg(L, H, Hq, W, n, d, lam), k.view(np.uint16), k.view(np.uint16), q.view(np.uint16))
    assert np.allclose(key, A * np.exp(-lam * (n - 1 - np.arange(n))), rtol=1e-13)
