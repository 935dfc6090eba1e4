"""CPU float64 oracle for one decode step of attention over a KV cache.

TEST INFRASTRUCTURE ONLY (see oracle.naive): the slow, plain definition the
HIP decode kernel is checked against. Nothing here is shared with the GPU path.

What is computed (Paper III: one new query token per head attends to the
keys and values cached for all earlier tokens plus its own, the cache growing
by one row per step; grouped heads share a cache head):

    for batch b with len_b tokens already cached and query head h,
    kv head  g = h // (Hq / Hkv)                 (GQA; Hkv = 1 is MQA)
    append:  K[b, g, len_b] = k_new[b, g],  V[b, g, len_b] = v_new[b, g]
    keys:    j = 0 .. T_b - 1 with T_b = len_b + 1 (len_b without an append)
    s_j   = scale * q[b, h] . K[b, g, j]
    p     = softmax(s),  L = log sum_j exp(s_j)   (natural log)
    O[b, h] = sum_j p_j V[b, g, j]

A step with no key at all (len_b = 0 and nothing appended) returns O = 0 and
L = -inf. The paper states the decode cost as O(n) per token and keeps the
KV-cache accumulation inside the step (Paper III, the decode kernel of
section sec:paper3); the formula is the last row of causal attention over the
same keys, which the pins in tests/test_oracle_decode.py check.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

__all__ = ["append_kv", "decode_head", "decode_step"]


def append_kv(k_cache, v_cache, k_new, v_new, lens):
    """Caches after writing the new token's key and value at row lens[b]
    (copies; float64)."""
    K = np.array(k_cache, dtype=np.float64)
    V = np.array(v_cache, dtype=np.float64)
    B = K.shape[0]
    for b in range(B):
        K[b, :, lens[b]] = k_new[b]
        V[b, :, lens[b]] = v_new[b]
    return K, V


def decode_head(q, K, V, T: int, scale: float):
    """One query row against the first T rows of K and V: (O, L)."""
    q = np.asarray(q, dtype=np.float64)
    if T == 0:
        return np.zeros(q.shape[-1]), -np.inf
    s = scale * (np.asarray(K[:T], dtype=np.float64) @ q)
    m = s.max()
    e = np.exp(s - m)
    z = e.sum()
    O = (e / z) @ np.asarray(V[:T], dtype=np.float64)
    return O, m + np.log(z)


def decode_step(q, k_cache, v_cache, lens, scale: float, k_new=None, v_new=None) -> Dict[str, np.ndarray]:
    """Decode step over [B, Hq, d] queries and [B, Hkv, n_cap, d] caches.

    ``lens`` holds the number of cached tokens per batch entry. With k_new and
    v_new ([B, Hkv, d]) the new token is appended first and attended to.
    Returns O [B, Hq, d], L [B, Hq] and the updated caches K, V (float64).
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv = k_cache.shape[1]
    assert Hq % Hkv == 0, "query heads must be a multiple of the cache heads"
    G = Hq // Hkv
    lens = [int(x) for x in lens]
    if k_new is not None:
        K, V = append_kv(k_cache, v_cache, k_new, v_new, lens)
        T = [x + 1 for x in lens]
    else:
        K = np.asarray(k_cache, dtype=np.float64)
        V = np.asarray(v_cache, dtype=np.float64)
        T = lens
    O = np.zeros((B, Hq, d))
    L = np.zeros((B, Hq))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            O[b, h], L[b, h] = decode_head(q[b, h], K[b, g], V[b, g], T[b], scale)
    return {"O": O, "L": L, "K": K, "V": V}
