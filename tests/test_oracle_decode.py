"""Pins for the decode-step oracle (no GPU).

The decode step is pinned to facts outside oracle.decode: the last row of the
(separately pinned) causal attention oracle over the same keys, PyTorch's
float64 scaled_dot_product_attention with the grouped heads expanded by
repeat_interleave (an independent derivation of the GQA head mapping),
closed forms, the cache update itself, and permutation invariance. The last
test plants typical mistakes and checks that a pin catches each.
"""
import math

import numpy as np
import pytest

from oracle import decode as dec
from oracle import naive as orc


def _case(seed, B, Hq, Hkv, n_cap, d, lens, append=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, Hq, d))
    kc = rng.standard_normal((B, Hkv, n_cap, d))
    vc = rng.standard_normal((B, Hkv, n_cap, d))
    kn = rng.standard_normal((B, Hkv, d)) if append else None
    vn = rng.standard_normal((B, Hkv, d)) if append else None
    return q, kc, vc, kn, vn, np.asarray(lens)


def test_equals_last_row_of_causal_attention():
    """Decoding token n-1 after n-1 cached tokens is row n-1 of causal
    attention over all n tokens (MHA)."""
    rng = np.random.default_rng(7)
    n, d, s = 9, 5, 0.6
    Q, K, V = (rng.standard_normal((n, d)) for _ in range(3))
    full = orc.attention_forward(Q[None, None], K[None, None], V[None, None], s, True)
    kc = np.zeros((1, 1, n + 3, d))
    vc = np.zeros((1, 1, n + 3, d))
    kc[0, 0, :n - 1] = K[:n - 1]
    vc[0, 0, :n - 1] = V[:n - 1]
    r = dec.decode_step(Q[None, None, n - 1], kc, vc, [n - 1], s, K[None, None, n - 1], V[None, None, n - 1])
    np.testing.assert_allclose(r["O"][0, 0], full["O"][0, 0, n - 1], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(r["L"][0, 0], full["L"][0, 0, n - 1], rtol=1e-13)


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (6, 1), (32, 4)])
@pytest.mark.parametrize("append", [True, False])
def test_matches_torch_sdpa_with_expanded_heads(Hq, Hkv, append):
    torch = pytest.importorskip("torch")
    B, n_cap, d, s = 3, 40, 8, 0.3
    lens = [5, 33, 17] if append else [6, 39, 1]
    q, kc, vc, kn, vn, lens = _case(11 + Hq + Hkv, B, Hq, Hkv, n_cap, d, lens, append)
    r = dec.decode_step(q, kc, vc, lens, s, kn, vn)
    G = Hq // Hkv
    for b in range(B):
        K = torch.from_numpy(kc[b].copy())
        V = torch.from_numpy(vc[b].copy())
        T = int(lens[b])
        if append:
            K[:, T] = torch.from_numpy(kn[b])
            V[:, T] = torch.from_numpy(vn[b])
            T += 1
        Ke = K[:, :T].repeat_interleave(G, dim=0)       # [Hq, T, d]
        Ve = V[:, :T].repeat_interleave(G, dim=0)
        qb = torch.from_numpy(q[b])[:, None, :]         # [Hq, 1, d]
        O = torch.nn.functional.scaled_dot_product_attention(qb, Ke, Ve, scale=s)[:, 0]
        Lt = torch.logsumexp(s * (qb @ Ke.transpose(1, 2))[:, 0], dim=-1)
        np.testing.assert_allclose(r["O"][b], O.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r["L"][b], Lt.numpy(), rtol=1e-12, atol=1e-12)


def test_closed_forms():
    d, s = 6, 0.9
    rng = np.random.default_rng(3)
    # constant V rows: O = v whatever the scores
    q = rng.standard_normal((1, 1, d))
    kc = rng.standard_normal((1, 1, 10, d))
    vc = np.tile(rng.standard_normal(d), (1, 1, 10, 1))
    r = dec.decode_step(q, kc, vc, [10], s)
    np.testing.assert_allclose(r["O"][0, 0], vc[0, 0, 0], rtol=1e-14)
    # q = 0: uniform weights, O = mean of the T rows, L = ln T
    vc = rng.standard_normal((1, 1, 10, d))
    r = dec.decode_step(np.zeros((1, 1, d)), kc, vc, [7], s)
    np.testing.assert_allclose(r["O"][0, 0], vc[0, 0, :7].mean(axis=0), rtol=1e-13)
    np.testing.assert_allclose(r["L"][0, 0], math.log(7), rtol=1e-14)
    # a single key (first token, appended): O = v_new, L = s q.k_new
    kn, vn = rng.standard_normal((1, 1, d)), rng.standard_normal((1, 1, d))
    r = dec.decode_step(q, kc, vc, [0], s, kn, vn)
    np.testing.assert_allclose(r["O"][0, 0], vn[0, 0], rtol=1e-14)
    np.testing.assert_allclose(r["L"][0, 0], s * float(q[0, 0] @ kn[0, 0]), rtol=1e-13)
    # no key at all: O = 0, L = -inf
    r = dec.decode_step(q, kc, vc, [0], s)
    assert np.all(r["O"] == 0) and r["L"][0, 0] == -np.inf


def test_append_writes_one_row_per_cache_head():
    q, kc, vc, kn, vn, lens = _case(5, 2, 4, 2, 12, 3, [4, 11])
    r = dec.decode_step(q, kc, vc, lens, 0.5, kn, vn)
    for b in range(2):
        for g in range(2):
            for j in range(12):
                want_k = kn[b, g] if j == lens[b] else kc[b, g, j]
                want_v = vn[b, g] if j == lens[b] else vc[b, g, j]
                assert np.array_equal(r["K"][b, g, j], want_k) and np.array_equal(r["V"][b, g, j], want_v)


def test_invariant_to_key_order():
    q, kc, vc, _, _, _ = _case(9, 1, 2, 1, 20, 4, [20], append=False)
    perm = np.random.default_rng(1).permutation(20)
    a = dec.decode_step(q, kc, vc, [20], 0.4)
    b = dec.decode_step(q, kc[:, :, perm], vc[:, :, perm], [20], 0.4)
    np.testing.assert_allclose(a["O"], b["O"], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(a["L"], b["L"], rtol=1e-14)


def test_planted_mistakes_are_caught(monkeypatch):
    """Each mistake below breaks the torch cross-check or the causal-row pin."""
    torch = pytest.importorskip("torch")
    B, Hq, Hkv, n_cap, d, s = 2, 8, 2, 16, 4, 0.7
    q, kc, vc, kn, vn, lens = _case(21, B, Hq, Hkv, n_cap, d, [5, 9])

    def reference():
        G = Hq // Hkv
        out = np.zeros((B, Hq, d))
        for b in range(B):
            K = torch.from_numpy(kc[b].copy())
            V = torch.from_numpy(vc[b].copy())
            T = int(lens[b])
            K[:, T] = torch.from_numpy(kn[b])
            V[:, T] = torch.from_numpy(vn[b])
            Ke = K[:, :T + 1].repeat_interleave(G, dim=0)
            Ve = V[:, :T + 1].repeat_interleave(G, dim=0)
            out[b] = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q[b])[:, None, :], Ke, Ve, scale=s)[:, 0].numpy()
        return out

    ref = reference()
    good = dec.decode_step(q, kc, vc, lens, s, kn, vn)["O"]
    np.testing.assert_allclose(good, ref, rtol=1e-12, atol=1e-12)

    def wrong_group(q_, k_cache, v_cache, lens_, scale, k_new=None, v_new=None):
        K, V = dec.append_kv(k_cache, v_cache, k_new, v_new, [int(x) for x in lens_])
        O = np.zeros(q_.shape)
        for b in range(B):
            for h in range(Hq):
                O[b, h] = dec.decode_head(q_[b, h], K[b, h % Hkv], V[b, h % Hkv], int(lens_[b]) + 1, scale)[0]
        return {"O": O}

    def drops_new_token(q_, k_cache, v_cache, lens_, scale, k_new=None, v_new=None):
        K, V = dec.append_kv(k_cache, v_cache, k_new, v_new, [int(x) for x in lens_])
        G = Hq // Hkv
        O = np.zeros(q_.shape)
        for b in range(B):
            for h in range(Hq):
                O[b, h] = dec.decode_head(q_[b, h], K[b, h // G], V[b, h // G], int(lens_[b]), scale)[0]
        return {"O": O}

    def unscaled(q_, k_cache, v_cache, lens_, scale, k_new=None, v_new=None):
        return dec.decode_step(q_, k_cache, v_cache, lens_, 1.0, k_new, v_new)

    for bad in (wrong_group, drops_new_token, unscaled):
        out = bad(q, kc, vc, lens, s, kn, vn)["O"]
        assert not np.allclose(out, ref, rtol=1e-6, atol=1e-8), bad.__name__
