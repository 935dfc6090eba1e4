"""Parity of the decode step (attn_decode, GPU) against the float64 oracle.

For every checked (batch, query head): max|O - O_ref| / max|O_ref| and the same
for L within the bfloat16 bound 2e-2; the cache after the step equals the
cache before it except for the appended row, which holds k_new / v_new bit
for bit. Cases cover MHA, GQA and MQA groupings (up to 64 query heads per
cache head, i.e. two 32-head chunks), d in {32, 64, 128}, lengths from an
empty cache to splits of a long one, ragged per-sequence lengths, and steps
with and without an append.
"""
import numpy as np
import pytest

import workloads
from helpers import TOL, gpu_available, max_rel, to_host64
from oracle import decode as dec

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _run_case(w, n=None, B=None, append=True, use_lens=True, scale=None, seed=None):
    import torch
    import paper_2609_33916_amd as lib
    inp = workloads.generate_decode(w, n=n, B=B, seed=seed)
    dev = workloads.decode_to_torch(inp, "cuda")
    kc0, vc0 = dev["k_cache"].clone(), dev["v_cache"].clone()
    nn = inp.lens.max() if use_lens else (w.n if n is None else n)
    lens = inp.lens if use_lens else np.full(len(inp.lens), nn, dtype=np.int32)
    s = w.scale if scale is None else scale
    O, L = lib.attn_decode(dev["q"], dev["k_cache"], dev["v_cache"],
                           dev["k_new"] if append else None, dev["v_new"] if append else None,
                           cache_lens=dev["lens"] if use_lens else None, n=int(nn), scale=s)
    torch.cuda.synchronize()
    ref = dec.decode_step(inp.q, inp.k_cache, inp.v_cache, lens, s,
                          inp.k_new if append else None, inp.v_new if append else None)
    errs = {"O": max_rel(to_host64(O), ref["O"])}
    Lg, Lr = to_host64(L), ref["L"]
    fin = np.isfinite(Lr)
    assert np.array_equal(np.isfinite(Lg), fin)
    errs["L"] = max_rel(Lg[fin], Lr[fin]) if fin.any() else 0.0
    # the caches: unchanged except the appended rows
    kc, vc = dev["k_cache"], dev["v_cache"]
    if append:
        for b in range(len(lens)):
            p = int(lens[b])
            assert torch.equal(kc[b, :, p], dev["k_new"][b]) and torch.equal(vc[b, :, p], dev["v_new"][b])
            kc[b, :, p] = kc0[b, :, p]
            vc[b, :, p] = vc0[b, :, p]
    assert torch.equal(kc, kc0) and torch.equal(vc, vc0)
    return errs


def _check(errs, label):
    print(label, {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    assert not bad, f"{label}: {bad} exceed {TOL['bf16']}"


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 2), (16, 2), (32, 1), (64, 1)])
def test_decode_groupings_and_lengths(d, Hq, Hkv):
    for n in (0, 1, 127, 128, 300, 3000):
        w = workloads.DecodeWorkload(f"dec_n{n}_d{d}_{Hq}x{Hkv}", 2, Hq, Hkv, n, n + 5, d, "bf16", False, 1.0,
                                     500 + n + d + Hq)
        _check(_run_case(w, use_lens=False), w.name)


@pytest.mark.parametrize("append", [True, False])
def test_decode_ragged_lengths(append):
    w = workloads.DecodeWorkload("dec_ragged", 6, 16, 4, 2000, 2001, 128, "bf16", True, 1.0, 77)
    _check(_run_case(w, append=append), f"ragged append={append}")


def test_decode_empty_cache_without_append():
    """No key at all: O = 0 and L = -inf (checked inside _run_case)."""
    w = workloads.DecodeWorkload("dec_empty", 2, 4, 2, 0, 3, 64, "bf16", False, 1.0, 5)
    _check(_run_case(w, append=False, use_lens=False), "empty")


@pytest.mark.parametrize("scale", [-0.2, 0.0, 0.5])
def test_decode_scale_values(scale):
    w = workloads.DecodeWorkload("dec_scale", 2, 8, 2, 700, 701, 64, "bf16", False, 1.0, 91)
    _check(_run_case(w, scale=scale, use_lens=False), f"scale={scale}")


def test_decode_long_cache_many_splits():
    w = workloads.DecodeWorkload("dec_long", 1, 8, 1, 50000, 50001, 128, "bf16", False, 1.0, 31)
    _check(_run_case(w, use_lens=False), "long")


@pytest.mark.parametrize("name", ["dec_b16_hq64_hkv8_n8192_d128_bf16", "dec_b32_hq32_hkv8_n4096_d128_bf16_ragged"])
def test_decode_workloads_sampled_batch(name):
    """The workloads' shapes with the batch cut to 3 sequences (the oracle
    keeps float64 copies of the caches)."""
    w = workloads.DECODE_WORKLOADS[name]
    _check(_run_case(w, B=3), name)


def test_decode_matches_last_row_of_forward():
    """GPU against GPU: decoding token n-1 equals row n-1 of attn_fwd with
    the causal mask (one cache head per query head)."""
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.Workload("dec_vs_fwd", 1, 4, 1000, 64, "bf16", True, 1.0, 1.0, 1.0, 8)
    inp = workloads.generate(w)
    dev = workloads.to_torch(inp, "cuda")
    O, L = lib.attn_fwd(dev["q"], dev["k"], dev["v"], causal=True)
    n = w.n
    kc = torch.zeros(1, 4, n, 64, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    kc[:, :, :n - 1] = dev["k"][:, :, :n - 1]
    vc[:, :, :n - 1] = dev["v"][:, :, :n - 1]
    Od, Ld = lib.attn_decode(dev["q"][:, :, n - 1].contiguous(), kc, vc, dev["k"][:, :, n - 1].contiguous(),
                             dev["v"][:, :, n - 1].contiguous(), n=n - 1)
    torch.cuda.synchronize()
    a, b = Od.float(), O[:, :, n - 1].float()
    assert (a - b).abs().max().item() <= 1e-2 * b.abs().max().item()
    assert (Ld - L[:, :, n - 1]).abs().max().item() <= 1e-4 * L[:, :, n - 1].abs().max().item()


def test_decode_workspace_reused_across_sizes():
    """One workspace, sized for the largest call, serves calls with different
    split counts in a row (its contents on entry are ignored); each call
    meets the oracle."""
    import torch
    import paper_2609_33916_amd as lib
    sizes = [(1, 8, 1, 50000), (3, 16, 4, 2000), (1, 8, 1, 9000), (2, 64, 1, 3000)]
    cap = max(lib.attn_decode_workspace_bytes(B, Hq, Hkv, n, 128, True) for B, Hq, Hkv, n in sizes)
    ws = torch.empty(cap, dtype=torch.uint8, device="cuda")
    for i, (B, Hq, Hkv, n) in enumerate(sizes + sizes[:1]):
        w = workloads.DecodeWorkload(f"dec_reuse{i}", B, Hq, Hkv, n, n + 1, 128, "bf16", False, 1.0, 700 + i)
        inp = workloads.generate_decode(w)
        dev = workloads.decode_to_torch(inp, "cuda")
        O, L = lib.attn_decode(dev["q"], dev["k_cache"], dev["v_cache"], dev["k_new"], dev["v_new"],
                               n=n, scale=w.scale, workspace=ws)
        torch.cuda.synchronize()
        lens = np.full(B, n, dtype=np.int32)
        ref = dec.decode_step(inp.q, inp.k_cache, inp.v_cache, lens, w.scale, inp.k_new, inp.v_new)
        errs = {"O": max_rel(to_host64(O), ref["O"]), "L": max_rel(to_host64(L), ref["L"])}
        _check(errs, f"reuse {i}: B={B} Hq={Hq} Hkv={Hkv} n={n}")
