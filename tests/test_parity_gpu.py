"""Parity of the HIP path against the float64 oracle (GPU).

Every case draws seeded inputs, runs the library through the C ABI and
compares each output T in {O, L, dQ, dK, dV} element by element with the
oracle: max|T - T_ref| / max|T_ref| <= 1e-4 for float32 inputs and 2e-2 for
bfloat16 inputs. The bfloat16 oracle consumes exactly the bfloat16 values the
GPU was given (widened to float64).
"""
import math

import numpy as np
import pytest

import oracle
import workloads
from helpers import OUTPUTS, TOL, compare, gpu_available, run_fwd_bwd, to_gpu, to_host64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _check(errs, dtype, label):
    print(label, {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= TOL[dtype]}
    assert not bad, f"{label}: {bad} exceed {TOL[dtype]}"


def _full_compare(w, inp, causal, scale=None, heads=None):
    scale = w.scale if scale is None else scale
    dev = to_gpu(inp)
    got = run_fwd_bwd(dev, scale, causal)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, scale, causal, heads=heads)
    host = {}
    for k in OUTPUTS:
        a = to_host64(got[k])
        if heads is not None:
            a = np.stack([a[b, h] for (b, h) in heads])
        host[k] = a
    return compare(host, ref), got


@pytest.mark.parametrize("name", ["h1_n128_d32_f32", "b4h8_n1024_d64_f32"])
def test_f32_workloads_every_head(name):
    w = workloads.WORKLOADS[name]
    inp = workloads.generate(w)
    errs, _ = _full_compare(w, inp, w.causal)
    _check(errs, w.dtype, name)


@pytest.mark.parametrize("name,heads", [
    ("b8h16_n4096_d64_bf16_causal", [(0, 0), (3, 7), (7, 15)]),
    ("b16h32_n2048_d128_bf16_peaked", [(0, 0), (5, 17), (15, 31)]),
    ("b2h32_n16384_d128_bf16_causal", [(1, 19), (0, 4)]),
])
def test_bf16_workloads_sampled_heads(name, heads):
    """Full-size launch; the oracle recomputes the listed heads in full."""
    w = workloads.WORKLOADS[name]
    inp = workloads.generate(w)
    errs, _ = _full_compare(w, inp, w.causal, heads=heads)
    _check(errs, w.dtype, f"{name} heads={heads}")


TAIL_N = [1, 2, 63, 65, 127, 129, 1000]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_ragged_lengths(dtype, d, causal):
    """Sequence lengths that are not multiples of any tile, down to n = 1."""
    for n in TAIL_N:
        w = workloads.Workload(f"tail_n{n}_d{d}_{dtype}", 1, 2, n, d, dtype, causal,
                               1.0, 1.0, 1.0 if dtype == "f32" else 0.1, 1000 + n + d)
        inp = workloads.generate(w)
        errs, _ = _full_compare(w, inp, causal)
        _check(errs, dtype, w.name + ("_causal" if causal else ""))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("scale", [-0.3, 0.0, 1.7])
@pytest.mark.parametrize("d,causal", [(64, True), (128, True), (128, False)])
def test_scale_values(dtype, scale, d, causal):
    """Negative, zero and large scales (zero gives uniform attention); at
    d = 128 the bf16 dK/dV kernel takes a negative scale as the sign of
    s log2(e) instead of a sign flip of K."""
    w = workloads.Workload(f"scale_{dtype}_d{d}", 1, 2, 200, d, dtype, causal, 1.0, 1.0, 1.0, 77 + d)
    inp = workloads.generate(w)
    errs, _ = _full_compare(w, inp, causal, scale=scale)
    _check(errs, dtype, f"scale={scale} {dtype} d={d} causal={causal}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("d", [64, 128])
def test_forward_entry_point(dtype, causal, d):
    """attn_fwd alone (no dO: the forward writes no D); at d = 128 in bf16
    this is the eight-wave forward, with 333 queries ending inside its
    second 256-query workgroup."""
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.Workload(f"fwd_{dtype}_d{d}", 2, 3, 333, d, dtype, causal, 1.0, 1.0, 1.0, 55 + d)
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    O, L = lib.attn_fwd(dev["q"], dev["k"], dev["v"], scale=w.scale, causal=causal)
    torch.cuda.synchronize()
    ref = oracle.attention_forward(inp.q, inp.k, inp.v, w.scale, causal)
    errs = compare({"O": to_host64(O), "L": to_host64(L)}, ref, keys=("O", "L"))
    _check(errs, dtype, f"attn_fwd {dtype} causal={causal}")
    # the forward of attn_fwd_bwd is the same kernel: identical bits
    full = run_fwd_bwd(dev, w.scale, causal)
    assert torch.equal(full["O"], O) and torch.equal(full["L"], L)


def test_repeat_calls_are_bitwise_identical():
    """No atomics and a fixed reduction order: results do not depend on
    scheduling. Three calls, including a differently ordered stream history."""
    import torch
    w = workloads.WORKLOADS["b8h16_n4096_d64_bf16_causal"]
    inp = workloads.generate(w, B=2)
    dev = to_gpu(inp)
    first = run_fwd_bwd(dev, w.scale, True)
    for _ in range(2):
        again = run_fwd_bwd(dev, w.scale, True)
        for k in OUTPUTS:
            assert torch.equal(first[k], again[k]), k


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("n,d", [(1, 64), (77, 32), (333, 64), (1000, 128)])
def test_backward_entry_point(dtype, causal, n, d):
    """attn_bwd from the oracle's O (stored in the input dtype) and L."""
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.Workload(f"bwd_{dtype}", 2, 2, n, d, dtype, causal, 1.0, 1.0,
                           1.0 if dtype == "f32" else 0.1, 300 + n + d)
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, causal)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    O = torch.from_numpy(ref["O"].astype(np.float32)).to("cuda").to(tdt)
    L = torch.from_numpy(ref["L"].astype(np.float32)).to("cuda")
    dQ, dK, dV = lib.attn_bwd(dev["q"], dev["k"], dev["v"], O, L, dev["do"], scale=w.scale,
                              causal=causal)
    torch.cuda.synchronize()
    errs = compare({"dQ": to_host64(dQ), "dK": to_host64(dK), "dV": to_host64(dV)}, ref,
                   keys=("dQ", "dK", "dV"))
    _check(errs, dtype, f"attn_bwd n={n} d={d} {dtype} causal={causal}")


def test_backward_entry_point_matches_fused_call():
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.WORKLOADS["b8h16_n4096_d64_bf16_causal"]
    inp = workloads.generate(w, B=1, H=4)
    dev = to_gpu(inp)
    O, L, dQ, dK, dV = lib.attn_fwd_bwd(dev["q"], dev["k"], dev["v"], dev["do"], scale=w.scale,
                                        causal=True)
    bQ, bK, bV = lib.attn_bwd(dev["q"], dev["k"], dev["v"], O, L, dev["do"], scale=w.scale,
                              causal=True)
    torch.cuda.synchronize()
    for a, b in ((dQ, bQ), (dK, bK), (dV, bV)):
        diff = (a.float() - b.float()).abs().max().item() / a.float().abs().max().item()
        assert diff <= 1e-2, diff


def test_longest_workload_sampled_rows_every_head():
    """n = 16384, d = 128, causal, all 64 heads: O, L and dQ of 48 sampled
    query rows per head against the oracle restricted to those rows (each
    depends only on its own row of S and P). The rows include the first, the
    last and rows next to tile boundaries."""
    import torch
    w = workloads.WORKLOADS["b2h32_n16384_d128_bf16_causal"]
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    got = run_fwd_bwd(dev, w.scale, True)
    n = w.n
    rng = np.random.default_rng(2024)
    fixed = np.array([0, 1, 63, 64, 127, 128, 8191, 8192, n - 129, n - 128, n - 2, n - 1])
    worst = {"O": 0.0, "L": 0.0, "dQ": 0.0}
    for b in range(w.B):
        for h in range(w.H):
            rows = np.unique(np.concatenate([fixed, rng.choice(n, 36, replace=False)]))
            ref = oracle.rows_forward_dq(inp.q[b, h], inp.k[b, h], inp.v[b, h], inp.do[b, h], rows,
                                         w.scale, True)
            idx = torch.from_numpy(rows).to(got["O"].device)
            for key in worst:
                x = to_host64(got[key][b, h].index_select(0, idx))
                worst[key] = max(worst[key], oracle.max_rel_err(x, ref[key]))
    _check(worst, w.dtype, "n=16384 d=128 causal, 48 rows x 64 heads")
