"""Parity of the atomic-dQ variant (attn_fwd_bwd_atomic, GPU).

The dK/dV kernel also accumulates dQ = dS K with float32 atomic adds; its
outputs must meet the same bound against the float64 oracle as the fused
path (bfloat16: max|T - T_ref| / max|T_ref| <= 2e-2), and agree with
attn_fwd_bwd: O and L bit for bit (same forward kernel), dK and dV bit for
bit (same products in the same order), dQ within the bound.
"""
import pytest

import oracle
import workloads
from helpers import OUTPUTS, TOL, compare, gpu_available, to_gpu, to_host64, run_fwd_bwd

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _run(dev, scale, causal):
    import torch
    import paper_2609_33916_amd as lib
    r = lib.attn_fwd_bwd_atomic(dev["q"], dev["k"], dev["v"], dev["do"], scale=scale, causal=causal)
    torch.cuda.synchronize()
    return dict(zip(OUTPUTS, r))


def _check(errs, label):
    print(label, {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= TOL["bf16"]}
    assert not bad, f"{label}: {bad} exceed {TOL['bf16']}"


@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_atomic_ragged_lengths(d, causal):
    import torch
    for n in (1, 2, 63, 65, 127, 129, 1000):
        w = workloads.Workload(f"aq_n{n}_d{d}", 1, 2, n, d, "bf16", causal, 1.0, 1.0, 0.1, 3000 + n + d)
        inp = workloads.generate(w)
        dev = to_gpu(inp)
        got = _run(dev, w.scale, causal)
        ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, causal)
        _check(compare({k: to_host64(got[k]) for k in OUTPUTS}, ref), w.name + ("_causal" if causal else ""))
        fused = run_fwd_bwd(dev, w.scale, causal)
        for k in ("O", "L", "dK", "dV"):
            assert torch.equal(fused[k], got[k]), (n, k)


@pytest.mark.parametrize("scale", [-0.3, 0.0])
def test_atomic_scale_values(scale):
    w = workloads.Workload("aq_scale", 1, 2, 200, 64, "bf16", True, 1.0, 1.0, 1.0, 79)
    inp = workloads.generate(w)
    got = _run(to_gpu(inp), scale, True)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, scale, True)
    _check(compare({k: to_host64(got[k]) for k in OUTPUTS}, ref), f"atomic scale={scale}")


@pytest.mark.parametrize("name,heads", [
    ("b8h16_n4096_d64_bf16_causal", [(0, 0), (7, 15)]),
    ("b16h32_n2048_d128_bf16_peaked", [(0, 0), (15, 31)]),
    ("b2h32_n16384_d128_bf16_causal", [(1, 19)]),
])
def test_atomic_workloads(name, heads):
    import numpy as np
    w = workloads.WORKLOADS[name]
    inp = workloads.generate(w)
    got = _run(to_gpu(inp), w.scale, w.causal)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, w.causal, heads=heads)
    host = {k: np.stack([to_host64(got[k])[b, h] for (b, h) in heads]) for k in OUTPUTS}
    _check(compare(host, ref), f"atomic {name}")


def test_atomic_rejects_float32():
    import torch
    import paper_2609_33916_amd as lib
    x = torch.zeros(1, 1, 8, 32, device="cuda")
    with pytest.raises(lib.AttnError):
        lib.attn_fwd_bwd_atomic(x, x, x, x)
