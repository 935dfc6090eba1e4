"""Parity of the naive (materialising) path against the float64 oracle (GPU).

attn_mat_fwd stores the attention matrix P and attn_mat_bwd reads it back
instead of recomputing it (the naive realisation the paper compares the fused
one against). Its outputs O, L, dQ, dK, dV must meet the same bound as the
fused path (max|T - T_ref| / max|T_ref| <= 1e-4 float32, 2e-2 bfloat16), and
the stored P itself must match the oracle's P on every entry the layout
defines (query i < n, key j < n, j <= i under the causal mask), with exact
zeros at the masked entries of the written diagonal blocks.
"""
import numpy as np
import pytest

import oracle
import workloads
from helpers import OUTPUTS, TOL, compare, gpu_available, to_gpu, to_host64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU"),
              # a NaN in a defined entry of P must fail, never pass as a warning
              pytest.mark.filterwarnings("error::RuntimeWarning")]


def _check(errs, dtype, label):
    print(label, {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    bad = {k: v for k, v in errs.items() if not v <= TOL[dtype]}
    assert not bad, f"{label}: {bad} exceed {TOL[dtype]}"


def _run_mat(dev, scale, causal):
    import torch
    import paper_2609_33916_amd as lib
    O, L, dQ, dK, dV, P = lib.attn_mat_fwd_bwd(dev["q"], dev["k"], dev["v"], dev["do"], scale=scale,
                                               causal=causal)
    torch.cuda.synchronize()
    return {"O": O, "L": L, "dQ": dQ, "dK": dK, "dV": dV}, P


def _p_checks(P_dev, inp, scale, causal, heads, dtype):
    """Stored P against the oracle's P on the defined entries; zeros above the
    diagonal inside each query's 32-row block under the causal mask."""
    import torch
    n = inp.q.shape[2]
    worst = 0.0
    if causal:
        # entries the checks read: key j < min(n, end of query i's 32-row
        # block); the forward writes them all. Entries past them were never
        # written (they hold whatever the buffer held) and are zeroed on the
        # device before widening, so no undefined value reaches the host.
        i = torch.arange(n, device=P_dev.device)[:, None]
        j = torch.arange(n, device=P_dev.device)[None, :]
        used = j < torch.clamp((i // 32 + 1) * 32, max=n)
    for (b, h) in heads:
        ref = oracle.attention_head(inp.q[b, h], inp.k[b, h], inp.v[b, h], inp.do[b, h], scale, causal,
                                    keep=True)["P"]
        blk = P_dev[b, h, :, :n]
        if causal:
            blk = torch.where(used, blk, torch.zeros((), dtype=blk.dtype, device=blk.device))
        got = to_host64(blk)
        if causal:
            lower = np.tril(np.ones((n, n), dtype=bool))
            worst = max(worst, float(np.abs(got[lower] - ref[lower]).max()))
            i = np.arange(n)[:, None]
            j = np.arange(n)[None, :]
            diag_block = (j > i) & (j < np.minimum(n, (i // 32 + 1) * 32))
            assert np.all(got[diag_block] == 0.0), (b, h)
        else:
            worst = max(worst, float(np.abs(got - ref).max()))
    # P entries are probabilities in [0, 1]: absolute error, same bound
    assert worst <= TOL[dtype], f"P max abs error {worst:.2e}"
    return worst


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_naive_ragged_lengths(dtype, d, causal):
    # 31/33 straddle the 32-query tiles of the d <= 64 dK/dV kernel, 63/65 the
    # 64-row tiles, 129 the 128-row ones
    for n in (1, 2, 31, 33, 63, 65, 129, 1000):
        w = workloads.Workload(f"mat_n{n}_d{d}_{dtype}", 1, 2, n, d, dtype, causal,
                               1.0, 1.0, 1.0 if dtype == "f32" else 0.1, 2000 + n + d)
        inp = workloads.generate(w)
        dev = to_gpu(inp)
        got, P = _run_mat(dev, w.scale, causal)
        ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, causal)
        errs = compare({k: to_host64(got[k]) for k in OUTPUTS}, ref)
        pe = _p_checks(P, inp, w.scale, causal, [(0, 0), (0, 1)], dtype)
        _check(dict(errs, P=pe), dtype, w.name + ("_causal" if causal else ""))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("scale", [-0.3, 0.0])
def test_naive_scale_values(dtype, scale):
    w = workloads.Workload(f"mat_scale_{dtype}", 1, 2, 200, 64, dtype, True, 1.0, 1.0, 1.0, 78)
    inp = workloads.generate(w)
    got, P = _run_mat(to_gpu(inp), scale, True)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, scale, True)
    errs = compare({k: to_host64(got[k]) for k in OUTPUTS}, ref)
    _check(errs, dtype, f"naive scale={scale} {dtype}")


@pytest.mark.parametrize("name,heads", [
    ("b4h8_n1024_d64_f32", None),
    ("b8h16_n4096_d64_bf16_causal", [(0, 0), (6, 11)]),
    ("b16h32_n2048_d128_bf16_peaked", [(0, 0), (9, 30)]),
])
def test_naive_workloads(name, heads):
    """Full-size launches of the workloads with n <= 4096 (P of every head
    stored: 4 GiB at n = 4096 and n = 2048 here)."""
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.generate(w)
    got, P = _run_mat(to_gpu(inp), w.scale, w.causal)
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, w.causal, heads=heads)
    host = {}
    for k in OUTPUTS:
        a = to_host64(got[k])
        if heads is not None:
            a = np.stack([a[b, h] for (b, h) in heads])
        host[k] = a
    errs = compare(host, ref)
    pe = _p_checks(P, inp, w.scale, w.causal, heads or [(0, 0), (3, 7)], w.dtype)
    _check(dict(errs, P=pe), w.dtype, f"naive {name}")
    del P
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("causal", [False, True])
def test_naive_split_entry_points(dtype, causal):
    """attn_mat_fwd then attn_mat_bwd (D from the stored O) against the
    one-call attn_mat_fwd_bwd: the forward's O, L and P are the same bits; the
    gradients agree within the bound and both meet the oracle."""
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.Workload(f"mat_split_{dtype}", 2, 2, 333, 64, dtype, causal, 1.0, 1.0,
                           1.0 if dtype == "f32" else 0.1, 99)
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    O, L, P = lib.attn_mat_fwd(dev["q"], dev["k"], dev["v"], scale=w.scale, causal=causal)
    dQ, dK, dV = lib.attn_mat_bwd(dev["q"], dev["k"], dev["v"], O, dev["do"], P, scale=w.scale,
                                  causal=causal)
    both, P2 = _run_mat(dev, w.scale, causal)
    torch.cuda.synchronize()
    assert torch.equal(O, both["O"]) and torch.equal(L, both["L"])
    n = w.n
    for b in range(2):
        for h in range(2):
            rows = P[b, h, :, :n]
            mask = torch.tril(torch.ones(n, n, dtype=torch.bool, device=rows.device)) if causal else \
                torch.ones(n, n, dtype=torch.bool, device=rows.device)
            assert torch.equal(rows[mask], P2[b, h, :, :n][mask])
    ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, causal)
    errs = compare({"dQ": to_host64(dQ), "dK": to_host64(dK), "dV": to_host64(dV)}, ref,
                   keys=("dQ", "dK", "dV"))
    _check(errs, dtype, f"attn_mat_bwd {dtype} causal={causal}")
