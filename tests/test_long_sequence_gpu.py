"""The longest sequence tested (GPU): one head of n = 2^20 keys (d = 64,
causal, bf16), the largest n the paper's decode sweep reaches and 64x the
forward/backward sizes it measures. No n x n buffer exists at any point (the
n x n float32 matrix would be 4 TiB). Checks:

* O, L and dQ of 40 sampled query rows (the first, the last, rows next to
  tile boundaries and random ones) against the float64 oracle restricted to
  those rows (each depends only on its own row of S and P);
* dK and dV through the whole-tensor identities that hold exactly for the
  true result: sum_j dK_j = 0, sum_j dV_j = sum_i dO_i, <Q, dQ> = <K, dK>,
  <V, dV> = <O, dO>;
* every output finite.
"""
import numpy as np
import pytest

import oracle
import workloads
from helpers import TOL, gpu_available, run_fwd_bwd, to_gpu, to_host64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def test_one_head_of_a_million_keys():
    import torch
    n, d = 1 << 20, 64
    w = workloads.Workload("n1048576_d64_causal", 1, 1, n, d, "bf16", True, 1.0, 1.0, 0.1, 2020)
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    print(f"one head, n = {n}, d = {d}, causal, bf16", flush=True)
    r = run_fwd_bwd(dev, w.scale, True)
    for k, t in r.items():
        assert torch.isfinite(t.float()).all().item(), k
    rng = np.random.default_rng(11)
    rows = np.unique(np.concatenate([[0, 1, 63, 64, 127, 128, n // 2 - 1, n // 2, n - 129, n - 128, n - 2, n - 1],
                                     rng.choice(n, 28, replace=False)]))
    ref = oracle.rows_forward_dq(inp.q[0, 0], inp.k[0, 0], inp.v[0, 0], inp.do[0, 0], rows, w.scale, True)
    idx = torch.from_numpy(rows).to(r["O"].device)
    errs = {k: oracle.max_rel_err(to_host64(r[k][0, 0].index_select(0, idx)), ref[k]) for k in ("O", "L", "dQ")}
    print("sampled rows", {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
    assert all(v <= TOL["bf16"] for v in errs.values()), errs
    f64 = lambda t: t[0, 0].to(torch.float64)
    Q, K, V, dO = (f64(dev[k]) for k in ("q", "k", "v", "do"))
    O, dQ, dK, dV = (f64(r[k]) for k in ("O", "dQ", "dK", "dV"))
    ident = {
        "sum_dK": (dK.sum(0).abs().max() / dK.abs().sum(0).max()).item(),
        "sum_dV": ((dV.sum(0) - dO.sum(0)).abs().max() / dO.abs().sum(0).max()).item(),
        "QdQ_KdK": (((Q * dQ).sum() - (K * dK).sum()).abs() / (K * dK).abs().sum()).item(),
        "VdV_OdO": (((V * dV).sum() - (O * dO).sum()).abs() / (O * dO).abs().sum()).item(),
    }
    print("identities", {k: f"{v:.2e}" for k, v in ident.items()}, flush=True)
    assert all(v <= TOL["bf16"] for v in ident.values()), ident
