"""Whole-tensor identities on every head of the full-size bf16 workloads (GPU).

For the exact result, on every head: sum_j dK_j = 0 (rows of dS sum to 0),
sum_j dV_j = sum_i dO_i (rows of P sum to 1), <Q, dQ> = <K, dK> (both equal
sum_ij dS_ij S_ij) and <V, dV> = <O, dO>. The GPU outputs carry bfloat16
rounding, so each identity is checked relative to the magnitude of the terms
it sums (e.g. |sum_j dK_j| against sum_j |dK_j|), with the bf16 bound 2e-2.
"""
import pytest

import workloads
from helpers import gpu_available, run_fwd_bwd, to_gpu

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

REL = 2e-2


@pytest.mark.parametrize("name", ["b8h16_n4096_d64_bf16_causal",
                                  "b16h32_n2048_d128_bf16_peaked",
                                  "b2h32_n16384_d128_bf16_causal"])
def test_identities_every_head(name):
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    r = run_fwd_bwd(dev, w.scale, w.causal)
    f64 = lambda t: t.to(torch.float64)
    Q, K, V, dO = (f64(dev[k]) for k in ("q", "k", "v", "do"))
    O, dQ, dK, dV = (f64(r[k]) for k in ("O", "dQ", "dK", "dV"))
    # [B, H, d] sums over the sequence
    sk = dK.sum(dim=2).abs().amax(dim=-1) / dK.abs().sum(dim=2).amax(dim=-1)
    sv = (dV.sum(dim=2) - dO.sum(dim=2)).abs().amax(dim=-1) / dO.abs().sum(dim=2).amax(dim=-1)
    qk = ((Q * dQ).sum(dim=(2, 3)) - (K * dK).sum(dim=(2, 3))).abs() / (K * dK).abs().sum(dim=(2, 3))
    vo = ((V * dV).sum(dim=(2, 3)) - (O * dO).sum(dim=(2, 3))).abs() / (O * dO).abs().sum(dim=(2, 3))
    worst = {"sum_dK": sk.max().item(), "sum_dV": sv.max().item(),
             "QdQ_KdK": qk.max().item(), "VdV_OdO": vo.max().item()}
    print(name, {k: f"{v:.2e}" for k, v in worst.items()}, flush=True)
    for k, v in worst.items():
        assert v <= REL, (k, v)
    for t in (O, dQ, dK, dV):
        assert torch.isfinite(t).all()
