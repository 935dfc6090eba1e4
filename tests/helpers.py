"""Shared helpers for the GPU tests: move seeded inputs to the device, call
the library, and compare against the oracle with the per-dtype bound."""
from __future__ import annotations

import numpy as np

import workloads

# max over a tensor of |x - ref| / max|ref| against the float64 oracle
TOL = {"f32": 1e-4, "bf16": 2e-2}
OUTPUTS = ("O", "L", "dQ", "dK", "dV")


def torch_mod():
    import torch
    return torch


def gpu_available() -> bool:
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def to_gpu(inp: workloads.Inputs, device="cuda"):
    """Seeded host inputs -> device tensors in the workload's element type."""
    return workloads.to_torch(inp, device)


def to_host64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def run_fwd_bwd(dev_inputs, scale, causal):
    import paper_2609_33916_amd as lib
    torch = torch_mod()
    r = lib.attn_fwd_bwd(dev_inputs["q"], dev_inputs["k"], dev_inputs["v"], dev_inputs["do"],
                         scale=scale, causal=causal)
    torch.cuda.synchronize()
    return dict(zip(OUTPUTS, r))


def max_rel(x: np.ndarray, ref: np.ndarray) -> float:
    den = np.abs(ref).max()
    diff = np.abs(np.asarray(x, np.float64) - ref).max()
    return float(diff / den) if den > 0 else float(diff)


def compare(got: dict, ref: dict, keys=OUTPUTS) -> dict:
    """Max relative error per output; `got` host float64 arrays aligned with ref."""
    return {k: max_rel(got[k], ref[k]) for k in keys}
