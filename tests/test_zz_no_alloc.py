"""attn_fwd_bwd_noalloc (GPU): the entry point for callers that cannot
allocate device memory. It runs the kernels of attn_fwd_bwd with the D and
log-sum-exp rows in the library's fixed per-GPU scratch instead of a caller
workspace, so its outputs must be bit-identical to attn_fwd_bwd's on the same
inputs. Two calls in a row, the second smaller, check that nothing of the
first call's scratch contents leaks into the second; both also meet the
float64 oracle's bound, and the size limit is rejected before any launch.
"""
import numpy as np
import pytest

import oracle
import workloads
from helpers import OUTPUTS, TOL, compare, gpu_available, to_gpu, to_host64

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _outputs_like(dev):
    import torch
    q = dev["q"]
    B, H, n, _ = q.shape
    return (torch.empty_like(q), torch.empty((B, H, n), dtype=torch.float32, device=q.device),
            torch.empty_like(q), torch.empty_like(q), torch.empty_like(q))


@pytest.mark.parametrize("dtype,d,causal", [("bf16", 128, True), ("bf16", 64, False), ("f32", 64, True),
                                            ("f32", 32, False)])
def test_noalloc_matches_workspace_entry_point(dtype, d, causal):
    import torch
    import paper_2609_33916_amd as lib
    sizes = [(2, 3, 1000), (1, 2, 333)]   # the second call is smaller
    for i, (B, H, n) in enumerate(sizes):
        w = workloads.Workload(f"noalloc_{dtype}_{d}_{i}", B, H, n, d, dtype, causal, 1.0, 1.0,
                               1.0 if dtype == "f32" else 0.1, 4100 + 10 * i + d)
        inp = workloads.generate(w)
        dev = to_gpu(inp)
        print(f"noalloc call {i}: B={B} H={H} n={n} d={d} {dtype} causal={causal}", flush=True)
        ref_out = lib.attn_fwd_bwd(dev["q"], dev["k"], dev["v"], dev["do"], scale=w.scale, causal=causal)
        got = lib.attn_fwd_bwd_noalloc(dev["q"], dev["k"], dev["v"], dev["do"], _outputs_like(dev),
                                       scale=w.scale, causal=causal)
        torch.cuda.synchronize()
        for name, a, b in zip(OUTPUTS, got, ref_out):
            assert torch.equal(a, b), (i, name)
        ref = oracle.attention(inp.q, inp.k, inp.v, inp.do, w.scale, causal)
        errs = compare({k: to_host64(t) for k, t in zip(OUTPUTS, got)}, ref)
        print(i, {k: f"{v:.2e}" for k, v in errs.items()}, flush=True)
        assert all(v <= TOL[dtype] for v in errs.values()), errs


def test_noalloc_full_size_matches_and_allocates_nothing():
    """n = 16384, d = 128, causal, 64 heads (half the scratch), then a smaller
    call: outputs equal attn_fwd_bwd's bit for bit and no device memory is
    allocated by the calls."""
    import torch
    import paper_2609_33916_amd as lib
    w = workloads.WORKLOADS["b2h32_n16384_d128_bf16_causal"]
    inp = workloads.generate(w)
    dev = to_gpu(inp)
    ref_out = lib.attn_fwd_bwd(dev["q"], dev["k"], dev["v"], dev["do"], scale=w.scale, causal=True)
    out = _outputs_like(dev)
    lib.attn_fwd_bwd_noalloc(dev["q"], dev["k"], dev["v"], dev["do"], out, scale=w.scale, causal=True)
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    torch.cuda.reset_peak_memory_stats()
    peak0 = torch.cuda.max_memory_allocated()
    got = lib.attn_fwd_bwd_noalloc(dev["q"], dev["k"], dev["v"], dev["do"], out, scale=w.scale, causal=True)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert torch.cuda.max_memory_allocated() == peak0
    assert free0 - free1 <= 4 << 20
    for name, a, b in zip(OUTPUTS, got, ref_out):
        assert torch.equal(a, b), name
    # second, smaller call: 2 heads of the same inputs
    small = {k: t[:1, :2].contiguous() for k, t in dev.items()}
    ref_small = lib.attn_fwd_bwd(small["q"], small["k"], small["v"], small["do"], scale=w.scale, causal=True)
    got_small = lib.attn_fwd_bwd_noalloc(small["q"], small["k"], small["v"], small["do"], _outputs_like(small),
                                         scale=w.scale, causal=True)
    torch.cuda.synchronize()
    for name, a, b in zip(OUTPUTS, got_small, ref_small):
        assert torch.equal(a, b), ("small", name)


def test_noalloc_rejects_sizes_beyond_the_scratch():
    import torch
    import paper_2609_33916_amd as lib
    rows = lib.attn_noalloc_max_rows()
    assert rows == (16 << 20) // 8
    L = lib.lib()
    # B * H * n one row past the limit: rejected before any launch, with
    # pointers that are never dereferenced
    fake = 1 << 20
    rc = L.attn_fwd_bwd_noalloc(fake, fake, fake, fake, fake, fake, fake, fake, fake,
                                1, 1, rows + 1, 64, 0.125, 0, 0, None)
    assert rc == -8
    assert "attn_noalloc_max_rows" in lib.attn_strerror(rc)
