"""Benchmark of the fused attention forward+backward pass on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--no-other-workloads]
    python bench.py --mode fwd|bwd      attn_fwd or attn_bwd alone
    python bench.py --mode naive        fused versus the naive materialising path
    python bench.py --mode atomic       attn_fwd_bwd versus the atomic-dQ variant
    python bench.py --mode decode [--decode-workload NAME] [--decode-sweep]
                                        one decode step over a KV cache (HBM-bound)

One step is one attn_fwd_bwd call (forward, dK/dV and dQ kernels) over the
whole workload, inputs resident in HBM before timing starts. Prints ONE JSON
line with whole-job TFLOP/s (algorithmic flops 14*d per (query, key) pair
that takes part), the roofline position of the dominant kernel measured with
HIP events on the launch stream, the max relative error of every output on
sampled heads against the float64 oracle, and the oracle itself timed on the
host as a CPU baseline. The other four workloads of the table follow, each
timed and checked the same way, under the key "other_workloads".
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402

METRIC = "fused attn fwd+bwd TFLOP/s and % of MI355X MFMA peak (1 GPU); max rel err"
DEFAULT_WORKLOAD = "b2h32_n16384_d128_bf16_causal"
# MI355X published dense peaks (TFLOP/s)
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}
HBM_PEAK_GBS = 8000.0
KERNELS = ("fwd", "dkdv", "dq")
# algorithmic flops per (query, key) pair and per d, by kernel: the forward's
# two products; the dK/dV kernel's S recompute, dP, dV and dK; the dQ kernel's
# dQ product (its S and dP recomputation is counted once, in dK/dV).
ALG_FLOPS_PER_PAIR_D = {"fwd": 4, "dkdv": 8, "dq": 2}
# flops the MFMA units execute per pair and per d, by kernel
EXEC_FLOPS_PER_PAIR_D = {"fwd": 4, "dkdv": 8, "dq": 6}


class HipEvents:
    """hipEvent_t handles from the HIP runtime that torch already loaded."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so.7")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        ev = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(ev))
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")
        return ev.value

    def elapsed_ms(self, a, b) -> float:
        out = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(out), a, b)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)

    def destroy(self, ev):
        self.hip.hipEventDestroy(ev)


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 summary
    (FETCH_SIZE + WRITE_SIZE, copy-calibrated), or None when there is none
    or the kernel sources changed since the counters were taken."""
    from paper_2609_33916_amd import profiling
    rec = profiling.read_traffic(os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md"))
    if not rec or rec.get("source_hash") != profiling.source_hash():
        return None
    k = next((v for name, v in rec["kernels"].items()
              if name in (f"{kernel}_kernel", f"{kernel}16_kernel")), None)
    if not k:
        return None
    return int(k["fetch_bytes"] + k["write_bytes"])


def cpu_model() -> str:
    """The host CPU's model name (first processor in /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def cpu_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        n = [p.get("num_threads", 0) for p in threadpool_info() if p.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def bench_entry(args, w, inp, dev, out, ws, hip, torch, attn) -> int:
    """Time attn_fwd (4 d flops per pair) or attn_bwd (10 d per pair) alone;
    the roofline entry then covers the whole call."""
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    O, L, dQ, dK, dV = out
    B, H, n, d = q.shape
    # attn_bwd consumes a real forward result
    attn.attn_fwd(q, k, v, scale=w.scale, causal=w.causal, out=(O, L))
    if args.mode == "fwd":
        call = lambda: attn.attn_fwd(q, k, v, scale=w.scale, causal=w.causal, out=(O, L))
        per_pair = 4
    else:
        call = lambda: attn.attn_bwd(q, k, v, O, L, do, scale=w.scale, causal=w.causal,
                                     out=(dQ, dK, dV), workspace=ws)
        per_pair = 10
    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = hip.create(), hip.create()
    stream = torch.cuda.current_stream().cuda_stream
    hip.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    t0 = time.perf_counter()
    hip.hip.hipEventRecord(e0, stream)
    for _ in range(args.steps):
        call()
    hip.hip.hipEventRecord(e1, stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    dev_ms = hip.elapsed_ms(e0, e1) / args.steps
    flops = per_pair * d * workloads.causal_pairs(n, w.causal) * B * H
    value = flops / (wall_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    achieved = flops / (dev_ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": f"attention {'forward' if args.mode == 'fwd' else 'backward'} TFLOP/s (1 GPU)",
        "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall_ms, 4), "device_ms_per_step": round(dev_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype,
        "data": "synthetic", "pct_of_peak": round(100 * value / peak, 2),
        "config": {"workload": w.name, "entry": "attn_" + args.mode, "B": B, "H": H, "n": n, "d": d,
                   "causal": w.causal, "alg_flops": flops},
        "roofline": {"kernel": "attn_" + args.mode + " (whole call)", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "traffic": None},
    }), flush=True)
    return 0


def _time_calls(call, steps, warmup, hip, torch):
    """(device ms, wall ms) per call over `steps` back-to-back calls."""
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = hip.create(), hip.create()
    stream = torch.cuda.current_stream().cuda_stream
    hip.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    t0 = time.perf_counter()
    hip.hip.hipEventRecord(e0, stream)
    for _ in range(steps):
        call()
    hip.hip.hipEventRecord(e1, stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    dev_ms = hip.elapsed_ms(e0, e1) / steps
    hip.destroy(e0)
    hip.destroy(e1)
    return dev_ms, wall


def mat_written_elems(n: int, causal: bool) -> int:
    """Elements of P the materialising forward writes per head: every 64-key
    tile a 32-query block visits, for the block's rows < n (its forward
    workgroups own 128 queries; under the causal mask a block visits the
    tiles that start at or before its last query)."""
    total = 0
    for qw0 in range(0, n, 32):
        rows = min(32, n - qw0)
        q0 = qw0 // 128 * 128
        kv_end = min(n, q0 + 128) if causal else n
        tiles = sum(1 for kv0 in range(0, kv_end, 64) if not causal or kv0 <= qw0 + 31)
        total += rows * 64 * tiles
    return total


def bench_naive(args, w, inp, dev, out, ws, hip, torch, attn) -> int:
    """The paper's central comparison on this GPU: the fused path (attn_fwd_bwd)
    against the naive path that stores the attention matrix, timed as forward
    alone + backward alone (attn_mat_fwd, attn_mat_bwd) and as one call."""
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    O, L, dQ, dK, dV = out
    B, H, n, d = q.shape
    e = 2 if w.dtype == "bf16" else 4
    P = torch.empty((B, H, n, attn.attn_mat_lda(n)), dtype=q.dtype, device=q.device)
    O2, L2 = torch.empty_like(O), torch.empty_like(L)
    g2 = tuple(torch.empty_like(q) for _ in range(3))
    fused = lambda: attn.attn_fwd_bwd(q, k, v, do, scale=w.scale, causal=w.causal, out=out, workspace=ws)
    mfwd = lambda: attn.attn_mat_fwd(q, k, v, scale=w.scale, causal=w.causal, out=(O2, L2), P=P)
    mbwd = lambda: attn.attn_mat_bwd(q, k, v, O2, do, P, scale=w.scale, causal=w.causal, out=g2,
                                     workspace=ws)
    mboth = lambda: attn.attn_mat_fwd_bwd(q, k, v, do, scale=w.scale, causal=w.causal,
                                          out=(O2, L2) + g2, P=P, workspace=ws)
    print("[bench] naive: fused, naive forward, naive backward, naive one call", file=sys.stderr, flush=True)
    t = {}
    t["fused"] = _time_calls(fused, args.steps, args.warmup, hip, torch)
    t["naive_fwd"] = _time_calls(mfwd, args.steps, args.warmup, hip, torch)
    t["naive_bwd"] = _time_calls(mbwd, args.steps, args.warmup, hip, torch)
    t["naive_call"] = _time_calls(mboth, args.steps, args.warmup, hip, torch)
    naive_ms = t["naive_fwd"][0] + t["naive_bwd"][0]
    f_alg = workloads.alg_flops(B, H, n, d, w.causal)
    heads = B * H
    p_elems = mat_written_elems(n, w.causal) * heads
    # naive forward element count (Table tab:paper1-dram's model): read Q, K, V
    # once, write P (the tiles written) and O once, plus the float32 L rows
    model = {"read": 3 * heads * n * d * e, "write": p_elems * e + heads * n * d * e + 4 * heads * n}
    rec = {
        "metric": "fused / naive device time, attention fwd+bwd (1 GPU)",
        "value": round(t["fused"][0] / naive_ms, 4), "unit": "ratio", "higher_is_better": False,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "n": n, "d": d, "causal": w.causal},
        "fused_ms": round(t["fused"][0], 4),
        "fused_tflops": round(f_alg / (t["fused"][0] * 1e-3) / 1e12, 2),
        "naive_fwd_ms": round(t["naive_fwd"][0], 4),
        "naive_bwd_ms": round(t["naive_bwd"][0], 4),
        "naive_ms": round(naive_ms, 4),
        "naive_one_call_ms": round(t["naive_call"][0], 4),
        "naive_tflops": round(f_alg / (naive_ms * 1e-3) / 1e12, 2),
        "fused_over_naive_one_call": round(t["fused"][0] / t["naive_call"][0], 4),
        "p_stored_bytes": p_elems * e,
        "naive_fwd_hbm_model_bytes": model,
        "naive_fwd_model_gbs": round((model["read"] + model["write"]) / (t["naive_fwd"][0] * 1e-3) / 1e9, 1),
    }
    tr = measured_traffic_kernel(w.name, "mat_fwd_kernel", prefix="hbm_traffic_naive")
    if tr is not None:
        rec["naive_fwd_hbm_measured_bytes"] = tr
        rec["naive_fwd_measured_over_model"] = {
            "read": round(tr["fetch_bytes"] / model["read"], 3),
            "write": round(tr["write_bytes"] / model["write"], 3),
            "total": round((tr["fetch_bytes"] + tr["write_bytes"]) / (model["read"] + model["write"]), 3)}
    if not args.no_cpu_baseline:
        import oracle
        torch.cuda.synchronize()
        b, h = B - 1, H // 2
        ref = oracle.attention_head(inp.q[b, h], inp.k[b, h], inp.v[b, h], inp.do[b, h], w.scale, w.causal)
        got = {"O": O2[b, h], "L": L2[b, h], "dQ": g2[0][b, h], "dK": g2[1][b, h], "dV": g2[2][b, h]}
        rec["naive_max_rel_err"] = {key: float(f"{oracle.max_rel_err(x.float().cpu().numpy(), ref[key]):.3e}")
                                    for key, x in got.items()}
        rec["naive_max_rel_err_sample"] = f"head ({b}, {h}) vs float64 oracle"
    print(json.dumps(rec), flush=True)
    return 0


def atomic_adds(B: int, H: int, n: int, d: int, causal: bool) -> int:
    """float32 atomic adds of attn_fwd_bwd_atomic: every 128-key workgroup adds
    d values for each query row < n of the tiles it sweeps (from its first
    key's 64-query tile under the causal mask, from 0 otherwise)."""
    rows = sum(n - ((k0 // 64) * 64 if causal else 0) for k0 in range(0, n, 128))
    return B * H * d * rows


def bench_atomic(args, w, inp, dev, out, ws, hip, torch, attn) -> int:
    """The paper's atomic-versus-recompute trade-off on this GPU: attn_fwd_bwd
    (dQ by a separate kernel that recomputes S and dP) against
    attn_fwd_bwd_atomic (dQ accumulated with float32 atomics in the dK/dV
    kernel)."""
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    B, H, n, d = q.shape
    wsa = torch.empty(attn.attn_workspace_bytes_atomic(B, H, n, d), dtype=torch.uint8, device=q.device)
    out2 = tuple(torch.empty_like(t) for t in out)
    fused = lambda: attn.attn_fwd_bwd(q, k, v, do, scale=w.scale, causal=w.causal, out=out, workspace=ws)
    atom = lambda: attn.attn_fwd_bwd_atomic(q, k, v, do, scale=w.scale, causal=w.causal, out=out2,
                                            workspace=wsa)
    print("[bench] atomic: fused, atomic-dQ", file=sys.stderr, flush=True)
    tf = _time_calls(fused, args.steps, args.warmup, hip, torch)
    ta = _time_calls(atom, args.steps, args.warmup, hip, torch)
    f_alg = workloads.alg_flops(B, H, n, d, w.causal)
    rec = {
        "metric": "attention fwd+bwd TFLOP/s, atomic-dQ variant (1 GPU)",
        "value": round(f_alg / (ta[1] * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": B, "H": H, "n": n, "d": d, "causal": w.causal},
        "atomic_ms": round(ta[0], 4), "fused_ms": round(tf[0], 4),
        "atomic_tflops": round(f_alg / (ta[0] * 1e-3) / 1e12, 2),
        "fused_tflops": round(f_alg / (tf[0] * 1e-3) / 1e12, 2),
        "atomic_over_fused_time": round(ta[0] / tf[0], 4),
        "predicted_atomic_adds": atomic_adds(B, H, n, d, w.causal),
    }
    torch.cuda.synchronize()
    diff = {name: float((a.float() - b.float()).abs().max() / b.float().abs().max())
            for name, a, b in zip(("O", "L", "dQ", "dK", "dV"), out2, out)}
    rec["max_rel_diff_vs_fused"] = {key: float(f"{val:.3e}") for key, val in diff.items()}
    print(json.dumps(rec), flush=True)
    return 0


def bench_decode(args, torch, attn, hip) -> int:
    """One decode step (append the new token, attend over the cache) timed on
    resident inputs; the step is HBM-bound, so the roofline is bytes per second
    against the 8 TB/s peak. --decode-sweep times the step over cache lengths
    1024 ... 2^20 (the paper's sweep) and reports the local scaling exponent."""
    w = workloads.DECODE_WORKLOADS[args.decode_workload]
    print(f"[bench] decode workload {w.name}: generating seeded inputs", file=sys.stderr, flush=True)

    def setup(n=None, B=None):
        inp = workloads.generate_decode(w, n=n, B=B)
        dev = workloads.decode_to_torch(inp, "cuda")
        n_max = int(inp.lens.max())
        ws_b = attn.attn_decode_workspace_bytes(len(inp.lens), w.Hq, w.Hkv, n_max, w.d, True)
        ws = torch.empty(max(ws_b, 16), dtype=torch.uint8, device="cuda")
        O = torch.empty_like(dev["q"])
        L = torch.empty(dev["q"].shape[:2], dtype=torch.float32, device="cuda")
        call = lambda: attn.attn_decode(dev["q"], dev["k_cache"], dev["v_cache"], dev["k_new"], dev["v_new"],
                                        cache_lens=dev["lens"], n=n_max, scale=w.scale, out=(O, L),
                                        workspace=ws)
        return inp, dev, call, O, L

    if args.decode_sweep:
        rows = []
        n = 1024
        while n <= 1 << 20:
            inp, dev, call, O, L = setup(n=n)
            t = _time_calls(call, args.steps, args.warmup, hip, torch)
            nbytes = workloads.decode_bytes(inp.lens, w.Hq, w.Hkv, w.d, w.elem_bytes)
            rows.append((n, t[0], nbytes / (t[0] * 1e-3) / 1e9))
            del inp, dev
            torch.cuda.empty_cache()
            n *= 4
        expo = [round(np.log(rows[i + 1][1] / rows[i][1]) / np.log(rows[i + 1][0] / rows[i][0]), 3)
                for i in range(len(rows) - 1)]
        print(json.dumps({"metric": "decode step time versus cache length (1 GPU)", "workload": w.name,
                          "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "d": w.d, "dtype": w.dtype,
                          "points": [{"n": r[0], "ms": round(r[1], 5), "GB/s": round(r[2], 1)} for r in rows],
                          "local_exponent": expo}), flush=True)
        return 0

    inp, dev, call, O, L = setup()
    t = _time_calls(call, args.steps, args.warmup, hip, torch)
    B = len(inp.lens)
    nbytes = workloads.decode_bytes(inp.lens, w.Hq, w.Hkv, w.d, w.elem_bytes)
    gbs = nbytes / (t[0] * 1e-3) / 1e9
    rec = {
        "metric": "decode step HBM bandwidth (1 GPU)", "value": round(gbs, 1), "unit": "GB/s",
        "higher_is_better": True, "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(t[1], 5), "device_ms_per_step": round(t[0], 5), "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "tokens_per_s": round(B / (t[0] * 1e-3), 1),
        "config": {"workload": w.name, "B": B, "Hq": w.Hq, "Hkv": w.Hkv, "n": w.n, "d": w.d,
                   "ragged": w.ragged, "alg_bytes": nbytes},
        "roofline": {"kernel": "attn_decode (whole call)", "bound": "hbm", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None},
    }
    if not args.no_cpu_baseline:
        from oracle import decode as dec
        torch.cuda.synchronize()
        bs = list(range(min(B, 2)))
        c0 = time.perf_counter()
        ref = dec.decode_step(inp.q[bs], inp.k_cache[bs], inp.v_cache[bs], inp.lens[bs], w.scale,
                              inp.k_new[bs], inp.v_new[bs])
        t_cpu = time.perf_counter() - c0
        import oracle
        rec["max_rel_err"] = {
            "O": float(f"{oracle.max_rel_err(O[bs].float().cpu().numpy(), ref['O']):.3e}"),
            "L": float(f"{oracle.max_rel_err(L[bs].cpu().numpy(), ref['L']):.3e}")}
        sample_bytes = workloads.decode_bytes(inp.lens[bs], w.Hq, w.Hkv, w.d, w.elem_bytes)
        rec["cpu_baseline"] = {"value": round(sample_bytes / t_cpu / 1e9, 3), "unit": "GB/s", "cores": cpu_threads(),
                               "kind": "oracle",
                               "sample": f"{len(bs)} of {B} sequences, float64 NumPy decode step, {t_cpu:.1f} s"}
    print(json.dumps(rec), flush=True)
    return 0


def measured_traffic_kernel(workload: str, kernel: str, prefix: str = "hbm_traffic"):
    """fetch/write bytes per launch of `kernel` from a committed summary, or None."""
    from paper_2609_33916_amd import profiling
    rec = profiling.read_traffic(os.path.join(ROOT, "profiles", f"{prefix}_{workload}.md"))
    if not rec or rec.get("source_hash") != profiling.source_hash():
        return None
    return rec["kernels"].get(kernel)




def oracle_sample(w, inp, out, budget_s: float):
    """The float64 oracle on whole heads of the workload, in a fixed order,
    until about `budget_s` seconds of host work: returns the max relative
    error of every output over those heads, the CPU baseline record and a
    description of the sample."""
    import oracle
    from oracle import naive
    O, L, dQ, dK, dV = out
    B, H = w.B, w.H
    threads = cpu_threads()
    order = [(B - 1, (H // 2 + 3) % H), (0, 0), (B // 2, H - 1), (B - 1, 1), (0, H // 3),
             (B // 2, 2 * H // 3 % H), (B - 1, H - 2 if H > 1 else 0), (0, H - 1)]
    order += [(b, h) for b in range(B) for h in range(H)]
    heads, errs, t_cpu = [], {}, 0.0
    print(f"[bench] {w.name}: float64 oracle with {threads} threads", file=sys.stderr, flush=True)
    for (b, h) in order:
        if (b, h) in heads:
            continue
        c0 = time.perf_counter()
        ref = naive.attention_head(inp.q[b, h], inp.k[b, h], inp.v[b, h], inp.do[b, h], w.scale, w.causal)
        t_cpu += time.perf_counter() - c0
        heads.append((b, h))
        got = {"O": O[b, h], "L": L[b, h], "dQ": dQ[b, h], "dK": dK[b, h], "dV": dV[b, h]}
        for key, t in got.items():
            errs[key] = max(errs.get(key, 0.0), oracle.max_rel_err(t.float().cpu().numpy(), ref[key]))
        if t_cpu >= budget_s or len(heads) >= B * H:
            break
    head_flops = workloads.alg_flops(1, 1, w.n, w.d, w.causal)
    nh = len(heads)
    shown = heads if nh <= 8 else heads[:8] + ["..."]
    sample = f"{nh} of {B * H} heads {shown}, all outputs, vs float64 oracle"
    base = {
        "value": round(nh * head_flops / t_cpu / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"{nh} of {B * H} heads (n={w.n}, d={w.d}), float64 NumPy naive fwd+bwd "
                  f"with explicit n x n S and P, {t_cpu:.2f} s on {cpu_model()} ({threads} BLAS "
                  f"threads)" + (f"; all {B * H} heads extrapolated: {t_cpu / nh * B * H:.1f} s"
                                 if nh < B * H else ""),
    }
    return {key: float(f"{val:.3e}") for key, val in errs.items()}, base, sample


def measure_workload(w, args, hip, torch, attn, with_oracle: bool) -> dict:
    """One workload timed like the headline one (warmup, then `steps`
    back-to-back attn_fwd_bwd calls with HIP events around every kernel),
    then checked against the oracle on a bounded sample of whole heads."""
    print(f"[bench] workload {w.name}: generating seeded inputs", file=sys.stderr, flush=True)
    inp = workloads.generate(w)
    dev = workloads.to_torch(inp, "cuda")
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    B, H, n, d = q.shape
    out = (torch.empty_like(q), torch.empty((B, H, n), dtype=torch.float32, device=q.device),
           torch.empty_like(q), torch.empty_like(q), torch.empty_like(q))
    ws = torch.empty(attn.attn_workspace_bytes(B, H, n, d), dtype=torch.uint8, device=q.device)
    wall_ms, step_dev, kstats = time_fwd_bwd(w, q, k, v, do, out, ws, args, hip, torch, attn)
    f_alg = workloads.alg_flops(B, H, n, d, w.causal)
    peak = PEAK_TFLOPS[w.dtype]
    dev_ms = statistics.median(step_dev)
    rec = {
        "ms_per_step": round(wall_ms, 4),
        "device_ms_per_step": round(dev_ms, 4),
        "tflops": round(f_alg / (wall_ms * 1e-3) / 1e12, 3),
        "tflops_device_median": round(f_alg / (dev_ms * 1e-3) / 1e12, 3),
        "frac_of_peak": round(f_alg / (wall_ms * 1e-3) / 1e12 / peak, 4),
        "peak": peak,
        "dtype": w.dtype,
        "config": {"B": B, "H": H, "n": n, "d": d, "causal": w.causal, "alg_flops": f_alg},
        "kernels": kstats,
    }
    if with_oracle:
        budget = 10.0 if w.heads * w.n * w.n > 1 << 32 else 3.0
        errs, base, sample = oracle_sample(w, inp, out, budget_s=budget)
        rec["max_rel_err"] = errs
        rec["max_rel_err_bound"] = 1e-4 if w.dtype == "f32" else 2e-2
        rec["max_rel_err_sample"] = sample
        rec["cpu_baseline"] = base
    return rec


def time_fwd_bwd(w, q, k, v, do, out, ws, args, hip, torch, attn):
    """(wall ms per call, device ms of every call, per-kernel statistics)
    over `args.steps` back-to-back calls after `args.warmup` untimed ones.
    The wall time brackets all calls between two device synchronisations;
    the device times come from HIP events recorded between the kernels."""
    B, H, n, d = q.shape
    evs = [[hip.create() for _ in range(4)] for _ in range(args.steps)]
    for _ in range(args.warmup):
        attn.attn_fwd_bwd(q, k, v, do, scale=w.scale, causal=w.causal, out=out, workspace=ws)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        attn.attn_fwd_bwd_timed(q, k, v, do, evs[i], scale=w.scale, causal=w.causal, out=out,
                                workspace=ws)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    per_kernel = {name: [hip.elapsed_ms(e[j], e[j + 1]) for e in evs] for j, name in enumerate(KERNELS)}
    step_dev = [hip.elapsed_ms(e[0], e[3]) for e in evs]
    for e in evs:
        for x in e:
            hip.destroy(x)
    pairs = workloads.causal_pairs(n, w.causal) * B * H
    kstats = {}
    for name in KERNELS:
        mean_ms = statistics.fmean(per_kernel[name])
        kstats[name] = {
            "mean_ms": round(mean_ms, 4),
            "alg_tflops": round(ALG_FLOPS_PER_PAIR_D[name] * d * pairs / (mean_ms * 1e-3) / 1e12, 2),
            "mfma_exec_tflops": round(EXEC_FLOPS_PER_PAIR_D[name] * d * pairs / (mean_ms * 1e-3) / 1e12, 2),
        }
    return wall_ms, step_dev, kstats


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=sorted(workloads.WORKLOADS))
    ap.add_argument("--decode-workload", default="dec_b16_hq64_hkv8_n8192_d128_bf16",
                    choices=sorted(workloads.DECODE_WORKLOADS))
    ap.add_argument("--decode-sweep", action="store_true",
                    help="with --mode decode: time cache lengths 1024 ... 2^20 of the workload's shape")
    ap.add_argument("--mode", default="fwd_bwd", choices=("fwd_bwd", "fwd", "bwd", "naive", "atomic", "decode"),
                    help="entry point timed: attn_fwd_bwd (default), attn_fwd, attn_bwd, or the "
                         "fused path against the naive materialising path")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip the host oracle (and with it the sampled-head error check)")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="measure only --workload (by default the other four workloads follow it, "
                         "reported under other_workloads)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="instead of the benchmark, run 5 device-to-device copies of MIB MiB "
                         "(reference kernel of known traffic for the HBM byte counters)")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): every (batch, head) is "
              "independent, so a multi-GPU run would shard heads with no communication; "
              "run with --gpus 1.", file=sys.stderr)
        return 2

    import torch
    import paper_2609_33916_amd as attn

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if args.copy_calibration:
        nbytes = args.copy_calibration << 20
        src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": nbytes, "copies": 5}), flush=True)
        return 0
    if args.mode == "decode":
        return bench_decode(args, torch, attn, HipEvents())
    w = workloads.WORKLOADS[args.workload]
    print(f"[bench] workload {w.name}: generating seeded inputs", file=sys.stderr, flush=True)
    inp = workloads.generate(w)
    dev = workloads.to_torch(inp, "cuda")
    q, k, v, do = dev["q"], dev["k"], dev["v"], dev["do"]
    B, H, n, d = q.shape
    O = torch.empty_like(q)
    L = torch.empty((B, H, n), dtype=torch.float32, device=q.device)
    dQ, dK, dV = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    ws = torch.empty(attn.attn_workspace_bytes(B, H, n, d), dtype=torch.uint8, device=q.device)
    out = (O, L, dQ, dK, dV)

    hip = HipEvents()
    if args.mode == "naive":
        return bench_naive(args, w, inp, dev, out, ws, hip, torch, attn)
    if args.mode == "atomic":
        return bench_atomic(args, w, inp, dev, out, ws, hip, torch, attn)
    if args.mode != "fwd_bwd":
        return bench_entry(args, w, inp, dev, out, ws, hip, torch, attn)
    print(f"[bench] warmup {args.warmup}, timing {args.steps} steps", file=sys.stderr, flush=True)
    wall_ms, step_dev, kstats = time_fwd_bwd(w, q, k, v, do, out, ws, args, hip, torch, attn)
    pairs = workloads.causal_pairs(n, w.causal) * B * H
    f_alg = workloads.alg_flops(B, H, n, d, w.causal)
    value = f_alg / (wall_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    dom = max(KERNELS, key=lambda nme: kstats[nme]["mean_ms"])
    dom_alg_flops = ALG_FLOPS_PER_PAIR_D[dom] * d * pairs
    achieved = dom_alg_flops / (kstats[dom]["mean_ms"] * 1e-3) / 1e12

    record = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 4),
        "device_ms_per_step": round(statistics.median(step_dev), 4),
        "timing": ("value and ms_per_step: wall clock over the timed calls (two device synchronisations "
                   "around them) divided by steps; device_ms_per_step: median of the per-call HIP event "
                   "time on the launch stream"),
        "tflops_device_median": round(f_alg / (statistics.median(step_dev) * 1e-3) / 1e12, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "pct_of_peak": round(100.0 * value / peak, 2),
        "config": {"workload": w.name, "B": B, "H": H, "n": n, "d": d, "causal": w.causal,
                   "dtype": w.dtype, "scale": w.scale, "alg_flops": f_alg,
                   "parallelism": "single GPU, one workgroup per (head, tile)"},
        "kernels": kstats,
        "roofline": {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(w.name, dom)},
    }

    if not args.no_cpu_baseline:
        errs, base, sample = oracle_sample(w, inp, out, budget_s=10.0)
        record["max_rel_err"] = errs
        record["max_rel_err_sample"] = sample
        record["cpu_baseline"] = base
    if not args.no_other_workloads:
        del dev, q, k, v, do, out, O, L, dQ, dK, dV, ws, inp
        torch.cuda.empty_cache()
        # the other workloads of the table, each timed and checked like the headline one
        record["other_workloads"] = {
            other.name: measure_workload(other, args, hip, torch, attn, with_oracle=not args.no_cpu_baseline)
            for other in workloads.WORKLOADS.values() if other.name != w.name}
    print(json.dumps(record), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
