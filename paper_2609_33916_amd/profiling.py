"""Summaries of rocprofv3 output for the attention kernels.

    python -m paper_2609_33916_amd.profiling trace DIR
        kernel-trace statistics (rocprofv3 --kernel-trace --stats
        --output-format csv -d DIR) as a markdown table
    python -m paper_2609_33916_amd.profiling counters DIR [DIR ...]
        per-kernel averages of PMC counter passes (--pmc ... -d DIR)
    python -m paper_2609_33916_amd.profiling traffic --fetch DIR --write DIR
            --cal-fetch DIR --cal-write DIR --copy-mib M
        HBM bytes per dispatch from FETCH_SIZE and WRITE_SIZE passes, each
        scaled by what the same counter reads for a device-to-device copy of
        M MiB (bench.py --copy-calibration M); prints a markdown summary with
        a machine-readable line that bench.py reads back.

The traffic summary records a hash of the kernel sources; bench.py reports
the figure only while the sources still hash the same.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re
import sys
from typing import Dict, List

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
TRAFFIC_TAG = "attn-traffic-json:"


def source_hash() -> str:
    """sha256 over the HIP sources (file names and contents, sorted) and the
    compiler flags of each translation unit."""
    from . import build as _build
    h = hashlib.sha256()
    h.update(repr((_build.HIPCC_FLAGS, sorted(_build.SOURCES.items()))).encode())
    for fn in sorted(os.listdir(CSRC)):
        if fn.endswith((".hip", ".hpp", ".h")):
            h.update(fn.encode())
            with open(os.path.join(CSRC, fn), "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def _template_args(kernel: str):
    """Template arguments of a demangled name ("true"/"false" for the bool
    parameters of a mangled one)."""
    m = re.search(r"<([^<>]*)>", kernel)
    if m:
        return [x.strip() for x in m.group(1).split(",")]
    return ["true" if b == "1" else "false" for b in re.findall(r"Lb([01])E", kernel)]


def _last_template_arg_true(kernel: str) -> bool:
    """Whether the last template argument is `true` (demangled or mangled name)."""
    m = re.search(r"<([^<>]*)>", kernel)
    if m:
        return m.group(1).split(",")[-1].strip() == "true"
    m = re.search(r"Lb([01])EEEvNS_", kernel)
    return bool(m and m.group(1) == "1")


def short_name(kernel: str) -> str:
    """Kernel name without template arguments; the backward kernels of the
    materialising path (template argument MAT = true) get a mat_ prefix, the
    dK/dV kernel of the atomic-dQ form (AQ = true) an atomic_dq_ prefix.
    dkdv16_kernel<D, CAUSAL, NW, BQ, MAT, AQ, KB>; dkdv_kernel and dq_kernel
    end in MAT."""
    k = kernel.replace("void ", "")
    for key in ("decode_append_kernel", "decode_combine_kernel", "decode_kernel",
                "mat_fwd_kernel", "bwd_prep_kernel", "zero_f32_kernel", "dq_finalize_kernel", "fwd_pp_kernel",
                "fwd_kernel",
                "dkdv16_kernel", "dkdv_kernel", "dq_kernel", "copyBuffer", "elementwise"):
        if key in k:
            if key == "dkdv16_kernel":
                args = _template_args(k)
                if len(args) >= 6 and args[5] == "true":
                    return "atomic_dq_" + key
                if len(args) >= 5 and args[4] == "true":
                    return "mat_" + key
                return key
            if key in ("dkdv_kernel", "dq_kernel") and _last_template_arg_true(k):
                return "mat_" + key
            return key
    return k.split("(")[0][:40]


def _csv_rows(d: str, suffix: str) -> List[dict]:
    rows = []
    for f in sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True)):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    return rows


def trace_table(d: str) -> str:
    rows = _csv_rows(d, "_kernel_stats.csv")
    out = ["| kernel | calls | average (us) | min (us) | max (us) | total (ms) | share |",
           "|---|---|---|---|---|---|---|"]
    for r in rows:
        ns = lambda k: float(r[k]) / 1e3
        out.append(f"| {short_name(r['Name'])} | {r['Calls']} | {ns('AverageNs'):.1f} | "
                   f"{ns('MinNs'):.1f} | {ns('MaxNs'):.1f} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['Percentage']):.1f}% |")
    return "\n".join(out)


def counter_means(dirs) -> Dict[str, Dict[str, float]]:
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in dirs:
        for r in _csv_rows(d, "_counter_collection.csv"):
            agg[short_name(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: sum(v) / len(v) for c, v in d.items()} for k, d in agg.items()}


def counters_table(dirs) -> str:
    m = counter_means(dirs)
    names = sorted({c for d in m.values() for c in d})
    out = ["| kernel | " + " | ".join(names) + " |", "|---|" + "---|" * len(names)]
    for k, d in m.items():
        out.append(f"| {k} | " + " | ".join(f"{d[c]:.4g}" if c in d else "" for c in names) + " |")
    # derived figures where the passes allow them
    lines = []
    for k, d in m.items():
        if "GRBM_GUI_ACTIVE" in d and "SQ_VALU_MFMA_BUSY_CYCLES" in d:
            cycles = d["GRBM_GUI_ACTIVE"] / 8.0        # summed over the 8 XCDs
            lines.append(f"- {k}: MFMA busy {d['SQ_VALU_MFMA_BUSY_CYCLES'] / (cycles * 1024):.3f} "
                         f"of SIMD cycles (1024 SIMDs)")
        if "SQ_LDS_BANK_CONFLICT" in d and "SQ_INSTS_LDS" in d:
            lines.append(f"- {k}: LDS bank conflict cycles per LDS instruction "
                         f"{d['SQ_LDS_BANK_CONFLICT'] / max(d['SQ_INSTS_LDS'], 1):.3f}")
    return "\n".join(out + [""] + lines)


def traffic(fetch: str, write: str, cal_fetch: str, cal_write: str, copy_mib: int) -> dict:
    f = counter_means([fetch])
    w = counter_means([write])
    cf = counter_means([cal_fetch])["copyBuffer"]["FETCH_SIZE"]
    cw = counter_means([cal_write])["copyBuffer"]["WRITE_SIZE"]
    copy_kib = copy_mib * 1024.0
    fetch_scale, write_scale = copy_kib / cf, copy_kib / cw
    per = {}
    for k in f:
        if k in ("copyBuffer", "elementwise"):
            continue
        per[k] = {"fetch_bytes": f[k]["FETCH_SIZE"] * 1024 * fetch_scale,
                  "write_bytes": w[k]["WRITE_SIZE"] * 1024 * write_scale}
    return {"source_hash": source_hash(), "fetch_scale": fetch_scale,
            "write_scale": write_scale, "kernels": per}


def read_traffic(path: str):
    """Traffic record from a summary written by `traffic`, or None."""
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        for line in fh:
            if TRAFFIC_TAG in line:
                return json.loads(line.split(TRAFFIC_TAG, 1)[1].strip().rstrip("->").strip())
    return None


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("dir")
    c = sub.add_parser("counters")
    c.add_argument("dirs", nargs="+")
    tr = sub.add_parser("traffic")
    tr.add_argument("--fetch", required=True)
    tr.add_argument("--write", required=True)
    tr.add_argument("--cal-fetch", required=True)
    tr.add_argument("--cal-write", required=True)
    tr.add_argument("--copy-mib", type=int, required=True)
    a = ap.parse_args(argv)
    if a.cmd == "trace":
        print(trace_table(a.dir))
    elif a.cmd == "counters":
        print(counters_table(a.dirs))
    else:
        rec = traffic(a.fetch, a.write, a.cal_fetch, a.cal_write, a.copy_mib)
        print("| kernel | HBM read (MB) | HBM write (MB) |\n|---|---|---|")
        for k, v in rec["kernels"].items():
            print(f"| {k} | {v['fetch_bytes'] / 1e6:.1f} | {v['write_bytes'] / 1e6:.1f} |")
        print(f"\nFETCH_SIZE scale {rec['fetch_scale']:.3f}, WRITE_SIZE scale "
              f"{rec['write_scale']:.3f} (true bytes / counter bytes of a {a.copy_mib} MiB copy)")
        print(f"\n<!-- {TRAFFIC_TAG} {json.dumps(rec)} -->")
    return 0


if __name__ == "__main__":
    sys.exit(main())
