"""Text summaries of rocprofv3 CSV output, for the profiles/ folder.

  python -m paper_2508_19078_amd.rocprof_summary stats STATS_CSV --cmd "..." [--top N]
  python -m paper_2508_19078_amd.rocprof_summary traffic --fetch CSV --write CSV \
      --cmd-fetch "..." --cmd-write "..." [--calib-bytes B]

``stats`` reads a ``--kernel-trace --stats`` kernel_stats.csv and prints a table
of the busiest kernels.  ``traffic`` reads two ``--pmc FETCH_SIZE`` /
``--pmc WRITE_SIZE`` counter_collection.csv files of the same bench command
(which ends with a device-to-device copy of ``calib_bytes``), scales each counter
by what it reads for that copy, and prints the HBM bytes per step of the grouped
SwiGLU forward + backward, with a hash of the kernel sources the counters were
taken on (bench.py reports the traffic only while the sources still match).
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os

PKG = os.path.dirname(os.path.abspath(__file__))

# The kernels of moe_grouped_swiglu_fwd + moe_grouped_swiglu_bwd (bf16 path).
FFN_KERNELS = ("k_build_sched", "kb_gate_up", "kb_down", "kb_dh", "kb_dx", "kb_dw_gu", "kb_dw_d")
# Sources those kernels are built from.
FFN_SOURCES = ("csrc/ffn.hip", "csrc/gemm_bf16.hpp", "csrc/gemm.hpp", "csrc/common.hpp")
CALIB_KERNEL = "copyBuffer"


def ffn_source_hash() -> str:
    h = hashlib.sha256()
    for rel in FFN_SOURCES:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(n: str) -> str:
    n = n.replace("fm::(anonymous namespace)::", "").replace("void ", "")
    return n.split("(")[0]


def base_name(n: str) -> str:
    """Kernel name without template arguments (kb_dw_gu<false> -> kb_dw_gu)."""
    return short_name(n).split("<")[0]


def stats_table(path: str, top: int) -> str:
    rows = list(csv.DictReader(open(path)))
    # PyTorch's own kernels (input generation, fills) are left out of the table
    lib = [r for r in rows if not short_name(r["Name"]).startswith("at::")]
    out = ["| kernel | calls | avg µs | total ms | % of all GPU time |", "|---|---|---|---|---|"]
    for r in lib[:top]:
        out.append(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['Percentage']):.1f} |")
    ffn = [r for r in rows if base_name(r["Name"]) in FFN_KERNELS]
    calls = [int(r["Calls"]) for r in ffn if base_name(r["Name"]) == "kb_gate_up"]
    if calls:
        steps = max(calls)
        tot = sum(float(r["TotalDurationNs"]) for r in ffn) / steps / 1e3
        out.append("")
        out.append(f"grouped SwiGLU fwd+bwd kernels per step (sum of averages over {steps} steps): {tot:.1f} µs")
    q8 = [r for r in rows if base_name(r["Name"]) in ("kq_gate_up", "kq_down")]
    if q8:
        layers = max(int(r["Calls"]) for r in q8)
        tot = sum(float(r["TotalDurationNs"]) for r in q8) / layers / 1e3
        out.append("")
        out.append(f"int8-code grouped forward kernels per layer (sum of averages over {layers} layer passes): "
                   f"{tot:.1f} µs")
    return "\n".join(out)


def counter_per_kernel(path: str, counter: str):
    """{kernel: [value per dispatch]} for one counter (KiB for *_SIZE)."""
    per = collections.defaultdict(dict)
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        per[base_name(r["Kernel_Name"])][r["Dispatch_Id"]] = \
            per[base_name(r["Kernel_Name"])].get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    return {k: list(v.values()) for k, v in per.items()}


def operand_bytes(rows: dict):
    """Distinct bytes each grouped-SwiGLU kernel must read and write in one step
    (every operand once, no padding): rows['total'] rows over rows['slots']
    slots with rows, rows['tuning'] rows of rows['tuning_slots'] tuning slots."""
    n, nt, s, st = rows["total"], rows["tuning"], rows["slots"], rows["tuning_slots"]
    d, I, b = rows["d"], rows["I"], rows["bytes"]
    w = d * I * b                      # one matrix of one slot
    return {
        "kb_gate_up": (n * d * b + 2 * s * w, 3 * n * I * b),
        "kb_down": (n * I * b + s * w, n * d * b),
        "kb_dh": (n * d * b + s * w + 2 * n * I * b, 2 * n * I * b),
        "kb_dx": (2 * n * I * b + 2 * s * w, n * d * b),
        "kb_dw_gu": (2 * nt * I * b + nt * d * b, 2 * st * d * I * 4),
        "kb_dw_d": (nt * (d + I) * b, st * d * I * 4),
    }


def traffic(fetch_csv: str, write_csv: str, calib_bytes: int):
    res = {}
    for name, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        per = counter_per_kernel(path, name)
        calib = [v for k, vs in per.items() if CALIB_KERNEL in k for v in vs]
        if not calib:
            raise SystemExit(f"no {CALIB_KERNEL} dispatch in {path}")
        kib = max(calib)
        factor = (calib_bytes / 1024.0) / kib
        steps = len(per.get("kb_gate_up", []))
        raw = sum(sum(per.get(k, [])) for k in FFN_KERNELS) / max(steps, 1)
        res[name] = {"calib_kib": kib, "factor": factor, "steps": steps, "kib_per_step": raw,
                     "bytes_per_step": raw * 1024.0 * factor,
                     "per_kernel_kib": {k: sum(per.get(k, [])) / max(steps, 1) for k in FFN_KERNELS},
                     # the library's other kernels: scaled bytes per dispatch (mean)
                     "other_bytes": {k: sum(vs) / len(vs) * 1024.0 * factor for k, vs in per.items()
                                     if k.startswith("k_") and k not in FFN_KERNELS}}
    return res


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--cmd", required=True)
    s.add_argument("--top", type=int, default=16)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--cmd-fetch", required=True)
    t.add_argument("--cmd-write", required=True)
    t.add_argument("--calib-bytes", type=int, default=256 << 20)
    t.add_argument("--bench-json", help="the bench's JSON line (roofline.rows: operand sizes of the step)")
    a = ap.parse_args()
    if a.what == "stats":
        print(f"command: `{a.cmd}`\n")
        print(stats_table(a.csv, a.top))
        return
    r = traffic(a.fetch, a.write, a.calib_bytes)
    f, w = r["FETCH_SIZE"], r["WRITE_SIZE"]
    print(f"commands:\n- `{a.cmd_fetch}`\n- `{a.cmd_write}`\n")
    print(f"Calibration: a device-to-device copy of {a.calib_bytes} bytes reads FETCH_SIZE "
          f"{f['calib_kib']:.0f} KiB (factor {f['factor']:.4f}) and WRITE_SIZE {w['calib_kib']:.0f} KiB "
          f"(factor {w['factor']:.4f}).\n")
    ops = None
    if a.bench_json:
        import json
        for line in open(a.bench_json):
            if line.startswith("{"):
                ops = operand_bytes(json.loads(line)["roofline"]["rows"])
    print("Per step.  Raw = the counter as read (KiB); scaled = raw x the copy's factor (bytes);"
          " operand = the distinct bytes the kernel must read or write (every operand once);"
          " ratio = scaled / operand.\n")
    print("| kernel | FETCH raw KiB | fetch scaled MB | operand read MB | read ratio | WRITE raw KiB | "
          "write scaled MB | operand write MB | write ratio |")
    print("|---|---|---|---|---|---|---|---|---|")
    for k in FFN_KERNELS:
        fr, wr = f["per_kernel_kib"][k], w["per_kernel_kib"][k]
        fs, ws_ = fr * 1024 * f["factor"], wr * 1024 * w["factor"]
        if ops and k in ops:
            ro, wo = ops[k]
            print(f"| {k} | {fr:.0f} | {fs / 1e6:.1f} | {ro / 1e6:.1f} | {fs / ro:.2f} | {wr:.0f} | {ws_ / 1e6:.1f} | "
                  f"{wo / 1e6:.1f} | {ws_ / wo:.2f} |")
        else:
            print(f"| {k} | {fr:.0f} | {fs / 1e6:.1f} | | | {wr:.0f} | {ws_ / 1e6:.1f} | | |")
    others = sorted(set(f["other_bytes"]) | set(w["other_bytes"]))
    if others:
        print("\nOther kernels of the library, scaled HBM bytes per dispatch (mean over dispatches):\n")
        print("| kernel | fetch MB | write MB |")
        print("|---|---|---|")
        for k in others:
            print(f"| {k} | {f['other_bytes'].get(k, 0) / 1e6:.2f} | {w['other_bytes'].get(k, 0) / 1e6:.2f} |")
    total = f["bytes_per_step"] + w["bytes_per_step"]
    print(f"\nHBM traffic of the grouped SwiGLU fwd+bwd per step (scaled): fetch {f['bytes_per_step']:.4g} B, "
          f"write {w['bytes_per_step']:.4g} B, total {total:.4g} B", end="")
    if ops:
        ro = sum(ops[k][0] for k in ops)
        wo = sum(ops[k][1] for k in ops)
        print(f"; operands {ro:.4g} B read and {wo:.4g} B written ({total / (ro + wo):.2f}x).\n")
    else:
        print(".\n")
    print("```")
    print(f"source_sha256: {ffn_source_hash()}")
    print(f"traffic_bytes: {total:.0f}")
    print("```")


if __name__ == "__main__":
    main()
