"""Summaries of rocprofv3 output for profiles/ (used by hand after a profiling run).

    python -m paper_2608_26430_amd.prof_summary stats <kernel_stats.csv>
        markdown table of a --kernel-trace --stats run
    python -m paper_2608_26430_amd.prof_summary traffic <fetch counter csv> <write counter csv> \\
        <copy probe MiB> <kernel hash> <workload>
        HBM bytes per launch of the fused kernels from a FETCH_SIZE pass and a WRITE_SIZE pass,
        each scaled by what the same counter reads for the known-size device copy that
        bench.py --copy-probe-mib issued first (the largest __amd_rocclr_copyBuffer dispatch)
"""
import csv
import json
import sys
from collections import defaultdict


def short_name(name: str) -> str:
    name = name.replace("ff::(anonymous namespace)::", "").replace("void ", "")
    if name.startswith("Custom_Cijk"):
        return "hipBLASLt bf16 GEMM (frozen W0, context)"
    return name.split("(")[0][:60]


def table(stats_csv: str) -> str:
    rows = list(csv.DictReader(open(stats_csv)))
    out = ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out)


KERNELS = {"fwd128": "fwd_kernel", "bwd128": "bwd_kernel", "bwd16": "bwd_kernel", "reduce128": "reduce_kernel",
           "fwd_kernel": "fwd_kernel", "bwd_kernel": "bwd_kernel", "dc_reduce": "reduce_kernel"}


def counter_kib(path: str, counter: str):
    """Per dispatch counter values (KiB): {kernel label: [values]}, and the copy probe's values."""
    per = defaultdict(list)
    copies = []
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        v = float(r["Counter_Value"])
        name = r["Kernel_Name"]
        if "__amd_rocclr_copyBuffer" in name:
            copies.append((int(r["Grid_Size"]), v))
            continue
        for key, label in KERNELS.items():
            if f"::{key}" in name or name.startswith(key):
                per[label].append(v)
                break
    big = max(g for g, _ in copies)
    probe = [v for g, v in copies if g == big]
    return per, probe


def traffic(fetch_csv: str, write_csv: str, probe_mib: float, kernel_hash: str, workload: str) -> dict:
    probe_kib = probe_mib * 1024.0
    f_per, f_probe = counter_kib(fetch_csv, "FETCH_SIZE")
    w_per, w_probe = counter_kib(write_csv, "WRITE_SIZE")
    f_scale = probe_kib / (sum(f_probe) / len(f_probe))
    w_scale = probe_kib / (sum(w_probe) / len(w_probe))
    out = {"workload": workload, "kernel_hash": kernel_hash, "copy_probe_mib": probe_mib,
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "bytes_per_launch": {}, "fetch_bytes_per_launch": {}, "write_bytes_per_launch": {}}
    for label in sorted(set(f_per) & set(w_per)):
        fb = 1024.0 * f_scale * sum(f_per[label]) / len(f_per[label])
        wb = 1024.0 * w_scale * sum(w_per[label]) / len(w_per[label])
        out["fetch_bytes_per_launch"][label] = round(fb)
        out["write_bytes_per_launch"][label] = round(wb)
        out["bytes_per_launch"][label] = round(fb + wb)
    return out


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        print(table(sys.argv[2]))
    elif sys.argv[1] == "traffic":
        print(json.dumps(traffic(sys.argv[2], sys.argv[3], float(sys.argv[4]), sys.argv[5], sys.argv[6]), indent=1))
    else:
        raise SystemExit(__doc__)
