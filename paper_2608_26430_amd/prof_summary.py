"""Turn a rocprofv3 kernel-stats CSV into a short markdown table (used for profiles/)."""
import csv
import sys


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


if __name__ == "__main__":
    print(table(sys.argv[1]))
