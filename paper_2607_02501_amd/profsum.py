"""Summarise a rocprofv3 --stats kernel CSV into a short markdown table.

    python -m paper_2607_02501_amd.profsum <kernel_stats.csv> "<command>" [title]
"""
import csv
import re
import sys


def short(name: str) -> str:
    m = re.search(r"(\w+_kernel)<([^>]*)>", name)
    return f"{m.group(1)}<{m.group(2)}>" if m else name[:70]


def main():
    path, cmd = sys.argv[1], sys.argv[2]
    title = sys.argv[3] if len(sys.argv) > 3 else "rocprofv3 kernel statistics"
    rows = list(csv.DictReader(open(path)))
    print(f"# {title}\n\nCommand:\n\n```\n{cmd}\n```\n")
    print("| kernel | calls | avg (us) | min (us) | max (us) | share of GPU time |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        print(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.3f} | "
              f"{float(r['MinNs']) / 1e3:.3f} | {float(r['MaxNs']) / 1e3:.3f} | {float(r['Percentage']):.1f}% |")


if __name__ == "__main__":
    main()
