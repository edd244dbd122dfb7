#!/usr/bin/env python3
"""Turns a rocprofv3 `--stats` kernel_stats.csv into the short markdown
summary kept in this folder.  Usage:
  summarize_rocprof.py KERNEL_STATS_CSV "COMMAND THAT PRODUCED IT" [--top N] > summary.md
"""
import csv
import re
import sys


def main():
    path, command = sys.argv[1], sys.argv[2]
    top = int(sys.argv[sys.argv.index("--top") + 1]) if "--top" in sys.argv else 20
    rows = list(csv.DictReader(open(path)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    print("# rocprofv3 kernel statistics\n")
    print("Command (one MI355X; the repository at /root/repo; `cd /tmp && export TMPDIR=/tmp` first):\n")
    print("```\n" + command + "\n```\n")
    print(f"Total kernel time {total / 1e6:.1f} ms over {sum(int(r['Calls']) for r in rows)} launches.\n")
    print("| total ms | % | calls | avg us | min us | max us | kernel |")
    print("|---:|---:|---:|---:|---:|---:|---|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"]))[:top]:
        name = re.sub(r"\(.*", "", r["Name"]).replace("sprk::", "").replace("HIP_vector_type<unsigned int, 4u>", "uint4")
        print(f"| {float(r['TotalDurationNs']) / 1e6:.1f} | {float(r['Percentage']):.2f} | {r['Calls']} | "
              f"{float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"`{name}` |")


if __name__ == "__main__":
    main()
