"""Turns a rocprofv3 --stats kernel_stats.csv into the markdown summaries kept in this folder.

    python profiles/make_summary.py STATS_CSV OUT_MD "title" "workload note" "command"
"""
import csv
import re
import sys


def main(src, out, title, note, cmd):
    rows = list(csv.DictReader(open(src)))
    lines = [f"# {title}", "", note, "", "Command (on the MI355X box, from /tmp with TMPDIR=/tmp; R = repository root):",
             "", f"    {cmd}", "", "| kernel | calls | total ns | average ns | % | min ns | max ns |",
             "|---|---|---|---|---|---|---|"]
    for r in rows:
        name = r["Name"]
        m = re.search(r"(gemm_kernel<[^(]*>|\w+_kernel|fillBufferAligned)", name)
        short = m.group(1) if m else name[:60]
        short = short.replace("bpk::(anonymous namespace)::", "")
        lines.append(f"| `{short}` | {r['Calls']} | {r['TotalDurationNs']} | {float(r['AverageNs']):.0f} | "
                     f"{float(r['Percentage']):.1f} | {r['MinNs']} | {r['MaxNs']} |")
    open(out, "w").write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main(*sys.argv[1:6])
