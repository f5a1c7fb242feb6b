"""Summarise a rocprofv3 --stats kernel table (and the bench line of the same run) as markdown.

    python profiles/make_summary.py <kernel_stats.csv> <bench.json> <title> <command> > profiles/<name>.md
"""
import csv
import json
import sys


def main(stats, bench, title, command):
    rows = list(csv.DictReader(open(stats)))
    b = json.load(open(bench))
    out = [f"# {title}", "", "Command (repo root, one MI355X):", "", f"    {command}", "",
           "Per-kernel statistics from rocprofv3 `--stats`:", "",
           "| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "")
        name = name.split("(")[0].replace("void ", "").replace("rubiconv::", "")
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.1f}% |")
    out += ["", "bench.py's live HIP-event timing of the library's stages in the same kind of run "
            "(avg us per step; a stage may be several launches): " +
            ", ".join(f"{k} {v['avg_us']:.1f}" for k, v in b["kernels"].items()), "",
            f"Step: {b['ms_per_step']} ms, {b['value']} Mtokens*channels/s, whole-step HBM roofline "
            f"fraction {b['hbm_roofline_frac_step']}; dominant stage {b['roofline']['kernel']} at "
            f"{b['roofline']['achieved']} GB/s of compulsory traffic ({b['roofline']['frac']} of 8 TB/s)."]
    print("\n".join(out))


if __name__ == "__main__":
    main(*sys.argv[1:5])
