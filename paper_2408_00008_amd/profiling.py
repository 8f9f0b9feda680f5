"""Summaries of rocprofv3 output for the MoE kernels.

    python -m paper_2408_00008_amd.profiling stats  STATS.csv  --title T --command C  > x.md
    python -m paper_2408_00008_amd.profiling traffic --fetch F.csv --write W.csv \\
        --calib-fetch CF.csv --calib-write CW.csv --calib-bytes N \\
        --match stream_kernel<true --kernel expert_up_stream --workload decode_t64 \\
        --source paper_2408_00008_amd/csrc/expert_stream.hip --out profiles/traffic_....json

`stats` turns a `--kernel-trace --stats` CSV into a markdown table.
`traffic` turns two `--pmc FETCH_SIZE` / `--pmc WRITE_SIZE` runs (KiB per
dispatch) into HBM bytes per launch of one kernel, scaled by what the same
counters read for a plain device copy of a known size (read N, write N), and
records the sha256 of the kernel's source so that stale counts are not used.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys


def _rows(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def short_name(n: str) -> str:
    n = n.replace("moe::(anonymous namespace)::", "")
    if n.startswith("void "):
        n = n[5:]
    return n.split("(")[0] if "(" in n and not n.startswith("at::") else n[:90]


def stats_md(path, title, command):
    rows = _rows(path)
    out = [f"# {title}", "", "Command:", "", f"    {command}", "",
           "| kernel | calls | avg us | min us | max us | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{short_name(r['Name'])[:90]}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                   f"{float(r['Percentage']):.1f}% |")
    return "\n".join(out) + "\n"


def counter_per_dispatch(path, counter, match):
    vals = [float(r["Counter_Value"]) for r in _rows(path)
            if r["Counter_Name"] == counter and match in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no {counter} rows for kernels matching {match!r} in {path}")
    return sum(vals) / len(vals), len(vals)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    for a in ("fetch", "write", "calib_fetch", "calib_write", "match", "kernel", "workload",
              "source", "out"):
        t.add_argument("--" + a.replace("_", "-"), required=True)
    t.add_argument("--calib-bytes", type=int, required=True)
    t.add_argument("--calib-match", default="copy")
    t.add_argument("--command", default="")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        sys.stdout.write(stats_md(a.csv, a.title, a.command))
        return
    fk, nf = counter_per_dispatch(a.fetch, "FETCH_SIZE", a.match)
    wk, nw = counter_per_dispatch(a.write, "WRITE_SIZE", a.match)
    cfk, _ = counter_per_dispatch(a.calib_fetch, "FETCH_SIZE", a.calib_match)
    cwk, _ = counter_per_dispatch(a.calib_write, "WRITE_SIZE", a.calib_match)
    f_scale = a.calib_bytes / (cfk * 1024.0)
    w_scale = a.calib_bytes / (cwk * 1024.0)
    fetch_b = fk * 1024.0 * f_scale
    write_b = wk * 1024.0 * w_scale
    with open(a.source, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()[:16]
    rec = {"kernel": a.kernel, "workload": a.workload, "match": a.match,
           "fetch_kib_per_dispatch": fk, "write_kib_per_dispatch": wk, "dispatches": [nf, nw],
           "copy_calibration": {"bytes": a.calib_bytes, "fetch_kib": cfk, "write_kib": cwk,
                                "fetch_scale": f_scale, "write_scale": w_scale},
           "hbm_read_bytes_per_launch": fetch_b, "hbm_write_bytes_per_launch": write_b,
           "hbm_bytes_per_launch": fetch_b + write_b,
           "source": a.source, "source_sha256_16": sha, "command": a.command}
    os.makedirs(os.path.dirname(a.out) or ".", exist_ok=True)
    with open(a.out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
