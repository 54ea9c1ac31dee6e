"""Summarise rocprofv3 output into the short text reports kept under profiles/.

  python -m paper_2605_31464_amd.rocprof_summary stats STATS_CSV OUT_MD --cmd "..."
      kernel table (calls, average and total duration, share of GPU time) from the
      --kernel-trace --stats summary.
  python -m paper_2605_31464_amd.rocprof_summary traffic FETCH_CSV WRITE_CSV OUT_MD \
      --kernel SUBSTR --copy-bytes N --source FILE --cmd "..."
      HBM bytes per launch of the kernel whose name contains SUBSTR, from one
      FETCH_SIZE run and one WRITE_SIZE run; each counter is scaled by the factor that
      makes a plain device-to-device copy of N bytes (the largest "copy" dispatch in the
      same run) read N and write N bytes.  The report records the sha256 of the kernel
      source so a reader can tell when the figure has gone stale.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib


def _per_dispatch(path):
    """{dispatch_id: (kernel_name, {counter: summed value})}."""
    out = collections.OrderedDict()
    with open(path) as f:
        for r in csv.DictReader(f):
            d = out.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], collections.Counter()])
            d[1][r["Counter_Name"]] += float(r["Counter_Value"])
    return out


def source_sha256(path: str) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def stats(args):
    rows = list(csv.DictReader(open(args.stats_csv)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = [f"# Kernel time: {args.title}", "", f"Command: `{args.cmd}`", "",
             "| kernel | calls | avg ms | total ms | share |", "|---|---|---|---|---|"]
    for r in rows[: args.top]:
        name = r["Name"]
        if len(name) > 110:
            name = name[:107] + "..."
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.3f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.1f} | "
                     f"{100 * float(r['TotalDurationNs']) / total:.1f}% |")
    lines.append("")
    open(args.out_md, "w").write("\n".join(lines) + "\n")


def traffic(args):
    fetch = _per_dispatch(args.fetch_csv)
    write = _per_dispatch(args.write_csv)

    def pick(table, counter, substr):
        return [v[1][counter] for v in table.values() if substr in v[0]]

    def copy_val(table, counter):
        vals = [v[1][counter] for v in table.values() if "copy" in v[0].lower()]
        return max(vals) if vals else None

    kib = 1024.0
    f_k = pick(fetch, "FETCH_SIZE", args.kernel)
    w_k = pick(write, "WRITE_SIZE", args.kernel)
    f_c, w_c = copy_val(fetch, "FETCH_SIZE"), copy_val(write, "WRITE_SIZE")
    if not f_k or not w_k or not f_c or not w_c:
        raise SystemExit("kernel or calibration copy not found in the counter files")
    f_scale = args.copy_bytes / (f_c * kib)
    w_scale = args.copy_bytes / (w_c * kib)
    fb = sum(f_k) / len(f_k) * kib * f_scale
    wb = sum(w_k) / len(w_k) * kib * w_scale
    sha = source_sha256(args.source)
    lines = [f"# HBM traffic: {args.title}", "", f"Commands: `{args.cmd}`", "",
             f"- kernel name contains: `{args.kernel}`; launches: {len(f_k)} (FETCH run), "
             f"{len(w_k)} (WRITE run)",
             f"- raw per launch: FETCH_SIZE {sum(f_k) / len(f_k):.4g} KiB, "
             f"WRITE_SIZE {sum(w_k) / len(w_k):.4g} KiB",
             f"- calibration copy of {args.copy_bytes} bytes read FETCH_SIZE {f_c:.4g} KiB, "
             f"WRITE_SIZE {w_c:.4g} KiB -> scale {f_scale:.4f} (fetch), {w_scale:.4f} (write)",
             f"- scaled HBM bytes per launch: read {fb:.4g}, write {wb:.4g}, total {fb + wb:.4g}",
             "", f"bench-traffic: {fb + wb:.6g} {sha}", ""]
    open(args.out_md, "w").write("\n".join(lines) + "\n")


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    s = sub.add_parser("stats")
    s.add_argument("stats_csv")
    s.add_argument("out_md")
    s.add_argument("--cmd", required=True)
    s.add_argument("--title", default="")
    s.add_argument("--top", type=int, default=20)
    t = sub.add_parser("traffic")
    t.add_argument("fetch_csv")
    t.add_argument("write_csv")
    t.add_argument("out_md")
    t.add_argument("--kernel", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--source", required=True)
    t.add_argument("--cmd", required=True)
    t.add_argument("--title", default="")
    a = ap.parse_args()
    (stats if a.mode == "stats" else traffic)(a)


if __name__ == "__main__":
    main()
