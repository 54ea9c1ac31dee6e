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
  python -m paper_2605_31464_amd.rocprof_summary counters MFMA_CSV FETCH_CSV WRITE_CSV OUT_MD \
      --copy-bytes N --cmd "..."
      per-phase table from three --pmc runs of the same program: MFMA work and busy
      cycles (SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE) for
      the MFMA kernels, copy-calibrated FETCH_SIZE + WRITE_SIZE bytes for the rest;
      durations from the dispatch timestamps of the same runs.
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


# Kernel groups of a scoring step: (label, name substring, kind).
PHASES = [
    ("gate/up GEMM (SwiGLU)", "gemm_bf16_kernel<256, 256, 32, 128, 64, 4, (surr::Epi)2", "mfma"),
    ("O and down GEMMs (fp32 residual add)", "gemm_bf16_kernel<256, 256, 32, 128, 64, 4, (surr::Epi)1", "mfma"),
    ("QKV GEMM (RoPE, V^T)", "gemm_bf16_kernel<256, 256, 32, 128, 64, 4, (surr::Epi)4", "mfma"),
    ("prefill attention", "attn_bf16_kernel<128, false>", "mfma"),
    ("RMSNorm", "rmsnorm_reg_kernel<true, 16, false>", "hbm"),
    ("embedding gather", "embed_kernel<true>", "hbm"),
    ("LM head (last rows)", "gemm_bf16_kernel<128, 128, 32, 64, 64, 4, (surr::Epi)3", "hbm"),
    ("verdict log-sum-exp", "lse_verdict_kernel", "hbm"),
]
N_XCD, SIMD_PER_XCD = 8, 128      # MI355X: 8 XCDs of 32 CUs x 4 SIMDs
MOP_FLOP = 512.0                  # SQ_INSTS_VALU_MFMA_MOPS_* counts units of 512 FLOP
PEAK_BF16_TFLOPS, PEAK_HBM_GBS = 2500.0, 8000.0


def _dispatches(path):
    """[(kernel_name, duration_ns, {counter: value})] in dispatch order."""
    out = collections.OrderedDict()
    with open(path) as f:
        for r in csv.DictReader(f):
            key = int(r["Dispatch_Id"])
            if key not in out:
                out[key] = [r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"]),
                            collections.Counter()]
            out[key][2][r["Counter_Name"]] += float(r["Counter_Value"])
    return list(out.values())


def counters(args):
    mf = _dispatches(args.mfma_csv)
    fe = _dispatches(args.fetch_csv)
    wr = _dispatches(args.write_csv)

    def copy_val(table, counter):
        vals = [d[2][counter] for d in table if "copy" in d[0].lower()]
        return max(vals) if vals else None

    kib = 1024.0
    f_scale = args.copy_bytes / (copy_val(fe, "FETCH_SIZE") * kib)
    w_scale = args.copy_bytes / (copy_val(wr, "WRITE_SIZE") * kib)
    lines = [f"# Counters per phase: {args.title}", "", f"Commands: `{args.cmd}`", "",
             "MFMA kernels: FLOP = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 per launch over its duration "
             f"(peak {PEAK_BF16_TFLOPS:.0f} TFLOP/s dense bf16); MFMA busy = "
             "SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x 128 SIMDs per XCD); clock = "
             "GRBM_GUI_ACTIVE / (8 XCDs x duration).  Memory kernels: (FETCH_SIZE + WRITE_SIZE) "
             f"per launch, scaled by a {args.copy_bytes}-byte device copy in the same runs "
             f"(x{f_scale:.3f} fetch, x{w_scale:.3f} write), over the launch's duration "
             f"(peak {PEAK_HBM_GBS:.0f} GB/s).  Launches run one at a time under counter "
             "collection.", "",
             "| phase | launches | avg ms | counter rate | of peak | MFMA busy | clock GHz | HBM GB/s |",
             "|---|---|---|---|---|---|---|---|"]
    for label, sub, kind in PHASES:
        m = [d for d in mf if sub in d[0]]
        f = [d for d in fe if sub in d[0]]
        w = [d for d in wr if sub in d[0]]
        if not m or not f or not w:
            continue
        dur = sum(d[1] for d in m) / len(m)  # ns, from the MFMA run
        gbs = ""
        fb = sum(d[2]["FETCH_SIZE"] for d in f) / len(f) * kib * f_scale
        wb = sum(d[2]["WRITE_SIZE"] for d in w) / len(w) * kib * w_scale
        fdur = sum(d[1] for d in f) / len(f)
        wdur = sum(d[1] for d in w) / len(w)
        gbs = f"{(fb / fdur + wb / wdur):.0f}"
        if kind == "mfma":
            mops = sum(d[2]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] for d in m) / len(m)
            busy = sum(d[2]["SQ_VALU_MFMA_BUSY_CYCLES"] for d in m) / len(m)
            gui = sum(d[2]["GRBM_GUI_ACTIVE"] for d in m) / len(m)
            tf = mops * MOP_FLOP / dur / 1e3
            lines.append(f"| {label} | {len(m)} | {dur / 1e6:.3f} | {tf:.0f} TFLOP/s | "
                         f"{100 * tf / PEAK_BF16_TFLOPS:.1f}% | {100 * busy / (gui * SIMD_PER_XCD):.1f}% | "
                         f"{gui / (N_XCD * dur):.2f} | {gbs} |")
        else:
            rate = float(gbs)
            lines.append(f"| {label} | {len(m)} | {dur / 1e6:.3f} | {rate:.0f} GB/s | "
                         f"{100 * rate / PEAK_HBM_GBS:.1f}% | | | {gbs} |")
    lines.append("")
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
    c = sub.add_parser("counters")
    c.add_argument("mfma_csv")
    c.add_argument("fetch_csv")
    c.add_argument("write_csv")
    c.add_argument("out_md")
    c.add_argument("--copy-bytes", type=int, required=True)
    c.add_argument("--cmd", required=True)
    c.add_argument("--title", default="")
    a = ap.parse_args()
    {"stats": stats, "traffic": traffic, "counters": counters}[a.mode](a)


if __name__ == "__main__":
    main()
