"""Summaries of rocprofv3 CSV output (``--output-format csv``) as the markdown
tables kept under ``profiles/``: kernel statistics, HBM traffic from the
FETCH_SIZE / WRITE_SIZE counters scaled by a device copy of known size, and
the host-to-device copies of a memory-copy trace.

    python -m paper_2607_24787_amd.profsum kernels TRACE_DIR
    python -m paper_2607_24787_amd.profsum traffic FETCH_DIR WRITE_DIR CAL_FETCH_DIR CAL_WRITE_DIR KERNEL \
        [--bytes ALGORITHMIC_BYTES_PER_LAUNCH]
    python -m paper_2607_24787_amd.profsum copies TRACE_DIR --blob BYTES [--overlap-kernel h2d_copy_kernel]
    python -m paper_2607_24787_amd.profsum overlap TRACE_DIR KERNEL [KERNEL ...]

Each reads the ``run_*.csv`` files rocprofv3 writes with ``-o run`` and prints
markdown.  Measurement tooling: not part of the decode path.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import statistics
from collections import defaultdict

CAL_BYTES = 256 << 20  # bench.py --copy-probe: a 256 MiB device-to-device copy


def _rows(d, name):
    with open(os.path.join(d, name)) as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    name = name.replace("spp::(anonymous namespace)::", "").replace("void ", "")
    return name.split("(")[0] if "(" in name else name


def kernels(trace_dir: str) -> str:
    rows = _rows(trace_dir, "run_kernel_stats.csv")
    out = ["| kernel | calls | avg µs | min µs | max µs | share % |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out)


def _counter(d):
    """kernel name -> (dispatches, average counter value in KiB)."""
    acc = defaultdict(list)
    for r in _rows(d, "run_counter_collection.csv"):
        acc[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: (len(v), statistics.fmean(v)) for k, v in acc.items()}


def traffic(fetch_dir, write_dir, cal_fetch_dir, cal_write_dir, kernel, algorithmic=None, source=None) -> str:
    f, w = _counter(fetch_dir), _counter(write_dir)
    cf, cw = _counter(cal_fetch_dir), _counter(cal_write_dir)
    cal = next(k for k in cf if "copyBuffer" in k)
    s_f = CAL_BYTES / 1024 / cf[cal][1]
    s_w = CAL_BYTES / 1024 / cw[cal][1]
    out = [f"calibration (256 MiB = {CAL_BYTES // 1024} KiB device copy, `{cal}`): FETCH_SIZE "
           f"{cf[cal][1]:.0f} KiB/dispatch -> scale {s_f:.3f}; WRITE_SIZE {cw[cal][1]:.0f} KiB/dispatch -> "
           f"scale {s_w:.3f}", "",
           "| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | scaled HBM KiB (fetch×s_f + write×s_w) |",
           "|---|---|---|---|---|"]
    for k in sorted(set(f) | set(w)):
        fv, wv = f.get(k, (0, 0.0))[1], w.get(k, (0, 0.0))[1]
        out.append(f"| `{k}` | {max(f.get(k, (0,))[0], w.get(k, (0,))[0])} | {fv:.1f} | {wv:.1f} | "
                   f"{fv * s_f + wv * s_w:.0f} |")
    match = [k for k in f if k.startswith(kernel)]
    if match:
        k = match[0]
        rd, wr = f[k][1] * s_f * 1024, w.get(k, (0, 0.0))[1] * s_w * 1024
        out += ["", f"`{k}`: {rd:,.0f} B read + {wr:,.0f} B written per launch."]
        if algorithmic:
            out.append(f"Algorithmic bytes per launch {algorithmic:,}: read / algorithmic = {rd / algorithmic:.3f}.")
        out += ["", f"traffic_bytes_per_launch: {int(round(rd + wr))}"]
        if source:
            with open(source, "rb") as fh:
                out.append(f"kernel_source_sha256_16: {hashlib.sha256(fh.read()).hexdigest()[:16]}")
    return "\n".join(out)


def copies(trace_dir: str, blob: int, overlap_kernel: str = "h2d_copy_kernel", after_kernel: str = "ffn_") -> str:
    """DMA host-to-device copies of a memory-copy trace, each `blob` bytes: the
    ones issued after the first kernel whose name contains `after_kernel` (the
    decode's prefetches) with their rate, and how much of each copy's time an
    `overlap_kernel` launch (on-demand loads by copy kernel) shared the link."""
    cps = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
           for r in _rows(trace_dir, "run_memory_copy_trace.csv") if r["Direction"].endswith("HOST_TO_DEVICE")]
    ks = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
          for r in _rows(trace_dir, "run_kernel_trace.csv")]
    t0 = min(s for s, _, n in ks if after_kernel in n)
    dec = [c for c in cps if c[0] >= t0]
    early = [c for c in cps if c[0] < t0]
    ovk = [(s, e) for s, e, n in ks if overlap_kernel in n and s >= t0]

    def gbs(c):
        return blob / (c[1] - c[0])

    def shared(c):
        return sum(max(0, min(c[1], e) - max(c[0], s)) for s, e in ovk) / (c[1] - c[0])

    out = [f"copies in the trace: {len(cps)} host-to-device ({len(early)} before the decode: resident-slot fills "
           f"and the per-expert cost profile; {len(dec)} during the decode: the prefetches), {blob:,} B each", ""]
    if early:
        med = statistics.median(e - s for s, e in early)
        out.append(f"- before the decode: median {med / 1e3:.1f} µs per copy -> {blob / med:.2f} GB/s")
    if dec:
        d_us = [(e - s) / 1e3 for s, e in dec]
        rates = [gbs(c) for c in dec]
        sh = [shared(c) for c in dec]
        alone = [gbs(c) for c in dec if shared(c) < 0.05]
        mostly = [gbs(c) for c in dec if shared(c) >= 0.5]
        out += [f"- prefetches: {len(dec)}; duration µs mean {statistics.fmean(d_us):.1f}, median "
                f"{statistics.median(d_us):.1f}, min {min(d_us):.1f}, max {max(d_us):.1f}; GB/s per copy median "
                f"{statistics.median(rates):.2f}, max {max(rates):.2f}",
                f"- share of each prefetch's time during which an on-demand copy kernel also used the link: mean "
                f"{statistics.fmean(sh):.3f}",
                f"- prefetches with the link to themselves (<5% shared): {len(alone)}, median "
                f"{statistics.median(alone) if alone else float('nan'):.2f} GB/s",
                f"- prefetches sharing the link for at least half their time: {len(mostly)}, median "
                f"{statistics.median(mostly) if mostly else float('nan'):.2f} GB/s"]
        span = max(e for _, e in dec) - min(s for s, _ in dec)
        busy = sum(e - s for s, e in dec)
        out.append(f"- prefetch copies in flight {100.0 * busy / span:.1f}% of the decode span "
                   f"({busy / 1e3:.0f} of {span / 1e3:.0f} µs); on-demand copy kernels: {len(ovk)} launches, "
                   f"{sum(e - s for s, e in ovk) / 1e3:.0f} µs")
    return "\n".join(out)


def overlap(trace_dir: str, names) -> str:
    """Durations of the kernels whose names contain each of `names`, split by
    whether a host-to-device DMA copy of the memory-copy trace ran during
    them (any overlap) or not."""
    cps = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
                 for r in _rows(trace_dir, "run_memory_copy_trace.csv") if r["Direction"].endswith("HOST_TO_DEVICE"))
    ks = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"]), _short(r["Kernel_Name"]))
          for r in _rows(trace_dir, "run_kernel_trace.csv")]

    def busy(s, e):
        return any(cs < e and ce > s for cs, ce in cps)

    out = ["| kernel | launches with a DMA copy beside them | median µs | launches without | median µs |",
           "|---|---|---|---|---|"]
    for name in names:
        w = [(e - s) / 1e3 for s, e, n in ks if name in n and busy(s, e)]
        wo = [(e - s) / 1e3 for s, e, n in ks if name in n and not busy(s, e)]
        med = lambda v: f"{statistics.median(v):.2f}" if v else "-"
        out.append(f"| `{name}` | {len(w)} | {med(w)} | {len(wo)} | {med(wo)} |")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    k = sub.add_parser("kernels")
    k.add_argument("trace_dir")
    t = sub.add_parser("traffic")
    for a in ("fetch_dir", "write_dir", "cal_fetch_dir", "cal_write_dir", "kernel"):
        t.add_argument(a)
    t.add_argument("--bytes", type=int, default=None)
    t.add_argument("--source", default=None, help="kernel source whose hash marks the counters' validity")
    c = sub.add_parser("copies")
    c.add_argument("trace_dir")
    c.add_argument("--blob", type=int, required=True)
    c.add_argument("--overlap-kernel", default="h2d_copy_kernel")
    o = sub.add_parser("overlap")
    o.add_argument("trace_dir")
    o.add_argument("kernels", nargs="+")
    a = ap.parse_args()
    if a.cmd == "kernels":
        print(kernels(a.trace_dir))
    elif a.cmd == "traffic":
        print(traffic(a.fetch_dir, a.write_dir, a.cal_fetch_dir, a.cal_write_dir, a.kernel, a.bytes, a.source))
    elif a.cmd == "copies":
        print(copies(a.trace_dir, a.blob, a.overlap_kernel))
    else:
        print(overlap(a.trace_dir, a.kernels))


if __name__ == "__main__":
    main()
