"""Summaries of rocprofv3 result databases for the ps_mf and ps_lda kernels.

    python -m paper_1410_8043_amd.rocprof_summary stats <dir>
        per-kernel calls, total and average duration from a --kernel-trace --stats run,
        and the average span of the sweep (its kernels of one clock run concurrently on
        two streams: from the first start to the last end);
    python -m paper_1410_8043_amd.rocprof_summary counters <dir> [<dir> ...]
        per-kernel counter values (sum over a dispatch's dimensions) of --pmc runs;
    python -m paper_1410_8043_amd.rocprof_summary derived <dir> [<dir> ...]
        per-kernel figures derived from --pmc runs (average over dispatches): duration in
        cycles (GRBM_GUI_ACTIVE counts every XCD), busy fractions of the texture address and
        data units (one per CU), of the L2 channels and of the matrix cores, the L2 hit rate
        and the average L1-to-L2 read latency -- whichever of them the runs collected;
    python -m paper_1410_8043_amd.rocprof_summary traffic --fetch <dir> --write <dir> \
            --copy-bytes N --out profiles/<name>.json [--kernels k_lda_sweep --step lda \
            --source paper_1410_8043_amd/csrc/ps_lda.hip]
        HBM bytes per clock of the sweep kernels from one FETCH_SIZE and one WRITE_SIZE run,
        scaled by what the same counters read for a plain copy kernel (torch's elementwise
        y = x * 2 over N bytes), written as JSON next to the sha256 of the kernel
        source, so that bench.py reports it only while the kernel is unchanged.

Each input directory is the -d directory of one rocprofv3 run (the *_results.db file
is found below it).
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import json
import os
import sqlite3
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(_HERE, "csrc", "ps_mf.hip")
SWEEP_KERNELS = ("k_dense", "k_cells", "k_units")  # the concurrent kernels of one clock's sweep


def kernel_source_sha256(path: str = KERNEL_SOURCE) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def _db(d: str) -> sqlite3.Connection:
    found = sorted(glob.glob(os.path.join(d, "**", "*results.db"), recursive=True))
    if not found:
        raise FileNotFoundError(f"no rocprofv3 results database under {d}")
    return sqlite3.connect(found[-1])


def short_name(kernel_name: str) -> str:
    name = kernel_name.replace("(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    return name.split("(")[0].strip()


def stats(d: str):
    con = _db(d)
    rows = con.execute("select name, total_calls, total_duration, average, percentage from top_kernels").fetchall()
    # the top_kernels view reports microseconds
    return [(short_name(n), int(c), tot / 1e3, avg / 1e3, pct) for n, c, tot, avg, pct in rows]


def _is_sweep(name: str, kernels=SWEEP_KERNELS) -> bool:
    return any(name.startswith(k) for k in kernels)


def sweep_spans(d: str):
    """Per clock: (span, [duration of each sweep kernel]) in ms.  Every distinct sweep kernel
    (by full name: the two dense passes are different instantiations) runs at most once per
    clock, so its i-th dispatch is taken as clock i."""
    con = _db(d)
    rows = con.execute("select name, start, end from kernels order by start").fetchall()
    per = collections.OrderedDict()
    for name, start, end in rows:
        sn = short_name(name)
        if _is_sweep(sn):
            per.setdefault(sn, []).append((start, end))
    if not per:
        return []
    clocks = min(len(v) for v in per.values())
    out = []
    for i in range(clocks):
        ivs = [v[i] for v in per.values()]
        out.append(((max(e for _, e in ivs) - min(s for s, _ in ivs)) / 1e6, [(e - s) / 1e6 for s, e in ivs]))
    return out


def counters(d: str):
    """{(kernel, counter): [value per dispatch, in dispatch order]}"""
    con = _db(d)
    rows = con.execute("select dispatch_id, kernel_name, counter_name, sum(value) from counters_collection "
                       "group by dispatch_id, counter_name order by dispatch_id").fetchall()
    out = collections.defaultdict(list)
    for _, kname, cname, val in rows:
        out[(kname, cname)].append(val)
    return out


# MI355X: 8 XCDs, 256 CUs (one texture address / data unit each), 16 L2 channels per XCD,
# 4 SIMDs per CU
XCDS, CUS, L2_CHANNELS, SIMDS = 8, 256, 128, 1024


def derived(dirs):
    """{kernel: {figure: value}} from the counters of one or more --pmc runs (each counter
    averaged over the kernel's dispatches)."""
    avg = collections.defaultdict(dict)
    for d in dirs:
        for (k, c), v in counters(d).items():
            avg[short_name(k)][c] = sum(v) / len(v)
    out = {}
    for k, c in avg.items():
        f = {}
        cyc = c.get("GRBM_GUI_ACTIVE")
        if cyc:
            cyc /= XCDS
            f["cycles"] = cyc
            if "TA_TA_BUSY_sum" in c:
                f["ta_busy"] = c["TA_TA_BUSY_sum"] / CUS / cyc
            if "TA_ADDR_STALLED_BY_TC_CYCLES_sum" in c:
                f["ta_stalled_by_l1"] = c["TA_ADDR_STALLED_BY_TC_CYCLES_sum"] / CUS / cyc
            if "TD_TD_BUSY_sum" in c:
                f["td_busy"] = c["TD_TD_BUSY_sum"] / CUS / cyc
            if "TCC_BUSY_sum" in c:
                f["l2_busy"] = c["TCC_BUSY_sum"] / L2_CHANNELS / cyc
            if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
                f["mfma_busy"] = c["SQ_VALU_MFMA_BUSY_CYCLES"] / SIMDS / cyc
        if c.get("TCC_REQ_sum"):
            f["l2_hit"] = c.get("TCC_HIT_sum", 0.0) / c["TCC_REQ_sum"]
            f["l2_requests"] = c["TCC_REQ_sum"]
        if c.get("TCP_TCC_READ_REQ_sum"):
            f["l1_l2_read_latency"] = c.get("TCP_TCC_READ_REQ_LATENCY_sum", 0.0) / c["TCP_TCC_READ_REQ_sum"]
        if c.get("SQ_WAVE_CYCLES"):
            f["wave_wait_frac"] = c.get("SQ_WAIT_INST_ANY", 0.0) / c["SQ_WAVE_CYCLES"]
        for name in ("SQ_INSTS_VALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_MFMA", "SQ_WAVES"):
            if name in c:
                f[name] = c[name]
        out[k] = f
    return out


def _find(cnt, kernel_prefix: str, counter: str):
    for (k, c), v in cnt.items():
        if c == counter and short_name(k).startswith(kernel_prefix):
            return v
    raise KeyError(f"{counter} of {kernel_prefix} not found")


COPY_KERNEL = "MulFunctor"  # torch's elementwise y = x * 2 (reads and writes copy_bytes)


def _copy_value(cnt, counter: str) -> float:
    for (k, c), v in cnt.items():
        if c == counter and COPY_KERNEL in k:
            return max(v)
    raise KeyError(f"{counter} of the calibration copy kernel not found")


def _sweep_values(cnt, counter: str, kernels=SWEEP_KERNELS):
    """[(kernel, [value per dispatch])] of the sweep kernels, one entry per distinct kernel"""
    out = [(short_name(k), v) for (k, c), v in cnt.items() if c == counter and _is_sweep(short_name(k), kernels)]
    if not out:
        raise KeyError(f"{counter} of the sweep kernels not found")
    return out


def traffic(fetch_dir: str, write_dir: str, copy_bytes: int, kernels=SWEEP_KERNELS, per_clock: int = 1,
            source: str = KERNEL_SOURCE):
    """HBM bytes per clock of the sweep (its kernels of one clock summed), calibrated.  Each
    distinct sweep kernel runs per_clock times a clock (the sequential step: once per
    sub-epoch)."""
    f, w = counters(fetch_dir), counters(write_dir)
    copy_f = _copy_value(f, "FETCH_SIZE")
    copy_w = _copy_value(w, "WRITE_SIZE")
    fetch_scale = copy_bytes / (copy_f * 1024.0)
    write_scale = copy_bytes / (copy_w * 1024.0)
    sf, sw = _sweep_values(f, "FETCH_SIZE", kernels), _sweep_values(w, "WRITE_SIZE", kernels)
    clocks = min(len(v) for _, v in sf + sw) // per_clock
    n = clocks * per_clock
    fetch = sum(sum(v[:n]) for _, v in sf) * 1024.0 * fetch_scale / clocks
    write = sum(sum(v[:n]) for _, v in sw) * 1024.0 * write_scale / clocks
    return {
        "kernels": [k for k, _ in sf],
        "clocks": clocks,
        "fetch_bytes_per_clock": fetch,
        "write_bytes_per_clock": write,
        "traffic_bytes_per_clock": fetch + write,
        "copy_calibration": {"bytes": copy_bytes, "fetch_kib": copy_f, "write_kib": copy_w,
                             "fetch_scale": fetch_scale, "write_scale": write_scale},
        "per_launch_fetch_kib": {k: v for k, v in sf},
        "per_launch_write_kib": {k: v for k, v in sw},
        "kernel_source": os.path.basename(source),
        "kernel_source_sha256": kernel_source_sha256(source),
    }


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("dir")
    b = sub.add_parser("counters")
    b.add_argument("dirs", nargs="+")
    e = sub.add_parser("derived")
    e.add_argument("dirs", nargs="+")
    c = sub.add_parser("traffic")
    c.add_argument("--fetch", required=True)
    c.add_argument("--write", required=True)
    c.add_argument("--copy-bytes", type=int, required=True)
    c.add_argument("--out", required=True)
    c.add_argument("--command", default="")
    c.add_argument("--config", default="full")
    c.add_argument("--s", type=int, default=3)
    c.add_argument("--policy", default="lazy")
    c.add_argument("--step", default="rowmean")
    c.add_argument("--kernels", default=",".join(SWEEP_KERNELS), help="comma-separated kernel name prefixes")
    c.add_argument("--per-clock", type=int, default=1, help="dispatches of each kernel per clock")
    c.add_argument("--source", default=KERNEL_SOURCE, help="the kernels' source file (its sha256 is recorded)")
    args = ap.parse_args(argv)
    if args.cmd == "stats":
        for name, calls, tot, avg, pct in stats(args.dir):
            print(f"{calls:6d} calls  total {tot:10.3f} ms  avg {avg:9.4f} ms  {pct:5.1f}%  {name}")
        spans = sweep_spans(args.dir)
        if spans:
            avg = sum(sp for sp, _ in spans) / len(spans)
            print(f"sweep span (first start to last end of the {' / '.join(SWEEP_KERNELS)} kernels of a clock): "
                  f"{len(spans)} clocks, avg {avg:.4f} ms, min {min(sp for sp, _ in spans):.4f} ms, "
                  f"max {max(sp for sp, _ in spans):.4f} ms")
    elif args.cmd == "derived":
        for k, f in sorted(derived(args.dirs).items()):
            print(k)
            for name, v in f.items():
                print(f"    {name:22s} {v:.4g}")
    elif args.cmd == "counters":
        for d in args.dirs:
            for (k, cname), vals in sorted(counters(d).items()):
                print(f"{short_name(k)[:48]:48s} {cname:18s} " + " ".join(f"{v:.5g}" for v in vals[:8]))
    else:
        t = traffic(args.fetch, args.write, args.copy_bytes, tuple(args.kernels.split(",")), args.per_clock,
                    args.source)
        t["command"] = args.command
        t["workload"] = {"config": args.config, "s": args.s, "policy": args.policy}
        if args.step != "rowmean":
            t["workload"]["step"] = args.step
        with open(args.out, "w") as f:
            json.dump(t, f, indent=1)
        print(json.dumps({k: v for k, v in t.items() if not k.startswith("per_launch")}, indent=1))


if __name__ == "__main__":
    sys.exit(main())
