"""Text summaries of rocprofv3 CSV output for the kernels of libherald.so.

    python -m paper_2606_21633_amd.profsum trace DIR [--kernel NAME --last N --skip-last M]
        per-kernel launch statistics from DIR/*kernel_trace.csv; with --kernel,
        also the average duration of N of that kernel's launches, the last N
        before its final M (the denoising phase that bench.py times with HIP
        events, followed by M launches timed one by one).

    python -m paper_2606_21633_amd.profsum traffic --fetch DIR --write DIR
            --copy-fetch DIR --copy-write DIR --copy-bytes B [--read-fetch DIR]
            --kernel NAME --last N --source-sha256 HEX
        FETCH_SIZE and WRITE_SIZE (KiB per dispatch) of the kernel's last N
        dispatches, each scaled by bytes / counter of a plain copy of B bytes
        read and B written, and the resulting HBM bytes per launch. With
        --read-fetch, FETCH_SIZE is scaled by that of a plain read of B bytes
        instead (a kernel that reads and hardly writes counts its reads like
        the read, not like the copy).

Only reads CSV files; nothing here touches the GPU.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import re
import sys


def _short(name: str) -> str:
    m = re.search(r"herald::\(anonymous namespace\)::(\w+)(<[^()]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    m = re.search(r"at::native::[\w:()\s]*?(\w+_kernel)", name)
    return (m.group(1) if m else name)[:60]


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        sys.exit(f"no file matches {pattern}")
    return files[0]


def _trace_rows(d: str):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*kernel_trace.csv")))))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    return rows


def trace(args) -> None:
    rows = _trace_rows(args.dir)
    stats = {}
    for r in rows:
        n = _short(r["Kernel_Name"])
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        stats.setdefault(n, []).append(d)
    print(f"{'kernel':52s} {'calls':>6s} {'avg us':>9s} {'min us':>9s} {'max us':>9s} {'total ms':>9s}")
    for n, v in sorted(stats.items(), key=lambda kv: -sum(kv[1])):
        print(f"{n:52s} {len(v):6d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f} "
              f"{sum(v) / 1e3:9.2f}")
    if args.kernel:
        v = [x for n, x in ((_short(r["Kernel_Name"]),
                             (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
                            for r in rows) if n.startswith(args.kernel)]
        if args.skip_last:
            v = v[:-args.skip_last]
        tail = v[-args.last:] if args.last else v
        print(f"\n{args.kernel}: {len(tail)} launches (the last {args.last} before the final "
              f"{args.skip_last}): avg {sum(tail) / len(tail):.2f} us, "
              f"min {min(tail):.2f} us, max {max(tail):.2f} us")


def _counter(d: str, counter: str, kernel: str, last: int, skip_last: int = 0):
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))))
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        n = _short(r["Kernel_Name"])
        if not n.startswith(kernel):
            continue
        per.setdefault(int(r["Dispatch_Id"]), 0.0)
        per[int(r["Dispatch_Id"])] += float(r["Counter_Value"])
    vals = [per[k] for k in sorted(per)]
    if skip_last:
        vals = vals[:-skip_last]
    if not vals:
        sys.exit(f"no {counter} values for {kernel} in {d}")
    vals = vals[-last:] if last else vals
    return sum(vals) / len(vals), len(vals)


def traffic(args) -> None:
    f_kib, nf = _counter(args.fetch, "FETCH_SIZE", args.kernel, args.last, args.skip_last)
    w_kib, nw = _counter(args.write, "WRITE_SIZE", args.kernel, args.last, args.skip_last)
    cf_kib, _ = _counter(args.copy_fetch, "FETCH_SIZE", args.copy_kernel, 0)
    cw_kib, _ = _counter(args.copy_write, "WRITE_SIZE", args.copy_kernel, 0)
    sfc = args.copy_bytes / (cf_kib * 1024.0)
    sw = args.copy_bytes / (cw_kib * 1024.0)
    sf = sfc
    fetch_b = f_kib * 1024.0 * sf
    write_b = w_kib * 1024.0 * sw
    print(f"{args.kernel}: FETCH_SIZE {f_kib:.1f} KiB/dispatch ({nf} dispatches), "
          f"WRITE_SIZE {w_kib:.1f} KiB/dispatch ({nw} dispatches)")
    print(f"copy calibration ({args.copy_kernel}, {args.copy_bytes} B read and written): "
          f"FETCH_SIZE {cf_kib:.1f} KiB -> factor {sfc:.4f}; WRITE_SIZE {cw_kib:.1f} KiB -> "
          f"factor {sw:.4f}")
    if args.read_fetch:
        rf_kib, _ = _counter(args.read_fetch, "FETCH_SIZE", args.read_kernel, 0)
        sf = args.copy_bytes / (rf_kib * 1024.0)
        print(f"read calibration ({args.read_kernel}, {args.copy_bytes} B read): FETCH_SIZE "
              f"{rf_kib:.1f} KiB -> factor {sf:.4f}, used for FETCH_SIZE")
        fetch_b = f_kib * 1024.0 * sf
    print(f"HBM bytes per launch: fetch {fetch_b:.0f} + write {write_b:.0f} = "
          f"{fetch_b + write_b:.0f}")
    print(f"traffic: source_sha256={args.source_sha256} bytes_per_launch={fetch_b + write_b:.0f} "
          f"fetch={fetch_b:.0f} write={write_b:.0f}")


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(prog="profsum")
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("dir")
    t.add_argument("--kernel", default="")
    t.add_argument("--last", type=int, default=0)
    t.add_argument("--skip-last", type=int, default=0)
    c = sub.add_parser("traffic")
    for k in ("fetch", "write", "copy_fetch", "copy_write"):
        c.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    c.add_argument("--copy-bytes", type=float, required=True)
    c.add_argument("--copy-kernel", default="vectorized_elementwise_kernel")
    c.add_argument("--read-fetch", default="")
    c.add_argument("--read-kernel", default="reduce_kernel")
    c.add_argument("--kernel", required=True)
    c.add_argument("--last", type=int, default=0)
    c.add_argument("--skip-last", type=int, default=0)
    c.add_argument("--source-sha256", default="")
    args = ap.parse_args(argv)
    (trace if args.cmd == "trace" else traffic)(args)


if __name__ == "__main__":
    main()
