#!/usr/bin/env python3
"""HBM traffic of the dominant kernel from rocprofv3 hardware counters.

Two modes:

  python3 pmc_traffic.py copy
      A plain device-to-device copy of 1 GiB (three times): the calibration
      kernel.  Profile it once with `--pmc FETCH_SIZE` and once with
      `--pmc WRITE_SIZE`; each copy dispatch should read and write 1 GiB.

  python3 pmc_traffic.py summarize --copy-fetch D1 --copy-write D2 \\
          --fetch D3 --write D4 --kernel NAME --workload W --out-dir profiles
      Reads the counter output of the four runs (rocprofv3 -d D -o run; the
      sqlite results or CSV), scales the kernel's per-dispatch FETCH_SIZE /
      WRITE_SIZE (KiB) by what the same counters read for the 1 GiB copy,
      and writes profiles/traffic_<W>.json (read by bench.py).
      The JSON records a hash of the GEMM sources: bench.py reports the
      traffic only while the kernel is unchanged since the counters were taken.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 1 << 30
# Sources whose change invalidates a stored traffic figure for the large-M GEMM.
GEMM_SOURCES = ["paper_2609_27547_amd/csrc/gemm.hip", "paper_2609_27547_amd/csrc/kernels.h",
                "paper_2609_27547_amd/csrc/common.h"]


def sources_hash(paths=GEMM_SOURCES) -> str:
    """Hash of the code (comments and blank lines dropped) of the sources."""
    import re
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p)) as f:
            text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        for line in text.splitlines():
            line = re.sub(r"//.*", "", line).strip()
            if line:
                h.update(line.encode() + b"\n")
    return h.hexdigest()[:16]


def _per_dispatch(d: str, counter: str, name_part: str):
    """Counter value (KiB) of every dispatch whose kernel name contains
    name_part, from the rocprofv3 output under d (sqlite or csv)."""
    vals = {}
    dbs = glob.glob(os.path.join(d, "**", "*results.db"), recursive=True)
    for db in dbs:
        import sqlite3
        cur = sqlite3.connect(db).cursor()
        for pid, disp, name, value in cur.execute(
                "select pid, dispatch_id, kernel_name, value from counters_collection where counter_name = ?",
                (counter,)):
            if name_part in name:
                vals[(db, pid, disp)] = float(value)
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter and name_part in r["Kernel_Name"]:
                    vals[(f, r["Process_Id"], r["Dispatch_Id"])] = float(r["Counter_Value"])
    if not dbs and not vals:
        sys.exit(f"no rocprofv3 counter output under {d}")
    return list(vals.values())


def copy_main():
    import torch
    n = COPY_BYTES // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(f"copied {COPY_BYTES} bytes x3", flush=True)


def summarize_main(args):
    cf = _per_dispatch(args.copy_fetch, "FETCH_SIZE", "copyBuffer")
    cw = _per_dispatch(args.copy_write, "WRITE_SIZE", "copyBuffer")
    # the three 1 GiB copy dispatches: their median reading
    copy_fetch_kib, copy_write_kib = sorted(cf)[len(cf) // 2], sorted(cw)[len(cw) // 2]
    f_scale = COPY_BYTES / (copy_fetch_kib * 1024.0)
    w_scale = COPY_BYTES / (copy_write_kib * 1024.0)
    kf = _per_dispatch(args.fetch, "FETCH_SIZE", args.kernel)
    kw = _per_dispatch(args.write, "WRITE_SIZE", args.kernel)
    if not kf or not kw:
        sys.exit(f"no dispatches of {args.kernel}")
    fetch = sum(kf) / len(kf) * 1024.0 * f_scale
    write = sum(kw) / len(kw) * 1024.0 * w_scale
    res = {
        "workload": args.workload,
        "kernel": args.kernel,
        "dispatches": {"fetch_run": len(kf), "write_run": len(kw)},
        "fetch_bytes_per_launch": round(fetch),
        "write_bytes_per_launch": round(write),
        "traffic_bytes_per_launch": round(fetch + write),
        "calibration": {"copy_bytes": COPY_BYTES, "copy_fetch_kib": copy_fetch_kib,
                        "copy_write_kib": copy_write_kib, "fetch_scale": round(f_scale, 4),
                        "write_scale": round(w_scale, 4)},
        "sources_sha": sources_hash(),
        "command": ("cd /tmp && export TMPDIR=/tmp; for C in FETCH_SIZE WRITE_SIZE: "
                    "rocprofv3 --pmc $C --kernel-trace -d <dir_copy_$C> -o run -- python3 <repo>/pmc_traffic.py copy; "
                    f"rocprofv3 --pmc $C --kernel-trace -d <dir_$C> -o run -- python3 <repo>/bench.py --workload "
                    f"{args.workload} --steps 1 --warmup 1 --cpu-sample 0; then pmc_traffic.py summarize"),
    }
    os.makedirs(args.out_dir, exist_ok=True)
    with open(os.path.join(args.out_dir, f"traffic_{args.workload}.json"), "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="mode", required=True)
    sub.add_parser("copy")
    s = sub.add_parser("summarize")
    for k in ["copy-fetch", "copy-write", "fetch", "write", "kernel", "workload"]:
        s.add_argument(f"--{k}", required=True)
    s.add_argument("--out-dir", default=os.path.join(ROOT, "profiles"))
    args = ap.parse_args()
    if args.mode == "copy":
        copy_main()
    else:
        summarize_main(args)


if __name__ == "__main__":
    main()
