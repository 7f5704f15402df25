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

  python3 pmc_traffic.py kstats --dir D --title T --command C --out F.md
      Per-kernel table (calls, total, average, share) of a rocprofv3
      --kernel-trace run, plus family averages of the large-M GEMM (every
      launch, as bench.py's GEMM class counts them), the decode GEMM and the
      attention kernels.

  python3 pmc_traffic.py counters --dir D [--dir D2 ...] --kernel K [--kernel K2 ...]
          --title T --command C --out F.md [--copy-fetch D --copy-write D]
      Per-dispatch averages of every counter found under the run dirs for
      the kernels whose names contain K; MfmaUtil is reported as is (percent
      of the MFMA pipes' cycles busy over the dispatch), FETCH_SIZE and
      WRITE_SIZE (KiB) also in bytes scaled by the 1 GiB copy when its two
      calibration runs are given.
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


def _all_counters(d: str):
    """{(kernel name, counter): [per-dispatch values]} from rocprofv3 output under d."""
    import sqlite3
    out = {}
    for db in glob.glob(os.path.join(d, "**", "*results.db"), recursive=True):
        cur = sqlite3.connect(db).cursor()
        seen = {}
        for pid, disp, name, cname, value in cur.execute(
                "select pid, dispatch_id, kernel_name, counter_name, value from counters_collection"):
            seen[(db, pid, disp, cname)] = (name, cname, float(value))
        for name, cname, value in seen.values():
            out.setdefault((name, cname), []).append(value)
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                out.setdefault((r["Kernel_Name"], r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    return out


def _dispatches(d: str):
    """[(kernel name, duration ns)] of every dispatch in a --kernel-trace run under d."""
    import sqlite3
    rows = []
    for db in glob.glob(os.path.join(d, "**", "*results.db"), recursive=True):
        cur = sqlite3.connect(db).cursor()
        rows += [(n, float(du)) for n, du in cur.execute("select name, duration from kernels")]
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                rows.append((r["Kernel_Name"], float(r["End_Timestamp"]) - float(r["Start_Timestamp"])))
    if not rows:
        sys.exit(f"no kernel trace under {d}")
    return rows


def kstats_main(args):
    rows = _dispatches(args.dir)
    per = {}
    for n, du in rows:
        c, t = per.get(n, (0, 0.0))
        per[n] = (c + 1, t + du)
    total = sum(t for _, t in per.values())
    lines = [f"# {args.title}", "", "Command (repository root on the GPU host; `cd /tmp && export TMPDIR=/tmp` first):",
             "", "```", args.command, "```", "",
             f"Total kernel time {total / 1e6:.1f} ms over {len(rows)} dispatches.", ""]
    fams = [("gemm_bf16_big_kernel (all epilogues: the bench's large-M GEMM class)",
             lambda n: "gemm_bf16_big_kernel" in n),
            ("gemm_bf16_decode_kernel (all epilogues)", lambda n: "gemm_bf16_decode_kernel" in n),
            ("attn_prefill_bf16_kernel", lambda n: "attn_prefill_bf16_kernel" in n),
            ("attn_decode_bf16_kernel", lambda n: "attn_decode" in n)]
    for title, pred in fams:
        c = sum(v[0] for n, v in per.items() if pred(n))
        t = sum(v[1] for n, v in per.items() if pred(n))
        if c:
            lines.append(f"Family `{title}`: {c} dispatches, average {t / c / 1e3:.2f} us, "
                         f"{100 * t / total:.1f} % of kernel time.")
            lines.append("")
    lines += ["| kernel | calls | total (us) | average (us) | % |", "|---|---:|---:|---:|---:|"]
    for n, (c, t) in sorted(per.items(), key=lambda kv: -kv[1][1]):
        if 100 * t / total < 0.01:
            continue
        lines.append(f"| `{_short(n)}` | {c} | {t / 1e3:.0f} | {t / c / 1e3:.2f} | {100 * t / total:.2f} |")
    _write(args.out, lines)


def counters_main(args):
    vals = {}
    for d in args.dir:
        for k, v in _all_counters(d).items():
            vals.setdefault(k, []).extend(v)
    scale = {}
    if args.copy_fetch and args.copy_write:
        cf = sorted(_per_dispatch(args.copy_fetch, "FETCH_SIZE", "copyBuffer"))
        cw = sorted(_per_dispatch(args.copy_write, "WRITE_SIZE", "copyBuffer"))
        scale = {"FETCH_SIZE": COPY_BYTES / (cf[len(cf) // 2] * 1024.0),
                 "WRITE_SIZE": COPY_BYTES / (cw[len(cw) // 2] * 1024.0)}
    lines = [f"# {args.title}", "", "Commands (repository root on the GPU host; `cd /tmp && export TMPDIR=/tmp` "
             "first; one rocprofv3 run per counter set):", "", "```", args.command, "```", ""]
    if scale:
        lines += [f"Calibration: a 1 GiB device copy reads FETCH_SIZE x {scale['FETCH_SIZE']:.3f} and "
                  f"WRITE_SIZE x {scale['WRITE_SIZE']:.3f} bytes per KiB counted.", ""]
    lines += ["| kernel | counter | dispatches | average per dispatch | scaled bytes per dispatch |",
              "|---|---|---:|---:|---:|"]
    for kpat in args.kernel:
        for (name, cname), v in sorted(vals.items()):
            if kpat not in name:
                continue
            avg = sum(v) / len(v)
            sb = f"{avg * 1024.0 * scale[cname] / 1e6:.2f} MB" if cname in scale else ""
            lines.append(f"| `{_short(name)}` | {cname} | {len(v)} | {avg:.4g} | {sb} |")
    _write(args.out, lines)


def _short(name: str) -> str:
    """Kernel name without its parameter list."""
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i]
    return name


def _write(path, lines):
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


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
    k = sub.add_parser("kstats")
    for a in ["dir", "title", "command", "out"]:
        k.add_argument(f"--{a}", required=True)
    c = sub.add_parser("counters")
    c.add_argument("--dir", action="append", required=True)
    c.add_argument("--kernel", action="append", required=True)
    for a in ["title", "command", "out"]:
        c.add_argument(f"--{a}", required=True)
    c.add_argument("--copy-fetch")
    c.add_argument("--copy-write")
    s = sub.add_parser("summarize")
    for k in ["copy-fetch", "copy-write", "fetch", "write", "kernel", "workload"]:
        s.add_argument(f"--{k}", required=True)
    s.add_argument("--out-dir", default=os.path.join(ROOT, "profiles"))
    args = ap.parse_args()
    if args.mode == "copy":
        copy_main()
    elif args.mode == "kstats":
        kstats_main(args)
    elif args.mode == "counters":
        counters_main(args)
    else:
        summarize_main(args)


if __name__ == "__main__":
    main()
