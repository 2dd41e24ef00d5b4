"""rocprofv3 output -> the summaries kept with the benchmark.

Subcommands (run from the repository root):

  copy --mib N
      A plain device-to-device copy of N MiB, five times: the known-size
      kernel whose FETCH_SIZE / WRITE_SIZE counters calibrate the HBM byte
      counts of the library's kernels.
  stats KERNEL_STATS_CSV --title T --command C
      Markdown table of a `rocprofv3 --kernel-trace --stats` summary.
  traffic --kernel NAME --fetch CSV --write CSV --copy-fetch CSV --copy-write CSV
          --copy-mib N --source FILE --out JSON
      Average HBM bytes per launch of one kernel (FETCH_SIZE and WRITE_SIZE
      per dispatch, each divided by the factor the same counter shows for the
      copy), stamped with the SHA-256 of the kernel's source file so that a
      reader can tell when the kernel has changed since the counters were
      taken.

Kernel names are normalized to the library's trace names: the namespace and
parameter list are dropped and template arguments written as in the trace
("unsigned short" -> bf16, "float" -> f32, true/false -> 1/0).
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re
import statistics
import sys

_ARG = {"unsigned short": "bf16", "float": "f32", "true": "1", "false": "0"}


def normalize(name: str) -> str:
    n = name.strip()
    if n.startswith("void "):
        n = n[5:]
    n = n.replace("singa::(anonymous namespace)::", "").replace("singa::", "")
    # drop the parameter list: the last top-level "(...)"
    depth, cut = 0, len(n)
    for i in range(len(n) - 1, -1, -1):
        if n[i] == ")":
            depth += 1
        elif n[i] == "(":
            depth -= 1
            if depth == 0:
                cut = i
                break
    n = n[:cut] if cut < len(n) and n.endswith(")") else n
    m = re.match(r"^([A-Za-z_0-9:]+)<(.*)>$", n)
    if not m:
        return n
    args = [a.strip() for a in m.group(2).split(",")]
    return "%s<%s>" % (m.group(1), ",".join(_ARG.get(a, a) for a in args))


def sha256_of(path: str) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def _counter_rows(path: str, counter: str):
    """{dispatch id: (kernel name, value)} of one counter."""
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            d = r["Dispatch_Id"]
            name, val = out.get(d, (r["Kernel_Name"], 0.0))
            out[d] = (name, val + float(r["Counter_Value"]))
    return out


def cmd_copy(args):
    import torch
    n = args.mib * (1 << 20) // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 5}))


def cmd_stats(args):
    rows = list(csv.DictReader(open(args.csv)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    print("# %s\n" % args.title)
    print("Command (from the repository root on one MI355X, with `TMPDIR=/tmp`):\n")
    print("```\n%s\n```\n" % args.command)
    print("Kernel statistics (`*_kernel_stats.csv`) over every launch of the run; names as in the library's "
          "trace (template arguments: dtype, load modes, flags).\n")
    print("| Kernel | Calls | Total ms | Average us | Min us | Max us | Share |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        print("| `%s` | %s | %.3f | %.1f | %.1f | %.1f | %.1f%% |" % (
            normalize(r["Name"]), r["Calls"], float(r["TotalDurationNs"]) / 1e6, float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, 100.0 * float(r["TotalDurationNs"]) / total))


def _copy_factor(path, counter, nbytes):
    rows = _counter_rows(path, counter)
    vals = [v * 1024.0 for _, v in rows.values() if v > 0]
    if not vals:
        raise SystemExit("no %s dispatches in %s" % (counter, path))
    # the copies are the only (and largest) dispatches of that run
    big = sorted(vals)[-5:]
    return statistics.median(big) / nbytes


def cmd_traffic(args):
    nbytes = args.copy_mib * (1 << 20)
    f_fetch = _copy_factor(args.copy_fetch, "FETCH_SIZE", nbytes)
    f_write = _copy_factor(args.copy_write, "WRITE_SIZE", nbytes)
    fetch = [v for n, v in _counter_rows(args.fetch, "FETCH_SIZE").values() if normalize(n) == args.kernel]
    write = [v for n, v in _counter_rows(args.write, "WRITE_SIZE").values() if normalize(n) == args.kernel]
    if not fetch or not write:
        raise SystemExit("kernel %s not found in the counter files" % args.kernel)
    fb = statistics.mean(fetch) * 1024.0 / f_fetch
    wb = statistics.mean(write) * 1024.0 / f_write
    out = {"kernel": args.kernel, "source": args.source, "source_sha256": sha256_of(args.source),
           "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb, "bytes_per_launch": fb + wb,
           "dispatches": len(fetch), "copy_factor_fetch": f_fetch, "copy_factor_write": f_write,
           "copy_mib": args.copy_mib}
    with open(args.out, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--mib", type=int, default=1024)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    t = sub.add_parser("traffic")
    for a in ("--kernel", "--fetch", "--write", "--copy-fetch", "--copy-write", "--source", "--out"):
        t.add_argument(a, required=True)
    t.add_argument("--copy-mib", type=int, default=1024)
    args = ap.parse_args(argv)
    {"copy": cmd_copy, "stats": cmd_stats, "traffic": cmd_traffic}[args.cmd](args)


if __name__ == "__main__":
    main()
