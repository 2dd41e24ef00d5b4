"""rocprofv3 output -> the summaries kept with the benchmark.

Subcommands (run from the repository root):

  copy --mib N
      A plain device-to-device copy of N MiB, five times: the known-size
      kernel whose FETCH_SIZE / WRITE_SIZE counters calibrate the HBM byte
      counts of the library's kernels.
  stats KERNEL_STATS_CSV --title T --command C [--trace KERNEL_TRACE_CSV]
      Markdown table of a `rocprofv3 --kernel-trace --stats` summary (with the
      per-kernel median launch time when the same run's trace is given).
  traffic --kernel NAME --fetch CSV --write CSV --copy-fetch CSV --copy-write CSV
          --copy-mib N --source FILE --out JSON
      Average HBM bytes per launch of one kernel (FETCH_SIZE and WRITE_SIZE
      per dispatch, each divided by the factor the same counter shows for the
      copy), stamped with the SHA-256 of the kernel's source file so that a
      reader can tell when the kernel has changed since the counters were
      taken.
  counters CSV [CSV ...] --kernels NAME [NAME ...] [--copy-fetch CSV --copy-write CSV --copy-mib N]
      Markdown table of derived figures per kernel from `rocprofv3 --pmc`
      counter passes (each pass its own run of the same program): MFMA busy
      fraction and MFMA rate, LDS bank conflicts, vector L1 stalls on
      outstanding misses, mean L2 read latency, L2 hit rate, HBM bytes, and
      the occupancy the kernel's registers and LDS allow.

  timeline KERNEL_TRACE_CSV [--marker NAME] [--back N]
      One step of a run as a markdown table, from a `rocprofv3 --kernel-trace`
      CSV: every launch between two consecutive launches of the marker kernel
      (the step's first kernel; by default the N-th step from the end, N = 2),
      with its stream (main: the marker's queue; second: any other), start and
      end in microseconds from the step's start, and duration; then each
      stream's busy time over the step.

  libgemm [--reps N]
      Times the vendor library's bf16 GEMM (torch.matmul, hipBLASLt) on the
      explicit-GEMM shapes of the AlexNet-shaped layers at batch 256 (the
      convolutions as im2col GEMMs: rows = output pixels, columns = filters,
      reduction = taps) and a large square GEMM, beside this library's own
      call for the same product (implicit GEMM: the im2col is never built),
      both on normal random bf16 data: a reference for what a plain library
      GEMM of the same shape reaches on the device.  Not part of the
      library's path (which calls no vendor GEMM).

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
    med = {}
    if args.trace:
        # per-launch durations from the same run's kernel trace -> medians
        durs = collections.defaultdict(list)
        with open(args.trace) as f:
            for r in csv.DictReader(f):
                durs[normalize(r["Kernel_Name"])].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        med = {k: statistics.median(v) for k, v in durs.items()}
    print("# %s\n" % args.title)
    print("Command (from the repository root on one MI355X, with `TMPDIR=/tmp`):\n")
    print("```\n%s\n```\n" % args.command)
    print("Kernel statistics (`*_kernel_stats.csv`) over every launch of the run; names as in the library's "
          "trace (template arguments: dtype, load modes, flags).\n")
    print("| Kernel | Calls | Total ms | Average us | Median us | Min us | Max us | Share |")
    print("|---|---:|---:|---:|---:|---:|---:|---:|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = normalize(r["Name"])
        m = med.get(name)
        print("| `%s` | %s | %.3f | %.1f | %s | %.1f | %.1f | %.1f%% |" % (
            name, r["Calls"], float(r["TotalDurationNs"]) / 1e6, float(r["AverageNs"]) / 1e3,
            "-" if m is None else "%.1f" % (m / 1e3), float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
            100.0 * float(r["TotalDurationNs"]) / total))


# (name, M, N, K, the same product as this library's call or None):
# forward x (N,H,W,C), w (K,R,S,C), pad; filter gradient x, dy, w shape, pad
LIBGEMM_SHAPES = [
    ("square 8192", 8192, 8192, 8192, None),
    ("conv1 forward", 256 * 55 * 55, 96, 11 * 11 * 3, None),
    ("conv2 forward", 256 * 27 * 27, 256, 5 * 5 * 96, ("fwd", (256, 27, 27, 96), (256, 5, 5, 96), 2)),
    ("conv3 forward", 256 * 13 * 13, 384, 3 * 3 * 256, ("fwd", (256, 13, 13, 256), (384, 3, 3, 256), 1)),
    ("conv4 forward", 256 * 13 * 13, 384, 3 * 3 * 384, ("fwd", (256, 13, 13, 384), (384, 3, 3, 384), 1)),
    ("conv5 forward", 256 * 13 * 13, 256, 3 * 3 * 384, ("fwd", (256, 13, 13, 384), (256, 3, 3, 384), 1)),
    ("conv2 filter gradient", 256, 5 * 5 * 96, 256 * 27 * 27, ("wgrad", (256, 27, 27, 96), (256, 5, 5, 96), 2)),
    ("conv4 filter gradient", 384, 3 * 3 * 384, 256 * 13 * 13, ("wgrad", (256, 13, 13, 384), (384, 3, 3, 384), 1)),
    ("fc6 forward", 256, 4096, 9216, ("fwd", (256, 6, 6, 256), (4096, 6, 6, 256), 0)),
    ("fc7 forward", 256, 4096, 4096, ("fwd", (256, 1, 1, 4096), (4096, 1, 1, 4096), 0)),
    ("fc8 forward", 256, 1000, 4096, ("fwd", (256, 1, 1, 4096), (1000, 1, 1, 4096), 0)),
]


def _time_ms(fn, reps):
    import torch
    for _ in range(3):
        fn()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(reps):
        fn()
    ev1.record()
    torch.cuda.synchronize()
    return ev0.elapsed_time(ev1) / reps


def cmd_libgemm(args):
    import torch
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    from paper_1603_07846_amd import singa
    torch.manual_seed(0)
    dev = torch.device("cuda:0")
    print("| GEMM | M | N | K | library ms | library TFLOP/s | this library ms | this library TFLOP/s |")
    print("|---|---:|---:|---:|---:|---:|---:|---:|")
    for name, m, n, k, ours in LIBGEMM_SHAPES:
        flop = 2.0 * m * n * k
        a = torch.randn(m, k, device=dev, dtype=torch.bfloat16)
        b = torch.randn(k, n, device=dev, dtype=torch.bfloat16)
        ms = _time_ms(lambda: a @ b, args.reps)
        del a, b
        cells = ["-", "-"]
        if ours is not None:
            op, xs, ws, pad = ours
            x = torch.randn(xs, device=dev, dtype=torch.bfloat16)
            w = torch.randn(ws, device=dev, dtype=torch.bfloat16)
            ys = singa.conv_out_shape(xs, ws, pad, 1)
            if op == "fwd":
                y = singa.empty(ys, torch.bfloat16, dev)
                ws_buf = singa.empty((max(1, singa.conv_workspace_bytes(singa.OP_FWD, singa.BF16, xs, ws, pad, 1)),),
                                     torch.uint8, dev)
                fn = lambda: singa.conv_fwd(x, w, None, pad=pad, out=y, workspace=ws_buf)
            else:
                dy = torch.randn(ys, device=dev, dtype=torch.bfloat16)
                dw = singa.empty(ws, torch.float32, dev)
                db = singa.empty((ws[0],), torch.float32, dev)
                ws_buf = singa.empty((max(1, singa.conv_workspace_bytes(singa.OP_BWD_FILTER, singa.BF16, xs, ws, pad,
                                                                         1)),), torch.uint8, dev)
                fn = lambda: singa.conv_bwd_filter(x, dy, ws, pad=pad, dw=dw, db=db, workspace=ws_buf)
            oms = _time_ms(fn, args.reps)
            cells = ["%.4f" % oms, "%.0f" % (flop / oms / 1e9)]
        print("| %s | %d | %d | %d | %.4f | %.0f | %s | %s |" % (name, m, n, k, ms, flop / ms / 1e9, cells[0], cells[1]),
              flush=True)


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


# gfx950: 8 XCDs of 32 compute units, 4 SIMDs per CU, 512 VGPRs (arch + acc)
# per lane per SIMD, 160 KiB of LDS per CU, at most 8 waves per SIMD.
N_XCD, N_CU, SIMD_PER_CU, VGPR_FILE, LDS_BYTES, MAX_WAVES = 8, 256, 4, 512, 160 * 1024, 8


def _dispatches(paths):
    """{(path index, dispatch id): {"name", "ns", "wg", "lds", "vgpr", "agpr", counter: value}}."""
    out = {}
    for i, path in enumerate(paths):
        with open(path) as f:
            for r in csv.DictReader(f):
                d = out.setdefault((i, r["Dispatch_Id"]), {
                    "name": normalize(r["Kernel_Name"]), "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"]),
                    "grid": int(r["Grid_Size"]),
                    "wg": int(r["Workgroup_Size"]), "lds": int(r["LDS_Block_Size"]),
                    "vgpr": int(r["VGPR_Count"]), "agpr": int(r.get("Accum_VGPR_Count") or 0)})
                d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return out


def _occupancy(wg, lds, vgpr, agpr):
    """Waves per SIMD that the kernel's resources allow (VGPRs and AGPRs share one
    file of 512 per lane, allocated in blocks of 8; LDS per CU)."""
    regs = -(-(vgpr + agpr) // 8) * 8
    by_regs = VGPR_FILE // regs if regs else MAX_WAVES
    waves_per_wg = -(-wg // 64)
    wg_per_cu = LDS_BYTES // lds if lds else 10 ** 9
    by_lds = wg_per_cu * waves_per_wg / SIMD_PER_CU
    return min(MAX_WAVES, by_regs, by_lds)


def cmd_counters(args):
    """MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cycles x SIMDs) (the counter is
    summed over the 1024 SIMDs); MFMA TFLOP/s issued = 512 x
    SQ_INSTS_VALU_MFMA_MOPS_* / duration (includes tile padding and the bias
    column, unlike the algorithmic figures); LDS bank-conflict cycles per
    cycle of LDS instruction activity; L1 miss-stall = TCP_PENDING_STALL_CYCLES
    / (cycles x CUs); L2 read latency = TCP_TCC_READ_REQ_LATENCY /
    TCP_TCC_READ_REQ (cycles per request, issued to returned)."""
    disp = _dispatches(args.csv)
    f_fetch = f_write = None
    if args.copy_fetch and args.copy_write:
        nbytes = args.copy_mib * (1 << 20)
        f_fetch = _copy_factor(args.copy_fetch, "FETCH_SIZE", nbytes)
        f_write = _copy_factor(args.copy_write, "WRITE_SIZE", nbytes)
    cols = ["Kernel", "Launches", "us / launch", "MFMA busy", "MFMA TFLOP/s issued", "LDS bank-conflict cycles",
            "L1 miss-stall", "L2 read latency (clk)", "L2 hit", "HBM read MB", "HBM write MB", "waves/SIMD (limit)"]
    print("| " + " | ".join(cols) + " |")
    print("|---|" + "---:|" * (len(cols) - 1))

    def mean(rows, key):
        vals = [r[key] for r in rows if key in r]
        return statistics.mean(vals) if vals else None

    def fmt(v, f):
        return "-" if v is None else f % v

    def pct(v):
        return "-" if v is None else "%.1f%%" % (100.0 * v)

    groups = []
    for kernel in args.kernels:
        rows = [d for d in disp.values() if d["name"] == kernel]
        if not rows:
            raise SystemExit("kernel %s not found in the counter files" % kernel)
        groups.append((kernel, None, rows))
        if args.by_grid:
            # one row per launch shape (each layer of the step has its own grid)
            for g in sorted({r["grid"] for r in rows}, reverse=True):
                groups.append((kernel, g, [r for r in rows if r["grid"] == g]))
    for kernel, grid, rows in groups:
        ns = statistics.mean(r["ns"] for r in rows)
        # GRBM_GUI_ACTIVE is summed over the XCDs: cycles of one = sum / N_XCD.
        # It also covers the dispatch's start-up and drain, so busy fractions
        # of launches shorter than a few tens of microseconds read low.
        per_pass = {}
        for r in rows:
            if "GRBM_GUI_ACTIVE" in r:
                for k, v in r.items():
                    if isinstance(v, float) and k != "GRBM_GUI_ACTIVE":
                        per_pass.setdefault(k, []).append((v, r["GRBM_GUI_ACTIVE"] / N_XCD))

        def frac(key, units):
            # counter / (cycles of the same dispatches x units)
            pairs = per_pass.get(key)
            if not pairs:
                return None
            return sum(v for v, _ in pairs) / (sum(c for _, c in pairs) * units)

        mops = [(r.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) + r.get("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0), r["ns"])
                for r in rows if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in r or "SQ_INSTS_VALU_MFMA_MOPS_F32" in r]
        # one MOP is 512 floating-point operations of a matrix instruction
        tflops = sum(m * 512.0 for m, _ in mops) / sum(t for _, t in mops) / 1e3 if mops else None
        lat = mean(rows, "TCP_TCC_READ_REQ_LATENCY_sum")
        req = mean(rows, "TCP_TCC_READ_REQ_sum")
        hit, miss = mean(rows, "TCC_HIT_sum"), mean(rows, "TCC_MISS_sum")
        fetch, write = mean(rows, "FETCH_SIZE"), mean(rows, "WRITE_SIZE")
        r0 = rows[0]
        cells = [
            ("`%s`" % kernel) if grid is None else ("&nbsp;&nbsp;grid %d threads" % grid),
            str(sum(1 for (i, _) in disp if i == 0 and disp[(i, _)]["name"] == kernel
                    and (grid is None or disp[(i, _)]["grid"] == grid))),
            "%.1f" % (ns / 1e3),
            pct(frac("SQ_VALU_MFMA_BUSY_CYCLES", N_CU * SIMD_PER_CU)), fmt(tflops, "%.0f"),
            pct(None if not mean(rows, "SQ_ACTIVE_INST_LDS") else
                mean(rows, "SQ_LDS_BANK_CONFLICT") / mean(rows, "SQ_ACTIVE_INST_LDS")),
            pct(frac("TCP_PENDING_STALL_CYCLES_sum", N_CU)),
            fmt(None if not req else lat / req, "%.0f"),
            pct(None if hit is None or miss is None or hit + miss == 0 else hit / (hit + miss)),
            fmt(None if fetch is None or f_fetch is None else fetch * 1024.0 / f_fetch / 1e6, "%.1f"),
            fmt(None if write is None or f_write is None else write * 1024.0 / f_write / 1e6, "%.1f"),
            "%g" % _occupancy(r0["wg"], r0["lds"], r0["vgpr"], r0["agpr"]),
        ]
        print("| " + " | ".join(cells) + " |")


def cmd_timeline(args):
    with open(args.csv) as f:
        rows = list(csv.DictReader(f))
    qkey = "Queue_Id" if rows and "Queue_Id" in rows[0] else "Stream_Id"
    ks = sorted((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), normalize(r["Kernel_Name"]), r[qkey])
                for r in rows)
    marks = [i for i, k in enumerate(ks) if k[2] == args.marker]
    if len(marks) < args.back + 1:
        raise SystemExit("fewer than %d launches of %s in the trace" % (args.back + 1, args.marker))
    a, b = marks[-args.back - 1], marks[-args.back]
    t0, main_q = ks[a][0], ks[a][3]
    busy = collections.defaultdict(float)
    print("| Stream | Start us | End us | us | Kernel |")
    print("|---|---:|---:|---:|---|")
    for s0, e0, name, q in ks[a:b]:
        st = "main" if q == main_q else "second"
        busy[st] += (e0 - s0) / 1e3
        print("| %s | %.1f | %.1f | %.1f | `%s` |" % (st, (s0 - t0) / 1e3, (e0 - t0) / 1e3, (e0 - s0) / 1e3, name))
    print("\nStep: %.1f us from one `%s` to the next; kernels busy %s." % (
        (ks[b][0] - t0) / 1e3, args.marker,
        ", ".join("%s stream %.1f us" % (k, v) for k, v in sorted(busy.items()))))


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("copy")
    c.add_argument("--mib", type=int, default=1024)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--trace", help="the run's kernel_trace.csv, for per-kernel medians")
    t = sub.add_parser("traffic")
    for a in ("--kernel", "--fetch", "--write", "--copy-fetch", "--copy-write", "--source", "--out"):
        t.add_argument(a, required=True)
    t.add_argument("--copy-mib", type=int, default=1024)
    k = sub.add_parser("counters")
    k.add_argument("csv", nargs="+")
    k.add_argument("--kernels", nargs="+", required=True)
    k.add_argument("--copy-fetch")
    k.add_argument("--copy-write")
    k.add_argument("--copy-mib", type=int, default=1024)
    k.add_argument("--by-grid", action="store_true", help="also one row per launch shape of each kernel")
    tl = sub.add_parser("timeline")
    tl.add_argument("csv")
    tl.add_argument("--marker", default="space_to_depth_kernel<bf16>")
    tl.add_argument("--back", type=int, default=2)
    g = sub.add_parser("libgemm")
    g.add_argument("--reps", type=int, default=20)
    args = ap.parse_args(argv)
    {"copy": cmd_copy, "stats": cmd_stats, "traffic": cmd_traffic, "counters": cmd_counters,
     "libgemm": cmd_libgemm, "timeline": cmd_timeline}[args.cmd](args)


if __name__ == "__main__":
    main()
