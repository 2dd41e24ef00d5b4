"""Host logic of the benchmark and of the profile summaries (CPU only).

* the flop accounting the conv TFLOP/s figures divide by, against the layer
  shapes written out by hand (2 x multiply-adds of the direct definition,
  Sec. 4.1.2's ComputeFeature / ComputeGradient passes);
* the one-GPU contract of bench.py;
* the HBM-traffic figure is dropped when the kernel source changed;
* the counter-table derivations (MFMA busy, L2 latency, occupancy limit) and
  kernel-name normalization of profiling.py on synthetic counter files.
"""
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_1603_07846_amd import profiling  # noqa: E402
from paper_1603_07846_amd import workloads as wl  # noqa: E402


def _alexnet_fwd(batch):
    """Forward flops of the AlexNet-shaped layers, each written out:
    output pixels x filters x taps x 2."""
    conv = [
        (55 * 55, 96, 11 * 11 * 3),
        (27 * 27, 256, 5 * 5 * 96),
        (13 * 13, 384, 3 * 3 * 256),
        (13 * 13, 384, 3 * 3 * 384),
        (13 * 13, 256, 3 * 3 * 384),
    ]
    fc = [(9216, 4096), (4096, 4096), (4096, 1000)]
    c = [2.0 * batch * pq * k * taps for pq, k, taps in conv]
    f = [2.0 * batch * i * o for i, o in fc]
    return c, f


def test_step_flops_of_the_alexnet_workloads():
    # conv stacks (workloads 3 and 4): three passes per layer but conv1's input gradient
    for idx, batch in ((3, 128), (4, 256)):
        c, _ = _alexnet_fwd(batch)
        want = 3 * sum(c) - c[0]
        assert bench.step_conv_flops(wl.WORKLOADS[idx], batch) == pytest.approx(want, rel=1e-12)
    c, f = _alexnet_fwd(256)
    assert bench.step_conv_flops(wl.CFG5, 256) == pytest.approx(3 * (sum(c) + sum(f)) - c[0], rel=1e-12)
    # with the first layer's input gradient: one more forward-sized pass
    assert bench.step_conv_flops(wl.CFG5, 256, True) - bench.step_conv_flops(wl.CFG5, 256) == pytest.approx(c[0])


def test_step_flops_of_the_single_layer_workload():
    # 16 x 3 x 32 x 32 through 32 filters 5 x 5, pad 2: fwd + input grad + filter grad
    one = 2.0 * 16 * 32 * 32 * 32 * 3 * 5 * 5
    assert bench.step_conv_flops(wl.WORKLOADS[1], 16, True) == pytest.approx(3 * one)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


def test_traffic_dropped_when_the_source_changed(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("kernel one\n")
    os.makedirs(tmp_path / "profiles")
    rec = {"kernel": "k<1>", "source": "k.hip", "source_sha256": profiling.sha256_of(str(src)),
           "bytes_per_launch": 1234.4}
    (tmp_path / "profiles" / "traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("k<1>") == 1234
    assert bench.measured_traffic("other<1>") is None
    src.write_text("kernel two\n")
    assert bench.measured_traffic("k<1>") is None


def test_kernel_names_normalized():
    n = profiling.normalize
    assert n("void singa::(anonymous namespace)::conv_wgrad_large_kernel<true, false>"
             "(singa::(anonymous namespace)::WgradArgs)") == "conv_wgrad_large_kernel<1,0>"
    assert n("void singa::(anonymous namespace)::pool_fwd_nhwc_vec_kernel<unsigned short, 8, 3, 0>"
             "(singa::(anonymous namespace)::PoolGeom, int)") == "pool_fwd_nhwc_vec_kernel<bf16,8,3,0>"
    assert n("sgd_kernel(unsigned long, float*)") == "sgd_kernel"


FIELDS = ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Workgroup_Size", "LDS_Block_Size", "VGPR_Count",
          "Accum_VGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _counter_csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_counter_table_derivations(tmp_path, capsys):
    base = {"Kernel_Name": "void singa::k<true>(int)", "Grid_Size": 1024, "Workgroup_Size": 256,
            "LDS_Block_Size": 73728, "VGPR_Count": 191, "Accum_VGPR_Count": 0,
            "Start_Timestamp": 0, "End_Timestamp": 100000}
    cycles = 200000.0  # per XCD
    rows = []
    for d in (1, 2):
        for name, val in (("GRBM_GUI_ACTIVE", 8 * cycles), ("SQ_VALU_MFMA_BUSY_CYCLES", 0.25 * cycles * 1024),
                          ("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6), ("TCP_PENDING_STALL_CYCLES_sum", 0.5 * cycles * 256),
                          ("TCP_TCC_READ_REQ_sum", 1000.0), ("TCP_TCC_READ_REQ_LATENCY_sum", 300000.0)):
            rows.append(dict(base, Dispatch_Id=d, Counter_Name=name, Counter_Value=val))
    p = tmp_path / "c.csv"
    _counter_csv(str(p), rows)
    profiling.main(["counters", str(p), "--kernels", "k<1>"])
    line = [l for l in capsys.readouterr().out.splitlines() if l.startswith("| `k<1>`")][0]
    cells = [c.strip() for c in line.strip("|").split("|")]
    assert cells[1] == "2"  # launches
    assert cells[2] == "100.0"  # us per launch
    assert cells[3] == "25.0%"  # MFMA busy: counter / (cycles x 1024 SIMDs)
    assert cells[4] == "%.0f" % (512e6 / 100000 / 1e3)  # 512 flops per MOP over the duration
    assert cells[6] == "50.0%"  # L1 miss stall: counter / (cycles x 256 CUs)
    assert cells[7] == "300"  # latency per request
    assert cells[-1] == "2"  # 191 VGPRs -> 192 per lane -> 2 waves; 72 KB LDS -> 2 workgroups of 4 waves


def test_occupancy_limits():
    occ = profiling._occupancy
    assert occ(256, 73728, 191, 0) == 2       # registers and LDS both allow 2 waves per SIMD
    assert occ(512, 98304, 207, 0) == 2       # one 8-wave workgroup per CU
    assert occ(256, 49152, 159, 0) == 3       # 160 registers -> 3 waves; LDS for 3 workgroups
    assert occ(256, 0, 24, 0) == 8            # bandwidth kernels: the 8-wave limit
    assert occ(256, 147456, 272, 128) == 1    # 400 registers, one workgroup


def test_timeline_of_one_step(tmp_path, capsys):
    """profiling.py timeline: the launches between two consecutive marker
    launches, main = the marker's queue, times from the step's start."""
    p = tmp_path / "trace.csv"
    rows = [("void singa::(anonymous namespace)::space_to_depth_kernel<unsigned short>(int)", 1, 0, 10),
            ("void singa::(anonymous namespace)::conv_fwd_large_kernel<true, 32, 4, false>(A)", 1, 10, 40),
            ("void singa::(anonymous namespace)::conv_wgrad_large_kernel<true, false>(W)", 2, 15, 55),
            ("void singa::(anonymous namespace)::space_to_depth_kernel<unsigned short>(int)", 1, 60, 70),
            ("void singa::(anonymous namespace)::sgd_kernel(unsigned long)", 1, 70, 75),
            ("void singa::(anonymous namespace)::space_to_depth_kernel<unsigned short>(int)", 1, 100, 110)]
    with open(p, "w") as f:
        f.write("Kernel_Name,Queue_Id,Start_Timestamp,End_Timestamp\n")
        for name, q, s, e in rows:
            f.write('"%s",%d,%d,%d\n' % (name, q, s * 1000, e * 1000))
    profiling.main(["timeline", str(p)])  # the second-to-last step: 0 .. 60 us
    out = capsys.readouterr().out
    lines = [l for l in out.splitlines() if l.startswith("| main") or l.startswith("| second")]
    assert lines == ["| main | 0.0 | 10.0 | 10.0 | `space_to_depth_kernel<bf16>` |",
                     "| main | 10.0 | 40.0 | 30.0 | `conv_fwd_large_kernel<1,32,4,0>` |",
                     "| second | 15.0 | 55.0 | 40.0 | `conv_wgrad_large_kernel<1,0>` |"]
    assert "Step: 60.0 us" in out and "main stream 40.0 us" in out and "second stream 40.0 us" in out
    profiling.main(["timeline", str(p), "--back", "1"])  # the last complete step: 60 .. 100 us
    out = capsys.readouterr().out
    assert "| main | 10.0 | 15.0 | 5.0 | `sgd_kernel` |" in out and "Step: 40.0 us" in out
