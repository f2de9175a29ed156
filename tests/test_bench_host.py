"""bench.py's host-side bookkeeping, on the CPU: attributing timed launches
to the workload's groups, and turning counter runs into traffic per launch."""
import csv
import os
import subprocess
import sys

import bench

NAMES = {0: "forward", 1: "backward_short", 2: "backward_dkdv", 3: "backward_dq", 4: "rope"}


def test_split_by_group_follows_launch_order():
    # two steps of three groups: RoPE + forward + dQ + dK/dV, forward +
    # one-kernel backward, forward + dQ + dK/dV
    step = [(4, 0.1), (4, 0.1), (0, 1.0), (3, 2.0), (2, 3.0), (0, 4.0), (1, 5.0),
            (0, 6.0), (3, 7.0), (2, 8.0)]
    g = bench.split_by_group(step * 2, NAMES, 3)
    assert g[0] == {"rope": [0.1] * 4, "forward": [1.0, 1.0], "backward_dq": [2.0, 2.0],
                    "backward_dkdv": [3.0, 3.0]}
    assert g[1] == {"forward": [4.0, 4.0], "backward_short": [5.0, 5.0]}
    assert g[2] == {"forward": [6.0, 6.0], "backward_dq": [7.0, 7.0],
                    "backward_dkdv": [8.0, 8.0]}


def _write_counters(path, counter, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, kib) in enumerate(rows):
            w.writerow([i + 1, name, counter, kib])


def test_traffic_summary_scales_by_the_copy(tmp_path, monkeypatch):
    # --buckets 8192,4096 of the D=64 sweep: per step forward, dQ, dK/dV per
    # group; one warm-up and one timed step.  The copies read half their
    # bytes (FETCH) and write all of them (WRITE), as measured on gfx950.
    def rows(per_kib, copy_kib):
        r = [("void at::native::normal_kernel", 10.0)]
        r += [("void at::native::copy_kernel", copy_kib)] * 3
        for _ in range(2):
            for base in (1000.0, 500.0):
                r += [("void dd::fwd_kernel<64, false>(...)", base * per_kib),
                      ("void dd::dq_kernel<64, false>(...)", 2 * base * per_kib),
                      ("void dd::dkdv1_kernel<64, false>(...)", 3 * base * per_kib)]
        return r
    _write_counters(tmp_path / "f", "FETCH_SIZE", rows(1.0, 2 ** 19))
    _write_counters(tmp_path / "w", "WRITE_SIZE", rows(0.5, 2 ** 20))
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--workload",
                          "dd_sweep_d64", "--buckets", "8192,4096", "--traffic-summary",
                          str(tmp_path / "f"), str(tmp_path / "w")],
                         capture_output=True, text=True, check=True).stdout
    kv = dict(l.split(" = ") for l in out.splitlines() if " = " in l and not l.startswith("#"))
    assert float(kv["fetch_scale"]) == 2.0 and float(kv["write_scale"]) == 1.0
    # dK/dV of the L=4096 group: 3 * 500 KiB read (x2), 3 * 250 KiB written
    assert int(kv["fetch_bytes_per_launch.backward_dkdv.L=4096"]) == 3 * 500 * 1024 * 2
    assert int(kv["write_bytes_per_launch.backward_dkdv.L=4096"]) == 3 * 250 * 1024
    assert int(kv["bytes_per_launch.forward.L=8192"]) == 1000 * 1024 * 2 + 500 * 1024
    # bench.measured_traffic reads such keys back (group names hold "=")
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "traffic_dd_sweep_d64.txt").write_text(out)
    h = bench.kernel_source_hash()  # the summary was stamped with the current sources
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: h)
    assert bench.measured_traffic("dd_sweep_d64", "backward_dkdv", "L=4096") == 3 * 500 * 1024 * 2 + 3 * 250 * 1024


def test_traffic_summary_names_the_short_row_backward(tmp_path):
    # --buckets 256 of the D=64 sweep: the forward and the one-kernel
    # backward, whose persistent form is not a template.
    def rows(per_kib):
        r = [("void at::native::copy_kernel", 2 ** 20)] * 3
        for _ in range(2):
            r += [("void dd::fwd_kernel<64, true, false>(...)", 100.0 * per_kib),
                  ("dd::bwd_short_persist_kernel(unsigned short const*, ...)", 300.0 * per_kib)]
        return r
    _write_counters(tmp_path / "f", "FETCH_SIZE", rows(1.0))
    _write_counters(tmp_path / "w", "WRITE_SIZE", rows(1.0))
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--workload",
                          "dd_sweep_d64", "--buckets", "256", "--traffic-summary",
                          str(tmp_path / "f"), str(tmp_path / "w")],
                         capture_output=True, text=True, check=True).stdout
    kv = dict(l.split(" = ") for l in out.splitlines() if " = " in l and not l.startswith("#"))
    assert int(kv["bytes_per_launch.backward_short.L=256"]) == 2 * 300 * 1024


def test_cpu_baseline_counts_every_sampled_slice():
    # 16 sampled (b, h) slices of full causal rows of 8192 tokens: 16 x
    # 8192*8193/2 pairs; with documents, each row's own segments count.
    pairs = [(0, h) for h in range(16)]
    assert bench.sample_flops(pairs, 1, 8192, 64) == 14 * 64 * 16 * 8192 * 8193 // 2
    cu = [0, 3, 10, 16]  # rows of 8: [0,3) [3,8) | [8,10) [10,16)
    assert list(bench.row_pairs(2, 8, cu)) == [6 + 15, 3 + 21]
    assert bench.sample_flops([(1, 0), (1, 5), (0, 2)], 2, 8, 64, cu) == 14 * 64 * (24 + 24 + 21)
