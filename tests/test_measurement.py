"""Host-side measurement helpers (no GPU): the benchmark's byte and flop
accounting, and the rocprofv3 summary tools, on synthetic CSV files."""

import csv
import os

import pytest

import bench
from paper_2502_11018_amd import profiling
from workloads.configs import get_workload


def test_algorithmic_bytes_of_the_8b_step():
    w = get_workload("llama3-8b")
    total, parts = bench.algorithmic_bytes(w)
    m = w.model
    # weights: per layer QKV 6144x4096, O 4096x4096, gate/up 2x14336x4096, down 4096x14336; LM head
    per_layer = 6144 * 4096 + 4096 * 4096 + 2 * 14336 * 4096 + 4096 * 14336
    assert parts["weights"] >= 2 * (per_layer * 32 + 128256 * 4096)
    # prefix KV read: 2048 positions x 8 KV heads x 128 dims x (K, V) x 2 bytes x 32 layers
    assert parts["kv_read"] == 2048 * 8 * 128 * 2 * 2 * 32
    assert abs(total / 1e9 - 15.29) < 0.02


def test_class_bytes_and_flops_per_launch():
    w = get_workload("llama3-8b")
    b = bench.class_bytes_per_launch(w)
    assert b["gate_up_gemm"] == 2 * 2 * 14336 * 4096
    assert b["down_gemm"] == 2 * 4096 * 14336
    f = bench.class_mfma_flops_per_launch(w)
    # 64 rows, split-bf16 (2 MFMAs per product), 2 flops per multiply-add
    assert f["gate_up_gemm"] == 2 * 2 * 64 * 2 * 14336 * 4096
    assert f["tree_attention"] == 2 * 2 * 2 * 32 * 64 * 2048 * 128


def _write_csv(path, header, rows):
    with open(path, "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(header)
        wr.writerows(rows)


def test_traffic_record_round_trip(tmp_path):
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    _write_csv(tmp_path / "f.csv", hdr, [[1, "void gemm_kernel<1, 2>()", "FETCH_SIZE", 1000.0],
                                        [2, "void gemm_kernel<1, 2>()", "FETCH_SIZE", 1200.0],
                                        [3, "void gemm_kernel<0, 1>()", "FETCH_SIZE", 5.0]])
    _write_csv(tmp_path / "w.csv", hdr, [[1, "void gemm_kernel<1, 2>()", "WRITE_SIZE", 10.0]])
    _write_csv(tmp_path / "cf.csv", hdr, [[1, "copyBuffer", "FETCH_SIZE", 512.0]])
    _write_csv(tmp_path / "cw.csv", hdr, [[1, "copyBuffer", "WRITE_SIZE", 1024.0]])
    src = tmp_path / "k.hip"
    src.write_text("kernel source")
    prof = tmp_path / "profiles"
    prof.mkdir()
    profiling.main(["traffic", "--kernel-regex", "gemm_kernel<1,", "--fetch", str(tmp_path / "f.csv"),
                    "--write", str(tmp_path / "w.csv"), "--copy-regex", "copyBuffer",
                    "--copy-fetch", str(tmp_path / "cf.csv"), "--copy-write", str(tmp_path / "cw.csv"),
                    "--copy-bytes", str(1024 * 1024), "--label", "gate_up_gemm", "--workload", "x",
                    "--source", str(src), "--out", str(prof / "t.md"), "--command", "cmd"])
    # fetch: mean 1100 KiB x scale (1 MiB / 512 KiB = 2); write: 10 KiB x 1.  The record stores the
    # source path relative to the repository root.
    rec = [l for l in (prof / "t.md").read_text().splitlines() if l.startswith("traffic-record:")][0]
    kv = dict(t.split("=", 1) for t in rec.split()[1:])
    assert float(kv["fetch_bytes"]) == pytest.approx(1100 * 1024 * 2)
    assert float(kv["write_bytes"]) == pytest.approx(10 * 1024)
    root = os.path.dirname(profiling.PKG)
    assert profiling.read_traffic_record(str(prof), "gate_up_gemm", "x", root) == pytest.approx(
        1100 * 1024 * 2 + 10 * 1024)
    src.write_text("kernel source, changed")       # a changed kernel voids the record
    assert profiling.read_traffic_record(str(prof), "gate_up_gemm", "x", root) is None


def test_stats_summary_groups_kernels_by_grid(tmp_path):
    hdr = ["Kernel_Name", "Start_Timestamp", "End_Timestamp", "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z",
           "Workgroup_Size_X", "Workgroup_Size_Y", "Workgroup_Size_Z"]
    rows, t = [], 0
    for step in range(3):
        for name, grid, dur in (("void griffin::gemm_kernel<0>(x)", 256, 1000), ("void griffin::gemm_kernel<0>(x)", 512, 3000),
                                ("void griffin::norm(x)", 64, 200), ("void griffin::gemm_kernel<0>(x)", 512, 2000),
                                ("void griffin::accept_kernel(x)", 64, 500)):
            rows.append([name, t, t + dur, grid, 1, 1, 64, 1, 1])
            t += dur + 100
    _write_csv(tmp_path / "trace.csv", hdr, rows)
    out = tmp_path / "s.md"
    profiling.main(["stats", str(tmp_path / "trace.csv"), "--steps", "2", "--out", str(out), "--title", "t",
                    "--command", "c"])
    text = out.read_text()
    # rows are keyed by kernel, grid and the kernel launched before it: the two
    # 8-workgroup launches of one step stay apart
    assert "| `gemm_kernel<0>` | 8x1x1 | `gemm_kernel<0>` | 1 | 3.00 |" in text
    assert "| `gemm_kernel<0>` | 8x1x1 | `norm` | 1 | 2.00 |" in text
    assert "| `gemm_kernel<0>` | 4x1x1 | `accept_kernel` | 1 | 1.00 |" in text


def test_ragged_batch_accounting():
    """A ragged batch counts each sequence's own prefix and tree: KV bytes
    follow the sum of the prefixes, and 16 chains in 3-row slots are one
    64-row tile for the GEMMs."""
    w = get_workload("llama3-8b-chain2-b16")
    m = w.model
    total, parts = bench.algorithmic_bytes(w)
    assert parts["kv_read"] == sum(w.prefixes()) * m.kv_bytes_per_position()
    assert parts["kv_write"] == 16 * 3 * m.kv_bytes_per_position()
    f = bench.class_mfma_flops_per_launch(w)
    assert f["qkv_gemm"] == 2 * 2 * 64 * m.qkv_rows * m.d_model
    keys = sum(-(-p // 32) * 32 for p in w.prefixes())
    assert f["tree_attention"] == 2 * 2 * 2 * m.n_q_heads * 32 * keys * m.head_dim
    assert bench.class_bytes_per_launch(w)["tree_attention"] == \
        sum(w.prefixes()) * m.kv_bytes_per_position() // m.n_layers
