"""Host logic of bench.py (no GPU): the algorithmic byte counts behind the reported GB/s, the
refusal of more than one GPU, and the source hash that keys committed counter data."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402
from paper_2607_06202_amd import workloads as W  # noqa: E402


def _bytes(name):
    w = W.WORKLOADS[name]
    return bench.algorithmic_bytes(w.T, w.k, w.H, w.R, w.E, w.T * w.k, w.payload)


def test_decode_bytes_from_the_sizes_of_x_and_recv():
    """EP=64 decode, no invalid ids: x is 8192 x 7168 bf16 = 117,440,512 B and the packed receive
    rows are 65,536 x 7168 bf16 = 939,524,096 B. Dispatch reads x and the row table and writes the
    rows; combine reads the rows, the weights and the row table and writes the output."""
    b = _bytes("decode_ep64")
    x, recv, table = 117_440_512, 939_524_096, 8192 * 8 * 4
    assert b["dispatch"] == x + table + recv
    assert b["combine"] == recv + 2 * table + x
    assert b["total"] == b["layout"] + b["dispatch"] + b["combine"] == 2_116_207_884
    # 70% of 8 TB/s on these bytes is 377.9 us per layer
    assert abs(b["total"] / (0.7 * 8e12) * 1e6 - 377.9) < 0.05


def test_fused_row_kernel_bytes_add_the_placement_metadata():
    """The row kernel with the layout's finalize step fused in writes the expert, rank and segment
    offsets, the pair rows and slots, and recv_src / recv_j on top of the dispatch's own bytes."""
    b = _bytes("decode_ep64")
    R, E, T, k, P = 64, 256, 8192, 8, 65536
    placement = 4 * ((E + 1) + (R + 1) + E * R + 2 * T * k + 2 * P)
    assert placement == 1_115_400
    assert b["rows_fused"] == b["dispatch"] + placement
    assert placement < b["layout"]  # the layout still accounts for them once in the total


def test_fp8_bytes_include_one_scale_per_128_elements():
    b = _bytes("skewed_fp8_ep64")
    P, H = 16384 * 8, 7168
    x = 16384 * H * 2
    assert b["dispatch"] == x + P * 4 + P * H + P * (H // 128) * 4
    assert P * (H // 128) * 4 == 29_360_128
    assert b["combine"] == P * H * 2 + 2 * P * 4 + x  # combine reads bf16 expert outputs


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "single-GPU" in r.stderr


def test_source_hash_ignores_comments_but_not_code(tmp_path, monkeypatch):
    src = tmp_path / "csrc"
    shutil.copytree(bench.CSRC, src)
    monkeypatch.setattr(bench, "CSRC", str(src))
    h0 = bench.source_hash("combine_kernel")
    f = src / "combine.hip"
    text = f.read_text()
    f.write_text("// a new comment\n" + text.replace("\n", "\n   ", 3) + "\n/* block\n comment */\n")
    assert bench.source_hash("combine_kernel") == h0
    assert bench.source_hash("dispatch_bf16_kernel") != h0  # other file
    f.write_text(text.replace("kGather = 8", "kGather = 4"))
    assert bench.source_hash("combine_kernel") != h0
