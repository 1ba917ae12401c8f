"""Host logic of bench.py (no GPU): the algorithmic byte counts behind the reported GB/s, the
refusal of more than one GPU, and the machine-code hash that keys committed counter data."""
import os
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


def test_per_rank_payload_matches_the_papers_bandwidth_table():
    """The paper's EPCL table (Table 4) gives latency and bandwidth but not the payload. This
    build reads the payload as 7,340,032 bytes per rank: 64 tokens x top-8 x 7168 x 2 bytes, one
    bf16 row per (token, expert) pair, the payload term P*H*2 (P = T*k) of the bench's dispatch
    byte model at the evaluation's default of 64 tokens per rank. Every printed bandwidth is
    consistent with that payload divided by the printed latency; two other plausible payloads are
    not."""
    path = os.path.join(os.path.dirname(__file__), "golden", "ep_comparison_latency_bw.txt")
    rows = [list(map(int, ln.split())) for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 5
    R, Tr, k, H = 128, 64, 8, 7168
    b = bench.algorithmic_bytes(R * Tr, k, H, R, R, R * Tr * k, "bf16")
    payload = (b["dispatch"] - R * Tr * H * 2 - R * Tr * k * 4) // R  # rows written per rank
    assert payload == 64 * 8 * 7168 * 2 == 7_340_032
    def consistent(nbytes, lat, bw):
        # Latencies are printed to the microsecond and bandwidths to the GB/s: the bandwidth
        # range the latency allows must meet the range the printed bandwidth stands for.
        lo, hi = nbytes / ((lat + 0.5) * 1e3), nbytes / ((lat - 0.5) * 1e3)
        return lo <= bw + 0.5 and hi >= bw - 0.5

    for ep, lat_cann, bw_cann, lat_ubep, bw_ubep in rows:
        for lat, bw in ((lat_cann, bw_cann), (lat_ubep, bw_ubep)):
            assert consistent(payload, lat, bw), (ep, lat, bw)
    # The table does not fit the byte counts of other plausible payloads: fp8 rows (half the
    # bytes), or rows with the 56 fp32 scales of a 128-element block quantiser added.
    for other in (payload // 2, payload + 64 * 8 * 56 * 4):
        assert not all(consistent(other, lat, bw) for r in rows for lat, bw in ((r[1], r[2]), (r[3], r[4])))


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


def test_code_hash_follows_the_machine_code(tmp_path):
    """The key of committed counter data is a hash of each kernel's gfx950 machine code and
    descriptor, read from the built object: unchanged by a comment that shifts every source
    line, changed by a change of code. (Compiles combine.hip three times with the library's
    own flags; hipcc cross-compiles without a GPU.)"""
    from concurrent.futures import ThreadPoolExecutor

    from paper_2607_06202_amd import _build

    text = open(os.path.join(_build.CSRC, "combine.hip")).read()
    variants = {"same": text,
                "comment": "// a new comment\n/* and a block\n comment */\n" + text.replace("\n", "\n   ", 3),
                "code": text.replace("kGather = 8", "kGather = 4")}
    assert variants["code"] != text

    def compile_variant(name):
        src = tmp_path / ("%s.hip" % name)
        src.write_text(variants[name])
        obj = tmp_path / ("%s.o" % name)
        subprocess.check_call([_build.HIPCC, *_build.FLAGS, "-I" + _build.CSRC, "-c", str(src), "-o", str(obj)])
        return bench.kernel_code_hashes(str(obj))

    with ThreadPoolExecutor(3) as ex:
        h = dict(zip(variants, ex.map(compile_variant, variants)))
    assert set(h["same"]) == {"combine_kernel", "debug_bf16_kernel"}
    assert all(len(v) == 16 for v in h["same"].values())
    assert h["comment"] == h["same"]
    assert h["code"]["combine_kernel"] != h["same"]["combine_kernel"]
    assert h["code"]["debug_bf16_kernel"] == h["same"]["debug_bf16_kernel"]


def test_code_hashes_of_the_built_library():
    """Every kernel of the library is found in its gfx950 code objects."""
    if not os.path.exists(bench.LIB_PATH):
        pytest.skip("libepl.so is not built")
    h = bench.kernel_code_hashes()
    assert {"route_hist_kernel", "route_scan_kernel", "route_finalize_kernel", "route_single_kernel",
            "dispatch_bf16_kernel", "dispatch_fp8_kernel", "fused_bf16_kernel", "combine_kernel",
            "locate_rows_kernel"} <= set(h)


@pytest.mark.parametrize("name", ["tiny", "skewed_fp8_small"])
def test_threaded_oracle_leg_matches_single_thread(name):
    """The CPU baseline's threaded leg calls the unchanged oracle functions on disjoint token
    ranges; its layer is bit-identical to the single-thread one, on bf16 and on fp8."""
    if name == "tiny":
        w = W.WORKLOADS["tiny"]
    else:
        base = W.WORKLOADS["skewed_fp8_ep64"]
        w = W.Workload(name, 8, 32, 8, 16, 512, "fp8", base.routing)
    idx = W.routing(w)
    x = W.tokens_bf16(w)
    gw = W.gate_weights(w)
    legs, identical, P = bench.cpu_baseline(w, idx, x, gw, 0.2, 4)
    assert identical
    assert legs["single"][2] == 1 and legs["threads"][2] == 4
    assert P == int(((idx >= 0) & (idx < w.E)).sum())
    assert 1 <= bench.host_threads() <= (os.cpu_count() or 1)
