#!/usr/bin/env python3
"""Benchmark: one MoE layer's dispatch + combine hot path on one MI355X.

A step is one pass of the whole hot path over one synthetic batch: the routing layout and the row
scatter (epl_layout_dispatch, or epl_layout then epl_dispatch with --separate), then the
gather-reduce (epl_combine), with identity experts in between (combine reads the receive buffer).
Steps that carry timing events issue epl_layout_dispatch as its two phases, epl_layout_counts then
epl_dispatch_rows (the same kernels), so that the row kernel is timed on its own. All inputs are
resident in HBM before timing starts. The token matrix x is read from byte-identical copies in
turn, at least 512 MB in total, so that no step finds its input in the 256 MB memory-side cache.

Default workload: EP=64 decode. 64 virtual ranks, 256 experts (4 per rank), top-8, 128
tokens per rank (8192 tokens), hidden 7168 bf16, uniform routing without replacement, softmax
gate weights.

Output: one JSON line. It carries:
* effective HBM GB/s, computed from the algorithmic bytes per layer;
* µs per layer and per call;
* the roofline entry of the dominant kernel, timed with HIP events on its own stream;
* the CPU oracle timed on the host as a reported baseline.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "dispatch+combine µs/MoE layer and effective HBM GB/s (% of peak), EP=64 decode"
HBM_PEAK_GBS = 8000.0
X_ROTATION_BYTES = 512 << 20  # twice the MI355X memory-side cache
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
ROOFLINE_SAMPLES = 20  # launches of the dominant kernel timed with HIP events, at least
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000  # hipEventDisableSystemFence


class FenceFreeEvent:
    """A HIP timing event created with hipEventDisableSystemFence. Recording a plain event (as
    torch.cuda.Event does) also issues a system-scope release, whose cache write-back lands in the
    interval the event brackets; this one only takes the timestamp. Read it after a device
    synchronize. Decode combine, one box, 20 launches: 186.8-187.6 us with these events,
    188.1-189.8 us with torch's, against 186.4 us averaged by rocprofv3 on another box; the
    layer's wall time was the same with either kind of marker."""

    _rt = None

    def __init__(self, epl):
        if FenceFreeEvent._rt is None:
            rt = epl._hip_runtime()
            rt.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            rt.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
            FenceFreeEvent._rt = rt
        self.h = ctypes.c_void_p()
        rc = self._rt.hipEventCreateWithFlags(ctypes.byref(self.h), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError("hipEventCreateWithFlags failed (%d)" % rc)

    def record(self, stream):
        rc = self._rt.hipEventRecord(self.h, ctypes.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError("hipEventRecord failed (%d)" % rc)

    def elapsed_time(self, end):
        ms = ctypes.c_float()
        rc = self._rt.hipEventElapsedTime(ctypes.byref(ms), self.h, end.h)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed (%d)" % rc)
        return ms.value

    def __del__(self):
        if self.h.value and self._rt is not None:
            try:
                self._rt.hipEventDestroy(self.h)
            except Exception:  # interpreter shutdown: the runtime may already be gone
                pass


def algorithmic_bytes(T, k, H, R, E, P, payload):
    """Bytes the method itself must move (each token row read once, each pair row written once
    by dispatch and read once by combine, the routing tables read and the metadata written)."""
    NB = H // 128
    b = 1 if payload == "fp8" else 2
    dispatch = T * H * 2 + T * k * 4 + P * H * b + (P * NB * 4 if payload == "fp8" else 0)
    combine = P * H * 2 + 2 * T * k * 4 + T * H * 2
    placement = 4 * ((E + 1) + (R + 1) + E * R + 2 * T * k + 2 * P)  # offsets, pair rows/slots, recv_src/j
    layout = T * k * 4 + 4 * (R * E + R * R + T + 1) + placement
    # The row kernel with the layout's finalize step fused in also writes the placement metadata.
    return {"layout": layout, "dispatch": dispatch, "combine": combine, "rows_fused": dispatch + placement,
            "total": layout + dispatch + combine}


LIB_PATH = os.path.join(ROOT, "paper_2607_06202_amd", "libepl.so")
_BUNDLE_MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def _elf_kernels(elf):
    """(mangled name, code bytes, kernel descriptor bytes) of every kernel in one AMDGPU code
    object (ELF64, little endian): the function symbols' bytes and their `.kd` objects."""
    import struct

    shoff, = struct.unpack_from("<Q", elf, 0x28)
    shentsize, shnum = struct.unpack_from("<HH", elf, 0x3A)
    secs = [struct.unpack_from("<IIQQQQIIQQ", elf, shoff + i * shentsize) for i in range(shnum)]
    syms = {}
    for sec in secs:
        if sec[1] not in (2, 11):  # SHT_SYMTAB, SHT_DYNSYM
            continue
        strtab = secs[sec[6]]
        for off in range(sec[4], sec[4] + sec[5], 24):
            name_off, info, _, shndx, value, size = struct.unpack_from("<IBBHQQ", elf, off)
            if shndx == 0 or shndx >= len(secs) or size == 0:
                continue
            start = strtab[4] + name_off
            name = elf[start:elf.index(b"\0", start)].decode()
            tgt = secs[shndx]
            syms[name] = (info & 0xF, bytes(elf[tgt[4] + value - tgt[3]:tgt[4] + value - tgt[3] + size]))
        break
    out = []
    for name, (typ, code) in syms.items():
        if typ == 2 and name + ".kd" in syms:  # STT_FUNC with a kernel descriptor
            kd = bytearray(syms[name + ".kd"][1])
            kd[16:24] = bytes(8)  # entry offset: depends on where the kernel sits, not on its code
            out.append((name, code, bytes(kd)))
    return out


def kernel_code_hashes(path=LIB_PATH):
    """Hash of each kernel's gfx950 machine code and descriptor in a built library or object,
    keyed by the kernel's unqualified name (template instances hashed together). Counter data
    taken on a kernel stays valid exactly as long as this hash does."""
    import re
    import struct

    data = open(path, "rb").read()
    parts = {}
    for m in re.finditer(re.escape(_BUNDLE_MAGIC), data):
        b = m.start()
        n, = struct.unpack_from("<Q", data, b + 24)
        pos = b + 32
        for _ in range(n):
            off, size, tlen = struct.unpack_from("<QQQ", data, pos)
            triple = data[pos + 24:pos + 24 + tlen].decode()
            pos += 24 + tlen
            if "amdgcn" in triple and "gfx950" in triple:
                for name, code, kd in _elf_kernels(data[b + off:b + off + size]):
                    mm = re.match(r"_ZN3epl(\d+)", name)
                    base = name[mm.end():mm.end() + int(mm.group(1))] if mm else name
                    parts.setdefault(base, []).append((name, code, kd))
    hashes = {}
    for base, items in parts.items():
        h = hashlib.sha256()
        for name, code, kd in sorted(items):
            h.update(name.encode() + code + kd)
        hashes[base] = h.hexdigest()[:16]
    return hashes


_CODE_HASHES = None


def code_hash(kernel):
    global _CODE_HASHES
    if _CODE_HASHES is None:
        _CODE_HASHES = kernel_code_hashes() if os.path.exists(LIB_PATH) else {}
    return _CODE_HASHES.get(kernel)


def load_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were taken on the
    kernel's current machine code; else None."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    ent = rec.get("kernels", {}).get("%s@%s" % (kernel, workload))
    if not ent or ent.get("code_hash") is None or ent.get("code_hash") != code_hash(kernel):
        return None
    return ent.get("bytes_per_launch")


def _counter_means(csv_path):
    """Mean counter value (KiB) per kernel name from a rocprofv3 --pmc counter_collection.csv."""
    import csv
    from collections import defaultdict

    vals = defaultdict(list)
    for r in csv.DictReader(open(csv_path)):
        name = r["Kernel_Name"].split("(")[0].replace("void ", "").strip()
        vals[name].append(float(r["Counter_Value"]))
    return vals


def ingest_counters(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, workload, command):
    """Turn four rocprofv3 --pmc runs (FETCH_SIZE and WRITE_SIZE over this bench, and over
    --calibrate-copy) into profiles/hbm_traffic.json and a text summary. The copy moves exactly
    2^30 bytes each way, so bytes/counter for it calibrates the kernels' readings."""
    n = float(1 << 30)
    cf = _counter_means(copy_fetch_csv)["__amd_rocclr_copyBuffer"]
    cw = _counter_means(copy_write_csv)["__amd_rocclr_copyBuffer"]
    fetch_factor = n / (float(np.median(cf)) * 1024)
    write_factor = n / (float(np.median(cw)) * 1024)
    fetch = _counter_means(fetch_csv)
    write = _counter_means(write_csv)
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        rec = {"kernels": {}}
    # Entries taken on older kernel sources no longer describe any kernel: drop them.
    rec["kernels"] = {k: v for k, v in rec.get("kernels", {}).items()
                      if v.get("code_hash") is not None and v.get("code_hash") == code_hash(k.split("@")[0])}
    rec["calibration"] = {"fetch_factor": round(fetch_factor, 4), "write_factor": round(write_factor, 4),
                          "copy_bytes_each_way": int(n), "copy_fetch_kib": float(np.median(cf)),
                          "copy_write_kib": float(np.median(cw))}
    lines = ["HBM traffic per launch, workload %s (rocprofv3 FETCH_SIZE / WRITE_SIZE, KiB per dispatch)" % workload,
             "commands:", *["  " + c for c in command],
             "calibration: 1 GiB device copy reads FETCH_SIZE %.1f KiB (factor %.4f), WRITE_SIZE %.1f KiB (factor %.4f)"
             % (np.median(cf), fetch_factor, np.median(cw), write_factor),
             "%-40s %8s %14s %14s %16s  %s" % ("kernel", "launches", "FETCH KiB", "WRITE KiB", "HBM bytes (cal.)",
                                                "code hash")]
    for name in fetch:
        if not name.startswith("epl::"):
            continue
        short = name.split("::")[1].split("<")[0]
        fk, wk = float(np.mean(fetch[name])), float(np.mean(write.get(name, [0.0])))
        b = fk * 1024 * fetch_factor + wk * 1024 * write_factor
        rec["kernels"]["%s@%s" % (short, workload)] = {"code_hash": code_hash(short), "fetch_kib": fk,
                                                        "write_kib": wk, "bytes_per_launch": int(round(b))}
        lines.append("%-40s %8d %14.1f %14.1f %16d  %s" % (name, len(fetch[name]), fk, wk, b, code_hash(short)))
    json.dump(rec, open(TRAFFIC_FILE, "w"), indent=1, sort_keys=True)
    txt = os.path.join(ROOT, "profiles", "hbm_counters_%s.txt" % workload)
    open(txt, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def device_info(torch):
    """The GPU's identity and the settings that move HBM-bound numbers between boxes (memory vendor,
    current memory clock, package power cap), read from torch and from the amdgpu driver's sysfs
    files of the same PCI device (no child process); missing fields are null."""
    import glob

    p = torch.cuda.get_device_properties(0)
    info = {"arch": p.gcnArchName.split(":")[0], "cus": p.multi_processor_count,
            "hbm_gib": round(p.total_memory / 2 ** 30, 1), "memory_vendor": None, "mclk_mhz": None,
            "max_package_power_w": None}
    bdf = "%04x:%02x:%02x." % (p.pci_domain_id, p.pci_bus_id, p.pci_device_id)
    for card in glob.glob("/sys/class/drm/card[0-9]*"):
        dev = os.path.join(card, "device")
        if "-" in os.path.basename(card) or not os.path.basename(os.path.realpath(dev)).startswith(bdf):
            continue
        try:
            info["memory_vendor"] = open(os.path.join(dev, "mem_info_vram_vendor")).read().strip()
        except OSError:
            pass
        try:
            for line in open(os.path.join(dev, "pp_dpm_mclk")).read().splitlines():
                if line.rstrip().endswith("*"):  # the current level
                    info["mclk_mhz"] = int(line.split(":")[1].strip(" *").lower().replace("mhz", ""))
        except (OSError, ValueError, IndexError):
            pass
        try:
            cap = sorted(glob.glob(os.path.join(dev, "hwmon", "hwmon*", "power1_cap")))
            if cap:
                info["max_package_power_w"] = int(open(cap[0]).read()) / 1e6  # microwatts
        except (OSError, ValueError):
            pass
        info["temp_c"] = gpu_temperatures(dev)
        info["_sysfs"] = dev
        break
    return info


def device_end(info):
    """The device fields for the output line, with the temperatures read again after the run."""
    out = dict(info)
    sysfs = out.pop("_sysfs", None)
    out["temp_c_end"] = gpu_temperatures(sysfs) if sysfs else {}
    return out


def gpu_temperatures(dev_dir):
    """The driver's temperature sensors of one GPU ({label: degrees C}, e.g. edge, junction,
    mem), from its hwmon files; empty if there are none."""
    import glob

    temps = {}
    for lab in sorted(glob.glob(os.path.join(dev_dir, "hwmon", "hwmon*", "temp*_label"))):
        try:
            name = open(lab).read().strip()
            temps[name] = int(open(lab.replace("_label", "_input")).read()) / 1000.0  # millidegrees
        except (OSError, ValueError):
            pass
    return temps


def host_threads():
    """Host threads the CPU baseline may use: the cores this process may run on, capped by
    OMP_NUM_THREADS when that is set (the share of the host given to one GPU's jobs)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit() and int(cap) > 0:
        n = min(n, int(cap))
    return max(1, n)


def cpu_baseline(w, idx, x, gw, budget_s, threads):
    """The oracle, unchanged, timed on this host's CPU on the same inputs, two ways:
    * single thread: oracle.layout, then the dispatch and the combine over all tokens;
    * `threads` threads: the same layout call, then the unchanged dispatch and combine functions
      called on disjoint token ranges from a thread pool (ctypes releases the GIL): scatter and
      combine split by token range, the layout kept serial.
    The threaded layer's receive rows and output must equal the single-thread ones bit for bit.
    For fp8 the combine reads a bf16 buffer of zeros, as the GPU layer does. Each leg runs whole
    layers until its half of the budget is spent (at least one)."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle

    fp8 = w.payload == "fp8"
    T, H, k = w.T, w.H, w.k

    def layer(recv, scale, out, pool=None, ranges=None):
        L = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
        y = recv if not fp8 else y_zero
        if pool is None:
            oracle.dispatch_range_into(x, L.pair_row, recv, 0, T, scale)
            oracle.combine_range_into(y, gw, L.pair_row, out, 0, T)
        else:
            list(pool.map(lambda r: oracle.dispatch_range_into(x, L.pair_row, recv, r[0], r[1], scale), ranges))
            list(pool.map(lambda r: oracle.combine_range_into(y, gw, L.pair_row, out, r[0], r[1]), ranges))
        return L.P

    rows = max(T * k, 1)
    y_zero = np.zeros((rows, H), np.uint16) if fp8 else None
    legs = {}
    outputs = {}
    for name, n in (("single", 1), ("threads", threads)):
        recv = np.zeros((rows, H), np.uint8 if fp8 else np.uint16)
        scale = np.zeros((rows, H // 128), np.float32) if fp8 else None
        out = np.zeros((T, H), np.uint16)
        step = max(1, -(-T // (4 * n)))  # a few ranges per thread
        ranges = [(g, min(T, g + step)) for g in range(0, T, step)]
        pool = ThreadPoolExecutor(n) if n > 1 else None
        t0 = time.perf_counter()
        reps = 0
        while True:
            P_ref = layer(recv, scale, out, pool, ranges)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s / 2 or reps >= 50:
                break
        if pool is not None:
            pool.shutdown()
        legs[name] = (el / reps, reps, n)
        outputs[name] = (recv[:P_ref], None if scale is None else scale[:P_ref], out)
    a, b = outputs["single"], outputs["threads"]
    identical = bool(np.array_equal(a[0], b[0]) and np.array_equal(a[2], b[2]) and
                     (a[1] is None or np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32))))
    return legs, identical, P_ref


def calibrate_replicate(torch, epl, w, dev, stream, steps):
    """The dispatch's byte pattern, one read and k writes per token row, with the k writes
    contiguous: x [T,H] -> [T,k,H]. Timed two ways on an x of the workload's shape (rotated
    copies, as in the layer):
    * torch's broadcast copy (a vendor elementwise kernel);
    * epl_dispatch itself, on a layout that sends every pair of every token to one expert of one
      rank, so pair (g, j) lands in row g*k + j (sequential rows instead of the routed scatter)."""
    x = torch.empty(w.T, w.H, dtype=torch.bfloat16, device=dev).normal_()
    n_x = max(2, -(-X_ROTATION_BYTES // (x.numel() * 2)))
    xs = [x] + [x.clone() for _ in range(n_x - 1)]
    dst = torch.empty(w.T, w.k, w.H, dtype=torch.bfloat16, device=dev)
    cfg = epl.config(1, 1, w.k, w.H, w.T, "bf16")
    L = epl.layout(cfg, torch.zeros(w.T, w.k, dtype=torch.int32, device=dev))
    recv = dst.view(w.T * w.k, w.H)
    runs = {"torch_broadcast_copy": lambda i: dst.copy_(xs[i % n_x].unsqueeze(1).expand(w.T, w.k, w.H)),
            "epl_dispatch_sequential_rows": lambda i: epl.dispatch(cfg, xs[i % n_x], L, recv)}
    nbytes = x.numel() * 2 + dst.numel() * 2
    out = {"calibration": "replicate x[T,H] -> [T,k,H]", "workload": w.name, "T": w.T, "k": w.k, "H": w.H,
           "bytes_read": x.numel() * 2, "bytes_written": dst.numel() * 2, "x_copies": n_x}
    for name, fn in runs.items():
        for i in range(5):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(steps):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / steps
        out[name] = {"us": round(us, 2), "GBps": round(nbytes / us / 1e3, 1),
                     "pct_of_peak": round(100 * nbytes / us / 1e3 / HBM_PEAK_GBS, 2)}
    ref = torch.empty_like(dst).copy_(xs[(steps - 1) % n_x].unsqueeze(1).expand(w.T, w.k, w.H))
    epl.dispatch(cfg, xs[(steps - 1) % n_x], L, recv)
    out["rows_equal"] = bool(torch.equal(ref.view(torch.int16), dst.view(torch.int16)))
    print(json.dumps(out))


def cpu_model():
    """The host CPU as /proc/cpuinfo names it, with its family, model and stepping numbers (a
    virtualised host may report only a short brand name), and the logical CPUs it lists."""
    fields = {}
    ncpu = 0
    try:
        for line in open("/proc/cpuinfo"):
            key, _, val = line.partition(":")
            key = key.strip()
            if key == "processor":
                ncpu += 1
            if key in ("model name", "cpu family", "model", "stepping", "vendor_id") and key not in fields:
                fields[key] = val.strip()
    except OSError:
        return None
    if not fields:
        return None
    return "%s (vendor %s, family %s, model %s, stepping %s; %d logical CPUs listed)" % (
        fields.get("model name", "?"), fields.get("vendor_id", "?"), fields.get("cpu family", "?"),
        fields.get("model", "?"), fields.get("stepping", "?"), ncpu)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="decode_ep64")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle CPU time (0 to skip)")
    ap.add_argument("--roofline-samples", type=int, default=ROOFLINE_SAMPLES,
                    help="launches of the dominant call timed with HIP events, at least: every 10th timed step, "
                         "topped up by steps right after the timed region")
    ap.add_argument("--separate", action="store_true",
                    help="time epl_layout, epl_dispatch and epl_combine as three calls instead of "
                         "epl_layout_dispatch + epl_combine")
    ap.add_argument("--decomposed", action="store_true",
                    help="time epl_layout_dispatch_decomposed (layout and dispatch in one launch of count and send "
                         "workgroups) + epl_combine")
    ap.add_argument("--sentinel-layer", action="store_true",
                    help="time epl_layer_sentinel: layout, dispatch and the combine of the dispatched rows in one "
                         "launch, synchronised per row by Sentinel Polling")
    ap.add_argument("--layer-flags", choices=["flag", "checksum"], default=None,
                    help="time epl_layer_data_as_flag: the one-launch layer synchronised per 1 KiB chunk by "
                         "Token-Flag Fusion (flag) or Data-for-Checksum (checksum), a new epoch every call")
    ap.add_argument("--scheduled", type=int, default=0, metavar="WORKERS",
                    help="time epl_layout + epl_dispatch_scheduled (WORKERS workgroups per source rank, each "
                         "sending one equal slice of the rank's pairs in the transposed expert order) + epl_combine")
    ap.add_argument("--remap-rows", type=int, default=0,
                    help="rows of the expert transposition of --scheduled (0: one per worker; 1: natural order)")
    ap.add_argument("--shape", type=int, nargs=5, metavar=("R", "E", "K", "TR", "H"),
                    help="a custom bf16 workload with uniform routing instead of --workload: R ranks, E experts, "
                         "top-K, TR tokens per rank, hidden size H")
    ap.add_argument("--count-groups", type=int, default=0,
                    help="count workgroups of the decomposed launch (0: the library's default split)")
    ap.add_argument("--graph", action="store_true",
                    help="time HIP graph replays of the layer (one graph per x copy) instead of eager launches")
    ap.add_argument("--recv-alloc", choices=["contiguous", "torch"], default="contiguous",
                    help="receive buffer: one physically contiguous HIP block (default) or torch's allocator")
    ap.add_argument("--row-pitch", default="auto",
                    help="elements from one receive row to the next: 'auto' (the measured pitch of the binding's "
                         "TUNED_PITCH table: 7936 for bf16 rows of 7168, else packed), 0 (packed, H) or a multiple "
                         "of 64 >= H")
    ap.add_argument("--warm", action="store_true",
                    help="read the same x every step (it may stay in the memory-side cache) instead of rotating copies")
    ap.add_argument("--calibrate-copy", action="store_true", help="time a plain 1 GiB device copy instead")
    ap.add_argument("--calibrate-replicate", action="store_true",
                    help="time the dispatch's 1-read : k-write byte pattern with sequential rows instead "
                         "(torch's broadcast copy, and epl_dispatch on an all-to-one layout)")
    ap.add_argument("--ingest-counters", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="write profiles/hbm_traffic.json from rocprofv3 --pmc runs (no GPU needed)")
    ap.add_argument("--command", action="append", default=[], help="profiler command recorded with --ingest-counters")
    args = ap.parse_args()
    args.fused = not args.separate
    if args.ingest_counters:
        ingest_counters(*args.ingest_counters, args.workload, args.command)
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU hot path only: every expert-parallel rank is a virtual rank "
              "in one GPU's HBM; --gpus %d (WORLD_SIZE %d) is not supported" % (args.gpus, world),
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_06202_amd import epl
    from paper_2607_06202_amd import workloads as W

    if not os.path.exists(epl.LIB_PATH):
        from paper_2607_06202_amd import _build
        _build.build()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream(dev)

    if args.calibrate_copy:
        n = 1 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev).random_(0, 255)
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            b.copy_(a)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "ms": ms,
                          "GBps": 2 * n / ms / 1e6}))
        return

    if args.shape:
        R, E, K, TR, H = args.shape
        w = W.Workload("custom_r%d_e%d_k%d_t%d_h%d" % (R, E, K, TR, H), R, E, K, TR, H, "bf16", "uniform")
    else:
        w = W.WORKLOADS[args.workload]
    dinfo = device_info(torch)  # read before the run: the temperatures are those at the start
    if args.calibrate_replicate:
        calibrate_replicate(torch, epl, w, dev, stream, args.steps)
        return
    idx = W.routing(w, args.seed)
    x = W.tokens_bf16(w, args.seed)
    gw = W.gate_weights(w, args.seed)
    pitch = epl.tuned_pitch(w.H, w.payload) if args.row_pitch == "auto" else int(args.row_pitch)
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload, row_pitch=pitch)

    idx_d = torch.from_numpy(idx).to(dev)
    x_d = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
    # Byte-identical copies of x at distinct addresses, used in turn, at least twice the
    # 256 MB memory-side cache (MALL) in total: every step's dispatch then reads its input from
    # HBM instead of finding the previous step's x still cached.
    x_bytes = x_d.numel() * x_d.element_size()
    n_x = max(2, -(-X_ROTATION_BYTES // x_bytes)) if x_bytes and not args.warm else 1
    xs = [x_d] + [x_d.clone() for _ in range(n_x - 1)]
    w_d = torch.from_numpy(gw).to(dev)
    L = epl.alloc_layout(cfg, dev)
    # The receive rows as one physically contiguous block, as a serving process would allocate them
    # once (torch's allocator if the driver has no such block, or with --recv-alloc torch).
    recv_alloc = args.recv_alloc
    if recv_alloc == "contiguous":
        try:
            recv, recv_scale = epl.alloc_recv(cfg, dev, contiguous=True)
        except (MemoryError, OSError):  # no contiguous block free, or the HIP runtime not found by name
            recv_alloc = "torch"
    if recv_alloc == "torch":
        recv, recv_scale = epl.alloc_recv(cfg, dev)
    out = torch.empty(w.T, w.H, dtype=torch.bfloat16, device=dev)
    if w.payload == "fp8":
        # combine reads bf16 expert outputs; identity experts would dequantise -- here a bf16
        # buffer of the same shape stands in for them (not timed)
        y = torch.zeros(epl.recv_rows_cap(cfg), cfg.pitch, dtype=torch.bfloat16, device=dev)[:, :w.H]
    else:
        y = recv

    mode = ("sentinel" if args.sentinel_layer else args.layer_flags if args.layer_flags else
            "decomposed" if args.decomposed else
            "scheduled" if args.scheduled else "fused" if args.fused else "separate")
    layer_modes = ("sentinel", "flag", "checksum")  # one launch for the whole layer, combine included
    if mode in layer_modes and w.payload != "bf16":
        raise SystemExit("the one-launch layers run bf16 layers only")
    if mode == "sentinel":
        epl.sentinel_fill(recv)  # once; every layer leaves the receive buffer so
    marks = None
    epoch = [0]
    if mode in ("flag", "checksum"):
        if args.graph:
            raise SystemExit("--layer-flags takes a new epoch on every call, which a graph replay cannot")
        marks = epl.alloc_marks(cfg, dev, recv.shape[0])
        variant = epl.DAF_TOKEN_FLAG_FUSION if mode == "flag" else epl.DAF_DATA_CHECKSUM
    status_d = torch.zeros(1, dtype=torch.int32, device=dev)

    def layout_dispatch(i, mark=None):
        """Layout and dispatch of step i. mark(), when given, runs between the layout's kernels and
        the row kernel; the decomposed call is one launch, so there it runs before it."""
        xi = xs[i % n_x]
        if mode == "sentinel":  # the whole layer, combine included, in one launch
            if mark is not None:
                mark()
            epl.layer_sentinel(cfg, idx_d, xi, w_d, recv, out=out, layout_out=L, count_groups=args.count_groups,
                               status=status_d)
        elif mode in ("flag", "checksum"):  # likewise, with a new epoch each call
            if mark is not None:
                mark()
            epoch[0] += 1
            epl.layer_data_as_flag(cfg, idx_d, xi, w_d, recv, marks, variant, epoch[0], out=out, layout_out=L,
                                   count_groups=args.count_groups, status=status_d)
        elif mode == "decomposed":
            if mark is not None:
                mark()
            epl.layout_dispatch_decomposed(cfg, idx_d, xi, out=L, recv=recv, count_groups=args.count_groups,
                                           status=status_d)
        elif mode == "scheduled":
            epl.layout(cfg, idx_d, out=L)
            if mark is not None:
                mark()
            epl.dispatch_scheduled(cfg, xi, L, args.scheduled, remap_rows=args.remap_rows, recv=recv,
                                   recv_scale=recv_scale)
        elif mode == "fused" and mark is None:
            epl.layout_dispatch(cfg, idx_d, xi, out=L, recv=recv, recv_scale=recv_scale)
        else:
            if mode == "fused":
                epl.layout_counts(cfg, idx_d, out=L)
            else:
                epl.layout(cfg, idx_d, out=L)
            if mark is not None:
                mark()
            if mode == "fused":
                epl.dispatch_rows(cfg, idx_d, xi, L, recv, recv_scale)
            else:
                epl.dispatch(cfg, xi, L, recv, recv_scale)

    def step(i, ev=None):
        # With events the fused call is issued as its two phases (the same kernels), so the legs
        # are epl_layout_counts and epl_dispatch_rows.
        if ev is not None:
            ev[0].record(stream)
        layout_dispatch(i, None if ev is None else (lambda: ev[1].record(stream)))
        if ev is not None:
            ev[2].record(stream)
        if mode not in layer_modes:
            epl.combine(cfg, y, w_d, L, out)
        if ev is not None:
            ev[3].record(stream)

    def timed_events(n):
        return [[FenceFreeEvent(epl) for _ in range(4)] for _ in range(n)]

    def per_call_us(evs):
        return np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3])] for e in evs]) * 1e3

    # Warm-up: all but the last step instrumented (they also pick the dominant call for the
    # roofline entry); the last one runs plain right before the timed region (below), so that the
    # GPU does not sit idle between warm-up and timing. A 20-step region after 20 ms of idle measured
    # 382.4 us per decode step, against 379.9 us with none and 380.1 us over 200 steps.
    n_warm = max(args.warmup, 1)
    n_instr = n_warm - 1 if n_warm > 1 else 1
    wev = timed_events(n_instr)
    for i in range(n_instr):
        step(i, wev[i])
    torch.cuda.synchronize()
    P = int(L.expert_off[-1].item())
    wper = np.median(per_call_us(wev), axis=0)  # robust to a slow first step
    dom = "dispatch" if wper[1] >= wper[2] else "combine"

    graphs = None
    if args.graph:
        # One captured layer per x copy; capture runs on a side stream after an eager warm-up there.
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            for i in range(n_x):
                step(i)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graphs = []
        for i in range(n_x):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(i)
            graphs.append(g)
        for i in range(max(args.warmup, 1)):
            graphs[i % n_x].replay()
        torch.cuda.synchronize()

    # The default call sequence through the binding's prepared calls: every argument checked and
    # converted once, so a step costs the host two C calls (the first step of a timed region
    # otherwise waits some 60 us for the binding's checks before its first kernel is enqueued).
    prep = (epl.PreparedLayer(cfg, idx_d, xs, w_d, L, recv, recv_scale, y=y, out=out)
            if mode == "fused" else None)

    def run_steps(first, n, dev_ev):
        """n plain steps starting at step index `first`; the steps in dev_ev bracket only the
        dominant call with two HIP events on the library's stream."""
        for i in range(first, first + n):
            if graphs is not None:
                graphs[i % n_x].replay()
                continue
            ev = dev_ev.get(i)
            if prep is not None:
                if ev is not None and dom == "dispatch":
                    prep.layout_counts()
                    ev[0].record(stream)
                    prep.dispatch_rows(i)
                    ev[1].record(stream)
                    prep.combine()
                    continue
                prep.layout_dispatch(i)
                if ev is not None:
                    ev[0].record(stream)
                prep.combine()
                if ev is not None:
                    ev[1].record(stream)
                continue
            if ev is not None and dom == "dispatch":
                layout_dispatch(i, lambda: ev[0].record(stream))
                ev[1].record(stream)
            else:
                layout_dispatch(i)
                if ev is not None:
                    ev[0].record(stream)
            if mode not in layer_modes:
                epl.combine(cfg, y, w_d, L, out)
            if ev is not None and dom == "combine":
                ev[1].record(stream)

    def events_for(indices):
        return {i: (FenceFreeEvent(epl), FenceFreeEvent(epl)) for i in indices}

    # Timed region: K plain steps. Every 10th of them (steps 5, 15, ...) brackets only the dominant call with two
    # fence-free HIP events (two plain markers per step cost about 6 us of wall time at decode, so not every step
    # carries them). When that gives fewer than --roofline-samples launches, as at K = 20, the
    # rest are sampled right after the timed region, on further steps of the same layer. Graph
    # replays take no markers; the dominant call's duration then comes from the instrumented
    # pass below.
    in_region = events_for([i for i in range(args.steps) if i % 10 == 5] if graphs is None else [])
    if n_warm > n_instr:  # the last warm-up step, plain, then straight into the timed region
        run_steps(n_warm - 1, 1, {})
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run_steps(0, args.steps, in_region)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    top_up = {}
    if graphs is None and len(in_region) < args.roofline_samples:
        n_more = args.roofline_samples - len(in_region)
        top_up = events_for(range(args.steps, args.steps + n_more))
        run_steps(args.steps, n_more, top_up)
        torch.cuda.synchronize()
    dev_ev = {**in_region, **top_up}

    decomposed_split = None
    if mode in layer_modes and int(status_d.item()) != 0:
        raise RuntimeError("a wait of the one-launch layer gave up (status %d)" % int(status_d.item()))
    if mode == "decomposed":
        if int(status_d.item()) != 0:
            raise RuntimeError("a wait of the decomposed launch gave up (status %d)" % int(status_d.item()))
        n_count, grid, capacity = epl.decomposed_plan(cfg, args.count_groups)
        decomposed_split = {"count": n_count, "send": grid - n_count, "capacity": capacity}

    # Per-call breakdown: a separate instrumented pass (events between every call).
    bev = timed_events(args.steps)
    for i in range(args.steps):
        step(i, bev[i])
    torch.cuda.synchronize()
    per = per_call_us(bev)
    us_layout, us_dispatch, us_combine = per.mean(axis=0).tolist()
    us_layer_events = float(per.sum(axis=1).mean())
    if dev_ev:
        dom_us = float(np.mean([a.elapsed_time(b) for a, b in dev_ev.values()]) * 1e3)
    else:
        dom_us = float(np.mean(per[:, 1 if dom == "dispatch" else 2]))

    pct = lambda a: [round(float(v), 2) for v in np.percentile(a, [10, 50, 90])]
    legs = {"decomposed": ("before_launch", "layout_dispatch_decomposed"), "fused": ("layout_counts", "dispatch_rows"),
            "separate": ("layout", "dispatch"), "sentinel": ("before_launch", "layer_sentinel"),
            "flag": ("before_launch", "layer_data_as_flag"), "checksum": ("before_launch", "layer_data_as_flag"),
            "scheduled": ("layout", "dispatch_scheduled")}[mode]
    percentiles = {legs[0]: pct(per[:, 0]), legs[1]: pct(per[:, 1]), "combine": pct(per[:, 2]),
                   "layer": pct(per.sum(axis=1))}

    nbytes = algorithmic_bytes(w.T, w.k, w.H, w.R, w.E, P, w.payload)
    value = nbytes["total"] / (ms_per_step * 1e-3) / 1e9
    # Bytes a multi-GPU dispatch would put on the fabric: one row per (token, destination rank)
    # pair after dedup, excluding a token's own rank (rank_cnt off the diagonal).
    rc = L.rank_cnt.cpu().numpy().astype(np.int64)
    fabric_pairs = int(rc.sum() - np.trace(rc))
    row_bytes = w.H * 2 if w.payload == "bf16" else w.H + (w.H // 128) * 4

    # The dispatch leg is one kernel: the plain dispatch kernel, or (epl_dispatch_rows with the
    # layout's finalize fused in) the fused row kernel, whose bytes include the placement metadata.
    launches = 1 if mode in ("decomposed",) + layer_modes else epl.layout_dispatch_launches(cfg) if mode == "fused" else None
    row_fused = mode == "fused" and launches == 3
    if mode == "decomposed" and dom == "dispatch":
        dom_bytes = nbytes["layout"] + nbytes["dispatch"]  # the one launch does the whole layout and dispatch
    elif mode in layer_modes:
        dom, dom_bytes = "dispatch", nbytes["total"]  # the one launch is the whole layer
    else:
        dom_bytes = nbytes["rows_fused" if row_fused and dom == "dispatch" else dom]
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9
    kname = {"dispatch": "decomposed_kernel" if mode in ("decomposed",) + layer_modes else
             "dispatch_scheduled_kernel" if mode == "scheduled" else
             "fused_bf16_kernel" if row_fused else
             "dispatch_fp8_kernel" if w.payload == "fp8" else "dispatch_bf16_kernel",
             "combine": "combine_kernel"}[dom]
    traffic = load_traffic(kname, w.name)
    roofline = {"bound": "hbm", "kernel": kname, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "algorithmic_bytes": dom_bytes,
                # the counter bytes over the same duration: the HBM rate the kernel really moved
                "traffic_GBps": None if traffic is None else round(traffic / (dom_us * 1e-6) / 1e9, 1),
                "avg_launch_us": round(dom_us, 2), "launches_sampled": len(dev_ev) if dev_ev else args.steps,
                "launches_sampled_in_timed_region": len(in_region) if dev_ev else 0}

    cpu = None
    if args.cpu_budget > 0:
        legs, identical, P_ref = cpu_baseline(w, idx, x, gw, args.cpu_budget, host_threads())
        assert P_ref == P
        if not identical:
            raise AssertionError("threaded oracle layer differs from the single-thread one")
        (sec1, reps1, _), (secn, repsn, nthr) = legs["single"], legs["threads"]
        cpu = {"value": round(nbytes["total"] / secn / 1e9, 3), "unit": "GB/s", "cores": nthr, "kind": "oracle",
               "cpu_model": cpu_model(), "us_per_layer": round(secn * 1e6, 1),
               "sample": "%d full %s layer(s) (layout+dispatch+combine) on the same inputs; layout on one thread, "
                         "dispatch and combine on %d threads over disjoint token ranges" % (repsn, w.name, nthr),
               "bit_identical_to_single_thread": identical,
               "single_thread": {"value": round(nbytes["total"] / sec1 / 1e9, 3), "unit": "GB/s", "cores": 1,
                                 "us_per_layer": round(sec1 * 1e6, 1),
                                 "sample": "%d full layer(s), one thread" % reps1}}

    rec = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.payload, "data": "synthetic",
        "config": {"workload": w.name, "ranks": w.R, "experts": w.E, "topk": w.k, "tokens_per_rank": w.T // w.R,
                   "hidden": w.H, "payload": w.payload, "routing": w.routing, "pairs": P, "seed": args.seed,
                   "row_pitch": cfg.pitch},
        "us_per_layer": round(ms_per_step * 1e3, 2), "us_per_layer_instrumented": round(us_layer_events, 2),
        "us_layout": round(us_layout, 2), "us_dispatch": round(us_dispatch, 2),
        "us_layout_dispatch": round(us_dispatch + us_layout, 2),
        "us_combine": round(us_combine, 2),
        "pct_of_peak": round(100 * value / HBM_PEAK_GBS, 2), "algorithmic_bytes_per_layer": nbytes["total"],
        "device": device_end(dinfo),
        "launch": "graph" if graphs is not None else "eager",
        "calls": {"decomposed": "epl_layout_dispatch_decomposed + epl_combine", "sentinel": "epl_layer_sentinel",
                  "flag": "epl_layer_data_as_flag (Token-Flag Fusion)",
                  "checksum": "epl_layer_data_as_flag (Data-for-Checksum)",
                  "fused": "epl_layout_dispatch + epl_combine",
                  "separate": "epl_layout + epl_dispatch + epl_combine",
                  "scheduled": "epl_layout + epl_dispatch_scheduled + epl_combine"}[mode],
        "count_groups": decomposed_split,
        "schedule": {"workers": args.scheduled, "remap_rows": args.remap_rows or args.scheduled}
        if mode == "scheduled" else None,
        "layout_dispatch_launches": launches,
        "per_call_us_p10_p50_p90": percentiles, "layout_launches": epl.layout_launches(cfg),
        "fabric_equivalent_bytes": fabric_pairs * row_bytes, "fabric_row_pairs": fabric_pairs,
        "roofline": roofline, "x_copies": n_x, "x_reuse": "warm" if args.warm else "rotated", "recv_alloc": recv_alloc,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
