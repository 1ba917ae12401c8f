"""Helpers shared by the GPU parity tests (host-side marshalling and comparisons only)."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W

LAYOUT_FIELDS = ["send_cnt", "rank_cnt", "expert_off", "rank_off", "seg_off", "tok_nranks", "pair_row",
                 "pair_rslot"]


def device():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a ROCm GPU")
    return torch.device("cuda:0")


def to_dev_bf16(x_u16: np.ndarray, dev) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x_u16).view(np.int16)).view(torch.bfloat16).to(dev)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def assert_layout_equal(L: epl.Layout, ref: oracle.RefLayout, what: str = "") -> None:
    for name in LAYOUT_FIELDS:
        want = getattr(ref, name)
        got = getattr(L, name).cpu().numpy()
        got = got.reshape(-1)[: want.size].reshape(want.shape)
        if not np.array_equal(got, want):
            bad = np.argwhere(got != want)[:5]
            raise AssertionError("%s layout.%s differs at %s: got %s want %s" % (
                what, name, bad.tolist(), got[tuple(bad.T)].tolist(), want[tuple(bad.T)].tolist()))
    P = ref.P
    np.testing.assert_array_equal(L.recv_src[:P].cpu().numpy(), ref.recv_src, err_msg=what + " recv_src")
    np.testing.assert_array_equal(L.recv_j[:P].cpu().numpy(), ref.recv_j, err_msg=what + " recv_j")
    assert int(L.num_invalid.item()) == ref.num_invalid, what + " num_invalid"


def bf16_ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance between bf16 bit patterns in units in the last place (+0 and -0 coincide)."""
    def ordered(h):
        h = h.astype(np.int32)
        return np.where(h & 0x8000, -(h & 0x7FFF), h & 0x7FFF)
    return np.abs(ordered(a) - ordered(b))


def run_layout(w: W.Workload, idx: np.ndarray, dev):
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload)
    idx_d = torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev)
    return cfg, epl.layout(cfg, idx_d)


def host_threads() -> int:
    """Threads for the host-side oracle runs of the full-size tests: the CPUs this process may
    use, at most 16 (one GPU's share of a box)."""
    import os

    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    return max(1, min(n, 16))


def _token_ranges(T: int, n: int):
    step = max(1, -(-T // (4 * n)))
    return [(g, min(T, g + step)) for g in range(0, T, step)]


def oracle_dispatch_threaded(x: np.ndarray, pair_row: np.ndarray, P: int, fp8: bool):
    """The oracle's dispatch of every token, its unchanged C function called on disjoint token
    ranges from a thread pool -> recv [P, H] (and scales [P, H/128] for fp8)."""
    from concurrent.futures import ThreadPoolExecutor

    T, H = x.shape
    recv = np.zeros((max(P, 1), H), np.uint8 if fp8 else np.uint16)
    scale = np.zeros((max(P, 1), H // 128), np.float32) if fp8 else None
    n = host_threads()
    with ThreadPoolExecutor(n) as ex:
        list(ex.map(lambda r: oracle.dispatch_range_into(x, pair_row, recv, r[0], r[1], scale), _token_ranges(T, n)))
    return recv[:P], None if scale is None else scale[:P]


def oracle_combine_threaded(y: np.ndarray, w: np.ndarray, pair_row: np.ndarray) -> np.ndarray:
    """The oracle's combine of every token, on disjoint token ranges from a thread pool -> [T, H]."""
    from concurrent.futures import ThreadPoolExecutor

    T = pair_row.shape[0]
    out = np.zeros((T, y.shape[1]), np.uint16)
    w = np.ascontiguousarray(w, np.float32)
    pair_row = np.ascontiguousarray(pair_row, np.int32)
    n = host_threads()
    with ThreadPoolExecutor(n) as ex:
        list(ex.map(lambda r: oracle.combine_range_into(y, w, pair_row, out, r[0], r[1]), _token_ranges(T, n)))
    return out
