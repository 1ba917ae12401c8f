"""CPU oracle for MoE dispatch / combine -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package. The product path (``paper_2607_06202_amd``) never does, and the two
share no code: the oracle is plain single-threaded C (``epl_oracle.c``) behind ctypes, over
numpy arrays.

Each function follows the definition cited in ``epl_oracle.c``; every one is pinned by the
non-GPU tests (brute force, closed forms, invariants, library routines).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "epl_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-fvisibility=hidden"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no GPU code involved)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        P = ctypes.c_void_p
        I, L = ctypes.c_int, ctypes.c_int64
        sig = {
            "eplref_layout": (I, [I, I, I, I] + [P] * 12),
            "eplref_dispatch_bf16": (None, [L, I, I, P, P, P]),
            "eplref_dispatch_fp8": (None, [L, I, I, P, P, P, P]),
            "eplref_quantize_row_e4m3": (None, [I, P, P, P]),
            "eplref_combine": (None, [L, I, I, P, P, P, P, L, P]),
            "eplref_combine_mapped": (None, [I, I, P, P, P, P, P, L, P]),
            "eplref_locate_rows": (None, [I, P, L, P, P, P]),
            "eplref_transposed_order": (None, [I, I, P]),
            "eplref_hop_schedule": (None, [I, I, I, I, P, P, P, P, P, P]),
            "eplref_f32_to_bf16_array": (None, [P, P, L]),
            "eplref_f32_to_e4m3_array": (None, [P, P, L]),
            "eplref_f32_to_bf16": (ctypes.c_uint16, [ctypes.c_float]),
            "eplref_f32_to_e4m3": (ctypes.c_uint8, [ctypes.c_float]),
            "eplref_bf16_to_f32": (ctypes.c_float, [ctypes.c_uint16]),
            "eplref_e4m3_to_f32": (ctypes.c_float, [ctypes.c_uint8]),
        }
        for name, (res, args) in sig.items():
            f = getattr(_lib, name)
            f.restype = res
            f.argtypes = args
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(ctypes.c_void_p)


@dataclass
class RefLayout:
    send_cnt: np.ndarray    # [R, E]
    rank_cnt: np.ndarray    # [R, R]
    expert_off: np.ndarray  # [E+1]
    rank_off: np.ndarray    # [R+1]
    seg_off: np.ndarray     # [E, R]
    tok_nranks: np.ndarray  # [T]
    pair_row: np.ndarray    # [T, k]
    pair_rslot: np.ndarray  # [T, k]
    recv_src: np.ndarray    # [P]
    recv_j: np.ndarray      # [P]
    num_invalid: int

    @property
    def P(self) -> int:
        return int(self.expert_off[-1])


def layout(R: int, E: int, k: int, Tr: int, idx: np.ndarray) -> RefLayout:
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(R * Tr, k)
    T = R * Tr
    send_cnt = np.zeros((R, E), np.int32)
    rank_cnt = np.zeros((R, R), np.int32)
    expert_off = np.zeros(E + 1, np.int32)
    rank_off = np.zeros(R + 1, np.int32)
    seg_off = np.zeros((E, R), np.int32)
    tok_nranks = np.zeros(T, np.int32)
    pair_row = np.zeros((T, k), np.int32)
    pair_rslot = np.zeros((T, k), np.int32)
    recv_src = np.full(max(T * k, 1), -7, np.int32)
    recv_j = np.full(max(T * k, 1), -7, np.int32)
    ninv = np.zeros(1, np.int32)
    rc = lib().eplref_layout(R, E, k, Tr, _p(idx), _p(send_cnt), _p(rank_cnt), _p(expert_off), _p(rank_off),
                             _p(seg_off), _p(tok_nranks), _p(pair_row), _p(pair_rslot), _p(recv_src), _p(recv_j),
                             _p(ninv))
    if rc != 0:
        raise ValueError("oracle layout rejected shape R=%d E=%d k=%d Tr=%d" % (R, E, k, Tr))
    P = int(expert_off[-1])
    return RefLayout(send_cnt, rank_cnt, expert_off, rank_off, seg_off, tok_nranks, pair_row, pair_rslot,
                     recv_src[:P].copy(), recv_j[:P].copy(), int(ninv[0]))


def dispatch_bf16(x: np.ndarray, pair_row: np.ndarray, rows: int, fill: int = 0) -> np.ndarray:
    """x: [T, H] uint16 (bf16 bits). Returns recv [rows, H] uint16 (rows not written keep ``fill``)."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    T, H = x.shape
    k = pair_row.shape[1]
    recv = np.full((rows, H), fill, np.uint16)
    lib().eplref_dispatch_bf16(T, k, H, _p(x), _p(np.ascontiguousarray(pair_row, dtype=np.int32)), _p(recv))
    return recv


def dispatch_fp8(x: np.ndarray, pair_row: np.ndarray, rows: int, fill: int = 0):
    """Returns (recv [rows, H] uint8, recv_scale [rows, H/128] float32)."""
    x = np.ascontiguousarray(x, dtype=np.uint16)
    T, H = x.shape
    k = pair_row.shape[1]
    recv = np.full((rows, H), fill, np.uint8)
    scale = np.full((rows, H // 128), np.nan, np.float32)
    lib().eplref_dispatch_fp8(T, k, H, _p(x), _p(np.ascontiguousarray(pair_row, dtype=np.int32)), _p(recv),
                              _p(scale))
    return recv, scale


def quantize_row_e4m3(xrow: np.ndarray):
    xrow = np.ascontiguousarray(xrow, dtype=np.uint16)
    H = xrow.shape[0]
    q = np.zeros(H, np.uint8)
    s = np.zeros(H // 128, np.float32)
    lib().eplref_quantize_row_e4m3(H, _p(xrow), _p(q), _p(s))
    return q, s


def combine(y: np.ndarray, w: np.ndarray, pair_row: np.ndarray, tokens=None) -> np.ndarray:
    """y: [rows, H] uint16; w, pair_row: [T, k]. Returns out [T or len(tokens), H] uint16."""
    y = np.ascontiguousarray(y, dtype=np.uint16)
    H = y.shape[1]
    T, k = pair_row.shape
    w = np.ascontiguousarray(w, dtype=np.float32)
    pr = np.ascontiguousarray(pair_row, dtype=np.int32)
    if tokens is None:
        out = np.zeros((T, H), np.uint16)
        lib().eplref_combine(T, k, H, _p(y), _p(w), _p(pr), None, 0, _p(out))
    else:
        tok = np.ascontiguousarray(tokens, dtype=np.int64)
        out = np.zeros((tok.shape[0], H), np.uint16)
        lib().eplref_combine(T, k, H, _p(y), _p(w), _p(pr), _p(tok), tok.shape[0], _p(out))
    return out


def combine_mapped(ys: np.ndarray, row_map: np.ndarray, w: np.ndarray, pair_row: np.ndarray,
                   tokens: np.ndarray) -> np.ndarray:
    """Combine for listed tokens when only some expert rows are on the host: row r of the full
    y is ys[row_map[r]]."""
    ys = np.ascontiguousarray(ys, dtype=np.uint16)
    H = ys.shape[1]
    T, k = pair_row.shape
    tok = np.ascontiguousarray(tokens, dtype=np.int64)
    out = np.zeros((tok.shape[0], H), np.uint16)
    lib().eplref_combine_mapped(k, H, _p(ys), _p(np.ascontiguousarray(row_map, dtype=np.int32)),
                                _p(np.ascontiguousarray(w, dtype=np.float32)),
                                _p(np.ascontiguousarray(pair_row, dtype=np.int32)), _p(tok), tok.shape[0],
                                _p(out))
    return out


def _at(a: np.ndarray, elem_offset: int):
    """Pointer to element elem_offset of a C-contiguous array (for calls on token sub-ranges)."""
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data + int(elem_offset) * a.itemsize)


def dispatch_range_into(x: np.ndarray, pair_row: np.ndarray, recv: np.ndarray, g0: int, g1: int,
                        recv_scale: np.ndarray | None = None) -> None:
    """eplref_dispatch_bf16 (or _fp8 when recv_scale is given) on tokens [g0, g1) only, writing
    into the caller's recv (and recv_scale). The C function is called unchanged on the token
    range's rows of x and pair_row; the rows it writes are the range's own, so calls on disjoint
    ranges may run at the same time (ctypes releases the GIL)."""
    T, H = x.shape
    k = pair_row.shape[1]
    if recv_scale is None:
        lib().eplref_dispatch_bf16(g1 - g0, k, H, _at(x, g0 * H), _at(pair_row, g0 * k), _p(recv))
    else:
        lib().eplref_dispatch_fp8(g1 - g0, k, H, _at(x, g0 * H), _at(pair_row, g0 * k), _p(recv),
                                  _p(recv_scale))


def combine_range_into(y: np.ndarray, w: np.ndarray, pair_row: np.ndarray, out: np.ndarray, g0: int,
                       g1: int) -> None:
    """eplref_combine on tokens [g0, g1) only, writing out[g0:g1] of the caller's out."""
    H = y.shape[1]
    k = pair_row.shape[1]
    lib().eplref_combine(g1 - g0, k, H, _p(y), _at(w, g0 * k), _at(pair_row, g0 * k), None, 0,
                         _at(out, g0 * H))


def locate_rows(expert_off: np.ndarray, rows=None, n: int | None = None):
    """Expert and in-expert offset of packed rows (Token-level Load Partition; Algorithm 1's
    result): rows, or 0..n-1 when rows is None. Positions outside [0, P) give (-1, -1)."""
    off = np.ascontiguousarray(expert_off, np.int32)
    E = off.size - 1
    if rows is not None:
        rows = np.ascontiguousarray(rows, np.int32)
        n = rows.size
    expert = np.empty(n, np.int32)
    offset = np.empty(n, np.int32)
    lib().eplref_locate_rows(E, _p(off), n, None if rows is None else _p(rows), _p(expert), _p(offset))
    return expert, offset


def transposed_order(E: int, rows: int) -> np.ndarray:
    """The remapped expert sequence of the logical matrix transposition: E experts laid row by row
    in a matrix of ``rows`` rows (the paper: one per worker), read column by column (Hierarchical
    Token-level Scheduling, Expert Remapping via Logical Matrix Transposition)."""
    order = np.zeros(E, np.int32)
    lib().eplref_transposed_order(E, rows, _p(order))
    return order


def hop_schedule(send_cnt: np.ndarray, order: np.ndarray, hop: np.ndarray, n: int, NH: int):
    """Equal slices of each source rank's pairs, taken in the expert sequence ``order``, for n workers
    -> (start_expert [R, n], start_offset [R, n], counts [R, n, NH]): each slice's first expert and
    offset, and its pairs per hop class hop[s, d] of their destination rank d (Token-level Load
    Partition; the per-hop counts v_{j,h} of Latency Homogenization)."""
    send_cnt = np.ascontiguousarray(send_cnt, np.int32)
    R, E = send_cnt.shape
    order = np.ascontiguousarray(order, np.int32)
    hop = np.ascontiguousarray(hop, np.int32).reshape(R, R)
    se = np.zeros((R, n), np.int32)
    so = np.zeros((R, n), np.int32)
    cnt = np.zeros((R, n, NH), np.int32)
    lib().eplref_hop_schedule(R, E, n, NH, _p(send_cnt), _p(order), _p(hop), _p(se), _p(so), _p(cnt))
    return se, so, cnt


def f32_to_bf16(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.zeros(v.shape, np.uint16)
    lib().eplref_f32_to_bf16_array(_p(v), _p(out), v.size)
    return out


def f32_to_e4m3(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.float32)
    out = np.zeros(v.shape, np.uint8)
    lib().eplref_f32_to_e4m3_array(_p(v), _p(out), v.size)
    return out


def e4m3_to_f32(c: np.ndarray) -> np.ndarray:
    f = lib().eplref_e4m3_to_f32
    return np.array([f(int(v)) for v in np.asarray(c).ravel()], dtype=np.float32).reshape(np.shape(c))


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    """Exact widening (bf16 is the upper half of binary32)."""
    return (np.asarray(h, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
