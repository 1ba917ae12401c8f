"""Python binding of libepl (MoE dispatch / combine on one MI355X): argument marshalling only.

Every step runs in the HIP kernels behind the C ABI declared in ``include/epl.h``. This module
allocates output tensors with torch on the tensors' device (the receive buffer, on request, as one
contiguous block from the HIP runtime), passes raw device pointers and the current HIP stream, and
turns status codes into exceptions. There is no fallback: if
``libepl.so`` is missing, or a tensor is not on the GPU, the call raises.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libepl.so")

PAYLOAD_BF16 = 0
PAYLOAD_FP8_E4M3 = 1
MAX_EXPERTS = 1024
MAX_TOPK = 32
MAX_HOP_CLASSES = 8  # EPL_MAX_HOP_CLASSES
STATIC_SCRATCH_BYTES = 8 << 20  # EPL_STATIC_SCRATCH_BYTES: the library's own workspace per GPU

STATUS = {0: "EPL_OK", 1: "EPL_ERR_INVALID_ARG", 2: "EPL_ERR_ALIGN", 3: "EPL_ERR_CAPACITY",
          4: "EPL_ERR_WORKSPACE", 5: "EPL_ERR_UNSUPPORTED", 6: "EPL_ERR_DEVICE"}


class EplError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s" % (what, STATUS.get(status, status)))


class Config(ctypes.Structure):
    _fields_ = [("num_ranks", ctypes.c_int32), ("num_experts", ctypes.c_int32), ("topk", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("tokens_per_rank", ctypes.c_int32), ("payload", ctypes.c_int32),
                ("row_pitch", ctypes.c_int32)]

    @property
    def T(self) -> int:
        return self.num_ranks * self.tokens_per_rank

    @property
    def pitch(self) -> int:
        """Elements from one recv (and y) row to the next."""
        return self.row_pitch or self.hidden

    def __repr__(self) -> str:
        return "Config(R=%d, E=%d, k=%d, H=%d, Tr=%d, payload=%d, row_pitch=%d)" % (
            self.num_ranks, self.num_experts, self.topk, self.hidden, self.tokens_per_rank, self.payload,
            self.row_pitch)


def config(R: int, E: int, k: int, H: int, Tr: int, payload: str | int = "bf16", row_pitch: int = 0) -> Config:
    """row_pitch: elements from one receive row to the next (0: H, rows packed without gaps)."""
    if isinstance(payload, str):
        payload = {"bf16": PAYLOAD_BF16, "fp8": PAYLOAD_FP8_E4M3}[payload]
    return Config(R, E, k, H, Tr, payload, row_pitch)


# Row pitches measured faster than packed rows on MI355X, by (H, payload); other shapes keep packed
# rows. Whole layer, one box, 200 steps per pitch (us per layer):
# * H = 7168 bf16, EP=64 decode: 7168 376.7-377.3, 7424 377.1, 7680 375.1, 7936 373.8, 8192 392.0,
#   8448 374.5, 9216 381.4 (on other boxes 7936 gained 0.6-3.6%); prefill and the DeepSeek shape
#   within 0.3% of packed rows; EP=256 0.2% faster at 7936 and 1.1% faster at 7680, which costs prefill
#   0.3% (one pitch per row size is kept);
# * H = 5120 bf16 (GLM-4.7 shape): 5120 131.8-132.2, 5248 131.6, 5632 134.5, 5888 144.5, 8192 141.9;
# * H = 2048 bf16 (Qwen3-30B shape): 39.5-40.1 at every pitch (bound by launches);
# * H = 7168 fp8: packed 556.0-556.3, every pitch from 7232 to 9216 bytes 556.5-563.2.
TUNED_PITCH = {(7168, PAYLOAD_BF16): 7936}


def tuned_pitch(H: int, payload: str | int = "bf16") -> int:
    """The row pitch the benchmark uses: a measured entry of TUNED_PITCH, else 0 (packed rows)."""
    if isinstance(payload, str):
        payload = {"bf16": PAYLOAD_BF16, "fp8": PAYLOAD_FP8_E4M3}[payload]
    return TUNED_PITCH.get((H, payload), 0)


class DecomposedOpts(ctypes.Structure):
    _fields_ = [("count_groups", ctypes.c_int32), ("spin_limit_us", ctypes.c_int32),
                ("test_ready_target", ctypes.c_int32)]


WAIT_GAVE_UP_COUNT = 1    # EPL_WAIT_GAVE_UP_COUNT
WAIT_GAVE_UP_SEND = 2     # EPL_WAIT_GAVE_UP_SEND
WAIT_GAVE_UP_COMBINE = 4  # EPL_WAIT_GAVE_UP_COMBINE
WAIT_SENTINEL_IN_X = 8    # EPL_WAIT_SENTINEL_IN_X
SENTINEL_BF16 = 0xFFFF    # EPL_SENTINEL_BF16
DAF_TOKEN_FLAG_FUSION = 1  # EPL_DAF_TOKEN_FLAG_FUSION
DAF_DATA_CHECKSUM = 2      # EPL_DAF_DATA_CHECKSUM


class LayoutBuffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("send_cnt", "rank_cnt", "expert_off", "rank_off", "seg_off",
                                               "tok_nranks", "pair_row", "pair_rslot", "recv_src", "recv_j",
                                               "num_invalid")]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libepl.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libepl.so is not built (run __graft_entry__.build()): %s" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, I64, S = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
        CP, LP = ctypes.POINTER(Config), ctypes.POINTER(LayoutBuffers)
        L.epl_workspace_bytes.restype = S
        L.epl_workspace_bytes.argtypes = [CP]
        L.epl_layout.restype = ctypes.c_int
        L.epl_layout.argtypes = [CP, P, LP, P, S, P]
        L.epl_dispatch.restype = ctypes.c_int
        L.epl_dispatch.argtypes = [CP, P, LP, P, P, I64, P]
        L.epl_combine.restype = ctypes.c_int
        L.epl_combine.argtypes = [CP, P, P, LP, P, P]
        L.epl_debug_f32_to_e4m3.restype = ctypes.c_int
        L.epl_debug_f32_to_e4m3.argtypes = [P, P, I64, P]
        L.epl_debug_f32_to_bf16.restype = ctypes.c_int
        L.epl_debug_f32_to_bf16.argtypes = [P, P, I64, P]
        L.epl_status_str.restype = ctypes.c_char_p
        L.epl_status_str.argtypes = [ctypes.c_int]
        L.epl_version.restype = ctypes.c_char_p
        L.epl_version.argtypes = []
        L.epl_layout_dispatch.restype = ctypes.c_int
        L.epl_layout_dispatch.argtypes = [CP, P, LP, P, S, P, P, P, I64, P]
        L.epl_layout_counts.restype = ctypes.c_int
        L.epl_layout_counts.argtypes = [CP, P, LP, P, S, P]
        L.epl_dispatch_rows.restype = ctypes.c_int
        L.epl_dispatch_rows.argtypes = [CP, P, LP, P, S, P, P, P, I64, P]
        L.epl_locate_rows.restype = ctypes.c_int
        L.epl_locate_rows.argtypes = [CP, P, P, I64, P, P, P]
        L.epl_layout_dispatch_launches.restype = ctypes.c_int
        L.epl_layout_dispatch_launches.argtypes = [CP]
        L.epl_layout_launches.restype = ctypes.c_int
        L.epl_layout_launches.argtypes = [CP]
        L.epl_layout_dispatch_decomposed.restype = ctypes.c_int
        L.epl_layout_dispatch_decomposed.argtypes = [CP, P, LP, P, S, P, P, P, I64, ctypes.POINTER(DecomposedOpts), P, P]
        L.epl_decomposed_plan.restype = ctypes.c_int
        L.epl_decomposed_plan.argtypes = [CP, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                          ctypes.POINTER(ctypes.c_int32)]
        L.epl_layer_sentinel.restype = ctypes.c_int
        L.epl_layer_sentinel.argtypes = [CP, P, LP, P, S, P, P, I64, P, P, ctypes.POINTER(DecomposedOpts), P, P]
        L.epl_layer_data_as_flag.restype = ctypes.c_int
        L.epl_layer_data_as_flag.argtypes = [CP, P, LP, P, S, P, P, I64, P, P, P, ctypes.c_int32, ctypes.c_uint64,
                                             ctypes.POINTER(DecomposedOpts), P, P]
        L.epl_layer_marks_bytes.restype = I64
        L.epl_layer_marks_bytes.argtypes = [CP, I64]
        L.epl_sentinel_fill.restype = ctypes.c_int
        L.epl_sentinel_fill.argtypes = [P, I64, P]
        L.epl_sentinel_find.restype = I64
        L.epl_sentinel_find.argtypes = [P, I64]
        L.epl_layout_dispatch_noalloc.restype = ctypes.c_int
        L.epl_layout_dispatch_noalloc.argtypes = [CP, P, LP, P, P, P, I64, P]
        I32 = ctypes.c_int32
        L.epl_hop_schedule.restype = ctypes.c_int
        L.epl_hop_schedule.argtypes = [CP, P, P, I32, P, I32, I32, P, P, P, P]
        L.epl_dispatch_scheduled.restype = ctypes.c_int
        L.epl_dispatch_scheduled.argtypes = [CP, P, LP, P, P, I64, I32, I32, P]
        _lib = L
    return _lib


def _check(status: int, what: str) -> None:
    if status != 0:
        raise EplError(status, what)


def _dev(t: torch.Tensor, name: str, dtype=None) -> int:
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return t.data_ptr()


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def workspace_bytes(cfg: Config) -> int:
    return int(lib().epl_workspace_bytes(ctypes.byref(cfg)))


@dataclass
class Layout:
    """Device outputs of epl_layout (int32 tensors)."""
    cfg: Config
    send_cnt: torch.Tensor    # [R, E]
    rank_cnt: torch.Tensor    # [R, R]
    expert_off: torch.Tensor  # [E+1]
    rank_off: torch.Tensor    # [R+1]
    seg_off: torch.Tensor     # [E, R]
    tok_nranks: torch.Tensor  # [T]
    pair_row: torch.Tensor    # [T, k]
    pair_rslot: torch.Tensor  # [T, k]
    recv_src: torch.Tensor    # [T*k] (first P valid)
    recv_j: torch.Tensor      # [T*k] (first P valid)
    num_invalid: torch.Tensor  # [1]
    workspace: torch.Tensor   # uint8 scratch

    def buffers(self) -> LayoutBuffers:
        """The C struct of device pointers, built once and rebuilt only after a field is replaced."""
        cached = self.__dict__.get("_buffers")
        if cached is None:
            cached = LayoutBuffers(*[getattr(self, n).data_ptr() for n, _ in LayoutBuffers._fields_])
            object.__setattr__(self, "_buffers", cached)
        return cached

    def workspace_needed(self) -> int:
        """epl_workspace_bytes of the layout's own config, computed once."""
        need = self.__dict__.get("_ws_need")
        if need is None:
            need = workspace_bytes(self.cfg)
            object.__setattr__(self, "_ws_need", need)
        return need

    def __setattr__(self, name, value):
        super().__setattr__(name, value)
        self.__dict__.pop("_buffers", None)
        if name == "cfg":
            self.__dict__.pop("_ws_need", None)


def alloc_layout(cfg: Config, device) -> Layout:
    R, E, k, T = cfg.num_ranks, cfg.num_experts, cfg.topk, cfg.T
    i32 = dict(dtype=torch.int32, device=device)
    ws = workspace_bytes(cfg)
    if ws == 0:
        raise EplError(1, "epl_workspace_bytes(%r)" % (cfg,))
    return Layout(cfg, torch.empty(R, E, **i32), torch.empty(R, R, **i32), torch.empty(E + 1, **i32),
                  torch.empty(R + 1, **i32), torch.empty(E, R, **i32), torch.empty(max(T, 1), **i32),
                  torch.empty(max(T, 1), k, **i32), torch.empty(max(T, 1), k, **i32), torch.empty(max(T * k, 1), **i32),
                  torch.empty(max(T * k, 1), **i32), torch.empty(1, **i32),
                  torch.zeros(ws, dtype=torch.uint8, device=device))  # zero: the decomposed call's sync words


def _on(dev):
    """Make dev the current device for a launch, switching only when it is not already."""
    return contextlib.nullcontext() if torch.cuda.current_device() == dev.index else torch.cuda.device(dev)


def _same_device(dev, **tensors) -> None:
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise ValueError("%s is on %s, expected %s" % (name, t.device, dev))


def _check_layout(cfg: Config, L: Layout, dev) -> None:
    """The layout buffers were sized for cfg (the kernels index them by cfg's shape)."""
    c = L.cfg
    if (c.num_ranks, c.num_experts, c.topk, c.tokens_per_rank) != (cfg.num_ranks, cfg.num_experts, cfg.topk,
                                                                    cfg.tokens_per_rank):
        raise ValueError("layout was allocated for %r, not %r" % (c, cfg))
    _same_device(dev, pair_row=L.pair_row, workspace=L.workspace)


def _rows_of(t: torch.Tensor, name: str, width: int) -> int:
    if t.dim() != 2 or t.shape[1] != width:
        raise ValueError("%s must be 2-D with %d columns, got shape %s" % (name, width, tuple(t.shape)))
    return t.shape[0]


def _pitched_rows(t, name: str, dtype, cfg: Config) -> int:
    """A receive-layout tensor (recv, or y for combine): 2-D [rows, H] on the GPU whose rows are
    cfg.pitch elements apart (a view of a [rows, pitch] buffer, or contiguous when the pitch is H).
    Returns its row count."""
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError("%s must be a GPU tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    rows = _rows_of(t, name, cfg.hidden)
    if (cfg.hidden > 1 and t.stride(1) != 1) or (rows > 1 and t.stride(0) != cfg.pitch):
        raise ValueError("%s rows must be %d elements apart and dense, got strides %s" % (name, cfg.pitch, t.stride()))
    return rows


def _layout_args(cfg: Config, topk_idx: torch.Tensor, out: Layout | None) -> Layout:
    """Checks shared by the calls that run the layout; returns the Layout to fill."""
    _dev(topk_idx, "topk_idx", torch.int32)
    if topk_idx.numel() != cfg.T * cfg.topk:
        raise ValueError("topk_idx has %d elements, expected T*k = %d" % (topk_idx.numel(), cfg.T * cfg.topk))
    L = out if out is not None else alloc_layout(cfg, topk_idx.device)
    _check_layout(cfg, L, topk_idx.device)
    if L.workspace.numel() < L.workspace_needed():  # cfg has the layout's shape (checked above)
        raise ValueError("layout workspace has %d bytes, needs %d" % (L.workspace.numel(), L.workspace_needed()))
    return L


def layout(cfg: Config, topk_idx: torch.Tensor, out: Layout | None = None) -> Layout:
    """epl_layout: topk_idx [T, k] int32 on the GPU -> Layout."""
    dev = topk_idx.device
    L = _layout_args(cfg, topk_idx, out)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layout(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs), L.workspace.data_ptr(),
                                L.workspace.numel(), _stream(dev)), "epl_layout")
    return L


def layout_counts(cfg: Config, topk_idx: torch.Tensor, out: Layout | None = None) -> Layout:
    """epl_layout_counts: first phase of layout_dispatch (the layout kernels the row kernel does
    not take over) -> Layout, complete only after dispatch_rows."""
    dev = topk_idx.device
    L = _layout_args(cfg, topk_idx, out)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layout_counts(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                       L.workspace.data_ptr(), L.workspace.numel(), _stream(dev)),
               "epl_layout_counts")
    return L


def recv_rows_cap(cfg: Config) -> int:
    return cfg.T * cfg.topk


_HIP_DEVICE_MALLOC_CONTIGUOUS = 0x4  # hipDeviceMallocContiguous
_hip = None


def _hip_runtime_path() -> str:
    """The HIP runtime this process already has mapped (torch's and libepl's), else its soname."""
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                path = line.split()[-1] if line.strip() else ""
                if os.path.basename(path).startswith("libamdhip64.so"):
                    return path
    except OSError:
        pass
    return "libamdhip64.so.7"


def _hip_runtime() -> ctypes.CDLL:
    """The HIP runtime that torch and libepl already share: the mapped file itself when it is found
    in the process's memory map (so no second copy is loaded), else by soname."""
    global _hip
    if _hip is None:
        lib()  # libepl links the runtime, so it is mapped from here on
        h = ctypes.CDLL(_hip_runtime_path())
        h.hipExtMallocWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t, ctypes.c_uint]
        h.hipExtMallocWithFlags.restype = ctypes.c_int
        h.hipFree.argtypes = [ctypes.c_void_p]
        h.hipFree.restype = ctypes.c_int
        _hip = h
    return _hip


class _ContiguousBlock:
    """One physically contiguous device allocation (hipExtMallocWithFlags with
    hipDeviceMallocContiguous), handed to torch through __cuda_array_interface__. torch holds a
    reference to the block for as long as a tensor uses its memory; hipFree runs after the last
    one is gone."""

    def __init__(self, nbytes: int, device: torch.device):
        self.ptr = ctypes.c_void_p()
        self.device = torch.device(device)
        with torch.cuda.device(self.device):
            rc = _hip_runtime().hipExtMallocWithFlags(ctypes.byref(self.ptr), nbytes, _HIP_DEVICE_MALLOC_CONTIGUOUS)
        if rc != 0 or not self.ptr.value:
            self.ptr = ctypes.c_void_p()
            raise MemoryError("no physically contiguous block of %d bytes on %s (hip status %d)" %
                              (nbytes, self.device, rc))
        self.nbytes = nbytes

    def tensor(self, shape, dtype: torch.dtype) -> torch.Tensor:
        """A tensor over the start of the block; its extent must fit in the block (the kernels
        write wherever a tensor says its rows are)."""
        n = dtype.itemsize
        for d in shape:
            n *= int(d)
        if n > self.nbytes:
            raise ValueError("a %s tensor of shape %s needs %d bytes; the block has %d" %
                             (dtype, tuple(shape), n, self.nbytes))
        typestr = {torch.bfloat16: "<i2", torch.uint8: "|u1"}[dtype]
        self.__cuda_array_interface__ = {"shape": tuple(shape), "typestr": typestr, "strides": None,
                                         "data": (self.ptr.value, False), "version": 2}
        t = torch.as_tensor(self, device=self.device)
        return t.view(dtype) if t.dtype != dtype else t

    def __del__(self):
        if self.ptr.value:
            try:
                with torch.cuda.device(self.device):
                    _hip_runtime().hipFree(self.ptr)  # synchronises with work still using the block
            except Exception:  # interpreter shutdown: the runtime may already be gone
                pass


def alloc_recv(cfg: Config, device, rows: int | None = None, contiguous: bool = False):
    """Receive buffer for dispatch: (recv [rows, H] bf16 | uint8, recv_scale [rows, H/128] fp32 |
    None), rows = T*k by default. recv is a view of a [rows, cfg.pitch] buffer, so its rows are
    cfg.pitch elements apart as the kernels expect (the whole buffer for packed rows). With contiguous=True the payload rows are one physically
    contiguous block from the HIP runtime instead of torch's allocator (MemoryError if the driver
    has no such block free). The rows are written in a scatter and gathered at random, and where
    they sit in HBM moves both kernels' times: on MI355X, decode-sized layers measured 377.0 us per
    layer (median of six allocations) on contiguous blocks against 379.9 us on torch's."""
    rows = max(recv_rows_cap(cfg) if rows is None else rows, 1)
    fp8 = cfg.payload == PAYLOAD_FP8_E4M3
    dtype = torch.uint8 if fp8 else torch.bfloat16
    P = cfg.pitch
    if contiguous:
        recv = _ContiguousBlock(rows * P * dtype.itemsize, device).tensor((rows, P), dtype)
    else:
        recv = torch.empty(rows, P, dtype=dtype, device=device)
    recv = recv[:, :cfg.hidden]  # rows P elements apart (the whole buffer when P == H)
    scale = torch.empty(rows, cfg.hidden // 128, dtype=torch.float32, device=device) if fp8 else None
    return recv, scale


def dispatch(cfg: Config, x: torch.Tensor, L: Layout, recv: torch.Tensor | None = None,
             recv_scale: torch.Tensor | None = None):
    """epl_dispatch: x [T, H] bf16 -> (recv [cap, H] bf16 | uint8, recv_scale [cap, H/128] fp32 | None)."""
    dev = x.device
    _dev(x, "x", torch.bfloat16)
    if _rows_of(x, "x", cfg.hidden) < cfg.T:
        raise ValueError("x has %d rows, needs T = %d" % (x.shape[0], cfg.T))
    _check_layout(cfg, L, dev)
    if recv is None:
        recv, recv_scale = alloc_recv(cfg, dev)
    fp8 = cfg.payload == PAYLOAD_FP8_E4M3
    rows = _pitched_rows(recv, "recv", torch.uint8 if fp8 else torch.bfloat16, cfg)
    sp = None
    if fp8:
        sp = _dev(recv_scale, "recv_scale", torch.float32)
        if _rows_of(recv_scale, "recv_scale", cfg.hidden // 128) < rows:
            raise ValueError("recv_scale has fewer rows than recv")
    _same_device(dev, recv=recv, recv_scale=recv_scale if fp8 else None)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_dispatch(ctypes.byref(cfg), x.data_ptr(), ctypes.byref(bufs), recv.data_ptr(), sp,
                                  rows if recv.numel() else 0, _stream(dev)), "epl_dispatch")
    return recv, recv_scale


def _recv_args(cfg: Config, x: torch.Tensor, recv, recv_scale, dev):
    """Checks of x, recv and recv_scale shared by the dispatching calls -> (recv, recv_scale,
    scale pointer or None, recv rows)."""
    _dev(x, "x", torch.bfloat16)
    if _rows_of(x, "x", cfg.hidden) < cfg.T:
        raise ValueError("x has %d rows, needs T = %d" % (x.shape[0], cfg.T))
    if recv is None:
        recv, recv_scale = alloc_recv(cfg, dev)
    fp8 = cfg.payload == PAYLOAD_FP8_E4M3
    rows = _pitched_rows(recv, "recv", torch.uint8 if fp8 else torch.bfloat16, cfg)
    sp = None
    if fp8:
        sp = _dev(recv_scale, "recv_scale", torch.float32)
        if _rows_of(recv_scale, "recv_scale", cfg.hidden // 128) < rows:
            raise ValueError("recv_scale has fewer rows than recv")
    _same_device(dev, x=x, recv=recv, recv_scale=recv_scale if fp8 else None)
    return recv, recv_scale, sp, rows if recv.numel() else 0


def layout_dispatch(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, out: Layout | None = None,
                    recv: torch.Tensor | None = None, recv_scale: torch.Tensor | None = None):
    """epl_layout_dispatch: layout and dispatch in one call -> (Layout, recv, recv_scale | None)."""
    dev = topk_idx.device
    L = _layout_args(cfg, topk_idx, out)
    recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layout_dispatch(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                         L.workspace.data_ptr(), L.workspace.numel(), x.data_ptr(), recv.data_ptr(),
                                         sp, rows, _stream(dev)), "epl_layout_dispatch")
    return L, recv, recv_scale


def layout_dispatch_noalloc(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, out: Layout,
                            recv: torch.Tensor, recv_scale: torch.Tensor | None = None):
    """epl_layout_dispatch_noalloc: layout and dispatch with the library's static per-GPU scratch
    as the workspace. Every output buffer comes from the caller (out, recv, recv_scale), so nothing
    is allocated here either; out.workspace is not used. -> (out, recv, recv_scale | None)."""
    dev = topk_idx.device
    _dev(topk_idx, "topk_idx", torch.int32)
    if topk_idx.numel() != cfg.T * cfg.topk:
        raise ValueError("topk_idx has %d elements, expected T*k = %d" % (topk_idx.numel(), cfg.T * cfg.topk))
    _check_layout(cfg, out, dev)
    recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
    bufs = out.buffers()
    with _on(dev):
        _check(lib().epl_layout_dispatch_noalloc(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                                 x.data_ptr(), recv.data_ptr(), sp, rows, _stream(dev)),
               "epl_layout_dispatch_noalloc")
    return out, recv, recv_scale


def layout_dispatch_decomposed(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, out: Layout | None = None,
                               recv: torch.Tensor | None = None, recv_scale: torch.Tensor | None = None,
                               count_groups: int = 0, spin_limit_us: int = 0, test_ready_target: int = 0,
                               status: torch.Tensor | None = None):
    """epl_layout_dispatch_decomposed: layout and dispatch in one launch of count and send
    workgroups -> (Layout, recv, recv_scale | None, status [1] int32: 0, or EPL_WAIT_* bits, once
    the stream reaches the end of the launch). The layout's workspace must have been allocated
    zero-filled (alloc_layout does)."""
    dev = topk_idx.device
    L = _layout_args(cfg, topk_idx, out)
    recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device=dev)
    _dev(status, "status", torch.int32)
    _same_device(dev, status=status)
    opts = DecomposedOpts(count_groups, spin_limit_us, test_ready_target)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layout_dispatch_decomposed(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                                    L.workspace.data_ptr(), L.workspace.numel(), x.data_ptr(),
                                                    recv.data_ptr(), sp, rows, ctypes.byref(opts), status.data_ptr(),
                                                    _stream(dev)), "epl_layout_dispatch_decomposed")
    return L, recv, recv_scale, status


def layer_sentinel(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, topk_w: torch.Tensor, recv: torch.Tensor,
                   out: torch.Tensor | None = None, layout_out: Layout | None = None, count_groups: int = 0,
                   spin_limit_us: int = 0, test_ready_target: int = 0, status: torch.Tensor | None = None):
    """epl_layer_sentinel: layout, dispatch and the combine of the dispatched rows in one launch,
    synchronised per row by Sentinel Polling. recv must hold the sentinel everywhere (sentinel_fill)
    and is left so. -> (Layout, out [T, H] bf16, status [1] int32)."""
    dev = topk_idx.device
    if cfg.payload != PAYLOAD_BF16:
        raise EplError(5, "epl_layer_sentinel (bf16 only)")
    L = _layout_args(cfg, topk_idx, layout_out)
    recv, _, _, rows = _recv_args(cfg, x, recv, None, dev)
    _dev(topk_w, "topk_w", torch.float32)
    if _rows_of(topk_w, "topk_w", cfg.topk) < cfg.T:
        raise ValueError("topk_w has %d rows, needs T = %d" % (topk_w.shape[0], cfg.T))
    if out is None:
        out = torch.empty(max(cfg.T, 1), cfg.hidden, dtype=torch.bfloat16, device=dev)
    _dev(out, "out", torch.bfloat16)
    if _rows_of(out, "out", cfg.hidden) < cfg.T:
        raise ValueError("out has %d rows, needs T = %d" % (out.shape[0], cfg.T))
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device=dev)
    _dev(status, "status", torch.int32)
    _same_device(dev, topk_w=topk_w, out=out, status=status)
    opts = DecomposedOpts(count_groups, spin_limit_us, test_ready_target)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layer_sentinel(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                        L.workspace.data_ptr(), L.workspace.numel(), x.data_ptr(), recv.data_ptr(),
                                        rows, topk_w.data_ptr(), out.data_ptr(), ctypes.byref(opts), status.data_ptr(),
                                        _stream(dev)), "epl_layer_sentinel")
    return L, out, status


def layer_marks_bytes(cfg: Config, rows: int | None = None) -> int:
    """epl_layer_marks_bytes: bytes of the marks buffer of layer_data_as_flag for `rows` receive
    rows (T*k by default)."""
    n = int(lib().epl_layer_marks_bytes(ctypes.byref(cfg), recv_rows_cap(cfg) if rows is None else rows))
    if n < 0:
        raise EplError(1, "epl_layer_marks_bytes(%r)" % (cfg,))
    return n


def alloc_marks(cfg: Config, device, rows: int | None = None) -> torch.Tensor:
    """A zero-filled marks buffer for layer_data_as_flag: one int64 word per (receive row, 1 KiB
    column chunk)."""
    n = layer_marks_bytes(cfg, rows) // 8
    return torch.zeros(max(n, 1), dtype=torch.int64, device=device)


def layer_data_as_flag(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, topk_w: torch.Tensor,
                       recv: torch.Tensor, marks: torch.Tensor, variant: int, epoch: int,
                       out: torch.Tensor | None = None, layout_out: Layout | None = None, count_groups: int = 0,
                       spin_limit_us: int = 0, test_ready_target: int = 0, status: torch.Tensor | None = None):
    """epl_layer_data_as_flag: the one-launch layer with the combine synchronised per 1 KiB chunk by
    Token-Flag Fusion (variant DAF_TOKEN_FLAG_FUSION) or Data-for-Checksum (DAF_DATA_CHECKSUM).
    marks: from alloc_marks (zero-filled), kept from call to call; epoch: nonzero, a new value on
    every call (for Token-Flag Fusion, never one used before on these marks). -> (Layout,
    out [T, H] bf16, status [1] int32)."""
    dev = topk_idx.device
    if cfg.payload != PAYLOAD_BF16:
        raise EplError(5, "epl_layer_data_as_flag (bf16 only)")
    L = _layout_args(cfg, topk_idx, layout_out)
    recv, _, _, rows = _recv_args(cfg, x, recv, None, dev)
    _dev(marks, "marks", torch.int64)
    if marks.numel() * 8 < layer_marks_bytes(cfg, rows):
        raise ValueError("marks has %d bytes, needs %d" % (marks.numel() * 8, layer_marks_bytes(cfg, rows)))
    _dev(topk_w, "topk_w", torch.float32)
    if _rows_of(topk_w, "topk_w", cfg.topk) < cfg.T:
        raise ValueError("topk_w has %d rows, needs T = %d" % (topk_w.shape[0], cfg.T))
    if out is None:
        out = torch.empty(max(cfg.T, 1), cfg.hidden, dtype=torch.bfloat16, device=dev)
    _dev(out, "out", torch.bfloat16)
    if _rows_of(out, "out", cfg.hidden) < cfg.T:
        raise ValueError("out has %d rows, needs T = %d" % (out.shape[0], cfg.T))
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device=dev)
    _dev(status, "status", torch.int32)
    _same_device(dev, topk_w=topk_w, out=out, status=status, marks=marks)
    opts = DecomposedOpts(count_groups, spin_limit_us, test_ready_target)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_layer_data_as_flag(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                            L.workspace.data_ptr(), L.workspace.numel(), x.data_ptr(), recv.data_ptr(),
                                            rows, topk_w.data_ptr(), out.data_ptr(), marks.data_ptr(), variant, epoch,
                                            ctypes.byref(opts), status.data_ptr(), _stream(dev)),
               "epl_layer_data_as_flag")
    return L, out, status


def sentinel_fill(buf: torch.Tensor) -> torch.Tensor:
    """epl_sentinel_fill over a bf16 GPU tensor: a contiguous one, or a 2-D view of rows with a
    pitch (as alloc_recv returns), filled from its first element to its last, the gaps between
    rows included."""
    if not isinstance(buf, torch.Tensor) or buf.device.type != "cuda" or buf.dtype != torch.bfloat16:
        raise ValueError("buf must be a bf16 GPU tensor")
    if buf.dim() == 2 and buf.shape[0] > 1 and buf.stride(1) == 1 and buf.stride(0) >= buf.shape[1]:
        n = (buf.shape[0] - 1) * buf.stride(0) + buf.shape[1]
    else:
        _dev(buf, "buf", torch.bfloat16)
        n = buf.numel()
    with _on(buf.device):
        _check(lib().epl_sentinel_fill(buf.data_ptr(), n, _stream(buf.device)), "epl_sentinel_fill")
    return buf


def sentinel_find(values) -> int:
    """epl_sentinel_find on HOST bf16 bit patterns (a numpy uint16/int16 array or a CPU bf16
    tensor): index of the first sentinel, or -1."""
    import numpy as np

    if isinstance(values, torch.Tensor):
        if values.device.type != "cpu":
            raise ValueError("sentinel_find checks host memory")
        values = values.contiguous().view(torch.int16).numpy()
    a = np.ascontiguousarray(values).view(np.uint16)
    return int(lib().epl_sentinel_find(a.ctypes.data_as(ctypes.c_void_p), a.size))


def decomposed_plan(cfg: Config, count_groups: int = 0):
    """epl_decomposed_plan on the current device -> (count workgroups, grid, co-resident capacity)."""
    grid, cap = ctypes.c_int32(0), ctypes.c_int32(0)
    n = lib().epl_decomposed_plan(ctypes.byref(cfg), count_groups, ctypes.byref(grid), ctypes.byref(cap))
    if n < 0:
        raise EplError(5, "epl_decomposed_plan(%r)" % (cfg,))
    return n, grid.value, cap.value


def dispatch_rows(cfg: Config, topk_idx: torch.Tensor, x: torch.Tensor, L: Layout, recv: torch.Tensor | None = None,
                  recv_scale: torch.Tensor | None = None):
    """epl_dispatch_rows: second phase of layout_dispatch, one kernel, after layout_counts on the
    same stream with the same topk_idx and L -> (recv, recv_scale | None)."""
    dev = topk_idx.device
    _layout_args(cfg, topk_idx, L)
    recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_dispatch_rows(ctypes.byref(cfg), topk_idx.data_ptr(), ctypes.byref(bufs),
                                       L.workspace.data_ptr(), L.workspace.numel(), x.data_ptr(), recv.data_ptr(),
                                       sp, rows, _stream(dev)), "epl_dispatch_rows")
    return recv, recv_scale


def locate_rows(cfg: Config, L: Layout, rows: torch.Tensor | None = None, n: int | None = None):
    """epl_locate_rows: expert and in-expert offset of packed rows (rows [n] int32 on the GPU, or
    the positions 0..n-1 when rows is None) -> (expert [n] int32, offset [n] int32)."""
    dev = L.expert_off.device
    if rows is not None:
        _dev(rows, "rows", torch.int32)
        _same_device(dev, rows=rows)
        n = rows.numel()
    elif n is None or n < 0:
        raise ValueError("give rows, or n >= 0 for the positions 0..n-1")
    if L.cfg.num_experts != cfg.num_experts:
        raise ValueError("layout was allocated for %r, not %r" % (L.cfg, cfg))
    expert = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    offset = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    with _on(dev):
        _check(lib().epl_locate_rows(ctypes.byref(cfg), L.expert_off.data_ptr(),
                                     None if rows is None else rows.data_ptr(), n, expert.data_ptr(),
                                     offset.data_ptr(), _stream(dev)), "epl_locate_rows")
    return expert[:n], offset[:n]


def hop_schedule(cfg: Config, send_cnt: torch.Tensor, hop_class: torch.Tensor, workers: int, num_classes: int,
                 remap_rows: int = 0, order: torch.Tensor | None = None):
    """epl_hop_schedule: send_cnt [R, E] and hop_class [R, R] int32 on the GPU (order [E] int32, or
    None for the transposition with remap_rows rows, 0 = one per worker) -> (start_expert [R, n],
    start_offset [R, n], class_cnt [R, n, num_classes]) int32, n = workers."""
    dev = send_cnt.device
    R, E = cfg.num_ranks, cfg.num_experts
    _dev(send_cnt, "send_cnt", torch.int32)
    _dev(hop_class, "hop_class", torch.int32)
    if send_cnt.numel() != R * E or hop_class.numel() != R * R:
        raise ValueError("send_cnt must hold R*E and hop_class R*R values")
    if order is not None:
        _dev(order, "order", torch.int32)
        if order.numel() != E:
            raise ValueError("order must hold E values")
    _same_device(dev, hop_class=hop_class, order=order)
    i32 = dict(dtype=torch.int32, device=dev)
    n = max(int(workers), 1)
    se = torch.empty(R, n, **i32)
    so = torch.empty(R, n, **i32)
    cnt = torch.empty(R, n, max(int(num_classes), 1), **i32)
    with _on(dev):
        _check(lib().epl_hop_schedule(ctypes.byref(cfg), send_cnt.data_ptr(),
                                      None if order is None else order.data_ptr(), remap_rows,
                                      hop_class.data_ptr(), workers, num_classes, se.data_ptr(), so.data_ptr(),
                                      cnt.data_ptr(), _stream(dev)), "epl_hop_schedule")
    return se, so, cnt


def dispatch_scheduled(cfg: Config, x: torch.Tensor, L: Layout, workers: int, remap_rows: int = 0,
                       recv: torch.Tensor | None = None, recv_scale: torch.Tensor | None = None):
    """epl_dispatch_scheduled: the rows of epl_dispatch, written by one workgroup per (source rank,
    worker) in the order of the hierarchical token-level schedule -> (recv [cap, H] bf16 | uint8,
    recv_scale [cap, H/128] fp32 | None)."""
    dev = x.device
    _check_layout(cfg, L, dev)
    recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_dispatch_scheduled(ctypes.byref(cfg), x.data_ptr(), ctypes.byref(bufs), recv.data_ptr(), sp,
                                            rows, remap_rows, workers, _stream(dev)), "epl_dispatch_scheduled")
    return recv, recv_scale


def combine(cfg: Config, y: torch.Tensor, topk_w: torch.Tensor, L: Layout, out: torch.Tensor | None = None):
    """epl_combine: y [>=P, H] bf16 with rows cfg.pitch apart, topk_w [T, k] fp32 -> out [T, H] bf16."""
    dev = y.device
    _pitched_rows(y, "y", torch.bfloat16, cfg)  # its row count must cover P, which only the device knows
    _dev(topk_w, "topk_w", torch.float32)
    if _rows_of(topk_w, "topk_w", cfg.topk) < cfg.T:
        raise ValueError("topk_w has %d rows, needs T = %d" % (topk_w.shape[0], cfg.T))
    _check_layout(cfg, L, dev)
    if out is None:
        out = torch.empty(max(cfg.T, 1), cfg.hidden, dtype=torch.bfloat16, device=dev)
    _dev(out, "out", torch.bfloat16)
    if _rows_of(out, "out", cfg.hidden) < cfg.T:
        raise ValueError("out has %d rows, needs T = %d" % (out.shape[0], cfg.T))
    _same_device(dev, topk_w=topk_w, out=out)
    bufs = L.buffers()
    with _on(dev):
        _check(lib().epl_combine(ctypes.byref(cfg), y.data_ptr(), topk_w.data_ptr(), ctypes.byref(bufs),
                                 out.data_ptr(), _stream(dev)), "epl_combine")
    return out


class PreparedLayer:
    """One MoE layer's calls with every argument checked and converted once, for loops that issue
    the same layer many times (a serving loop, a benchmark). layout_dispatch(i) is
    epl_layout_dispatch with x = xs[i % len(xs)], layout_counts() and dispatch_rows(i) are its two
    phases, combine() is epl_combine, and run(i) is layout_dispatch(i) then combine(); each is one
    C call with prebuilt arguments on the stream current at construction. Construction makes the
    checks the plain calls make; afterwards the tensors must stay alive and keep their shapes, and
    the calls must be made with the same current device."""

    def __init__(self, cfg: Config, topk_idx: torch.Tensor, xs, topk_w: torch.Tensor, L: Layout,
                 recv: torch.Tensor, recv_scale: torch.Tensor | None = None, y: torch.Tensor | None = None,
                 out: torch.Tensor | None = None):
        dev = topk_idx.device
        xs = list(xs)
        if not xs:
            raise ValueError("give at least one x")
        L = _layout_args(cfg, topk_idx, L)
        sp = rows = None
        for x in xs:
            recv, recv_scale, sp, rows = _recv_args(cfg, x, recv, recv_scale, dev)
        y = recv if y is None else y
        _pitched_rows(y, "y", torch.bfloat16, cfg)
        _dev(topk_w, "topk_w", torch.float32)
        if _rows_of(topk_w, "topk_w", cfg.topk) < cfg.T:
            raise ValueError("topk_w has %d rows, needs T = %d" % (topk_w.shape[0], cfg.T))
        if out is None:
            out = torch.empty(max(cfg.T, 1), cfg.hidden, dtype=torch.bfloat16, device=dev)
        _dev(out, "out", torch.bfloat16)
        if _rows_of(out, "out", cfg.hidden) < cfg.T:
            raise ValueError("out has %d rows, needs T = %d" % (out.shape[0], cfg.T))
        _same_device(dev, y=y, topk_w=topk_w, out=out)
        if torch.cuda.current_device() != dev.index:
            raise ValueError("make %s the current device before preparing its layer" % dev)
        self.L, self.recv, self.recv_scale, self.y, self.out = L, recv, recv_scale, y, out
        # A private copy of the config and of the pointer struct, and a reference to every tensor
        # whose address is baked into the calls: changing the caller's cfg, or replacing a field
        # of L, later leaves these calls as they were checked.
        self.cfg = Config(*[getattr(cfg, f) for f, _ in Config._fields_])
        self._bufs = LayoutBuffers(*[getattr(L, n).data_ptr() for n, _ in LayoutBuffers._fields_])
        self._keep = (topk_idx, xs, topk_w, [getattr(L, n) for n, _ in LayoutBuffers._fields_], L.workspace)
        cp, bp, st = ctypes.byref(self.cfg), ctypes.byref(self._bufs), _stream(dev)
        ws, wsn = L.workspace.data_ptr(), L.workspace.numel()
        lb = lib()
        self._ld, self._lc, self._dr, self._cb = (lb.epl_layout_dispatch, lb.epl_layout_counts, lb.epl_dispatch_rows,
                                                  lb.epl_combine)
        self._ld_args = [(cp, topk_idx.data_ptr(), bp, ws, wsn, x.data_ptr(), recv.data_ptr(), sp, rows, st)
                         for x in xs]
        self._lc_args = (cp, topk_idx.data_ptr(), bp, ws, wsn, st)
        self._cb_args = (cp, y.data_ptr(), topk_w.data_ptr(), bp, out.data_ptr(), st)

    def layout_dispatch(self, i: int = 0) -> None:
        s = self._ld(*self._ld_args[i % len(self._ld_args)])
        if s:
            raise EplError(s, "epl_layout_dispatch")

    def layout_counts(self) -> None:
        s = self._lc(*self._lc_args)
        if s:
            raise EplError(s, "epl_layout_counts")

    def dispatch_rows(self, i: int = 0) -> None:
        s = self._dr(*self._ld_args[i % len(self._ld_args)])
        if s:
            raise EplError(s, "epl_dispatch_rows")

    def combine(self) -> None:
        s = self._cb(*self._cb_args)
        if s:
            raise EplError(s, "epl_combine")

    def run(self, i: int = 0) -> None:
        self.layout_dispatch(i)
        self.combine()


def debug_f32_to_e4m3(v: torch.Tensor) -> torch.Tensor:
    _dev(v, "v", torch.float32)
    out = torch.empty(v.numel(), dtype=torch.uint8, device=v.device)
    _check(lib().epl_debug_f32_to_e4m3(v.data_ptr(), out.data_ptr(), v.numel(), _stream(v.device)),
           "epl_debug_f32_to_e4m3")
    return out


def debug_f32_to_bf16(v: torch.Tensor) -> torch.Tensor:
    _dev(v, "v", torch.float32)
    out = torch.empty(v.numel(), dtype=torch.int16, device=v.device)
    _check(lib().epl_debug_f32_to_bf16(v.data_ptr(), out.data_ptr(), v.numel(), _stream(v.device)),
           "epl_debug_f32_to_bf16")
    return out


def layout_launches(cfg: Config) -> int:
    """Kernel launches epl_layout issues for cfg: 1 (single-launch layout) or 3."""
    n = lib().epl_layout_launches(ctypes.byref(cfg))
    if n < 0:
        raise EplError(1, "epl_layout_launches")
    return n


def layout_dispatch_launches(cfg: Config) -> int:
    """Kernel launches epl_layout_dispatch issues for cfg: 2, 3 (finalize fused into dispatch) or 4;
    layout_counts issues all but the last."""
    n = lib().epl_layout_dispatch_launches(ctypes.byref(cfg))
    if n < 0:
        raise EplError(1, "epl_layout_dispatch_launches")
    return n


def version() -> str:
    return lib().epl_version().decode()
