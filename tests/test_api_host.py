"""Host-side checks of the C ABI that need no GPU.

* libepl.so loads and exports every function include/epl.h declares.
* Argument errors are reported with the documented status BEFORE any HIP call. The pointers
  below are fake addresses that the library must never dereference or launch on.
* Workspace sizing follows the documented chunking.
"""
import ctypes
import os
import re

import pytest

from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "epl.h")

OK, INVALID, ALIGN, CAPACITY, WORKSPACE, UNSUPPORTED = 0, 1, 2, 3, 4, 5


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(epl.LIB_PATH):
        from paper_2607_06202_amd import _build
        _build.build()
    return epl.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(epl_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"epl_layout", "epl_dispatch", "epl_combine", "epl_workspace_bytes", "epl_status_str",
            "epl_version"} <= set(names)
    for n in names:
        assert hasattr(lib, n), "libepl.so does not export " + n


def test_layout_launch_count():
    """One launch up to T*k = 16384, Tr*k = 4096 and 64 KiB of LDS; three beyond."""
    for name, want in [("tiny", 1), ("decode_ep64", 3), ("prefill_ep32", 3), ("skewed_fp8_ep64", 3),
                       ("large_ep256", 3)]:
        w = W.WORKLOADS[name]
        assert epl.layout_launches(epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload)) == want, name
    assert epl.layout_launches(epl.config(32, 256, 8, 64, 64)) == 1      # T*k = 16384
    assert epl.layout_launches(epl.config(32, 256, 8, 64, 65)) == 3      # T*k = 16640
    assert epl.layout_launches(epl.config(2, 16, 8, 64, 512)) == 1       # Tr*k = 4096
    assert epl.layout_launches(epl.config(2, 16, 8, 64, 513)) == 3       # Tr*k = 4104
    assert epl.layout_launches(epl.config(64, 1024, 8, 64, 32)) == 1     # LDS 53.5 KiB
    assert epl.layout_launches(epl.config(1024, 1024, 2, 64, 2)) == 3    # LDS 76 KiB
    assert epl.layout_launches(epl.config(2, 16, 8, 64, 0)) == 1         # no tokens
    with pytest.raises(epl.EplError):
        epl.layout_launches(epl.config(3, 16, 8, 64, 4))                 # E % R != 0


def test_layout_dispatch_launch_count():
    """The finalize step runs inside the dispatch for bf16 with at most 256 pairs per chunk and 256
    experts (3 launches); small layouts take 2, everything else 4."""
    want = {"tiny": 2, "decode_ep64": 3, "prefill_ep32": 4, "skewed_fp8_ep64": 4, "large_ep256": 4}
    for name, n in want.items():
        w = W.WORKLOADS[name]
        assert epl.layout_dispatch_launches(epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload)) == n, name
    assert epl.layout_dispatch_launches(epl.config(64, 256, 8, 7168, 128, "fp8")) == 4  # decode shape, fp8
    assert epl.layout_dispatch_launches(epl.config(64, 512, 8, 7168, 128)) == 4         # 512 experts
    assert epl.layout_dispatch_launches(epl.config(64, 256, 8, 7168, 130)) == 4         # 264 pairs per chunk
    with pytest.raises(epl.EplError):
        epl.layout_dispatch_launches(epl.config(3, 16, 8, 64, 4))


def test_version_and_status_strings(lib):
    assert "gfx950" in epl.version()
    for code in range(7):
        s = lib.epl_status_str(code).decode()
        assert s.startswith(epl.STATUS[code])


class Fake:
    """Distinct, 256-byte aligned fake device addresses (never dereferenced)."""
    base = 0x7F0000000000

    @classmethod
    def ptr(cls, i, misalign=0):
        return cls.base + 0x100000 * (i + 1) + misalign


def fake_layout(misalign_field=None, null_field=None):
    vals = []
    for i, (n, _) in enumerate(epl.LayoutBuffers._fields_):
        p = Fake.ptr(i, 2 if n == misalign_field else 0)
        vals.append(None if n == null_field else p)
    return epl.LayoutBuffers(*vals)


def call_layout(lib, cfg, idx=Fake.ptr(50), L=None, ws=Fake.ptr(60), ws_bytes=1 << 30):
    L = L if L is not None else fake_layout()
    return lib.epl_layout(ctypes.byref(cfg), idx, ctypes.byref(L), ws, ws_bytes, None)


GOOD = dict(R=8, E=64, k=8, H=7168, Tr=16)


def cfg(**kw):
    a = dict(GOOD)
    a.update(kw)
    return epl.config(a["R"], a["E"], a["k"], a["H"], a["Tr"], a.get("payload", "bf16"))


@pytest.mark.parametrize("bad", [dict(R=0), dict(E=7), dict(E=4), dict(k=0), dict(k=33), dict(E=2048, R=8),
                                 dict(H=7), dict(H=0), dict(H=1 << 21), dict(Tr=-1), dict(R=64, E=256, k=32, Tr=1 << 21)])
def test_layout_rejects_bad_config(lib, bad):
    assert call_layout(lib, cfg(**bad)) == INVALID
    assert lib.epl_workspace_bytes(ctypes.byref(cfg(**bad))) == 0


def test_unknown_payload(lib):
    c = cfg()
    c.payload = 7
    assert call_layout(lib, c) == UNSUPPORTED


def test_layout_buffer_errors(lib):
    assert lib.epl_layout(ctypes.byref(cfg()), Fake.ptr(50), None, Fake.ptr(60), 1 << 30, None) == INVALID
    for n, _ in epl.LayoutBuffers._fields_:
        assert call_layout(lib, cfg(), L=fake_layout(null_field=n)) == INVALID, n
        assert call_layout(lib, cfg(), L=fake_layout(misalign_field=n)) == ALIGN, n
    assert call_layout(lib, cfg(), idx=None) == INVALID
    assert call_layout(lib, cfg(), idx=Fake.ptr(50, 1)) == ALIGN
    assert call_layout(lib, cfg(), ws=None) == WORKSPACE
    assert call_layout(lib, cfg(), ws=Fake.ptr(60, 2)) == ALIGN
    need = lib.epl_workspace_bytes(ctypes.byref(cfg()))
    assert call_layout(lib, cfg(), ws_bytes=need - 1) == WORKSPACE


def test_workspace_formula(lib):
    # Chunks hold whole tokens. There are at most 1024 pairs per chunk. The target is >= 256
    # workgroups and >= 64 pairs per workgroup.
    for (R, E, k, Tr) in [(64, 256, 8, 128), (32, 256, 8, 4096), (256, 256, 8, 64), (4, 16, 2, 128), (3, 9, 5, 0),
                          (2, 8, 1, 2500), (1024, 1024, 32, 3)]:
        T = R * Tr
        want = max(-(-T // 256), -(-64 // k))
        CT = min(min(want, 1024 // k), Tr) if Tr > 0 else 1
        NC = -(-Tr // CT) if Tr > 0 else 1
        nblk = R * NC
        before_sync = E * nblk + nblk * R + E + nblk + E * R + T + nblk * E  # counts, totals, offsets, masks
        want_bytes = 4 * (-(-before_sync // 64) * 64 + 256)  # then 1 KiB of synchronisation words
        assert lib.epl_workspace_bytes(ctypes.byref(epl.config(R, E, k, 64, Tr))) == want_bytes


def test_dispatch_errors(lib):
    L = fake_layout()
    x, recv, sc = Fake.ptr(70), Fake.ptr(71), Fake.ptr(72)
    c = cfg()
    cap = 8 * 16 * 8
    d = lambda c, x=x, recv=recv, sc=sc, cap=cap, L=L: lib.epl_dispatch(ctypes.byref(c), x, ctypes.byref(L), recv, sc,
                                                                        cap, None)
    assert d(c, cap=cap - 1) == CAPACITY
    assert d(c, x=Fake.ptr(70, 8)) == ALIGN
    assert d(c, recv=Fake.ptr(71, 4)) == ALIGN
    assert d(c, x=None) == INVALID
    assert d(c, L=fake_layout(null_field="pair_row")) == INVALID
    f8 = cfg(payload="fp8", H=7168 + 64)
    assert d(f8) == UNSUPPORTED
    f8 = cfg(payload="fp8")
    assert d(f8, sc=None) == INVALID
    assert d(f8, sc=Fake.ptr(72, 2)) == ALIGN


def test_combine_errors(lib):
    L = fake_layout()
    c = cfg()
    y, w, out = Fake.ptr(80), Fake.ptr(81), Fake.ptr(82)
    cb = lambda y=y, w=w, out=out: lib.epl_combine(ctypes.byref(c), y, w, ctypes.byref(L), out, None)
    assert cb(out=Fake.ptr(82, 8)) == ALIGN
    assert cb(y=Fake.ptr(80, 2)) == ALIGN
    assert cb(w=Fake.ptr(81, 2)) == ALIGN
    assert cb(w=None) == INVALID


def test_noalloc_errors_before_any_hip_call(lib):
    """epl_layout_dispatch_noalloc reports argument errors, and a workspace beyond its static
    scratch (1024 ranks of one expert: 12 MiB > 8 MiB), before it touches the HIP runtime."""
    L = fake_layout()
    idx, x, recv = Fake.ptr(50), Fake.ptr(70), Fake.ptr(71)
    f = lambda c, idx=idx, x=x, recv=recv, sc=None, cap=1 << 20, L=L: lib.epl_layout_dispatch_noalloc(
        ctypes.byref(c), idx, ctypes.byref(L) if L is not None else None, x, recv, sc, cap, None)
    big = epl.config(1024, 1024, 8, 64, 16)
    assert lib.epl_workspace_bytes(ctypes.byref(big)) > epl.STATIC_SCRATCH_BYTES
    assert f(big, cap=1024 * 16 * 8) == WORKSPACE
    c = cfg()
    assert lib.epl_workspace_bytes(ctypes.byref(c)) <= epl.STATIC_SCRATCH_BYTES
    assert f(epl.config(3, 8, 2, 64, 4)) == INVALID  # E % R != 0
    assert f(c, cap=8 * 16 * 8 - 1) == CAPACITY
    assert f(c, x=Fake.ptr(70, 8)) == ALIGN
    assert f(c, idx=None) == INVALID
    assert f(c, L=None) == INVALID
    assert f(cfg(payload="fp8", H=7168 + 64)) == UNSUPPORTED
    assert f(cfg(payload="fp8")) == INVALID  # no scale buffer


def test_decomposed_errors_before_any_hip_call(lib):
    """epl_layout_dispatch_decomposed reports bad options, unsupported payloads and shapes, and a
    missing status word before it touches the HIP runtime."""
    L = fake_layout()
    idx, ws, x, recv, st = Fake.ptr(50), Fake.ptr(60), Fake.ptr(70), Fake.ptr(71), Fake.ptr(90)
    c = epl.config(64, 256, 8, 7168, 128)
    need = lib.epl_workspace_bytes(ctypes.byref(c))

    def f(c=c, opts=None, st=st, cap=64 * 128 * 8, sc=None):
        return lib.epl_layout_dispatch_decomposed(ctypes.byref(c), idx, ctypes.byref(L), ws, 1 << 30, x, recv, sc, cap,
                                                  ctypes.byref(opts) if opts is not None else None, st, None)
    assert f(opts=epl.DecomposedOpts(-1, 0, 0)) == INVALID
    assert f(opts=epl.DecomposedOpts(0, -5, 0)) == INVALID
    assert f(opts=epl.DecomposedOpts(0, 0, -1)) == INVALID
    assert f(c=epl.config(64, 256, 8, 7168, 128, "fp8"), sc=Fake.ptr(72)) == UNSUPPORTED
    assert f(c=epl.config(64, 512, 8, 7168, 128)) == UNSUPPORTED          # 512 experts
    assert f(c=epl.config(64, 256, 8, 7168, 130), cap=64 * 130 * 8) == UNSUPPORTED  # 264 pairs per chunk
    assert f(st=None) == INVALID
    assert f(st=Fake.ptr(90, 2)) == ALIGN
    assert f(cap=64 * 128 * 8 - 1) == CAPACITY


def test_debug_errors(lib):
    assert lib.epl_debug_f32_to_e4m3(Fake.ptr(1), Fake.ptr(2), -1, None) == INVALID
    assert lib.epl_debug_f32_to_bf16(None, Fake.ptr(2), 5, None) == INVALID
    assert lib.epl_debug_f32_to_bf16(Fake.ptr(1, 2), Fake.ptr(2), 5, None) == ALIGN


def test_binding_rejects_host_tensors_before_any_call():
    """The Python binding only marshals: a CPU tensor is refused before the library is entered."""
    import torch
    cfg_ = epl.config(2, 4, 2, 64, 3)
    with pytest.raises(ValueError):
        epl.layout(cfg_, torch.zeros(6, 2, dtype=torch.int32))
    with pytest.raises(ValueError):
        epl.debug_f32_to_e4m3(torch.zeros(4))
    L = epl.Layout(cfg_, *[torch.zeros(1, dtype=torch.int32)] * 11, torch.zeros(1, dtype=torch.uint8))
    with pytest.raises(ValueError):
        epl.PreparedLayer(cfg_, torch.zeros(6, 2, dtype=torch.int32), [torch.zeros(6, 64, dtype=torch.bfloat16)],
                          torch.zeros(6, 2), L, torch.zeros(12, 64, dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        epl.PreparedLayer(cfg_, torch.zeros(6, 2, dtype=torch.int32), [], torch.zeros(6, 2), L,
                          torch.zeros(12, 64, dtype=torch.bfloat16))


from hypothesis import given, settings, strategies as st  # noqa: E402


def _valid(R, E, k, H, Tr, payload, P=0):
    """The config rules documented in include/epl.h."""
    return (R >= 1 and R <= E <= epl.MAX_EXPERTS and E % R == 0 and 1 <= k <= 32 and Tr >= 0 and 8 <= H <= 1 << 20
            and H % 8 == 0 and R * Tr * k < 2 ** 31 - 1 and payload in (0, 1)
            and (P == 0 or (H <= P <= 1 << 20 and P % 64 == 0)))


@settings(max_examples=400, deadline=None)
@given(R=st.one_of(st.integers(-2, 70), st.sampled_from([128, 256, 1024, 1025])),
       E=st.one_of(st.integers(-2, 300), st.sampled_from([512, 1024, 1025, 2048])),
       k=st.integers(-1, 34), H=st.one_of(st.integers(-8, 300), st.sampled_from([7168, 1 << 20, (1 << 20) + 8])),
       Tr=st.one_of(st.integers(-2, 5000), st.sampled_from([1 << 20, 1 << 24])), payload=st.integers(-1, 2),
       P=st.one_of(st.just(0), st.integers(-70, 400),
                   st.sampled_from([7168, 7168 + 768, 7168 + 8, 7104, 1 << 20, (1 << 20) + 64])))
def test_config_rules_property(lib, R, E, k, H, Tr, payload, P):
    """Host-side validation follows the documented rules for any config, row pitch included;
    rejected configs never reach a launch (the calls below use fake pointers and would fault if
    they did)."""
    c = epl.Config(R, E, k, H, Tr, payload, P)
    ok = _valid(R, E, k, H, Tr, payload, P)
    assert (lib.epl_workspace_bytes(ctypes.byref(c)) > 0) == ok
    n = lib.epl_layout_launches(ctypes.byref(c))
    assert (n in (1, 3)) if ok else n == -1
    if not ok:
        st_ = call_layout(lib, c)
        assert st_ in (INVALID, UNSUPPORTED)
        assert (st_ == UNSUPPORTED) == (payload not in (0, 1) and _valid(R, E, k, H, Tr, 0, P))


def test_row_pitch_rule_and_tuned_pitch(lib):
    """The pitch rule at its edges, for every call that takes a config, and the benchmark's tuned
    pitches: valid pitches, and packed rows for every shape without a measured entry."""
    for P, ok in ((0, True), (7168, True), (7168 + 64, True), (7168 + 768, True), (1 << 20, True),
                  (7104, False), (7168 + 8, False), (7168 + 32, False), (-64, False), ((1 << 20) + 64, False)):
        for payload in (0, 1):
            c = epl.Config(64, 256, 8, 7168, 128, payload, P)
            assert (lib.epl_workspace_bytes(ctypes.byref(c)) > 0) == ok, (P, payload)
            if not ok:
                assert call_layout(lib, c) == INVALID
    assert epl.tuned_pitch(7168) == 7936 and epl.tuned_pitch(7168, "fp8") == 0
    assert epl.tuned_pitch(5120) == 0 and epl.tuned_pitch(2048) == 0 and epl.tuned_pitch(256) == 0
    for (H, payload), P in epl.TUNED_PITCH.items():
        c = epl.Config(64, 256, 8, H, 128, payload, P)
        assert lib.epl_workspace_bytes(ctypes.byref(c)) > 0
    assert epl.config(2, 4, 1, 64, 3).pitch == 64 and epl.config(2, 4, 1, 64, 3, row_pitch=128).pitch == 128


def test_contiguous_block_views_must_fit_the_block():
    """A tensor over a contiguous HIP block may not claim more bytes than the block holds: the
    kernels write wherever the tensor says its rows are. The check runs on the host, before any
    memory is touched (an object without a device allocation stands in for the block here)."""
    import torch

    b = object.__new__(epl._ContiguousBlock)
    b.ptr, b.nbytes, b.device = ctypes.c_void_p(), 100, torch.device("cuda:0")
    with pytest.raises(ValueError):
        b.tensor((51,), torch.bfloat16)  # 102 bytes
    with pytest.raises(ValueError):
        b.tensor((3, 34), torch.uint8)  # 102 bytes


def test_sentinel_find_on_the_host(lib):
    """The initialisation check for Sentinel Polling runs on the host: the first index of the
    reserved bf16 pattern, or -1; other NaNs, infinities and every other pattern pass."""
    import numpy as np

    assert epl.SENTINEL_BF16 == 0xFFFF
    every = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    assert epl.sentinel_find(every) == 0xFFFF
    others = every[every != 0xFFFF]
    assert epl.sentinel_find(others) == -1
    x = W.normal_bf16(3, W.STREAM_X, 4096)
    assert epl.sentinel_find(x) == -1
    x[1234] = 0xFFFF
    x[3000] = 0xFFFF
    assert epl.sentinel_find(x) == 1234
    assert lib.epl_sentinel_find(None, 5) == -1
    assert epl.sentinel_find(np.zeros(0, np.uint16)) == -1


def test_layer_sentinel_errors_before_any_hip_call(lib):
    L = fake_layout()
    c = epl.config(4, 16, 2, 256, 128)
    idx, ws, x, recv, w, out, st = (Fake.ptr(i) for i in (50, 60, 70, 71, 80, 81, 90))

    def f(c=c, w=w, out=out, st=st, opts=None):
        return lib.epl_layer_sentinel(ctypes.byref(c), idx, ctypes.byref(L), ws, 1 << 30, x, recv, 4 * 128 * 2, w, out,
                                      ctypes.byref(opts) if opts is not None else None, st, None)
    assert f(w=None) == INVALID
    assert f(out=Fake.ptr(81, 8)) == ALIGN
    assert f(st=None) == INVALID
    assert f(opts=epl.DecomposedOpts(-1, 0, 0)) == INVALID
    assert f(c=epl.config(4, 16, 2, 256, 128, "fp8")) == INVALID  # fp8 needs a scale buffer first
    assert lib.epl_sentinel_fill(Fake.ptr(1), 12, None) == INVALID  # not a multiple of 8 elements
    assert lib.epl_sentinel_fill(Fake.ptr(1, 8), 16, None) == ALIGN


def test_layer_data_as_flag_errors_before_any_hip_call(lib):
    """The flag and checksum layer: every argument error is reported before the call touches the
    GPU (the calls below use fake pointers and would fault if they launched)."""
    L = fake_layout()
    c = epl.config(4, 16, 2, 256, 128)
    idx, ws, x, recv, w, out, st, marks = (Fake.ptr(i) for i in (50, 60, 70, 71, 80, 81, 90, 91))

    def f(c=c, w=w, out=out, st=st, marks=marks, variant=epl.DAF_DATA_CHECKSUM, epoch=1, opts=None):
        return lib.epl_layer_data_as_flag(ctypes.byref(c), idx, ctypes.byref(L), ws, 1 << 30, x, recv, 4 * 128 * 2, w,
                                          out, marks, variant, epoch, ctypes.byref(opts) if opts is not None else None,
                                          st, None)
    for variant in (epl.DAF_TOKEN_FLAG_FUSION, epl.DAF_DATA_CHECKSUM):
        assert f(variant=variant, marks=None) == INVALID
        assert f(variant=variant, marks=Fake.ptr(91, 4)) == ALIGN
        assert f(variant=variant, epoch=0) == INVALID
        assert f(variant=variant, w=None) == INVALID
        assert f(variant=variant, out=Fake.ptr(81, 8)) == ALIGN
        assert f(variant=variant, st=None) == INVALID
        assert f(variant=variant, opts=epl.DecomposedOpts(-1, 0, 0)) == INVALID
        assert f(variant=variant, c=epl.config(4, 16, 2, 256, 128, "fp8")) == INVALID  # no scale buffer
        assert f(variant=variant, c=epl.config(4, 16, 2, 256, 128, row_pitch=300)) == INVALID
    for variant in (0, 3, -1):
        assert f(variant=variant) == INVALID
    assert f(variant=0, c=epl.config(4, 15, 2, 256, 128)) == INVALID  # the config is checked first
    assert lib.epl_layer_marks_bytes(ctypes.byref(c), 1024) == 1024 * 1 * 8  # H = 256: one 1 KiB chunk
    assert lib.epl_layer_marks_bytes(ctypes.byref(epl.config(64, 256, 8, 7168, 128)), 65536) == 65536 * 14 * 8
    assert lib.epl_layer_marks_bytes(ctypes.byref(epl.config(2, 4, 1, 520, 3)), 7) == 7 * 2 * 8  # a ragged chunk
    assert lib.epl_layer_marks_bytes(ctypes.byref(c), -1) == -1
    assert lib.epl_layer_marks_bytes(ctypes.byref(epl.config(4, 15, 2, 256, 128)), 8) == -1


def test_schedule_errors_before_any_hip_call(lib):
    """epl_hop_schedule and epl_dispatch_scheduled report bad worker counts, class counts, remap
    rows, payloads, missing buffers, misalignment and capacity before they touch the HIP runtime."""
    c = epl.config(64, 256, 8, 7168, 128)
    sc, hop, se, so, cc = Fake.ptr(10), Fake.ptr(11), Fake.ptr(12), Fake.ptr(13), Fake.ptr(14)

    def hs(c=c, sc=sc, order=None, rows=0, hop=hop, n=32, nh=2, se=se, so=so, cc=cc):
        return lib.epl_hop_schedule(ctypes.byref(c), sc, order, rows, hop, n, nh, se, so, cc, None)
    assert hs(n=0) == INVALID
    assert hs(n=1 << 30) == INVALID          # R * workers >= 2^31
    assert hs(nh=0) == INVALID
    assert hs(nh=epl.MAX_HOP_CLASSES + 1) == INVALID
    assert hs(rows=-1) == INVALID
    assert hs(sc=None) == INVALID
    assert hs(hop=None) == INVALID
    assert hs(cc=None) == INVALID
    assert hs(order=Fake.ptr(15, 2)) == ALIGN
    assert hs(se=Fake.ptr(12, 1)) == ALIGN
    assert hs(c=epl.config(3, 16, 8, 64, 4)) == INVALID  # E % R != 0

    L = fake_layout()
    x, recv = Fake.ptr(70), Fake.ptr(71)

    def ds(c=c, x=x, recv=recv, sc=None, cap=64 * 128 * 8, rows=0, n=32, L=L):
        return lib.epl_dispatch_scheduled(ctypes.byref(c), x, ctypes.byref(L) if L is not None else None, recv, sc,
                                          cap, rows, n, None)
    assert ds(c=epl.config(64, 256, 8, 7168 + 64, 128, "fp8"), sc=Fake.ptr(72)) == UNSUPPORTED  # H % 128 != 0
    assert ds(c=epl.config(64, 256, 8, 7168, 128, "fp8")) == INVALID  # no scale buffer
    assert ds(c=epl.config(64, 256, 8, 7168, 128, "fp8"), sc=Fake.ptr(72, 2)) == ALIGN
    assert ds(n=0) == INVALID
    assert ds(rows=-2) == INVALID
    assert ds(L=None) == INVALID
    assert ds(L=fake_layout(null_field="seg_off")) == INVALID
    assert ds(L=fake_layout(null_field="recv_src")) == INVALID
    assert ds(x=None) == INVALID
    assert ds(x=Fake.ptr(70, 8)) == ALIGN
    assert ds(cap=64 * 128 * 8 - 1) == CAPACITY
