"""The receive layout with a row pitch above H (epl_config.row_pitch): every entry point that writes
receive rows or reads expert-output rows, against the CPU oracle on the same inputs.

The receive buffer is a [rows, pitch] block viewed as [rows, H]. Before each call the whole block
holds a canary; afterwards the gaps between rows (elements H..pitch-1) and the rows past P must
still hold it, and the payload rows must equal the oracle's. The expert outputs y given to the
combine carry NaN patterns in their gaps, which must not reach the output."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import assert_layout_equal, bf16_bits, device, oracle_combine_threaded, to_dev_bf16

pytestmark = pytest.mark.gpu

CANARY_BF16 = 0x7FC1  # a quiet NaN, not the Sentinel Polling pattern
CANARY_FP8 = 0x5A
GAP_NAN = 0x7FC3      # what y holds between its rows


def _block(rows, H, pitch, fp8, dev):
    """(block [rows, pitch], view [rows, H]) filled with the canary."""
    if fp8:
        blk = torch.full((rows, pitch), CANARY_FP8, dtype=torch.uint8, device=dev)
    else:
        blk = torch.full((rows, pitch), CANARY_BF16, dtype=torch.int16, device=dev).view(torch.bfloat16)
    return blk, blk[:, :H]


def _bits(t):
    return t.cpu().numpy() if t.dtype == torch.uint8 else bf16_bits(t)


def _check_block(blk, H, P, want_rows, fp8, what):
    """Payload rows 0..P-1 equal want_rows; every other element still holds the canary."""
    got = _bits(blk)
    canary = CANARY_FP8 if fp8 else CANARY_BF16
    np.testing.assert_array_equal(got[:P, :H], want_rows[:P], err_msg=what + ": payload rows")
    gaps = got[:, H:]
    assert (gaps == canary).all(), "%s: a gap between rows was written (first at %s)" % (
        what, np.argwhere(gaps != canary)[:1].tolist())
    assert (got[P:, :H] == canary).all(), what + ": a row past P was written"


def _case(R, E, k, Tr, H, seed):
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)  # duplicates and invalid ids
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    return idx, x


def _pitched_y(rows, H, pitch, seed, dev):
    """Expert outputs [rows, H] with rows pitch apart and NaN patterns in the gaps -> (view, host bits)."""
    blk = torch.full((rows, pitch), GAP_NAN, dtype=torch.int16, device=dev).view(torch.bfloat16)
    yh = W.normal_bf16(seed, W.STREAM_X + 7, rows * H).reshape(rows, H)
    blk[:, :H].copy_(to_dev_bf16(yh, dev))
    return blk[:, :H], yh


# (R, E, k, Tr, H, pitch, seed, payload, launches of epl_layout_dispatch)
CASES = [
    (4, 16, 2, 128, 256, 320, 0, "bf16", 2),       # the one-launch layout
    (64, 256, 8, 40, 1032, 1088, 1, "bf16", 3),    # the fused finalize; a ragged last column chunk
    (32, 256, 8, 72, 7168, 7936, 2, "bf16", 3),    # the decode row size at the benchmark's pitch
    (8, 512, 4, 2048, 264, 320, 3, "bf16", 4),     # 512 experts: layout K1-K3, then the plain kernel
    (16, 64, 4, 512, 1024, 1088, 4, "fp8", 4),     # fp8 rows of 1 KiB at a pitch of 1,088 bytes
    (8, 32, 3, 300, 2048, 2048 + 512, 5, "fp8", 2),  # fp8 after the one-launch layout
]


@pytest.mark.parametrize("R,E,k,Tr,H,pitch,seed,payload,launches", CASES)
def test_layout_dispatch_and_combine_with_a_pitch(R, E, k, Tr, H, pitch, seed, payload, launches):
    dev = device()
    fp8 = payload == "fp8"
    T = R * Tr
    idx, x = _case(R, E, k, Tr, H, seed)
    cfg = epl.config(R, E, k, H, Tr, payload, row_pitch=pitch)
    assert epl.layout_dispatch_launches(cfg) == launches
    ref = oracle.layout(R, E, k, Tr, idx)
    P = ref.P
    idx_d, x_d = torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev)
    if fp8:
        want_rows, want_scale = oracle.dispatch_fp8(x, ref.pair_row, P)
    else:
        want_rows = oracle.dispatch_bf16(x, ref.pair_row, P)
    what = "R=%d E=%d k=%d Tr=%d H=%d pitch=%d %s" % (R, E, k, Tr, H, pitch, payload)

    def scale_buf():
        return torch.full((T * k, H // 128), float("nan"), device=dev) if fp8 else None

    # epl_layout_dispatch
    blk, recv = _block(T * k, H, pitch, fp8, dev)
    sc = scale_buf()
    L, _, _ = epl.layout_dispatch(cfg, idx_d, x_d, recv=recv, recv_scale=sc)
    torch.cuda.synchronize()
    assert_layout_equal(L, ref, what)
    _check_block(blk, H, P, want_rows, fp8, what + " layout_dispatch")
    if fp8:
        np.testing.assert_array_equal(sc[:P].cpu().numpy().view(np.uint32), want_scale.view(np.uint32))
    # epl_layout_counts + epl_dispatch_rows
    blk2, recv2 = _block(T * k, H, pitch, fp8, dev)
    L2 = epl.layout_counts(cfg, idx_d)
    epl.dispatch_rows(cfg, idx_d, x_d, L2, recv=recv2, recv_scale=scale_buf())
    torch.cuda.synchronize()
    _check_block(blk2, H, P, want_rows, fp8, what + " dispatch_rows")
    # epl_dispatch on the layout of epl_layout
    blk3, recv3 = _block(T * k, H, pitch, fp8, dev)
    epl.dispatch(cfg, x_d, epl.layout(cfg, idx_d), recv=recv3, recv_scale=scale_buf())
    torch.cuda.synchronize()
    _check_block(blk3, H, P, want_rows, fp8, what + " dispatch")
    # epl_layout_dispatch_noalloc
    blk4, recv4 = _block(T * k, H, pitch, fp8, dev)
    L4 = epl.alloc_layout(cfg, dev)
    epl.layout_dispatch_noalloc(cfg, idx_d, x_d, L4, recv4, scale_buf())
    torch.cuda.synchronize()
    _check_block(blk4, H, P, want_rows, fp8, what + " noalloc")
    # epl_dispatch_scheduled
    blk5, recv5 = _block(T * k, H, pitch, fp8, dev)
    sc5 = scale_buf()
    epl.dispatch_scheduled(cfg, x_d, L, workers=5, recv=recv5, recv_scale=sc5)
    torch.cuda.synchronize()
    _check_block(blk5, H, P, want_rows, fp8, what + " dispatch_scheduled")
    if fp8:
        np.testing.assert_array_equal(sc5[:P].cpu().numpy().view(np.uint32), want_scale.view(np.uint32))
    # epl_combine: of the received rows (bf16), and of independent rows with NaN gaps
    gw = W.softmax_gate_weights(seed, T, k)
    w_d = torch.from_numpy(gw).to(dev)
    if not fp8:
        out = epl.combine(cfg, recv, w_d, L)
        torch.cuda.synchronize()
        want = oracle_combine_threaded(x[ref.recv_src] if P else np.zeros((1, H), np.uint16), gw, ref.pair_row)
        np.testing.assert_array_equal(bf16_bits(out[:T]), want, err_msg=what + " combine of the received rows")
    y, yh = _pitched_y(max(P, 1), H, pitch, seed, dev)
    out = epl.combine(cfg, y, w_d, L)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out[:T]), oracle_combine_threaded(yh, gw, ref.pair_row),
                                  err_msg=what + " combine of rows with NaN gaps")


def test_prepared_layer_with_a_pitch():
    """The prepared calls with pitched recv and y: the same rows and output as the plain calls."""
    dev = device()
    R, E, k, Tr, H, pitch = 32, 256, 8, 64, 7168, 7936
    T = R * Tr
    idx, x = _case(R, E, k, Tr, H, 9)
    cfg = epl.config(R, E, k, H, Tr, row_pitch=pitch)
    ref = oracle.layout(R, E, k, Tr, idx)
    gw = W.softmax_gate_weights(9, T, k)
    idx_d, x_d, w_d = torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev), torch.from_numpy(gw).to(dev)
    blk, recv = _block(T * k, H, pitch, False, dev)
    prep = epl.PreparedLayer(cfg, idx_d, [x_d], w_d, epl.alloc_layout(cfg, dev), recv)
    prep.run(0)
    torch.cuda.synchronize()
    _check_block(blk, H, ref.P, oracle.dispatch_bf16(x, ref.pair_row, ref.P), False, "prepared layer")
    want = oracle_combine_threaded(x[ref.recv_src], gw, ref.pair_row)
    np.testing.assert_array_equal(bf16_bits(prep.out[:T]), want)


def test_alloc_recv_gives_the_pitch():
    dev = device()
    for payload, contiguous in (("bf16", False), ("bf16", True), ("fp8", False)):
        cfg = epl.config(4, 16, 2, 256, 128, payload, row_pitch=320)
        try:
            recv, scale = epl.alloc_recv(cfg, dev, contiguous=contiguous)
        except MemoryError:
            continue
        assert recv.shape == (4 * 128 * 2, 256) and recv.stride() == (320, 1)
        assert (scale is not None) == (payload == "fp8")


def test_layer_sentinel_with_a_pitch():
    """Sentinel Polling over pitched rows: the fill covers the gaps, the layer reads only payload
    elements, and leaves the payload elements at the sentinel."""
    dev = device()
    R, E, k, Tr, H, pitch = 16, 128, 8, 128, 2048, 2048 + 768
    T = R * Tr
    idx, x = _case(R, E, k, Tr, H, 6)
    gw = W.softmax_gate_weights(6, T, k)
    cfg = epl.config(R, E, k, H, Tr, row_pitch=pitch)
    recv, _ = epl.alloc_recv(cfg, dev)
    epl.sentinel_fill(recv)
    L, out, status = epl.layer_sentinel(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                        torch.from_numpy(gw).to(dev), recv)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, "layer_sentinel pitch")
    want = oracle_combine_threaded(x[ref.recv_src], gw, ref.pair_row)
    np.testing.assert_array_equal(bf16_bits(out[:T]), want)
    assert bool((recv.view(torch.int16) == -1).all())


def test_decomposed_with_a_pitch():
    dev = device()
    R, E, k, Tr, H, pitch = 64, 256, 8, 40, 1032, 1088
    T = R * Tr
    idx, x = _case(R, E, k, Tr, H, 7)
    cfg = epl.config(R, E, k, H, Tr, row_pitch=pitch)
    blk, recv = _block(T * k, H, pitch, False, dev)
    L, _, _, status = epl.layout_dispatch_decomposed(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                                     recv=recv)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, "decomposed pitch")
    _check_block(blk, H, ref.P, oracle.dispatch_bf16(x, ref.pair_row, ref.P), False, "decomposed")


def test_pitch_mismatch_is_refused_before_any_launch():
    dev = device()
    cfg = epl.config(4, 16, 2, 256, 128, row_pitch=320)
    idx_d = torch.zeros(512, 2, dtype=torch.int32, device=dev)
    x_d = torch.zeros(512, 256, dtype=torch.bfloat16, device=dev)
    dense = torch.zeros(1024, 256, dtype=torch.bfloat16, device=dev)
    with pytest.raises(ValueError):
        epl.layout_dispatch(cfg, idx_d, x_d, recv=dense)
    L = epl.layout(cfg, idx_d)
    with pytest.raises(ValueError):
        epl.combine(cfg, dense, torch.zeros(512, 2, device=dev), L)
    with pytest.raises(epl.EplError):
        epl.layout(epl.config(4, 16, 2, 256, 128, row_pitch=300), idx_d)


def _random_pitched_case(seed):
    rng = np.random.default_rng(9000 + seed)
    fp8 = seed % 3 == 2
    R = int(rng.choice([1, 2, 3, 8, 16, 64]))
    El = int(rng.integers(1, 5))
    E = R * El
    k = int(rng.integers(1, 9))
    Tr = 0 if seed % 6 == 0 else int(rng.integers(1, 300))
    H = 128 * int(rng.integers(1, 40)) if fp8 else 8 * int(rng.integers(1, 300))
    pitch = (H + 63) // 64 * 64 + 64 * int(rng.integers(0, 40))
    return R, E, k, Tr, H, pitch, "fp8" if fp8 else "bf16"


@pytest.mark.parametrize("seed", range(12))
def test_random_shapes_and_pitches(seed):
    """Random shapes (no tokens, a single rank, ragged rows) at random valid pitches: layout and
    dispatch in one call, then combine, against the oracle, with the canary checks."""
    dev = device()
    R, E, k, Tr, H, pitch, payload = _random_pitched_case(seed)
    fp8 = payload == "fp8"
    T = R * Tr
    idx, x = _case(R, E, k, Tr, H, seed)
    cfg = epl.config(R, E, k, H, Tr, payload, row_pitch=pitch)
    ref = oracle.layout(R, E, k, Tr, idx)
    P = ref.P
    rows = max(T * k, 1)
    blk, recv = _block(rows, H, pitch, fp8, dev)
    sc = torch.full((rows, H // 128), float("nan"), device=dev) if fp8 else None
    L, _, _ = epl.layout_dispatch(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev), recv=recv,
                                  recv_scale=sc)
    torch.cuda.synchronize()
    what = "seed %d: R=%d E=%d k=%d Tr=%d H=%d pitch=%d %s" % (seed, R, E, k, Tr, H, pitch, payload)
    assert_layout_equal(L, ref, what)
    if fp8:
        want_rows, want_scale = oracle.dispatch_fp8(x, ref.pair_row, P)
        np.testing.assert_array_equal(sc[:P].cpu().numpy().view(np.uint32), want_scale.view(np.uint32))
    else:
        want_rows = oracle.dispatch_bf16(x, ref.pair_row, P)
    _check_block(blk, H, P, want_rows, fp8, what)
    gw = W.softmax_gate_weights(seed, max(T, 1), k)[:T]
    y, yh = _pitched_y(max(P, 1), H, pitch, seed, dev)
    out = epl.combine(cfg, y, torch.from_numpy(np.ascontiguousarray(gw)).to(dev) if T else
                      torch.zeros(1, k, device=dev), L)
    torch.cuda.synchronize()
    if T:
        np.testing.assert_array_equal(bf16_bits(out[:T]), oracle_combine_threaded(yh, gw, ref.pair_row),
                                      err_msg=what + " combine")
