"""epl_layer_data_as_flag: the one-launch layer with the combine synchronised per 1 KiB chunk by
Token-Flag Fusion or Data-for-Checksum (the paper's Data-as-Flag variants beside Sentinel
Polling). Against the CPU oracle, bit for bit: the layout, the dispatched rows, and the combine of
x's rows with the gate weights. Consecutive layers reuse one marks buffer and one receive buffer
with new epochs and nothing refilled; the checksum variant also starts from random marks and rows.
A give-up is forced from the host (a ready target the count role never publishes, a short wait
bound): the launch completes, reports it, and the next call is exact."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import assert_layout_equal, bf16_bits, device, oracle_combine_threaded, to_dev_bf16

pytestmark = pytest.mark.gpu

VARIANTS = [pytest.param(epl.DAF_TOKEN_FLAG_FUSION, id="flag"), pytest.param(epl.DAF_DATA_CHECKSUM, id="checksum")]


def _layer(variant, R, E, k, Tr, H, seed, epoch, idx=None, x=None, L=None, recv=None, marks=None, pitch=0, what=""):
    dev = device()
    T = R * Tr
    if idx is None:
        idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)  # duplicates and invalid ids
    if x is None:
        x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    gw = W.softmax_gate_weights(seed, T, k)
    gw[::7] *= -0.5  # weights that do not sum to one
    cfg = epl.config(R, E, k, H, Tr, row_pitch=pitch)
    if recv is None:
        recv, _ = epl.alloc_recv(cfg, dev)
    if marks is None:
        marks = epl.alloc_marks(cfg, dev)
    x_d = to_dev_bf16(x, dev)
    L, out, status = epl.layer_data_as_flag(cfg, torch.from_numpy(idx).to(dev), x_d, torch.from_numpy(gw).to(dev),
                                            recv, marks, variant, epoch, layout_out=L)
    torch.cuda.synchronize()
    what = what or "variant %d R=%d E=%d k=%d Tr=%d H=%d" % (variant, R, E, k, Tr, H)
    assert int(status.item()) == 0, "%s: status %d" % (what, int(status.item()))
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, what)
    if ref.P:
        src = torch.from_numpy(ref.recv_src.astype(np.int64)).to(dev)
        assert torch.equal(recv[:ref.P].view(torch.int16), x_d[src].view(torch.int16)), what + ": dispatched rows"
    y = x[ref.recv_src] if ref.P else np.zeros((1, H), np.uint16)
    want = oracle_combine_threaded(np.ascontiguousarray(y), gw, ref.pair_row)
    np.testing.assert_array_equal(bf16_bits(out[:T]), want, err_msg=what)
    return cfg, L, recv, marks


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("R,E,k,Tr,H,seed", [
    (4, 16, 2, 128, 256, 0),      # the small workload's shape
    (16, 128, 8, 128, 2048, 1),   # the Qwen3-30B shape
    (64, 256, 8, 40, 1032, 2),    # ragged rows (a last column chunk of one vector)
    (32, 256, 8, 130, 520, 3),    # ragged last chunk
    (2, 4, 5, 300, 64, 4),        # more choices than experts, duplicates
    (4, 32, 20, 40, 520, 5),      # top-20: a send wave marks its chunks in two rounds of 64 lanes
])
def test_layer_matches_oracle(variant, R, E, k, Tr, H, seed):
    _layer(variant, R, E, k, Tr, H, seed, epoch=1)


@pytest.mark.parametrize("variant", VARIANTS)
def test_consecutive_layers_on_one_marks_buffer(variant):
    """Three layers through one workspace, one receive buffer and one marks buffer, epochs 1, 2, 3:
    every layer exact, with nothing refilled in between."""
    dev = device()
    R, E, k, Tr, H = 16, 128, 8, 128, 2048
    cfg = epl.config(R, E, k, H, Tr)
    recv, _ = epl.alloc_recv(cfg, dev)
    marks = epl.alloc_marks(cfg, dev)
    L = epl.alloc_layout(cfg, dev)
    for epoch, seed in ((1, 10), (2, 11), (3, 12)):
        _layer(variant, R, E, k, Tr, H, seed, epoch, L=L, recv=recv, marks=marks, what="epoch %d" % epoch)


def test_checksum_from_random_marks_and_rows():
    """Data-for-Checksum accepts a chunk only on a matching hash, so it needs no initialised marks
    or rows: both start random, and a second call with the same inputs and a new epoch is exact
    too (the rows then already hold the right data, the marks the old epoch's hashes)."""
    dev = device()
    R, E, k, Tr, H = 32, 256, 8, 130, 520
    cfg = epl.config(R, E, k, H, Tr)
    recv, _ = epl.alloc_recv(cfg, dev)
    recv.view(torch.int16).random_(-32768, 32767)
    marks = epl.alloc_marks(cfg, dev).random_()
    idx = W.with_replacement(31, R * Tr, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(31, W.STREAM_X, R * Tr * H).reshape(R * Tr, H)
    for epoch in (7, 8):
        _layer(epl.DAF_DATA_CHECKSUM, R, E, k, Tr, H, 31, epoch, idx=idx, x=x, recv=recv, marks=marks,
               what="checksum epoch %d" % epoch)


def test_flag_from_random_rows():
    """Token-Flag Fusion needs zero-filled marks but any receive rows."""
    dev = device()
    R, E, k, Tr, H = 64, 256, 8, 40, 1032
    cfg = epl.config(R, E, k, H, Tr)
    recv, _ = epl.alloc_recv(cfg, dev)
    recv.view(torch.int16).random_(-32768, 32767)
    _layer(epl.DAF_TOKEN_FLAG_FUSION, R, E, k, Tr, H, 32, 1, recv=recv)


@pytest.mark.parametrize("variant", VARIANTS)
def test_decode_shape(variant):
    """The decode layer's routing shape (64 ranks, 256 experts, 8,192 tokens, top-8) at H 7168, with
    the receive rows at the tuned pitch."""
    w = W.WORKLOADS["decode_ep64"]
    _layer(variant, w.R, w.E, w.k, w.Tr, w.H, 0, 1, idx=W.routing(w), x=W.tokens_bf16(w),
           pitch=epl.tuned_pitch(w.H, w.payload))


@pytest.mark.parametrize("variant", VARIANTS)
def test_forced_give_up_then_exact(variant):
    """A ready target the count role never publishes (2) with a 2 ms wait bound: every send and
    combine workgroup gives up, the launch completes and reports it, and the next call, with a new
    epoch, is exact."""
    dev = device()
    R, E, k, Tr, H = 4, 16, 2, 128, 256
    T = R * Tr
    idx = W.distinct_uniform(41, np.arange(T), k, E).astype(np.int32)
    x = W.normal_bf16(41, W.STREAM_X, T * H).reshape(T, H)
    gw = W.softmax_gate_weights(41, T, k)
    cfg = epl.config(R, E, k, H, Tr)
    recv, _ = epl.alloc_recv(cfg, dev)
    marks = epl.alloc_marks(cfg, dev)
    L, _, status = epl.layer_data_as_flag(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                          torch.from_numpy(gw).to(dev), recv, marks, variant, 1,
                                          spin_limit_us=2000, test_ready_target=2)
    torch.cuda.synchronize()
    st = int(status.item())
    assert st & epl.WAIT_GAVE_UP_SEND and st & epl.WAIT_GAVE_UP_COMBINE, st
    _layer(variant, R, E, k, Tr, H, 41, 2, idx=idx, x=x, L=L, recv=recv, marks=marks, what="after a give-up")
