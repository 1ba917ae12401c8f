"""epl_layer_sentinel: one launch that lays out, dispatches and combines the dispatched rows
(identity experts), with each combine wave waiting for its rows by Sentinel Polling. Against the
CPU oracle, bit for bit: the layout, and the combine of x's rows with the gate weights. The
receive buffer must hold the sentinel everywhere before the call and is left so. A sentinel
collision is forced from the host (an input element equal to the sentinel, with a short wait
bound): the launch completes, reports the collision and the combine give-up, and a refilled
buffer gives an exact layer again."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import assert_layout_equal, bf16_bits, device, oracle_combine_threaded, to_dev_bf16

pytestmark = pytest.mark.gpu


def _all_sentinel(recv):
    return bool((recv.view(torch.int16) == -1).all())  # 0xFFFF


def _layer(R, E, k, Tr, H, seed, idx=None, x=None, L=None, recv=None, count_groups=0, what=""):
    dev = device()
    T = R * Tr
    if idx is None:
        idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    if x is None:
        x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    assert epl.sentinel_find(x) == -1  # the initialisation check
    gw = W.softmax_gate_weights(seed, T, k)
    gw[::7] *= -0.5  # weights that do not sum to one
    cfg = epl.config(R, E, k, H, Tr)
    if recv is None:
        recv = epl.sentinel_fill(torch.empty(T * k, H, dtype=torch.bfloat16, device=dev))
    L, out, status = epl.layer_sentinel(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                        torch.from_numpy(gw).to(dev), recv, layout_out=L, count_groups=count_groups)
    torch.cuda.synchronize()
    what = what or "R=%d E=%d k=%d Tr=%d H=%d" % (R, E, k, Tr, H)
    assert int(status.item()) == 0, "%s: status %d" % (what, int(status.item()))
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, what)
    y = x[ref.recv_src] if ref.P else np.zeros((1, H), np.uint16)
    want = oracle_combine_threaded(np.ascontiguousarray(y), gw, ref.pair_row)
    np.testing.assert_array_equal(bf16_bits(out[:T]), want, err_msg=what)
    assert _all_sentinel(recv), what + ": the consumed rows were not reset to the sentinel"
    return cfg, L, recv


@pytest.mark.parametrize("R,E,k,Tr,H,seed", [
    (4, 16, 2, 128, 256, 0),      # the small workload's shape
    (16, 128, 8, 128, 2048, 1),   # the Qwen3-30B shape
    (64, 256, 8, 40, 1032, 2),    # ragged rows (a last column chunk of one vector)
    (32, 256, 8, 130, 520, 3),    # ragged last chunk
    (2, 4, 5, 300, 64, 4),        # more choices than experts, duplicates
])
def test_layer_sentinel_matches_oracle(R, E, k, Tr, H, seed):
    _layer(R, E, k, Tr, H, seed)


def test_layer_sentinel_consecutive_layers():
    """Three layers through one workspace and one receive buffer, filled once: every layer exact,
    the buffer back to the sentinel after each."""
    dev = device()
    R, E, k, Tr, H = 16, 128, 8, 128, 2048
    recv = epl.sentinel_fill(torch.empty(R * Tr * k, H, dtype=torch.bfloat16, device=dev))
    L = epl.alloc_layout(epl.config(R, E, k, H, Tr), dev)
    for seed in (10, 11, 12):
        _layer(R, E, k, Tr, H, seed, L=L, recv=recv, what="layer seed %d" % seed)


def test_layer_sentinel_decode_shape():
    """The decode layer's routing shape (64 ranks, 256 experts, 8,192 tokens, top-8) at H 7168."""
    w = W.WORKLOADS["decode_ep64"]
    _layer(w.R, w.E, w.k, w.Tr, w.H, 0, idx=W.routing(w), x=W.tokens_bf16(w))


def test_layer_sentinel_collision_is_reported():
    """Token 5's row holds the sentinel in one element. Its dispatched rows never count as arrived
    there: the launch still completes within the 2 ms wait bound, the status word reports the input
    collision and the combine give-up, and after a refill the next layer is exact."""
    dev = device()
    R, E, k, Tr, H = 4, 16, 2, 128, 256
    T = R * Tr
    idx = W.distinct_uniform(21, np.arange(T), k, E).astype(np.int32)
    x = W.normal_bf16(21, W.STREAM_X, T * H).reshape(T, H).copy()
    x[5, 100] = epl.SENTINEL_BF16
    assert epl.sentinel_find(x) == 5 * H + 100
    gw = W.softmax_gate_weights(21, T, k)
    cfg = epl.config(R, E, k, H, Tr)
    recv = epl.sentinel_fill(torch.empty(T * k, H, dtype=torch.bfloat16, device=dev))
    L, out, status = epl.layer_sentinel(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                        torch.from_numpy(gw).to(dev), recv, spin_limit_us=2000)
    torch.cuda.synchronize()
    st = int(status.item())
    assert st & epl.WAIT_SENTINEL_IN_X and st & epl.WAIT_GAVE_UP_COMBINE, st
    assert not st & (epl.WAIT_GAVE_UP_COUNT | epl.WAIT_GAVE_UP_SEND), st
    epl.sentinel_fill(recv)
    x[5, 100] = 0
    _layer(R, E, k, Tr, H, 21, idx=idx, x=x, L=L, recv=recv, what="after a collision")
