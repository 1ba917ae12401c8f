"""epl_layout_dispatch_decomposed: layout and dispatch in one launch of count and send workgroups,
against the CPU oracle, bit for bit, over the count/send splits; consecutive calls on one
workspace (every call returns the synchronisation words to zero); and the give-up path, forced
from the host with a published value no workgroup writes and a short wait bound: the launch still
completes, stores no row, reports the give-up in its status word, and the next call is exact."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import assert_layout_equal, bf16_bits, device, to_dev_bf16

pytestmark = pytest.mark.gpu


def _check(R, E, k, Tr, H, seed, count_groups=0, idx=None, L=None, recv=None, what=""):
    dev = device()
    T = R * Tr
    if idx is None:
        idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    cfg = epl.config(R, E, k, H, Tr)
    L, recv, _, status = epl.layout_dispatch_decomposed(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev),
                                                        out=L, recv=recv, count_groups=count_groups)
    torch.cuda.synchronize()
    what = what or "R=%d E=%d k=%d Tr=%d H=%d count_groups=%d" % (R, E, k, Tr, H, count_groups)
    assert int(status.item()) == 0, what + ": a wait gave up"
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, what)
    np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P), err_msg=what)
    return cfg, L, recv


@pytest.mark.parametrize("R,E,k,Tr,H,seed", [
    (4, 16, 2, 128, 256, 0),      # the small workload's shape
    (16, 128, 8, 128, 2048, 1),   # the Qwen3-30B shape
    (64, 256, 8, 40, 1032, 2),    # chunks of 10 tokens, ragged rows
    (32, 256, 8, 130, 520, 3),    # ragged last chunk
    (256, 256, 8, 16, 264, 4),    # one expert per rank
    (2, 4, 5, 300, 64, 5),        # more choices than experts
])
@pytest.mark.parametrize("split", ["default", "one", "three", "more_than_chunks"])
def test_decomposed_matches_oracle(R, E, k, Tr, H, seed, split):
    """Count/send splits: the default (one count workgroup per layout chunk here), one count
    workgroup doing every chunk and scan item, three, and more count workgroups than chunks."""
    cfg = epl.config(R, E, k, H, Tr)
    n_default, grid, cap = epl.decomposed_plan(cfg)
    assert grid <= cap and n_default >= 1
    count_groups = {"default": 0, "one": 1, "three": 3, "more_than_chunks": n_default + 7}[split]
    got, grid, _ = epl.decomposed_plan(cfg, count_groups)
    assert got == (count_groups or n_default) and grid <= cap
    _check(R, E, k, Tr, H, seed, count_groups)


def test_decomposed_decode_size_and_consecutive_calls():
    """The decode layer's shape (8,192 tokens, 256 experts, 64 ranks, H 7168) three times on one
    workspace and one receive buffer, with three routings: every call exact, status 0."""
    dev = device()
    w = W.WORKLOADS["decode_ep64"]
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr)
    L = epl.alloc_layout(cfg, dev)
    recv, _ = epl.alloc_recv(cfg, dev)
    x_d = W.device_normal_bf16((w.T, w.H), seed=5, device=dev)
    for seed in (0, 1, 2):
        idx = W.routing(w, seed)
        _, _, _, status = epl.layout_dispatch_decomposed(cfg, torch.from_numpy(idx).to(dev), x_d, out=L, recv=recv)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
        assert_layout_equal(L, ref, "decode seed %d" % seed)
        src = torch.from_numpy(ref.recv_src.astype(np.int64)).to(dev)
        assert torch.equal(recv[:ref.P].view(torch.int16), x_d[src].view(torch.int16)), "decode seed %d" % seed
    assert not L.workspace[-1024:].any(), "synchronisation words not returned to zero"


def test_decomposed_forced_give_up_then_exact():
    """The send workgroups wait for a value that no workgroup publishes, with a 2 ms bound: the
    launch completes (the host's synchronize returns), no row is stored, the status word has the
    send give-up bit, the synchronisation words are zero again, and the next call is exact."""
    dev = device()
    R, E, k, Tr, H = 16, 128, 8, 128, 2048
    T = R * Tr
    cfg = epl.config(R, E, k, H, Tr)
    idx = W.distinct_uniform(9, np.arange(T), k, E).astype(np.int32)
    idx_d = torch.from_numpy(idx).to(dev)
    x = W.normal_bf16(9, W.STREAM_X, T * H).reshape(T, H)
    x_d = to_dev_bf16(x, dev)
    L = epl.alloc_layout(cfg, dev)
    recv = torch.full((T * k, H), -3.0, dtype=torch.bfloat16, device=dev)  # canary
    _, _, _, status = epl.layout_dispatch_decomposed(cfg, idx_d, x_d, out=L, recv=recv, spin_limit_us=2000,
                                                     test_ready_target=2)
    torch.cuda.synchronize()
    assert int(status.item()) == epl.WAIT_GAVE_UP_SEND
    assert bool((recv.float() == -3.0).all()), "a send workgroup stored rows after giving up"
    assert not L.workspace[-1024:].any()
    _check(R, E, k, Tr, H, 9, idx=idx, L=L, recv=recv, what="after a forced give-up")


def test_decomposed_unsupported():
    dev = device()
    x = torch.zeros(64 * 8, 128, dtype=torch.bfloat16, device=dev)
    idx = torch.zeros(64 * 8, 8, dtype=torch.int32, device=dev)
    for cfg in (epl.config(64, 512, 8, 128, 8), epl.config(64, 256, 8, 128, 8, "fp8")):
        with pytest.raises(epl.EplError) as ei:
            epl.layout_dispatch_decomposed(cfg, idx, x)
        assert ei.value.status == 5
    cfg = epl.config(64, 256, 8, 128, 8)
    _, _, cap = epl.decomposed_plan(cfg)
    with pytest.raises(epl.EplError) as ei:
        epl.layout_dispatch_decomposed(cfg, idx, x, count_groups=cap)  # no room left for send workgroups
    assert ei.value.status == 5
