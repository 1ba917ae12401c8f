"""epl_layout_dispatch, and its two phases epl_layout_counts + epl_dispatch_rows, against the CPU
oracle: every layout output and the bf16 / fp8 payload, bit for bit. It takes three paths, and every
case asserts which one it exercises:
* 3 launches, the layout's finalize step fused into the bf16 dispatch (at most 256 pairs per
  chunk and 256 experts): ragged last chunks, duplicates, invalid ids, 1 and 2 experts per rank,
  more choices than experts, rows of 1, 2, 4 (ragged) and 5 column chunks, so that a
  workgroup's waves cover four, two, one or parts of two tokens;
* 4 launches, the layout then the dispatch (larger chunks, more experts, fp8);
* 2 launches for small layouts."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import LAYOUT_FIELDS, assert_layout_equal, bf16_bits, device, to_dev_bf16

pytestmark = pytest.mark.gpu


def _run(cfg, idx_d, x_d, phases):
    if not phases:
        return epl.layout_dispatch(cfg, idx_d, x_d)
    L = epl.layout_counts(cfg, idx_d)
    recv, sc = epl.dispatch_rows(cfg, idx_d, x_d, L)
    return L, recv, sc


def _check(R, E, k, Tr, H, payload, seed, idx=None, phases=False):
    dev = device()
    T = R * Tr
    if idx is None:
        idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    cfg = epl.config(R, E, k, H, Tr, payload)
    L, recv, sc = _run(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev), phases)
    torch.cuda.synchronize()
    what = "R=%d E=%d k=%d Tr=%d H=%d %s%s" % (R, E, k, Tr, H, payload, " (two phases)" if phases else "")
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, what)
    if payload == "bf16":
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P),
                                      err_msg=what)
    else:
        q, s = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q, err_msg=what)
        np.testing.assert_array_equal(sc[:ref.P].cpu().numpy().view(np.uint32), s.view(np.uint32), err_msg=what)
    return cfg, L, ref


@pytest.mark.parametrize("R,E,k,Tr,H,seed,launches", [
    (64, 256, 8, 40, 1024, 0, 3),    # chunks of 10 tokens (80 pairs)
    (32, 256, 8, 130, 512, 1, 3),    # chunks of 17 tokens, ragged last chunk
    (128, 256, 4, 50, 2048, 2, 3),   # two experts per rank
    (256, 256, 8, 16, 520, 3, 3),    # one expert per rank
    (2, 4, 5, 2000, 64, 4, 3),       # more choices than experts
    (64, 256, 8, 100, 8, 5, 3),      # 200 pairs per chunk; one 16-byte vector per row
    (16, 64, 8, 1024, 64, 6, 4),     # 512 pairs per chunk
    (8, 1024, 32, 1024, 64, 7, 4),   # k = 32, E = 1024
    (256, 256, 8, 64, 1032, 11, 4),  # the EP=256 chunking: 512 pairs per chunk, ragged last column chunk
    (4, 1024, 32, 300, 1032, 12, 4), # 1024 pairs per chunk, 1024 experts, ragged chunks
    (1024, 1024, 2, 40, 64, 13, 4),  # 1024 ranks of one expert
    (64, 256, 8, 40, 4096, 8, 3),    # 2 column chunks per row: 2 tokens per workgroup
    (32, 256, 8, 130, 6152, 9, 3),   # 4 chunks, the last one ragged (769 vectors per row)
    (64, 256, 8, 40, 10240, 10, 3),  # 5 chunks: a workgroup's waves straddle two tokens
])
@pytest.mark.parametrize("phases", [False, True])
def test_layout_dispatch_bf16(R, E, k, Tr, H, seed, launches, phases):
    cfg, _, _ = _check(R, E, k, Tr, H, "bf16", seed, phases=phases)
    assert epl.layout_dispatch_launches(cfg) == launches


@pytest.mark.parametrize("R,E,k,Tr,H,seed", [(64, 256, 8, 40, 1024, 10), (16, 160, 8, 257, 1152, 11)])
@pytest.mark.parametrize("phases", [False, True])
def test_layout_dispatch_fp8(R, E, k, Tr, H, seed, phases):
    cfg, _, _ = _check(R, E, k, Tr, H, "fp8", seed, phases=phases)
    assert epl.layout_dispatch_launches(cfg) == 4


@pytest.mark.parametrize("phases", [False, True])
def test_layout_dispatch_small_layout(phases):
    cfg, _, _ = _check(4, 16, 2, 128, 256, "bf16", 20, phases=phases)
    assert epl.layout_dispatch_launches(cfg) == 2


@pytest.mark.parametrize("phases", [False, True])
def test_layout_dispatch_all_invalid_and_empty(phases):
    cfg, _, _ = _check(64, 256, 8, 40, 128, "bf16", 30, idx=np.full((64 * 40, 8), -1, np.int32), phases=phases)
    assert epl.layout_dispatch_launches(cfg) == 3
    _check(64, 256, 8, 0, 128, "bf16", 31, idx=np.zeros((0, 8), np.int32), phases=phases)


@pytest.mark.parametrize("name", ["decode_ep64", "skewed_fp8_ep64", "large_ep256", "prefill_ep32"] + W.MODEL_ORDER)
def test_layout_dispatch_matches_separate_calls_at_full_size(name):
    """The named workloads in the benchmark's configuration: the fused call, its two phases and
    epl_layout then epl_dispatch give identical layouts and identical payloads (compared on the
    device)."""
    dev = device()
    w = W.WORKLOADS[name]
    idx_d = torch.from_numpy(W.routing(w)).to(dev)
    x_d = W.device_normal_bf16((w.T, w.H), seed=3, device=dev)
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload)
    L1 = epl.layout(cfg, idx_d)
    r1, s1 = epl.dispatch(cfg, x_d, L1)
    torch.cuda.synchronize()
    P = int(L1.expert_off[-1])
    r1p = r1[:P].clone()
    s1p = None if s1 is None else s1[:P].clone()
    del r1, s1
    for phases in (False, True):
        L2, r2, s2 = _run(cfg, idx_d, x_d, phases)
        torch.cuda.synchronize()
        what = "%s%s" % (name, " (two phases)" if phases else "")
        for n, _ in epl.LayoutBuffers._fields_:
            a, b = getattr(L1, n), getattr(L2, n)
            if n in ("recv_src", "recv_j"):
                a, b = a[:P], b[:P]
            assert torch.equal(a, b), "%s: %s differs" % (what, n)
        assert torch.equal(r1p.view(torch.uint8), r2[:P].view(torch.uint8)), what
        if s1p is not None:
            assert torch.equal(s1p.view(torch.int32), s2[:P].view(torch.int32)), what
        del L2, r2, s2


@pytest.mark.parametrize("seed", range(12))
def test_layout_dispatch_random_shapes(seed):
    """Random shapes through epl_layout_dispatch and its two phases (alternating by seed):
    ranks, experts per rank, k, tokens per rank, hidden sizes of 1 to 5 column chunks with ragged
    tails, bf16 or fp8, with duplicates and invalid ids; every path the call can take appears."""
    rng = np.random.default_rng(1300 + seed)
    R = int(rng.choice([1, 4, 16, 32, 64, 128]))
    El = int(rng.choice([1, 2, 4]))
    E = R * El
    k = int(rng.choice([1, 3, 8, 9]))
    Tr = int(rng.choice([3, 16, 40, 100, 257]))
    while R * Tr * k > 300_000:
        Tr = max(1, Tr // 2)
    payload = "fp8" if seed % 4 == 3 else "bf16"
    H = int(rng.choice([128, 1152, 2176])) if payload == "fp8" else int(rng.choice([8, 1032, 2056, 4104, 9224]))
    while R * Tr * k * H * 2 > 400_000_000:  # keep the host-side comparison small
        Tr = max(1, Tr // 2)
    lo, hi = (-1, E + 1) if seed % 2 else (0, E)
    idx = W.with_replacement(seed, R * Tr, k, lo, hi).astype(np.int32)
    _check(R, E, k, Tr, H, payload, seed, idx=idx, phases=bool(seed % 3 == 1))



def test_fused_row_kernel_with_buffer_loads():
    """An x of 200 MB or more is read through buffer loads, in the fused row kernel as in the
    plain dispatch: 64 ranks of 100 tokens at H = 16,384 (210 MB of x, chunks of 25 tokens, so the
    finalize step is still fused). The layout against the oracle; every packed row against its
    source row, bit for bit."""
    dev = device()
    R, E, k, Tr, H = 64, 256, 8, 100, 16384
    T = R * Tr
    cfg = epl.config(R, E, k, H, Tr)
    assert T * H * 2 >= 200 << 20 and epl.layout_dispatch_launches(cfg) == 3
    idx = W.distinct_uniform(21, np.arange(T), k, E).astype(np.int32)
    idx[::37, 2] = -1
    x_d = W.device_normal_bf16((T, H), seed=21, device=dev)
    for phases in (False, True):
        if phases:
            L = epl.layout_counts(cfg, torch.from_numpy(idx).to(dev))
            recv, _ = epl.dispatch_rows(cfg, torch.from_numpy(idx).to(dev), x_d, L)
        else:
            L, recv, _ = epl.layout_dispatch(cfg, torch.from_numpy(idx).to(dev), x_d)
        torch.cuda.synchronize()
        ref = oracle.layout(R, E, k, Tr, idx)
        assert_layout_equal(L, ref, "fused, buffer loads, phases=%s" % phases)
        src = torch.from_numpy(ref.recv_src.astype(np.int64)).to(dev)
        assert torch.equal(recv[:ref.P].view(torch.int16), x_d[src].view(torch.int16))
        del L, recv


@pytest.mark.parametrize("R,E,k,Tr,H,seed,payload", [
    (64, 256, 8, 40, 1024, 20, "bf16"),   # finalize fused into the row kernel
    (4, 16, 2, 128, 256, 21, "bf16"),     # one-launch layout
    (16, 64, 8, 300, 1032, 22, "bf16"),   # three-launch layout, then the plain dispatch
    (16, 64, 8, 40, 1152, 23, "fp8"),     # fp8: three-launch layout, then the fp8 dispatch
])
def test_prepared_layer_matches_the_plain_calls(R, E, k, Tr, H, seed, payload):
    """PreparedLayer (arguments checked and converted once) issues the same calls as
    epl_layout_dispatch + epl_combine: identical layout, rows and output, for every x it rotates
    through, both as run(i) and as the two phases plus combine."""
    dev = device()
    T = R * Tr
    cfg = epl.config(R, E, k, H, Tr, payload)
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    idx_d = torch.from_numpy(idx).to(dev)
    xs = [to_dev_bf16(W.normal_bf16(seed + i, W.STREAM_X, T * H).reshape(T, H), dev) for i in range(2)]
    w_d = torch.from_numpy(W.softmax_gate_weights(seed, T, k)).to(dev)
    fp8 = payload == "fp8"
    y = torch.from_numpy(W.normal_bf16(seed, W.STREAM_Y, T * k * H).reshape(T * k, H).view(np.int16)).view(
        torch.bfloat16).to(dev) if fp8 else None
    L = epl.alloc_layout(cfg, dev)
    recv, scale = epl.alloc_recv(cfg, dev)
    prep = epl.PreparedLayer(cfg, idx_d, xs, w_d, L, recv, scale, y=y)
    for i, x in enumerate(xs):
        L2, r2, s2 = epl.layout_dispatch(cfg, idx_d, x)
        o2 = epl.combine(cfg, r2 if not fp8 else y, w_d, L2)
        for phases in (False, True):
            if phases:
                prep.layout_counts()
                prep.dispatch_rows(i)
                prep.combine()
            else:
                prep.run(i)
            torch.cuda.synchronize()
            P = int(L2.expert_off[-1].item())
            for name in LAYOUT_FIELDS:
                assert torch.equal(getattr(prep.L, name), getattr(L2, name)), (name, i, phases)
            assert torch.equal(prep.recv[:P].view(torch.uint8), r2[:P].view(torch.uint8)), (i, phases)
            if fp8:
                assert torch.equal(prep.recv_scale[:P].view(torch.int32), s2[:P].view(torch.int32)), (i, phases)
            assert torch.equal(prep.out[:T].view(torch.int16), o2[:T].view(torch.int16)), (i, phases)
