"""The hierarchical token-level schedule on the GPU (Hierarchical Token-level Scheduling: Latency
Homogenization; Hardware-Accelerated Mapper) against the CPU oracle.

* epl_hop_schedule: every slice's first expert and offset and its pairs per hop class, element by
  element against the oracle's schedule, for transposed orders of many shapes (one row, one row
  per worker, more rows than experts), explicit permutations, empty slices (more workers than
  pairs), ranks with no pairs, and the counts of the named workloads' own layouts on a two-tier
  topology of 8-rank nodes. The closed-form case where the transposition meets the per-hop bound
  ceil(V_h / n) exactly is checked as well.
* epl_dispatch_scheduled: the packed rows, bit for bit against the oracle's dispatch (canary-filled
  tail untouched) on random shapes with invalid and duplicate ids and several worker counts, and at
  the decode and EP=256 sizes every packed row against x[recv_src] and against epl_dispatch.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import bf16_bits, device, run_layout, to_dev_bf16

pytestmark = pytest.mark.gpu


def _schedule_both(send, hop, n, NH, rows=0, order=None):
    dev = device()
    R, E = send.shape
    cfg = epl.config(R, E, 1, 64, 1)
    order_d = None if order is None else torch.from_numpy(np.ascontiguousarray(order, np.int32)).to(dev)
    se, so, cnt = epl.hop_schedule(cfg, torch.from_numpy(np.ascontiguousarray(send, np.int32)).to(dev),
                                   torch.from_numpy(np.ascontiguousarray(hop, np.int32)).to(dev), n, NH,
                                   remap_rows=rows, order=order_d)
    torch.cuda.synchronize()
    ref_order = order if order is not None else oracle.transposed_order(E, rows if rows else n)
    want = oracle.hop_schedule(send, ref_order, hop, n, NH)
    got = (se.cpu().numpy(), so.cpu().numpy(), cnt.cpu().numpy())
    return got, want


def _assert_same(got, want, what):
    for g, w, name in zip(got, want, ("start_expert", "start_offset", "class_cnt")):
        if not np.array_equal(g, w):
            bad = np.argwhere(g != w)[:5]
            raise AssertionError("%s %s differs at %s: got %s want %s" % (
                what, name, bad.tolist(), g[tuple(bad.T)].tolist(), w[tuple(bad.T)].tolist()))


@pytest.mark.parametrize("R,El,NH,n,rows,max_cnt", [
    (2, 2, 1, 3, 3, 3), (4, 4, 2, 5, 0, 4), (4, 4, 2, 40, 40, 2), (8, 2, 3, 7, 2, 6), (16, 4, 2, 12, 1, 3),
    (6, 1, 4, 1, 1, 5), (5, 3, 2, 16, 4, 1), (64, 4, 2, 32, 0, 9), (32, 8, 2, 48, 0, 300), (1, 1024, 8, 300, 0, 3),
    (1024, 1, 2, 2, 0, 7), (128, 2, 3, 2000, 5000, 2), (16, 64, 8, 1, 0, 40),
])
def test_schedule_matches_oracle_transposed(R, El, NH, n, rows, max_cnt):
    rng = np.random.default_rng(R * 7 + El * 131 + n)
    E = R * El
    for trial in range(3):
        send = rng.integers(0, max_cnt + 1, size=(R, E)).astype(np.int32)
        send[rng.random((R, E)) < 0.3] = 0
        if trial == 2:
            send[: R // 2] = 0  # ranks with no pairs at all
        hop = rng.integers(-1, NH + 1, size=(R, R)).astype(np.int32)  # some classes outside [0, NH)
        got, want = _schedule_both(send, hop, n, NH, rows=rows)
        _assert_same(got, want, "R=%d El=%d n=%d rows=%d trial %d" % (R, El, n, rows, trial))


@pytest.mark.parametrize("seed", range(4))
def test_schedule_matches_oracle_explicit_order(seed):
    rng = np.random.default_rng(900 + seed)
    R, El, NH, n = [(4, 4, 2, 6), (16, 16, 3, 33), (8, 128, 2, 64), (2, 2, 2, 9)][seed]
    E = R * El
    send = rng.integers(0, 6, size=(R, E)).astype(np.int32)
    hop = rng.integers(0, NH, size=(R, R)).astype(np.int32)
    order = rng.permutation(E).astype(np.int32)
    got, want = _schedule_both(send, hop, n, NH, order=order)
    _assert_same(got, want, "seed %d" % seed)


@pytest.mark.parametrize("name", ["decode_ep64", "skewed_fp8_ep64", "large_ep256", "prefill_ep32"])
@pytest.mark.parametrize("n", [32, 48])
@pytest.mark.parametrize("rows_per", ["worker", "node"])
def test_schedule_on_the_named_layouts(name, n, rows_per):
    """The counts of each named workload's own layout, 8-rank nodes as the two hop classes, the
    transposition with one matrix row per worker or one per node."""
    dev = device()
    w = W.WORKLOADS[name]
    idx = W.routing(w)
    _, L = run_layout(w, idx, dev)
    send = L.send_cnt.cpu().numpy()
    hop = W.node_hop_classes(w.R)
    got, want = _schedule_both(send, hop, n, 2, rows=0 if rows_per == "worker" else w.R // 8)
    _assert_same(got, want, name)
    # every slice holds floor(m/n) or ceil(m/n) pairs, and the classes add up to the rank's pairs
    sizes = got[2].sum(axis=2)
    m = send.sum(axis=1)
    assert np.all((sizes == (m // n)[:, None]) | (sizes == (-(-m // n))[:, None]))


def test_transposition_meets_the_per_hop_bound():
    """64 ranks in 4 nodes of 16, every expert u pairs from every source, 16 workers and a 4-row
    matrix: each slice holds exactly V_h / n pairs of each class."""
    R, E, u, n = 64, 256, 2, 16
    node = np.arange(R) // 16
    hop = (node[:, None] != node[None, :]).astype(np.int32)
    send = np.full((R, E), u, np.int32)
    got, want = _schedule_both(send, hop, n, 2, rows=4)
    _assert_same(got, want, "bound case")
    V = np.array([64 * u, 192 * u])
    assert np.all(got[2] == V // n)


# ---------------------------------------------------------------------- scheduled dispatch
@pytest.mark.parametrize("R,E,k,Tr,H,seed,workers,rows", [
    (4, 16, 2, 128, 256, 0, 4, 0), (3, 9, 5, 37, 264, 1, 7, 3), (8, 64, 8, 20, 7168, 2, 16, 0),
    (2, 2, 32, 9, 1032, 3, 1, 1), (16, 256, 8, 5, 2048, 4, 64, 0), (4, 16, 3, 10, 64, 5, 100, 0),
    (64, 256, 8, 4, 520, 6, 3, 256),
])
def test_dispatch_scheduled_parity(R, E, k, Tr, H, seed, workers, rows):
    dev = device()
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    w = W.Workload("d", R, E, k, Tr, H, "bf16", "-")
    cfg, L = run_layout(w, idx, dev)
    cap = T * k
    recv = torch.full((cap, H), -7.0, dtype=torch.bfloat16, device=dev)  # canary
    epl.dispatch_scheduled(cfg, to_dev_bf16(x, dev), L, workers, remap_rows=rows, recv=recv)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    canary = bf16_bits(torch.tensor([-7.0], dtype=torch.bfloat16))[0]
    want = oracle.dispatch_bf16(x, ref.pair_row, cap, fill=canary)
    np.testing.assert_array_equal(bf16_bits(recv), want)


def test_dispatch_scheduled_empty_and_all_invalid():
    dev = device()
    w = W.Workload("d", 4, 16, 2, 0, 64, "bf16", "-")
    cfg, L = run_layout(w, np.zeros((0, 2), np.int32), dev)
    x = torch.zeros(1, 64, dtype=torch.bfloat16, device=dev)
    epl.dispatch_scheduled(cfg, x, L, 8)  # T = 0: nothing to do
    w = W.Workload("d", 4, 16, 2, 8, 64, "bf16", "-")
    idx = np.full((32, 2), 99, np.int32)
    cfg, L = run_layout(w, idx, dev)
    recv = torch.full((64, 64), 3.0, dtype=torch.bfloat16, device=dev)
    epl.dispatch_scheduled(cfg, torch.ones(32, 64, dtype=torch.bfloat16, device=dev), L, 8, recv=recv)
    torch.cuda.synchronize()
    assert torch.all(recv == 3.0)


@pytest.mark.parametrize("name", ["decode_ep64", "large_ep256"])
def test_dispatch_scheduled_full_size(name):
    """Every packed row equals its source token's row and epl_dispatch's row."""
    dev = device()
    w = W.WORKLOADS[name]
    idx = W.routing(w)
    cfg, L = run_layout(w, idx, dev)
    x = W.device_normal_bf16((w.T, w.H), 3, dev)
    a, _ = epl.dispatch_scheduled(cfg, x, L, 32)
    b, _ = epl.dispatch(cfg, x, L)
    torch.cuda.synchronize()
    P = int(L.expert_off[-1].item())
    src = L.recv_src[:P].long()
    for lo in range(0, P, 1 << 14):
        hi = min(P, lo + (1 << 14))
        assert torch.equal(a[lo:hi].view(torch.int16), x[src[lo:hi]].view(torch.int16)), (name, lo)
        assert torch.equal(a[lo:hi].view(torch.int16), b[lo:hi].view(torch.int16)), (name, lo)


@pytest.mark.parametrize("R,E,k,Tr,H,seed,workers,rows", [
    (4, 16, 3, 24, 256, 0, 4, 0), (64, 256, 8, 4, 7168, 1, 16, 8), (2, 4, 5, 30, 1152, 2, 7, 1),
])
def test_dispatch_scheduled_fp8_parity(R, E, k, Tr, H, seed, workers, rows):
    """fp8 payloads: every packed row's codes and scales, bit for bit against the oracle's quantiser."""
    dev = device()
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    w = W.Workload("d", R, E, k, Tr, H, "fp8", "-")
    cfg, L = run_layout(w, idx, dev)
    recv, scale = epl.dispatch_scheduled(cfg, to_dev_bf16(x, dev), L, workers, remap_rows=rows)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    q, s = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
    np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q)
    np.testing.assert_array_equal(scale[:ref.P].cpu().numpy().view(np.uint32), s.view(np.uint32))


def test_dispatch_scheduled_fp8_full_size_skewed():
    """The skewed fp8 workload: every packed row and scale equal to epl_dispatch's."""
    dev = device()
    w = W.WORKLOADS["skewed_fp8_ep64"]
    cfg, L = run_layout(w, W.routing(w), dev)
    x = W.device_normal_bf16((w.T, w.H), 4, dev)
    a, sa = epl.dispatch_scheduled(cfg, x, L, 64, remap_rows=8)
    b, sb = epl.dispatch(cfg, x, L)
    torch.cuda.synchronize()
    P = int(L.expert_off[-1].item())
    assert torch.equal(a[:P], b[:P]) and torch.equal(sa[:P].view(torch.int32), sb[:P].view(torch.int32))
