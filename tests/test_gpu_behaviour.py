"""GPU behaviour beyond element parity:
* graph capture and replay;
* bitwise determinism of dispatch and combine;
* no stores past the P packed rows at full size;
* non-default streams;
* combine writing its output over x;
* the receive buffer as one contiguous HIP block;
* the paper's other model shapes: Qwen3-30B (hidden 2048, 128 experts), GLM-4.7 (hidden 5120,
  160 routed experts) and DeepSeek at 128 ranks, from the model-configuration table and the
  end-to-end deployments.

Every comparison is against the CPU oracle or against an eager run of the same HIP path.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import assert_layout_equal, bf16_bits, bf16_ulp_distance, device, to_dev_bf16

pytestmark = pytest.mark.gpu


def _inputs(R, E, k, Tr, H, seed, dev):
    T = R * Tr
    idx = W.distinct_uniform(seed, np.arange(T), k, E).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    gw = W.softmax_gate_weights(seed, T, k)
    return idx, x, gw, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev), torch.from_numpy(gw).to(dev)


@pytest.mark.parametrize("R,E,k,Tr,H,calls", [
    (16, 64, 8, 24, 1024, "separate"),   # one-launch layout, then dispatch, combine
    (64, 256, 8, 40, 1024, "fused"),     # counts, fused row kernel, combine, row location
    (16, 512, 8, 256, 512, "phases"),    # three-launch layout then dispatch, as epl_layout_counts + epl_dispatch_rows
])
def test_graph_capture_replays_match_eager(R, E, k, Tr, H, calls):
    """The calls allocate nothing and issue no memsets, so they can be captured in a graph.
    Replays with eager work in between must match the eager result every time."""
    dev = device()
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 3, dev)
    cfg = epl.config(R, E, k, H, Tr)
    L = epl.alloc_layout(cfg, dev)
    recv, _ = epl.alloc_recv(cfg, dev)
    out = torch.empty(R * Tr, H, dtype=torch.bfloat16, device=dev)
    where = torch.empty(R * Tr * k, dtype=torch.int32, device=dev)

    def layer():
        if calls == "separate":
            epl.layout(cfg, idx_d, out=L)
            epl.dispatch(cfg, x_d, L, recv)
        elif calls == "fused":
            epl.layout_dispatch(cfg, idx_d, x_d, out=L, recv=recv)
        else:
            epl.layout_counts(cfg, idx_d, out=L)
            epl.dispatch_rows(cfg, idx_d, x_d, L, recv)
        epl.combine(cfg, recv, w_d, L, out)
        e, _ = epl.locate_rows(cfg, L, n=R * Tr * k)
        where.copy_(e)

    layer()
    torch.cuda.synchronize()
    want_rows = L.pair_row.clone()
    want_out = out.clone()
    want_where = where.clone()
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        layer()  # warm the capture stream
    torch.cuda.current_stream(dev).wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer()
    for rep in range(4):
        L.pair_row.fill_(-5)
        out.zero_()
        recv.zero_()
        where.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(L.pair_row, want_rows), "replay %d: layout differs" % rep
        assert torch.equal(out.view(torch.int16), want_out.view(torch.int16)), "replay %d: combine differs" % rep
        assert torch.equal(where, want_where), "replay %d: row location differs" % rep
        _ = (x_d.float() * 2).sum()  # unrelated eager work between replays
    ref = oracle.layout(R, E, k, Tr, idx)
    np.testing.assert_array_equal(want_rows.cpu().numpy(), ref.pair_row)


def test_dispatch_and_combine_bitwise_deterministic():
    dev = device()
    w = W.WORKLOADS["skewed_fp8_ep64"]
    R, E, k, Tr, H = w.R, w.E, w.k, 32, w.H
    idx = W.zipf_group_limited(0, R * Tr, E, R, k).astype(np.int32)
    x = W.normal_bf16(2, W.STREAM_X, R * Tr * H).reshape(R * Tr, H)
    gw = W.softmax_gate_weights(2, R * Tr, k)
    idx_d, x_d, w_d = torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev), torch.from_numpy(gw).to(dev)
    for payload in ["bf16", "fp8"]:
        cfg = epl.config(R, E, k, H, Tr, payload)
        L = epl.layout(cfg, idx_d)
        outs = []
        for _ in range(3):
            recv, sc = epl.dispatch(cfg, x_d, L)
            y = recv if payload == "bf16" else torch.ones(recv.shape, dtype=torch.bfloat16, device=dev)
            o = epl.combine(cfg, y, w_d, L)
            torch.cuda.synchronize()
            P = int(L.expert_off[-1])
            outs.append((recv[:P].clone(), None if sc is None else sc[:P].clone(), o.clone()))
        for r, s_, o in outs[1:]:
            assert torch.equal(r.view(torch.uint8), outs[0][0].view(torch.uint8))
            assert s_ is None or torch.equal(s_, outs[0][1])
            assert torch.equal(o.view(torch.int16), outs[0][2].view(torch.int16))


def test_full_size_decode_writes_nothing_past_P():
    dev = device()
    w = W.WORKLOADS["decode_ep64"]
    idx = W.routing(w)
    idx[::97, 3] = -1  # some invalid pairs so that P < T*k
    idx_d = torch.from_numpy(idx).to(dev)
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr)
    L = epl.layout(cfg, idx_d)
    cap = w.T * w.k
    recv = torch.full((cap, w.H), -9.0, dtype=torch.bfloat16, device=dev)
    x_d = W.device_normal_bf16((w.T, w.H), seed=5, device=dev)
    epl.dispatch(cfg, x_d, L, recv)
    torch.cuda.synchronize()
    P = int(L.expert_off[-1])
    assert P == cap - len(idx[::97])
    assert bool((recv[P:].float() == -9.0).all()), "dispatch wrote past the packed rows"
    ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    assert_layout_equal(L, ref, "decode with invalid ids")


def test_side_stream_dispatch_and_combine():
    dev = device()
    R, E, k, Tr, H = 8, 32, 4, 40, 512
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 9, dev)
    cfg = epl.config(R, E, k, H, Tr)
    side = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(side):
        L = epl.layout(cfg, idx_d)
        recv, _ = epl.dispatch(cfg, x_d, L)
        out = epl.combine(cfg, recv, w_d, L)
    side.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    rr = oracle.dispatch_bf16(x, ref.pair_row, ref.P)
    np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), rr)
    np.testing.assert_array_equal(bf16_bits(out), oracle.combine(rr, gw, ref.pair_row))


@pytest.mark.parametrize("fused", [False, True])
def test_combine_output_over_x(fused):
    """epl_combine may write its output over x (dispatch is done with it, on the same stream). With
    identity experts and softmax weights the layer then leaves x's own storage holding x again, and
    the packed rows are untouched."""
    dev = device()
    R, E, k, Tr, H = 64, 256, 8, 24, 1024
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 12, dev)
    cfg = epl.config(R, E, k, H, Tr)
    if fused:
        L, recv, _ = epl.layout_dispatch(cfg, idx_d, x_d)
    else:
        L = epl.layout(cfg, idx_d)
        recv, _ = epl.dispatch(cfg, x_d, L)
    ptr = x_d.data_ptr()
    out = epl.combine(cfg, recv, w_d, L, out=x_d)
    torch.cuda.synchronize()
    assert out.data_ptr() == ptr
    assert torch.equal(x_d.float(), to_dev_bf16(x, dev).float())  # +0 == -0: a -0 input comes back as +0
    ref = oracle.layout(R, E, k, Tr, idx)
    np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P))


@pytest.mark.parametrize("payload", ["bf16", "fp8"])
def test_contiguous_receive_buffer(payload):
    """alloc_recv(contiguous=True): the payload rows live in one HIP block handed to torch. The
    layer on it matches the oracle."""
    dev = device()
    R, E, k, Tr, H = 16, 64, 4, 20, 1024
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 13, dev)
    cfg = epl.config(R, E, k, H, Tr, payload)
    recv, scale = epl.alloc_recv(cfg, dev, contiguous=True)
    assert recv.shape == (R * Tr * k, H) and recv.device == dev and recv.is_contiguous()
    assert recv.dtype == (torch.uint8 if payload == "fp8" else torch.bfloat16)
    L = epl.layout(cfg, idx_d)
    epl.dispatch(cfg, x_d, L, recv, scale)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    if payload == "bf16":
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P))
        out = epl.combine(cfg, recv, w_d, L)
        torch.cuda.synchronize()
        assert torch.equal(out.float(), x_d.float())
    else:
        q, sc = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q)
        np.testing.assert_array_equal(scale[:ref.P].cpu().numpy().view(np.uint32), sc.view(np.uint32))


def test_contiguous_block_lives_as_long_as_its_tensors():
    """torch keeps the HIP block alive while a tensor (or a view of one) uses it, and the block is
    freed once the last one is gone."""
    import gc
    import weakref
    dev = device()
    b = epl._ContiguousBlock(64 << 20, dev)
    t = b.tensor((1 << 15, 1024), torch.bfloat16)
    v = t[7:9]
    alive = weakref.ref(b)
    del b, t
    gc.collect()
    assert alive() is not None, "the block was dropped while a view still uses it"
    v.fill_(3.0)
    torch.cuda.synchronize()
    assert bool((v.float() == 3.0).all())
    del v
    gc.collect()
    assert alive() is None, "the block outlived its tensors"


@pytest.mark.parametrize("name,R,E,H,Tr", [("qwen3_30b_ep16", 16, 128, 2048, 64), ("glm47_ep32", 32, 160, 5120, 16),
                                           ("glm47_ep160", 160, 160, 5120, 4), ("deepseek_ep128", 128, 256, 7168, 16)])
@pytest.mark.parametrize("payload", ["bf16", "fp8"])
def test_other_model_shapes(name, R, E, H, Tr, payload):
    """Shapes of the paper's evaluated deployments, top-8, with uniform routing: Qwen3-30B on 16
    ranks, GLM-4.7's 160 experts on 32 ranks (5 each) or 160 ranks (1 each), and DeepSeek's 256
    experts on 128 ranks (2 each)."""
    dev = device()
    k = 8
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 11, dev)
    cfg = epl.config(R, E, k, H, Tr, payload)
    L = epl.layout(cfg, idx_d)
    recv, sc = epl.dispatch(cfg, x_d, L)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, name)
    if payload == "bf16":
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P))
        y = recv
        yh = bf16_bits(recv[:ref.P])
    else:
        q, s = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q)
        np.testing.assert_array_equal(sc[:ref.P].cpu().numpy().view(np.uint32), s.view(np.uint32))
        yh = W.normal_bf16(12, W.STREAM_Y, ref.P * H).reshape(ref.P, H)
        y = to_dev_bf16(yh, dev)
    out = epl.combine(cfg, y, w_d, L)
    torch.cuda.synchronize()
    want = oracle.combine(yh, gw, ref.pair_row)
    got = bf16_bits(out)
    assert bf16_ulp_distance(got, want).max() <= 1
    assert (got == want).all()


def test_binding_rejects_mismatched_tensors():
    """Tensors that do not match the config are refused on the host, before any launch: a kernel
    would otherwise read or write past them."""
    dev = device()
    R, E, k, Tr, H = 4, 16, 2, 8, 64
    T = R * Tr
    idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, 21, dev)
    cfg = epl.config(R, E, k, H, Tr)
    L = epl.layout(cfg, idx_d)
    bf = dict(dtype=torch.bfloat16, device=dev)
    bad_calls = [
        lambda: epl.layout(cfg, idx_d[:-1]),                                           # T*k - k ids
        lambda: epl.layout(cfg, idx_d, out=epl.alloc_layout(epl.config(R, E, k, H, Tr + 1), dev)),
        lambda: epl.dispatch(cfg, torch.zeros(T - 1, H, **bf), L),                     # too few rows of x
        lambda: epl.dispatch(cfg, torch.zeros(T, H + 8, **bf), L),                     # wrong width
        lambda: epl.dispatch(cfg, x_d, L, torch.empty(T * k, H + 8, **bf)),            # recv width
        lambda: epl.dispatch(cfg, x_d, epl.alloc_layout(epl.config(R, E, k, H, Tr + 1), dev)),
        lambda: epl.combine(cfg, torch.zeros(T * k, H - 8, **bf), w_d, L),             # y width
        lambda: epl.combine(cfg, torch.zeros(T * k, H, **bf), w_d[:-1], L),            # too few weight rows
        lambda: epl.combine(cfg, torch.zeros(T * k, H, **bf), torch.zeros(T, k + 1, device=dev), L),
        lambda: epl.combine(cfg, torch.zeros(T * k, H, **bf), w_d, L, torch.empty(T - 1, H, **bf)),
    ]
    for i, call in enumerate(bad_calls):
        with pytest.raises(ValueError):
            call()
            pytest.fail("call %d was accepted" % i)
    cfg8 = epl.config(R, E, k, 128, Tr, "fp8")
    L8 = epl.layout(cfg8, idx_d)
    x8 = torch.zeros(T, 128, **bf)
    recv8 = torch.empty(T * k, 128, dtype=torch.uint8, device=dev)
    with pytest.raises(ValueError):
        epl.dispatch(cfg8, x8, L8, recv8, torch.empty(T * k - 1, 1, dtype=torch.float32, device=dev))
    torch.cuda.synchronize()
    # the well-formed calls still work after the refusals
    recv, _ = epl.dispatch(cfg, x_d, L)
    out = epl.combine(cfg, recv, w_d, L)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    np.testing.assert_array_equal(bf16_bits(out), oracle.combine(oracle.dispatch_bf16(x, ref.pair_row, ref.P), gw,
                                                                  ref.pair_row))


def test_two_layers_concurrently_on_two_streams():
    """The library keeps no state between calls: two different layers enqueued on two streams at
    once (their kernels may overlap on the GPU) each match the oracle."""
    dev = device()
    specs = [(8, 32, 4, 60, 512, 31), (16, 64, 8, 20, 1024, 32)]
    streams = [torch.cuda.Stream(device=dev) for _ in specs]
    runs = []
    for (R, E, k, Tr, H, seed) in specs:
        idx, x, gw, idx_d, x_d, w_d = _inputs(R, E, k, Tr, H, seed, dev)
        runs.append((R, E, k, Tr, H, idx, x, gw, idx_d, x_d, w_d))
    torch.cuda.synchronize()
    outs = []
    for _ in range(3):  # interleave the enqueues of the two layers
        for (R, E, k, Tr, H, idx, x, gw, idx_d, x_d, w_d), s in zip(runs, streams):
            with torch.cuda.stream(s):
                cfg = epl.config(R, E, k, H, Tr)
                L = epl.layout(cfg, idx_d)
                recv, _ = epl.dispatch(cfg, x_d, L)
                outs.append((cfg, L, recv, epl.combine(cfg, recv, w_d, L)))
    torch.cuda.synchronize()
    for i, (cfg, L, recv, out) in enumerate(outs):
        R, E, k, Tr, H, idx, x, gw = runs[i % 2][:8]
        ref = oracle.layout(R, E, k, Tr, idx)
        assert_layout_equal(L, ref, "stream %d" % (i % 2))
        rr = oracle.dispatch_bf16(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), rr)
        np.testing.assert_array_equal(bf16_bits(out), oracle.combine(rr, gw, ref.pair_row))
