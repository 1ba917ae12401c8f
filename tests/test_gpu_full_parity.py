"""Full-size parity on the benchmark's own call path, element by element.

The benchmark's layer is epl_layout_dispatch (the layout's counts, then the row kernel, with the
finalize step fused in where it applies) into a receive buffer allocated as one physically
contiguous block at the benchmark's row pitch, then epl_combine reading that buffer (identity
experts). These tests run
exactly that sequence, at the named workloads' full sizes, after a first layer with other
routing has left its data in every buffer, and compare with the CPU oracle:
* every layout output;
* every packed payload row: bf16 rows on the device against x[oracle recv_src]; fp8 codes and
  scales against the oracle's quantised rows of every token;
* the complete combine output against the oracle's combine (run on the host over token ranges
  in parallel), on the identity rows and on independent expert rows.
Prefill (15 GB of receive rows) is compared the same way, streamed in token chunks.

Also: the fused row kernel with all four of its pair slots in use (256 pairs per chunk) against
the oracle directly, and the layout of every named workload at seeds 0-9.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import (assert_layout_equal, bf16_bits, device, oracle_combine_threaded,
                            oracle_dispatch_threaded, to_dev_bf16)

pytestmark = pytest.mark.gpu


def _recv(cfg, dev):
    try:
        return epl.alloc_recv(cfg, dev, contiguous=True)
    except (MemoryError, OSError):
        return epl.alloc_recv(cfg, dev)


def _bench_cfg(w):
    """The benchmark's config of a workload: its default (tuned) row pitch included."""
    return epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload, row_pitch=epl.tuned_pitch(w.H, w.payload))


def _pitched_like(cfg, y):
    """y [P, H] copied into rows cfg.pitch apart (the gaps hold NaN patterns)."""
    blk = torch.full((y.shape[0], cfg.pitch), 0x7FC3, dtype=torch.int16, device=y.device).view(torch.bfloat16)
    blk[:, :cfg.hidden].copy_(y)
    return blk[:, :cfg.hidden]


def _bench_layer(cfg, idx_d, x_d, w_d, L, recv, scale, y, out):
    """One step as bench.py issues it: epl_layout_dispatch, then epl_combine."""
    epl.layout_dispatch(cfg, idx_d, x_d, out=L, recv=recv, recv_scale=scale)
    epl.combine(cfg, y, w_d, L, out)


def _rows_equal_on_device(recv, x_d, src, what, slice_rows=1 << 15):
    """recv[r] == x_d[src[r]] for every r, bit for bit, compared in slices on the device."""
    src_d = torch.from_numpy(src.astype(np.int64)).to(recv.device)
    for r0 in range(0, src.size, slice_rows):
        r1 = min(src.size, r0 + slice_rows)
        if not torch.equal(recv[r0:r1].view(torch.int16), x_d[src_d[r0:r1]].view(torch.int16)):
            bad = (recv[r0:r1].view(torch.int16) != x_d[src_d[r0:r1]].view(torch.int16)).any(dim=1)
            first = int(torch.nonzero(bad)[0]) + r0
            raise AssertionError("%s: packed row %d differs from its source token %d" % (what, first, src[first]))


@pytest.mark.parametrize("name", ["decode_ep64", "large_ep256", "skewed_fp8_ep64"])
def test_bench_layer_full_size_every_element(name):
    dev = device()
    w = W.WORKLOADS[name]
    fp8 = w.payload == "fp8"
    cfg = _bench_cfg(w)
    assert cfg.pitch == (w.H if fp8 else w.H + 768)
    x = W.tokens_bf16(w)
    x_d = to_dev_bf16(x, dev)
    gw = W.gate_weights(w)
    w_d = torch.from_numpy(gw).to(dev)
    L = epl.alloc_layout(cfg, dev)
    recv, scale = _recv(cfg, dev)
    out = torch.empty(w.T, w.H, dtype=torch.bfloat16, device=dev)
    y_zero = torch.zeros(epl.recv_rows_cap(cfg), cfg.pitch, dtype=torch.bfloat16, device=dev)[:, :w.H] if fp8 else None
    # a first layer with other routing leaves its rows, metadata and output behind
    idx1 = W.routing(w, 1)
    _bench_layer(cfg, torch.from_numpy(idx1).to(dev), x_d, w_d, L, recv, scale, y_zero if fp8 else recv, out)
    idx = W.routing(w)
    idx_d = torch.from_numpy(idx).to(dev)
    _bench_layer(cfg, idx_d, x_d, w_d, L, recv, scale, y_zero if fp8 else recv, out)
    torch.cuda.synchronize()
    assert epl.layout_dispatch_launches(cfg) == {"decode_ep64": 3, "large_ep256": 4, "skewed_fp8_ep64": 4}[name]

    ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    P = ref.P
    assert_layout_equal(L, ref, name)
    if fp8:
        want_q, want_s = oracle_dispatch_threaded(x, ref.pair_row, P, fp8=True)
        got_q = recv[:P].cpu().numpy()
        bad = np.argwhere(got_q != want_q)
        assert bad.size == 0, "%s: fp8 codes differ at %s" % (name, bad[:5].tolist())
        np.testing.assert_array_equal(scale[:P].cpu().numpy().view(np.uint32), want_s.view(np.uint32))
        assert bool((out.view(torch.int16) == 0).all()), "combine of all-zero expert rows is not +0"
        yh = None
    else:
        _rows_equal_on_device(recv[:P], x_d, ref.recv_src, name)
        # combine of the identity rows, every element against the oracle
        yh = x[ref.recv_src]
        want = oracle_combine_threaded(yh, gw, ref.pair_row)
        np.testing.assert_array_equal(bf16_bits(out), want, err_msg=name + ": combine of the identity rows")
        assert torch.equal(out.float(), x_d.float())  # and that is x back (numerically: -0 == +0)
    # combine of independent expert rows through the same buffers
    y_d = W.device_normal_bf16((P, w.H), seed=11, device=dev)
    epl.combine(cfg, _pitched_like(cfg, y_d), w_d, L, out)
    torch.cuda.synchronize()
    want = oracle_combine_threaded(bf16_bits(y_d), gw, ref.pair_row)
    np.testing.assert_array_equal(bf16_bits(out), want, err_msg=name + ": combine of independent rows")


@pytest.mark.timeout(900)
def test_bench_layer_prefill_streamed():
    """Prefill (131,072 tokens, 1,048,576 packed rows of 14 KiB): the bench's layer, then every
    packed row against its source token on the device, and the combine of the identity rows and of
    independent rows against the oracle for every token, in chunks of 8,192 tokens whose expert
    rows are gathered on the device and copied to the host."""
    dev = device()
    w = W.WORKLOADS["prefill_ep32"]
    cfg = _bench_cfg(w)
    idx = W.routing(w)
    idx_d = torch.from_numpy(idx).to(dev)
    x_d = W.device_normal_bf16((w.T, w.H), seed=1, device=dev)
    gw = W.gate_weights(w)
    w_d = torch.from_numpy(gw).to(dev)
    L = epl.alloc_layout(cfg, dev)
    recv, scale = _recv(cfg, dev)
    out = torch.empty(w.T, w.H, dtype=torch.bfloat16, device=dev)
    _bench_layer(cfg, idx_d, x_d, w_d, L, recv, scale, recv, out)
    torch.cuda.synchronize()
    ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    P = ref.P
    assert_layout_equal(L, ref, "prefill")
    _rows_equal_on_device(recv[:P], x_d, ref.recv_src, "prefill")
    y_d = W.device_normal_bf16((P, w.H), seed=12, device=dev)
    out2 = epl.combine(epl.config(w.R, w.E, w.k, w.H, w.Tr), y_d, w_d, L)  # packed independent rows
    torch.cuda.synchronize()
    chunk = 8192
    for g0 in range(0, w.T, chunk):
        g1 = min(w.T, g0 + chunk)
        pr = ref.pair_row[g0:g1]
        ok = pr >= 0
        rows_d = torch.from_numpy(pr[ok].astype(np.int64)).to(dev)
        local = np.full(pr.shape, -1, np.int32)
        local[ok] = np.arange(int(ok.sum()), dtype=np.int32)  # position in the gathered block
        for y, o, what in ((recv, out, "identity rows"), (y_d, out2, "independent rows")):
            ys = bf16_bits(y[rows_d])
            want = oracle_combine_threaded(ys, gw[g0:g1], local)
            np.testing.assert_array_equal(bf16_bits(o[g0:g1]), want,
                                          err_msg="prefill combine of %s, tokens %d..%d" % (what, g0, g1))
        print("prefill combine: tokens %d..%d match the oracle" % (g0, g1), flush=True)
    del y_d, out2


@pytest.mark.parametrize("R,Tr,H,seed", [(32, 256, 264, 0), (64, 128, 8, 1), (16, 512, 1032, 2)])
def test_fused_row_kernel_with_every_pair_slot_in_use(R, Tr, H, seed):
    """8,192 tokens of top-8 give chunks of 32 tokens, 256 pairs: the fused row kernel's four
    64-pair slots are all in use, as in the decode layer. Layout and every payload row against the
    oracle, with invalid ids and duplicates among the choices."""
    dev = device()
    E, k = 256, 8
    T = R * Tr
    cfg = epl.config(R, E, k, H, Tr)
    assert epl.layout_dispatch_launches(cfg) == 3
    idx = W.distinct_uniform(seed, np.arange(T), k, E).astype(np.int32)
    idx[::13, 3] = -1
    idx[::17, 5] = idx[::17, 1]  # a duplicate id in one token
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    L, recv, _ = epl.layout_dispatch(cfg, torch.from_numpy(idx).to(dev), to_dev_bf16(x, dev))
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    per_chunk = np.bincount(np.arange(T) // 32, minlength=T // 32)
    assert (per_chunk * k == 256).all()
    assert_layout_equal(L, ref, "R=%d Tr=%d" % (R, Tr))
    np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), oracle.dispatch_bf16(x, ref.pair_row, ref.P))


@pytest.mark.parametrize("name", W.WORKLOAD_ORDER)
def test_layout_named_workloads_seeds_0_to_9(name):
    """The layout of each named workload, routing drawn with seeds 0-9, against the oracle: through
    epl_layout, and for the bf16 workloads also through the bench's epl_layout_dispatch (at a
    one-vector hidden size, which leaves the layout unchanged)."""
    dev = device()
    w = W.WORKLOADS[name]
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr, w.payload)
    cfg8 = epl.config(w.R, w.E, w.k, 8, w.Tr, "bf16")
    x8 = torch.zeros(w.T, 8, dtype=torch.bfloat16, device=dev)
    for seed in range(10):
        idx = W.routing(w, seed)
        idx_d = torch.from_numpy(idx).to(dev)
        L = epl.layout(cfg, idx_d)
        L2, _, _ = epl.layout_dispatch(cfg8, idx_d, x8)
        torch.cuda.synchronize()
        ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
        assert_layout_equal(L, ref, "%s seed %d" % (name, seed))
        assert_layout_equal(L2, ref, "%s seed %d (layout_dispatch)" % (name, seed))
        del L, L2
