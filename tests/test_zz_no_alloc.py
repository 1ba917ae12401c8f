"""epl_layout_dispatch_noalloc (the library's static per-GPU scratch as the layout workspace)
against epl_layout_dispatch with a caller workspace, through the C ABI: every layout output and
every payload row must be identical, on consecutive calls with shrinking inputs, so that a call
finds the previous call's contents in the shared scratch; and the same call captured into a HIP
graph and replayed on new inputs. Also the host-side refusal of a shape whose workspace exceeds the
static array, before any launch."""
import numpy as np
import pytest
import torch

from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import device, to_dev_bf16

pytestmark = pytest.mark.gpu

FIELDS = [n for n, _ in epl.LayoutBuffers._fields_]


def _case(name, R, E, k, Tr, H, payload, seed):
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32) if name == "random" else \
        W.distinct_uniform(seed, np.arange(T), k, E).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    return epl.config(R, E, k, H, Tr, payload), idx, x


def _compare(cfg, idx, x, dev, what):
    idx_d = torch.from_numpy(idx).to(dev)
    x_d = to_dev_bf16(x, dev)
    L_ref, r_ref, s_ref = epl.layout_dispatch(cfg, idx_d, x_d)
    L = epl.alloc_layout(cfg, dev)
    recv, scale = epl.alloc_recv(cfg, dev)
    epl.layout_dispatch_noalloc(cfg, idx_d, x_d, L, recv, scale)
    torch.cuda.synchronize()
    P = int(L_ref.expert_off[-1])
    for n in FIELDS:
        a, b = getattr(L_ref, n), getattr(L, n)
        if n in ("recv_src", "recv_j"):
            a, b = a[:P], b[:P]
        assert torch.equal(a, b), "%s: %s differs" % (what, n)
    assert torch.equal(r_ref[:P].view(torch.uint8), recv[:P].view(torch.uint8)), what + ": payload"
    if s_ref is not None:
        assert torch.equal(s_ref[:P].view(torch.int32), scale[:P].view(torch.int32)), what + ": scales"


def test_noalloc_matches_workspace_call_on_shrinking_inputs():
    dev = device()
    cases = [
        ("decode", 64, 256, 8, 128, 7168, "bf16", 0),   # fused finalize path, 0.41 MiB of scratch
        ("random", 16, 64, 8, 1024, 1152, "fp8", 1),    # four launches, fp8; smaller
        ("random", 8, 32, 5, 300, 264, "bf16", 2),      # smaller again, ragged chunks, invalid ids
        ("tiny", 4, 16, 2, 128, 256, "bf16", 3),        # one-launch layout (scratch unused)
    ]
    sizes = []
    for name, R, E, k, Tr, H, payload, seed in cases:
        cfg, idx, x = _case(name, R, E, k, Tr, H, payload, seed)
        sizes.append(epl.workspace_bytes(cfg))
        _compare(cfg, idx, x, dev, "%s R=%d E=%d k=%d Tr=%d %s" % (name, R, E, k, Tr, payload))
    assert sizes == sorted(sizes, reverse=True) and sizes[0] <= epl.STATIC_SCRATCH_BYTES


def test_noalloc_refuses_a_workspace_beyond_the_static_array():
    """1024 ranks of one expert each, 16 tokens per rank: 12 MiB of workspace > 8 MiB. The call
    returns EPL_ERR_WORKSPACE before launching anything (the outputs keep their fill)."""
    dev = device()
    R = E = 1024
    k, Tr, H = 8, 16, 8
    cfg = epl.config(R, E, k, H, Tr)
    assert epl.workspace_bytes(cfg) > epl.STATIC_SCRATCH_BYTES
    T = R * Tr
    idx_d = torch.zeros(T, k, dtype=torch.int32, device=dev)
    x_d = torch.zeros(T, H, dtype=torch.bfloat16, device=dev)
    L = epl.alloc_layout(cfg, dev)
    L.send_cnt.fill_(-5)
    recv, _ = epl.alloc_recv(cfg, dev)
    with pytest.raises(epl.EplError) as ei:
        epl.layout_dispatch_noalloc(cfg, idx_d, x_d, L, recv)
    assert ei.value.status == 4
    torch.cuda.synchronize()
    assert bool((L.send_cnt == -5).all())


@pytest.mark.parametrize("R,E,k,Tr,H,pitch", [
    (64, 256, 8, 40, 1032, 1088),  # finalize fused into the row kernel, rows a pitch apart
    (8, 512, 4, 512, 264, 0),      # 512 experts: layout K1-K3, then the plain row kernel
])
def test_noalloc_under_graph_capture(R, E, k, Tr, H, pitch):
    """The allocation-free call captured into a HIP graph together with the combine after it (it
    allocates nothing and issues no memset). Three replays, each after new routing, tokens and
    weights are copied into the captured buffers and other eager work has run, each against the
    eager workspace call on the same inputs: every layout output, the packed rows and the combine."""
    dev = device()
    cfg = epl.config(R, E, k, H, Tr, row_pitch=pitch)
    T = R * Tr
    idx_s = torch.zeros(T, k, dtype=torch.int32, device=dev)
    x_s = torch.zeros(T, H, dtype=torch.bfloat16, device=dev)
    w_s = torch.zeros(T, k, dtype=torch.float32, device=dev)
    L = epl.alloc_layout(cfg, dev)
    recv, _ = epl.alloc_recv(cfg, dev)
    out = torch.empty(T, H, dtype=torch.bfloat16, device=dev)

    def step():
        epl.layout_dispatch_noalloc(cfg, idx_s, x_s, L, recv)
        epl.combine(cfg, recv, w_s, L, out)

    side = torch.cuda.Stream(device=dev)  # eager warm-up off the default stream, as capture requires
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        step()  # the first call on the device looks up its scratch array, outside the capture
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for seed in (1, 2, 3):
        idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
        idx_s.copy_(torch.from_numpy(idx))
        x_s.copy_(to_dev_bf16(W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H), dev))
        w_s.copy_(torch.from_numpy(W.softmax_gate_weights(seed, T, k)))
        L_ref, r_ref, _ = epl.layout_dispatch(cfg, idx_s, x_s)
        out_ref = epl.combine(cfg, r_ref, w_s, L_ref)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        P = int(L_ref.expert_off[-1])
        what = "replay %d" % seed
        for n in FIELDS:
            a, b = getattr(L_ref, n), getattr(L, n)
            if n in ("recv_src", "recv_j"):
                a, b = a[:P], b[:P]
            assert torch.equal(a, b), "%s: %s differs" % (what, n)
        assert torch.equal(r_ref[:P].view(torch.int16), recv[:P].view(torch.int16)), what + ": payload"
        assert torch.equal(out_ref[:T].view(torch.int16), out.view(torch.int16)), what + ": combine"
