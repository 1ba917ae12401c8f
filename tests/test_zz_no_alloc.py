"""epl_layout_dispatch_noalloc (the library's static per-GPU scratch as the layout workspace)
against epl_layout_dispatch with a caller workspace, through the C ABI: every layout output and
every payload row must be identical, on consecutive calls with shrinking inputs, so that a call
finds the previous call's contents in the shared scratch. Also the host-side refusal of a shape
whose workspace exceeds the static array, before any launch."""
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
