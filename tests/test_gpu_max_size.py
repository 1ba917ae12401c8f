"""The layer at the index limit: T*k = 2^31 - 256 pairs (8 ranks of 8,388,607 tokens, top-32: just
below the int32 bound the config accepts), with small rows (H = 8) so that it fits in HBM (about
110 GB in all). The oracle cannot run at this size, so the layout, the dispatch and the combine are checked
on the GPU against properties that fix them:
* counts: send_cnt equals a bincount of each source rank's ids, expert_off its prefix sum;
* placement: pair_row is a bijection onto [0, P), recv_src / recv_j invert it, and the packed rows
  run in (expert, token, choice) order;
* dedup: tok_nranks equals the number of distinct destination ranks of each token (sampled);
* payload: every packed row equals its source row, bit for bit;
* combine: identity experts with softmax weights give x back, bit for bit.
Every index the kernels form here exceeds 2^31 when counted in bytes."""
import numpy as np
import pytest
import torch

from paper_2607_06202_amd import epl
from tests.gpu_util import device

pytestmark = pytest.mark.gpu

R, E, k, H = 8, 16, 32, 8
Tr = ((1 << 31) - 1) // (R * k)  # 8,388,607 tokens per rank
T = R * Tr


@pytest.fixture(scope="module")
def big():
    dev = device()
    if torch.cuda.get_device_properties(dev).total_memory < 200 * 2 ** 30:
        pytest.skip("needs about 110 GB of device memory")
    assert T * k < 2 ** 31 and T * k > 2 ** 31 - 512
    g = torch.Generator(device=dev)
    g.manual_seed(2026)
    idx = torch.randint(0, E, (T, k), generator=g, device=dev, dtype=torch.int32)
    x = torch.randn(T, H, generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
    cfg = epl.config(R, E, k, H, Tr, "bf16")
    L, recv, _ = epl.layout_dispatch(cfg, idx, x)
    torch.cuda.synchronize()
    yield cfg, idx, x, L, recv
    del L, recv, idx, x
    torch.cuda.empty_cache()


def test_counts_and_offsets(big):
    cfg, idx, x, L, recv = big
    per_rank = idx.view(R, Tr * k)
    for s in range(R):
        want = torch.bincount(per_rank[s].long(), minlength=E).to(torch.int32)
        assert torch.equal(L.send_cnt[s], want), "send_cnt of rank %d" % s
    recv_cnt = L.send_cnt.sum(0, dtype=torch.int64)
    assert int(recv_cnt.sum()) == T * k and int(L.num_invalid[0]) == 0
    want_off = torch.cat([torch.zeros(1, dtype=torch.int64, device=idx.device), recv_cnt.cumsum(0)])
    assert torch.equal(L.expert_off.long(), want_off)


def test_placement_is_a_sorted_bijection(big):
    cfg, idx, x, L, recv = big
    P = T * k
    rows = L.pair_row.view(-1)
    assert int(rows.min()) == 0 and int(rows.max()) == P - 1
    hit = torch.zeros(P, dtype=torch.int32, device=rows.device)
    hit.scatter_add_(0, rows.long(), torch.ones_like(rows))
    assert bool((hit == 1).all()), "pair_row is not a bijection onto [0, P)"
    del hit
    step = 1 << 28  # check recv_src / recv_j and the row order in slices
    prev_key = None
    for r0 in range(0, P, step):
        r1 = min(P, r0 + step)
        src = L.recv_src[r0:r1].long()
        j = L.recv_j[r0:r1].long()
        pair = src * k + j
        assert torch.equal(rows[pair], torch.arange(r0, r1, device=rows.device, dtype=torch.int32))
        key = idx.view(-1)[pair].long() * (T * k) + pair  # (expert, token, choice)
        assert bool((key[1:] > key[:-1]).all()), "rows out of order in [%d, %d)" % (r0, r1)
        if prev_key is not None:
            assert int(key[0]) > prev_key
        prev_key = int(key[-1])


def test_dedup_sampled(big):
    cfg, idx, x, L, recv = big
    gs = torch.from_numpy(np.random.default_rng(1).integers(0, T, 4096)).to(idx.device)
    ranks = (idx[gs] // (E // R)).cpu().numpy()
    want = np.array([len(set(r)) for r in ranks], np.int32)
    np.testing.assert_array_equal(L.tok_nranks[gs].cpu().numpy(), want)


def test_payload_rows_equal_source_rows(big):
    cfg, idx, x, L, recv = big
    P = T * k
    xv = x.view(torch.int16)
    rv = recv.view(torch.int16)
    step = 1 << 24  # rows per slice: torch's row gather fails to launch from 2^26 rows of this x
    for r0 in range(0, P, step):
        r1 = min(P, r0 + step)
        assert torch.equal(rv[r0:r1], xv[L.recv_src[r0:r1].long()]), "rows [%d, %d)" % (r0, r1)


def test_identity_combine_returns_x(big):
    cfg, idx, x, L, recv = big
    g = torch.Generator(device=idx.device)
    g.manual_seed(7)
    w = torch.empty(T, k, dtype=torch.float32, device=idx.device)
    step = 1 << 24  # tokens per slice of the softmax
    for t0 in range(0, T, step):
        t1 = min(T, t0 + step)
        w[t0:t1] = torch.softmax(torch.randn(t1 - t0, k, generator=g, device=idx.device, dtype=torch.float32), dim=1)
    out = epl.combine(cfg, recv, w, L)
    torch.cuda.synchronize()
    assert torch.equal(out.float(), x.float()), "identity round trip does not give x back"
