"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded inputs.

Bar:
* layout, metadata and bf16/fp8 payloads are bit-exact;
* combine is within 1 bf16 ulp, and a separate test also demands bit-exactness, since the
  fold is fixed-order fmaf on both sides.

Sizes:
* Small and medium shapes compare every element. They span several layout chunks and ragged
  tails.
* The five named workloads run at full size in the benchmark's launch configuration. There the
  test compares:
  - the whole layout;
  - sampled payload rows;
  - the identity round trip (dispatch, then identity experts, then combine reproduces x);
  - a sampled combine on independent expert rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from paper_2607_06202_amd import workloads as W
from tests.gpu_util import (assert_layout_equal, bf16_bits, bf16_ulp_distance, device, run_layout, to_dev_bf16)

pytestmark = pytest.mark.gpu


def _random_shape(seed):
    rng = np.random.default_rng(500 + seed)
    R = int(rng.choice([1, 2, 3, 4, 7, 8, 16, 33, 64]))
    El = int(rng.choice([1, 2, 3, 4, 8]))
    El = min(El, epl.MAX_EXPERTS // R)
    k = int(rng.choice([1, 2, 3, 5, 8, 9, 16, 32]))
    Tr = int(rng.choice([0, 1, 3, 17, 64, 100, 129, 300, 1100]))
    if R * Tr * k > 400_000:
        Tr = max(1, 400_000 // (R * k))
    return R, R * El, k, Tr


@pytest.mark.parametrize("seed", range(24))
def test_layout_random_shapes(seed):
    dev = device()
    R, E, k, Tr = _random_shape(seed)
    T = R * Tr
    if seed % 3 == 0:
        idx = W.with_replacement(seed, T, k, -2, E + 2)  # duplicates and invalid ids
    elif seed % 3 == 1 and k <= E:
        idx = W.distinct_uniform(seed, np.arange(T), k, E)
    else:
        idx = W.with_replacement(seed, T, k, 0, max(1, E // 3))  # hot low experts, duplicates
    idx = np.ascontiguousarray(idx, np.int32).reshape(T, k)
    w = W.Workload("rand", R, E, k, Tr, 64, "bf16", "-")
    _, L = run_layout(w, idx, dev)
    torch.cuda.synchronize()
    assert_layout_equal(L, oracle.layout(R, E, k, Tr, idx), "R=%d E=%d k=%d Tr=%d" % (R, E, k, Tr))


def test_layout_chunked_ragged_and_max_experts():
    dev = device()
    cases = [(2, 8, 1, 2500), (3, 12, 3, 700), (8, 1024, 32, 40), (1024, 1024, 2, 3), (5, 1000, 7, 301)]
    for i, (R, E, k, Tr) in enumerate(cases):
        T = R * Tr
        idx = W.with_replacement(100 + i, T, k, -1, E + 1).astype(np.int32)
        w = W.Workload("c", R, E, k, Tr, 64, "bf16", "-")
        _, L = run_layout(w, idx, dev)
        torch.cuda.synchronize()
        assert_layout_equal(L, oracle.layout(R, E, k, Tr, idx), "case %d" % i)


@pytest.mark.parametrize("R,E,k,Tr,launches", [
    (16, 64, 8, 100, 1),    # many chunks per rank, ragged last chunk
    (64, 1024, 8, 32, 1),   # E = 1024
    (4, 64, 32, 100, 1),    # k = 32: fifty 2-token chunks per rank
    (8, 8, 1, 500, 1),      # k = 1
    (32, 256, 8, 64, 1),    # T*k = 16384, the single-launch limit
    (32, 256, 8, 65, 3),    # T*k above the limit
    (64, 256, 8, 300, 3),   # decode-like, three launches
    (2, 16, 8, 1000, 3),    # Tr*k above the limit
    (1024, 1024, 2, 2, 3),  # LDS above the limit
])
@pytest.mark.parametrize("vec_ids", [True, False])
def test_layout_both_launch_paths(R, E, k, Tr, launches, vec_ids):
    """The one-launch and three-launch layouts against the oracle. The ids sit at a 16-byte
    aligned address (vector loads in the one-launch pass) or 4 bytes past one (scalar loads)."""
    dev = device()
    cfg = epl.config(R, E, k, 64, Tr)
    assert epl.layout_launches(cfg) == launches
    T = R * Tr
    idx = W.with_replacement(700 + R + k, T, k, -1, E + 1).astype(np.int32)  # duplicates and invalid ids
    buf = torch.zeros(T * k + 1, dtype=torch.int32, device=dev)
    off = 0 if vec_ids else 1
    idx_d = buf[off:off + T * k].view(T, k)
    idx_d.copy_(torch.from_numpy(idx))
    assert idx_d.data_ptr() % 16 == (0 if vec_ids else 4)
    L = epl.layout(cfg, idx_d)
    torch.cuda.synchronize()
    assert_layout_equal(L, oracle.layout(R, E, k, Tr, idx), "R=%d E=%d k=%d Tr=%d" % (R, E, k, Tr))


@pytest.mark.parametrize("R,Tr", [(1, 16384), (2, 8192)])
def test_every_pair_to_one_expert_per_rank(R, Tr):
    """k copies of one expert per token, on one expert per rank (E = R), the layout the replicate
    calibration uses: pair (g, j) of rank s lands in row s*Tr*k + (g - s*Tr)*k + j, i.e. each
    token's k rows are contiguous and the rows are sequential, for every rank's own tokens. The
    layout equals the oracle's and that closed form; the payload is x repeated k times."""
    dev = device()
    k, H = 8, 64
    T = R * Tr
    idx = np.repeat(np.arange(T) // Tr, k).reshape(T, k).astype(np.int32)  # token of rank s -> expert s
    w = W.Workload("one", R, R, k, Tr, H, "bf16", "-")
    cfg, L = run_layout(w, idx, dev)
    x = W.normal_bf16(7, W.STREAM_X, T * H).reshape(T, H)
    recv, _ = epl.dispatch(cfg, to_dev_bf16(x, dev), L)
    torch.cuda.synchronize()
    ref = oracle.layout(R, R, k, Tr, idx)
    assert_layout_equal(L, ref, "one expert per rank, R=%d" % R)
    np.testing.assert_array_equal(ref.pair_row.reshape(-1), np.arange(T * k))
    np.testing.assert_array_equal(bf16_bits(recv[:T * k]), np.repeat(x, k, axis=0))


def test_layout_empty_and_all_invalid():
    dev = device()
    w = W.Workload("empty", 4, 8, 3, 0, 64, "bf16", "-")
    idx = np.zeros((0, 3), np.int32)
    cfg, L = run_layout(w, idx, dev)
    x = torch.zeros(1, 64, dtype=torch.bfloat16, device=dev)
    recv, _ = epl.dispatch(cfg, x, L)
    out = epl.combine(cfg, recv, torch.zeros(1, 3, device=dev), L)
    torch.cuda.synchronize()
    assert_layout_equal(L, oracle.layout(4, 8, 3, 0, idx), "empty")
    w = W.Workload("inv", 2, 4, 2, 5, 64, "bf16", "-")
    idx = np.where(np.arange(20).reshape(10, 2) % 2 == 0, -1, 4).astype(np.int32)
    cfg, L = run_layout(w, idx, dev)
    x = to_dev_bf16(W.normal_bf16(1, 1, 10 * 64).reshape(10, 64), dev)
    recv, _ = epl.dispatch(cfg, x, L)
    out = epl.combine(cfg, recv, torch.ones(10, 2, device=dev), L)
    torch.cuda.synchronize()
    ref = oracle.layout(2, 4, 2, 5, idx)
    assert_layout_equal(L, ref, "all invalid")
    assert ref.num_invalid == 20
    assert (out.float() == 0).all() and not torch.signbit(out.float()).any()  # +0 for tokens without pairs


@pytest.mark.parametrize("name", W.WORKLOAD_ORDER + W.MODEL_ORDER)
def test_layout_named_full_size(name):
    dev = device()
    w = W.WORKLOADS[name]
    idx = W.routing(w)
    _, L = run_layout(w, idx, dev)
    torch.cuda.synchronize()
    assert_layout_equal(L, oracle.layout(w.R, w.E, w.k, w.Tr, idx), name)


# ---------------------------------------------------------------------- dispatch
@pytest.mark.parametrize("R,E,k,Tr,H,seed", [(4, 16, 2, 128, 256, 0), (3, 9, 5, 37, 264, 1), (8, 64, 8, 20, 7168, 2),
                                             (2, 2, 32, 9, 1032, 3), (16, 256, 8, 5, 2048, 4)])
def test_dispatch_bf16_parity(R, E, k, Tr, H, seed):
    dev = device()
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    w = W.Workload("d", R, E, k, Tr, H, "bf16", "-")
    cfg, L = run_layout(w, idx, dev)
    cap = T * k
    recv = torch.full((cap, H), -7.0, dtype=torch.bfloat16, device=dev)  # canary
    epl.dispatch(cfg, to_dev_bf16(x, dev), L, recv)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    canary = bf16_bits(torch.tensor([-7.0], dtype=torch.bfloat16))[0]
    want = oracle.dispatch_bf16(x, ref.pair_row, cap, fill=canary)
    np.testing.assert_array_equal(bf16_bits(recv), want)


def _adversarial_rows(H, n_rows, seed):
    """bf16 rows that sweep every finite bf16 pattern through the quantiser at many scales,
    plus zero blocks, single-spike blocks and subnormal-heavy blocks."""
    rng = np.random.default_rng(seed)
    pats = np.arange(1 << 16, dtype=np.uint32)
    exp = (pats >> 7) & 0xFF
    pats = pats[exp != 0xFF].astype(np.uint16)  # drop Inf/NaN
    rows = []
    for r in range(n_rows):
        row = pats[rng.integers(0, pats.size, H)]
        nb = H // 128
        kind = r % 6
        if kind == 1:
            row[: H // 2] = 0  # zero blocks
        if kind == 2:
            row = np.where(rng.random(H) < 0.9, np.uint16(0), row).astype(np.uint16)
        if kind == 3:  # spike per block makes every other value tiny relative to s
            row = (rng.integers(0, 0x80, H)).astype(np.uint16)  # bf16 subnormals
        if kind == 4:  # exact powers of two scale: amax = 448 * 2^m
            m = rng.integers(-30, 30, nb)
            f = oracle.bf16_to_f32(row).reshape(nb, 128).copy()
            f[:, 0] = np.float32(448.0) * (2.0 ** m).astype(np.float32)
            row = W.f32_to_bf16_bits(f.reshape(-1))
        rows.append(row.astype(np.uint16))
    return np.stack(rows)


@pytest.mark.parametrize("R,E,k,Tr,H,seed", [(4, 16, 3, 24, 256, 0), (64, 256, 8, 4, 7168, 1), (2, 4, 5, 30, 1152, 2)])
def test_dispatch_fp8_parity(R, E, k, Tr, H, seed):
    dev = device()
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    x[: min(T, 24)] = _adversarial_rows(H, min(T, 24), seed)
    w = W.Workload("f", R, E, k, Tr, H, "fp8", "-")
    cfg, L = run_layout(w, idx, dev)
    cap = T * k
    recv = torch.full((cap, H), 0xA5, dtype=torch.uint8, device=dev)
    scale = torch.full((cap, H // 128), -3.0, dtype=torch.float32, device=dev)
    epl.dispatch(cfg, to_dev_bf16(x, dev), L, recv, scale)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    want_q, want_s = oracle.dispatch_fp8(x, ref.pair_row, cap, fill=0xA5)
    want_s[ref.P:] = -3.0
    got_q = recv.cpu().numpy()
    bad = np.argwhere(got_q != want_q)
    assert bad.size == 0, "fp8 codes differ at %s: got %s want %s" % (
        bad[:5].tolist(), got_q[tuple(bad[:5].T)], want_q[tuple(bad[:5].T)])
    np.testing.assert_array_equal(scale.cpu().numpy().view(np.uint32), want_s.view(np.uint32))


def _special_rows(H, n, seed):
    """Rows whose 128-element blocks hold non-finite and extreme bf16 values: a NaN among normal
    values, +Inf, -Inf with a NaN, only zeros of both signs, only subnormals, the largest finite
    magnitude, only NaNs, and a lone tiny value."""
    rng = np.random.default_rng(seed)
    nan, pinf, ninf = 0x7FC1, 0x7F80, 0xFF80
    rows = W.normal_bf16(seed, W.STREAM_X, n * H).reshape(n, H).copy()
    for r in range(n):
        blocks = rows[r].reshape(-1, 128)
        for b in range(blocks.shape[0]):
            kind = (b + r) % 8
            blk = blocks[b]
            if kind == 0:
                blk[rng.integers(0, 128)] = nan | (0x8000 if r % 2 else 0)
            elif kind == 1:
                blk[rng.integers(0, 128)] = pinf
            elif kind == 2:
                blk[rng.integers(0, 128)] = ninf
                blk[rng.integers(0, 128)] = nan
            elif kind == 3:
                blk[:] = np.where(rng.random(128) < 0.5, 0x0000, 0x8000)
            elif kind == 4:
                blk[:] = rng.integers(1, 0x80, 128) | np.where(rng.random(128) < 0.5, 0, 0x8000)
            elif kind == 5:
                blk[rng.integers(0, 128)] = 0x7F7F  # largest finite bf16
            elif kind == 6:
                blk[:] = nan | np.where(rng.random(128) < 0.5, 0, 0x8000)
            else:
                blk[:] = 0
                blk[rng.integers(0, 128)] = 0x0001  # smallest subnormal
    return rows.astype(np.uint16)


@pytest.mark.parametrize("H", [1024, 1152])
def test_dispatch_fp8_special_values(H):
    """The quantiser on NaN, infinities, signed zeros, subnormals and the largest magnitude,
    against the oracle. A block's amax ignores NaNs (so an all-NaN block gets s = 0, q = 0). With
    an infinite amax the scale is +Inf; finite values then quantise to signed zeros and an
    infinite value's quotient Inf/Inf is a NaN whose sign IEEE 754 leaves open, so for those
    elements only the NaN code (low 7 bits 0x7F) is compared. Everything else is bit-exact."""
    dev = device()
    R, E, k, Tr = 2, 4, 3, 8
    T = R * Tr
    idx = W.with_replacement(11, T, k, 0, E).astype(np.int32)
    x = _special_rows(H, T, 5)
    w = W.Workload("sv", R, E, k, Tr, H, "fp8", "-")
    cfg, L = run_layout(w, idx, dev)
    recv, scale = epl.dispatch(cfg, to_dev_bf16(x, dev), L)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    want_q, want_s = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
    got_q, got_s = recv[:ref.P].cpu().numpy(), scale[:ref.P].cpu().numpy()
    np.testing.assert_array_equal(got_s.view(np.uint32), want_s.view(np.uint32))
    src = ref.recv_src
    xi = x[src]  # the source row of every packed row
    inf_quot = ((xi & 0x7FFF) == 0x7F80) & np.repeat(np.isinf(want_s), 128, axis=1)
    exact = ~inf_quot
    np.testing.assert_array_equal(got_q[exact], want_q[exact])
    assert ((got_q[inf_quot] & 0x7F) == 0x7F).all() and ((want_q[inf_quot] & 0x7F) == 0x7F).all()
    assert inf_quot.any() and np.isnan(oracle.bf16_to_f32(xi)).any()  # the cases are really there


# ---------------------------------------------------------------------- combine
@pytest.mark.parametrize("R,E,k,Tr,H,seed", [(4, 16, 2, 128, 256, 0), (3, 9, 5, 37, 264, 1), (8, 64, 8, 20, 7168, 2),
                                             (2, 2, 32, 9, 1032, 3), (16, 256, 9, 5, 520, 4)])
def test_combine_parity(R, E, k, Tr, H, seed):
    dev = device()
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    gw = W.softmax_gate_weights(seed, T, k)
    gw[::7] *= -1.5  # signs and weights that do not sum to one
    w = W.Workload("c", R, E, k, Tr, H, "bf16", "-")
    cfg, L = run_layout(w, idx, dev)
    ref = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(seed, W.STREAM_Y, max(ref.P, 1) * H).reshape(-1, H)
    out = epl.combine(cfg, to_dev_bf16(y, dev), torch.from_numpy(gw).to(dev), L)
    torch.cuda.synchronize()
    want = oracle.combine(y, gw, ref.pair_row)
    got = bf16_bits(out)
    d = bf16_ulp_distance(got, want)
    assert d.max() <= 1, "combine off by %d ulp" % d.max()
    assert (got == want).all(), "combine within 1 ulp but %d elements not bit-exact" % (got != want).sum()


def test_combine_special_values():
    """Combine on expert rows with NaNs, infinities, signed zeros, subnormals and magnitudes whose
    weighted sum overflows fp32 or rounds past the largest bf16, with zero, negative and
    subnormal weights, against the oracle. Finite and infinite outputs are bit-exact; where the
    output is a NaN only NaN-ness is compared, since IEEE 754 fixes no payload or sign for the
    NaN an operation returns."""
    dev = device()
    R, E, k, Tr, H = 2, 8, 6, 64, 264
    T = R * Tr
    idx = W.with_replacement(21, T, k, -1, E + 1).astype(np.int32)
    w = W.Workload("cs", R, E, k, Tr, H, "bf16", "-")
    cfg, L = run_layout(w, idx, dev)
    ref = oracle.layout(R, E, k, Tr, idx)
    rng = np.random.default_rng(21)
    y = W.normal_bf16(21, W.STREAM_Y, ref.P * H).reshape(ref.P, H).copy()
    pick = rng.random(y.shape)
    specials = np.array([0x7FC1, 0xFFC3, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x0001, 0x807F, 0x7F7F, 0xFF7F, 0x7F00],
                        np.uint16)
    y = np.where(pick < 0.15, specials[rng.integers(0, specials.size, y.shape)], y).astype(np.uint16)
    gw = W.softmax_gate_weights(21, T, k)
    gw[::5] = 0.0
    gw[1::7] *= -3.0
    gw[2::11] = np.float32(1e-40)  # subnormal weight
    gw[3::13] = np.float32(3.0)    # large weights push sums of big rows past the fp32 range
    out = epl.combine(cfg, to_dev_bf16(y, dev), torch.from_numpy(gw).to(dev), L)
    torch.cuda.synchronize()
    want = oracle.combine(y, gw, ref.pair_row)
    got = bf16_bits(out)
    nan_w = np.isnan(oracle.bf16_to_f32(want))
    nan_g = np.isnan(oracle.bf16_to_f32(got))
    np.testing.assert_array_equal(nan_g, nan_w)
    np.testing.assert_array_equal(got[~nan_w], want[~nan_w])
    f = oracle.bf16_to_f32(want)
    assert nan_w.any() and np.isinf(f).any() and (want == 0x8000).any()  # the cases are really there


# ---------------------------------------------------------------------- randomised whole layers
@pytest.mark.parametrize("seed", range(16))
def test_random_layer_parity(seed):
    """Random shapes, payloads and routings (duplicates, invalid ids, hot experts) through the whole
    layer: layout, dispatch (bf16 or fp8) and combine, each compared element by element."""
    dev = device()
    rng = np.random.default_rng(900 + seed)
    R = int(rng.choice([1, 2, 5, 8, 16, 64]))
    El = int(rng.choice([1, 2, 3, 4]))
    E = R * El
    k = int(rng.choice([1, 2, 4, 6, 8, 13]))
    Tr = int(rng.choice([1, 7, 33, 100]))
    payload = "fp8" if seed % 2 else "bf16"
    H = int(rng.choice([128, 384, 1024, 2176])) if payload == "fp8" else int(rng.choice([8, 264, 1032, 2048]))
    T = R * Tr
    lo, hi = (-1, E + 1) if seed % 3 else (0, max(1, E // 4))
    idx = W.with_replacement(seed, T, k, lo, hi).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    gw = W.softmax_gate_weights(seed, T, k)
    w = W.Workload("r", R, E, k, Tr, H, payload, "-")
    cfg, L = run_layout(w, idx, dev)
    ref = oracle.layout(R, E, k, Tr, idx)
    recv, scale = epl.dispatch(cfg, to_dev_bf16(x, dev), L)
    torch.cuda.synchronize()
    what = "seed %d: R=%d E=%d k=%d Tr=%d H=%d %s" % (seed, R, E, k, Tr, H, payload)
    assert_layout_equal(L, ref, what)
    if payload == "bf16":
        yh = oracle.dispatch_bf16(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), yh, err_msg=what)
        y = recv
    else:
        q, sc = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q, err_msg=what)
        np.testing.assert_array_equal(scale[:ref.P].cpu().numpy().view(np.uint32), sc.view(np.uint32), err_msg=what)
        yh = W.normal_bf16(seed, W.STREAM_Y, max(ref.P, 1) * H).reshape(-1, H)
        y = to_dev_bf16(yh, dev)
    out = epl.combine(cfg, y, torch.from_numpy(gw).to(dev), L)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out), oracle.combine(yh, gw, ref.pair_row), err_msg=what)


# ---------------------------------------------------------------------- extreme hidden sizes
@pytest.mark.parametrize("H,payload", [(8, "bf16"), (128, "fp8"), (1 << 20, "bf16"), (1 << 20, "fp8")])
def test_extreme_hidden_sizes(H, payload):
    """The smallest hidden size of each payload (one 16-byte vector per bf16 row, one 128-element
    block per fp8 row) and EPL_MAX_HIDDEN. Dispatch and combine compared element by element."""
    dev = device()
    R, E, k, Tr, seed = 2, 4, 3, 3, 7
    T = R * Tr
    idx = W.with_replacement(seed, T, k, -1, E + 1).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    if payload == "fp8":
        x[:2] = _adversarial_rows(H, 2, seed)
    gw = W.softmax_gate_weights(seed, T, k)
    w = W.Workload("h", R, E, k, Tr, H, payload, "-")
    cfg, L = run_layout(w, idx, dev)
    ref = oracle.layout(R, E, k, Tr, idx)
    recv, scale = epl.dispatch(cfg, to_dev_bf16(x, dev), L)
    torch.cuda.synchronize()
    if payload == "bf16":
        rr = oracle.dispatch_bf16(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(bf16_bits(recv[:ref.P]), rr)
        y, yh = recv, rr
    else:
        q, sc = oracle.dispatch_fp8(x, ref.pair_row, ref.P)
        np.testing.assert_array_equal(recv[:ref.P].cpu().numpy(), q)
        np.testing.assert_array_equal(scale[:ref.P].cpu().numpy().view(np.uint32), sc.view(np.uint32))
        yh = W.normal_bf16(seed, W.STREAM_Y, max(ref.P, 1) * H).reshape(-1, H)
        y = to_dev_bf16(yh, dev)
    out = epl.combine(cfg, y, torch.from_numpy(gw).to(dev), L)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bf16_bits(out), oracle.combine(yh, gw, ref.pair_row))


# ---------------------------------------------------------------------- full-size named workloads
def _full_inputs(w, dev):
    idx = W.routing(w)
    if w.T * w.H > 200_000_000:
        x_d = W.device_normal_bf16((w.T, w.H), seed=1, device=dev)
    else:
        x_d = to_dev_bf16(W.tokens_bf16(w), dev)
    gw = W.gate_weights(w)
    return idx, x_d, gw


@pytest.mark.parametrize("name", ["tiny", "decode_ep64", "prefill_ep32", "large_ep256"] + W.MODEL_ORDER)
def test_bf16_full_size_round_trip_and_samples(name):
    dev = device()
    w = W.WORKLOADS[name]
    idx, x_d, gw = _full_inputs(w, dev)
    cfg, L = run_layout(w, idx, dev)
    recv, _ = epl.dispatch(cfg, x_d, L)
    out = epl.combine(cfg, recv, torch.from_numpy(gw).to(dev), L)  # identity experts
    torch.cuda.synchronize()
    ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    assert_layout_equal(L, ref, name)
    # invariant: identity experts + softmax weights give x back, bitwise (+0 == -0)
    assert torch.equal(out.float(), x_d.float()), name + ": identity round trip does not reproduce x"
    # sampled payload rows against their source rows
    rng = np.random.default_rng(0)
    rows = rng.integers(0, ref.P, size=min(ref.P, 4096))
    src = torch.from_numpy(ref.recv_src[rows].astype(np.int64)).to(dev)
    rr = torch.from_numpy(rows.astype(np.int64)).to(dev)
    assert torch.equal(recv[rr].view(torch.int16), x_d[src].view(torch.int16)), name + ": dispatch rows differ"
    # sampled combine on independent expert rows (device-drawn y), oracle on the needed rows
    y = W.device_normal_bf16((ref.P, w.H), seed=7, device=dev)
    out2 = epl.combine(cfg, y, torch.from_numpy(gw).to(dev), L)
    toks = rng.integers(0, w.T, size=min(w.T, 256))
    need = np.unique(ref.pair_row[toks][ref.pair_row[toks] >= 0])
    row_map = np.full(ref.P, -1, np.int32)
    row_map[need] = np.arange(need.size)
    ys = bf16_bits(y[torch.from_numpy(need.astype(np.int64)).to(dev)])
    want = oracle.combine_mapped(ys, row_map, gw, ref.pair_row, toks)
    got = bf16_bits(out2[torch.from_numpy(toks).to(dev)])
    assert bf16_ulp_distance(got, want).max() <= 1
    assert (got == want).all(), name + ": sampled combine not bit-exact"


def test_wide_combine_large_k_and_ragged_chunk():
    """The wide combine form (2 KiB column chunks, taken from 4 GiB of expert rows) with k = 13,
    so the choices are folded in two groups of gathers, and H = 20,488, so the last column chunk
    holds a single vector: 8 ranks of 1,024 tokens give T*k*H*2 = 4.36 GB. Sampled tokens (the
    first and last among them) against the oracle, on the dispatched rows and on independent
    expert rows."""
    dev = device()
    R, E, k, Tr, H = 8, 64, 13, 1024, 20488
    T = R * Tr
    assert T * k * H * 2 >= 4 << 30 and (H // 8) % 128 == 1
    idx = W.distinct_uniform(5, np.arange(T), k, E).astype(np.int32)
    idx[::101, 4] = -1  # a few invalid pairs
    x_d = W.device_normal_bf16((T, H), seed=3, device=dev)
    gw = W.softmax_gate_weights(5, T, k)
    cfg = epl.config(R, E, k, H, Tr)
    idx_d = torch.from_numpy(idx).to(dev)
    L, recv, _ = epl.layout_dispatch(cfg, idx_d, x_d)
    w_d = torch.from_numpy(gw).to(dev)
    out = epl.combine(cfg, recv, w_d, L)
    torch.cuda.synchronize()
    ref = oracle.layout(R, E, k, Tr, idx)
    assert_layout_equal(L, ref, "wide combine case")
    # the dispatched rows as expert outputs (tokens with an invalid pair do not get x back)
    rng = np.random.default_rng(3)
    toks = np.unique(np.concatenate([rng.integers(0, T, 96), [0, T - 1]]))
    need = np.unique(ref.pair_row[toks][ref.pair_row[toks] >= 0])
    row_map = np.full(ref.P, -1, np.int32)
    row_map[need] = np.arange(need.size)
    sel = torch.from_numpy(need.astype(np.int64)).to(dev)
    want = oracle.combine_mapped(bf16_bits(recv[sel]), row_map, gw, ref.pair_row, toks)
    got = bf16_bits(out[torch.from_numpy(toks).to(dev)])
    np.testing.assert_array_equal(got, want)
    # independent expert rows
    y = W.device_normal_bf16((ref.P, H), seed=8, device=dev)
    out2 = epl.combine(cfg, y, w_d, L)
    torch.cuda.synchronize()
    want2 = oracle.combine_mapped(bf16_bits(y[sel]), row_map, gw, ref.pair_row, toks)
    np.testing.assert_array_equal(bf16_bits(out2[torch.from_numpy(toks).to(dev)]), want2)


def test_fp8_full_size_skewed():
    dev = device()
    w = W.WORKLOADS["skewed_fp8_ep64"]
    idx, x_d, gw = _full_inputs(w, dev)
    x = bf16_bits(x_d)
    cfg, L = run_layout(w, idx, dev)
    recv, scale = epl.dispatch(cfg, x_d, L)
    torch.cuda.synchronize()
    ref = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    assert_layout_equal(L, ref, w.name)
    rng = np.random.default_rng(1)
    toks = np.unique(np.concatenate([rng.integers(0, w.T, 192), [0, w.T - 1]]))
    rows = ref.pair_row[toks]
    got_q = recv[torch.from_numpy(rows.ravel().astype(np.int64)).to(dev)].cpu().numpy().reshape(len(toks), w.k, -1)
    got_s = scale[torch.from_numpy(rows.ravel().astype(np.int64)).to(dev)].cpu().numpy().reshape(len(toks), w.k, -1)
    for i, g in enumerate(toks):
        q, s = oracle.quantize_row_e4m3(x[g])
        for j in range(w.k):
            np.testing.assert_array_equal(got_q[i, j], q)
            np.testing.assert_array_equal(got_s[i, j].view(np.uint32), s.view(np.uint32))
    # skew is real: the hottest expert receives far more than the mean
    cnt = np.diff(ref.expert_off)
    assert cnt.max() > 8 * cnt.mean()


# ---------------------------------------------------------------------- behaviour
def test_deterministic_and_stream_ordered():
    dev = device()
    w = W.WORKLOADS["skewed_fp8_ep64"]
    idx = W.routing(w)
    cfg = epl.config(w.R, w.E, w.k, w.H, w.Tr, "bf16")
    idx_d = torch.from_numpy(idx).to(dev)
    L1 = epl.layout(cfg, idx_d)
    side = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(side):
        L2 = epl.layout(cfg, idx_d)
    side.synchronize()
    torch.cuda.synchronize()
    for f in ["pair_row", "pair_rslot", "seg_off", "rank_cnt", "tok_nranks"]:
        assert torch.equal(getattr(L1, f), getattr(L2, f)), f
    for _ in range(3):
        L3 = epl.layout(cfg, idx_d, out=L2)
        torch.cuda.synchronize()
        assert torch.equal(L1.pair_row, L3.pair_row)


def _e4m3_sweep():
    """Every (sign, exponent, top-11 mantissa bits) with four low-bit patterns, restricted to the
    range where E4M3 rounding and saturation happen, plus every bf16 pattern."""
    s = np.arange(2, dtype=np.uint32)
    e = np.arange(100, 140, dtype=np.uint32)  # 2^-27 .. 2^12
    m = np.arange(1 << 11, dtype=np.uint32)
    lo = np.array([0, 1, 0x7FF, 0xFFF], dtype=np.uint32)
    bits = (s[:, None, None, None] << 31) | (e[None, :, None, None] << 23) | (m[None, None, :, None] << 12) | \
        lo[None, None, None, :]
    bf = np.arange(1 << 16, dtype=np.uint32) << 16
    allb = np.concatenate([bits.ravel(), bf, np.array([0, 0x80000000, 1, 0x80000001], np.uint32)])
    v = allb.view(np.float32)
    return v[np.isfinite(v)]


def test_device_e4m3_conversion_matches_oracle():
    dev = device()
    v = _e4m3_sweep()
    got = epl.debug_f32_to_e4m3(torch.from_numpy(v).to(dev)).cpu().numpy()
    want = oracle.f32_to_e4m3(v)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "e4m3 differs for %s: got %s want %s" % (v[bad[:8]], got[bad[:8]], want[bad[:8]])


def test_device_bf16_conversion_matches_oracle():
    dev = device()
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2 ** 32, size=1 << 24, dtype=np.uint64).astype(np.uint32)
    hi = rng.integers(0, 1 << 16, size=1 << 20, dtype=np.uint32) << 16
    ties = np.concatenate([hi | 0x8000, hi | 0x7FFF, hi | 0x8001])
    v = np.concatenate([bits, ties]).view(np.float32)
    v = v[~np.isnan(v)]
    got = epl.debug_f32_to_bf16(torch.from_numpy(v).to(dev)).cpu().numpy().view(np.uint16)
    want = oracle.f32_to_bf16(v)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, "bf16 differs for %s: got %s want %s" % (v[bad[:8]], got[bad[:8]], want[bad[:8]])
