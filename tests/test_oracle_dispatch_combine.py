"""Pins for the oracle's dispatch (bf16 copy, fp8 quantise) and combine (fp32 fold, bf16 out).

* Dispatch: every packed row equals its source token row, found through the inverse map. Rows
  past P are never written.
* FP8 quantise:
  - scale s = a/448 in fp32, checked with numpy's IEEE float32 division;
  - every block with a > 0 holds a code of magnitude 448 (I10);
  - the reconstruction error is within half an E4M3 ulp (I11);
  - all-zero blocks give zero codes and s = 0.
* Combine:
  - identity experts with gate weights summing to 1 reproduce x bit for bit;
  - k = 1 with w = 1 copies y;
  - zero weights change nothing;
  - the result is within 1 bf16 ulp of the exact fp64 sum;
  - the result equals bf16(fp32 sequential sum) when the products are exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import workloads as W


def small_case(R=4, El=3, k=4, Tr=20, H=256, seed=0, invalid=True):
    E = R * El
    T = R * Tr
    lo, hi = (-1, E + 1) if invalid else (0, E)
    idx = W.with_replacement(seed, T, k, lo, hi).astype(np.int32)
    x = W.normal_bf16(seed, W.STREAM_X, T * H).reshape(T, H)
    w = W.softmax_gate_weights(seed, T, k)
    return R, E, k, Tr, H, idx, x, w


def f32(h):
    return oracle.bf16_to_f32(h)


def test_dispatch_bf16_rows_are_source_rows():
    R, E, k, Tr, H, idx, x, w = small_case()
    L = oracle.layout(R, E, k, Tr, idx)
    cap = R * Tr * k
    recv = oracle.dispatch_bf16(x, L.pair_row, cap, fill=0xDEAD)
    P = L.P
    np.testing.assert_array_equal(recv[:P], x[L.recv_src])
    assert (recv[P:] == 0xDEAD).all()  # I9: nothing beyond P is written


def test_quantize_block_rules():
    rng = np.random.default_rng(2)
    H = 1024
    xf = (rng.standard_normal(H) * np.repeat(2.0 ** rng.integers(-20, 20, H // 128), 128)).astype(np.float32)
    xf[256:384] = 0.0                       # all-zero block
    xf[384:512] = -0.0
    xf[512] = 3.0e-39                        # bf16 subnormal-range value in a tiny block
    xf[513:640] = 0.0
    xb = W.f32_to_bf16_bits(xf)
    q, s = oracle.quantize_row_e4m3(xb)
    xv = f32(xb).astype(np.float64)
    tab = np.array([float(oracle.lib().eplref_e4m3_to_f32(c)) for c in range(256)])
    for b in range(H // 128):
        blk = xv[b * 128:(b + 1) * 128]
        a = np.float32(np.abs(blk).max())
        assert s[b] == np.float32(a) / np.float32(448.0)  # IEEE fp32 division
        qb = q[b * 128:(b + 1) * 128]
        if a == 0:
            assert (qb == 0).all() and s[b] == 0
            continue
        assert ((qb & 0x7F) == 0x7E).any()            # I10
        dec = tab[qb] * float(s[b])
        err = np.abs(dec - blk)
        # I11: half an E4M3 ulp at |x/s| (2^-4 relative for normals, 2^-10 absolute for
        # subnormals, in units of s), plus fp32 slack for the division and the multiply
        xs = np.abs(blk) / float(s[b])
        half_ulp = np.where(xs >= 2.0 ** -6, 2.0 ** (np.floor(np.log2(np.maximum(xs, 1e-300))) - 4), 2.0 ** -10)
        assert (err <= (half_ulp * (1 + 2 ** -20) + xs * 2 ** -22) * float(s[b]) + 1e-45).all()


def test_dispatch_fp8_rows_are_quantised_source_rows():
    R, E, k, Tr, H, idx, x, w = small_case(H=512)
    L = oracle.layout(R, E, k, Tr, idx)
    cap = R * Tr * k
    recv, scale = oracle.dispatch_fp8(x, L.pair_row, cap, fill=0xAB)
    for row in range(L.P):
        q, s = oracle.quantize_row_e4m3(x[L.recv_src[row]])
        np.testing.assert_array_equal(recv[row], q)
        np.testing.assert_array_equal(scale[row], s)
    assert (recv[L.P:] == 0xAB).all() and np.isnan(scale[L.P:]).all()


@pytest.mark.parametrize("name", ["tiny", "large_ep256"])
def test_identity_round_trip_reproduces_x(name):
    """Dispatch -> identity experts -> combine with softmax weights reproduces x bitwise
    (numerically: -0 comes back as +0)."""
    w_ = W.WORKLOADS[name]
    if name == "large_ep256":
        w_ = W.Workload("large_ep256_h256", w_.R, w_.E, w_.k, 8, 256, "bf16", "hot_group")
    idx = W.routing(w_)
    x = W.tokens_bf16(w_)
    gw = W.gate_weights(w_)
    L = oracle.layout(w_.R, w_.E, w_.k, w_.Tr, idx)
    recv = oracle.dispatch_bf16(x, L.pair_row, L.P)
    out = oracle.combine(recv, gw, L.pair_row)
    np.testing.assert_array_equal(f32(out), f32(x))


def test_identity_round_trip_random_weights_sum_to_one():
    R, E, k, Tr, H, idx, x, w = small_case(k=8, invalid=False, seed=4)
    L = oracle.layout(R, E, k, Tr, idx)
    recv = oracle.dispatch_bf16(x, L.pair_row, L.P)
    out = oracle.combine(recv, w, L.pair_row)
    np.testing.assert_array_equal(f32(out), f32(x))


def test_combine_k1_unit_weight_copies_rows():
    R, E, k, Tr, H, idx, x, w = small_case(k=1, invalid=True, seed=6)
    L = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(9, W.STREAM_Y, max(L.P, 1) * H).reshape(-1, H)
    out = oracle.combine(y, np.ones((R * Tr, 1), np.float32), L.pair_row)
    for g in range(R * Tr):
        r = L.pair_row[g, 0]
        want = f32(y[r]) if r >= 0 else np.zeros(H, np.float32)
        np.testing.assert_array_equal(f32(out[g]), want)


def test_combine_zero_weights_change_nothing():
    R, E, k, Tr, H, idx, x, w = small_case(k=6, invalid=True, seed=8)
    L = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(9, W.STREAM_Y, L.P * H).reshape(L.P, H)
    w2 = w.copy()
    w2[:, 3:] = 0.0
    out = oracle.combine(y, w2, L.pair_row)
    pr = L.pair_row.copy()
    pr[:, 3:] = -1
    out_trunc = oracle.combine(y, w2, pr)
    np.testing.assert_array_equal(out, out_trunc)


def test_combine_within_one_ulp_of_fp64():
    R, E, k, Tr, H, idx, x, w = small_case(k=8, invalid=True, seed=10, H=512)
    L = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(9, W.STREAM_Y, L.P * H).reshape(L.P, H)
    out = oracle.combine(y, w, L.pair_row)
    yf = f32(y).astype(np.float64)
    ref = np.zeros((R * Tr, H))
    for j in range(k):
        r = L.pair_row[:, j]
        ok = r >= 0
        ref[ok] += w[ok, j, None].astype(np.float64) * yf[r[ok]]
    # distance in bf16 units-in-the-last-place between out and the exact value
    o = f32(out).astype(np.float64)
    ulp = 2.0 ** (np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126))) - 7)
    assert (np.abs(o - ref) <= ulp).all()


def test_combine_exact_products_match_sequential_fp32():
    """With weights that are powers of two the products are exact; then fmaf == add, and the
    result must equal torch's bf16 rounding of the fp32 sequential sum."""
    R, E, k, Tr, H, idx, x, w = small_case(k=5, invalid=True, seed=12)
    L = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(13, W.STREAM_Y, L.P * H).reshape(L.P, H)
    rng = np.random.default_rng(1)
    w2 = (2.0 ** rng.integers(-3, 2, size=w.shape) * rng.choice([-1, 1], size=w.shape)).astype(np.float32)
    out = oracle.combine(y, w2, L.pair_row)
    yf = torch.from_numpy(f32(y))
    acc = torch.zeros(R * Tr, H, dtype=torch.float32)
    for j in range(k):
        r = torch.from_numpy(L.pair_row[:, j].astype(np.int64))
        ok = r >= 0
        acc[ok] = acc[ok] + torch.from_numpy(w2[:, j])[ok, None] * yf[r[ok]]
    want = acc.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(f32(out), f32(want))


def test_combine_sampled_tokens_and_mapped_rows_agree():
    R, E, k, Tr, H, idx, x, w = small_case(k=4, seed=14)
    L = oracle.layout(R, E, k, Tr, idx)
    y = W.normal_bf16(15, W.STREAM_Y, L.P * H).reshape(L.P, H)
    full = oracle.combine(y, w, L.pair_row)
    toks = np.array([0, 5, 17, R * Tr - 1])
    np.testing.assert_array_equal(oracle.combine(y, w, L.pair_row, tokens=toks), full[toks])
    rows = np.unique(L.pair_row[toks][L.pair_row[toks] >= 0])
    row_map = np.full(L.P, -1, np.int32)
    row_map[rows] = np.arange(rows.size)
    np.testing.assert_array_equal(oracle.combine_mapped(y[rows], row_map, w, L.pair_row, toks), full[toks])


def test_combine_is_fused_multiply_add():
    """The fold is acc = fmaf(w, y, acc), a single rounding per term, not a rounded product
    followed by a rounded add. Construction, with A = 1 + 2^-7 (a bf16 whose last bit is odd)
    and M = A + 2^-8 (the bf16 midpoint above A):
    * pick fp32 w and bf16 y whose exact product p lies just below 2^-8 - 2^-24, but which
      rounds to exactly 2^-8 - 2^-24 in fp32;
    * fused: A + p rounds in fp32 to M - 2^-23, which is below the midpoint, so bf16 gives A;
    * unfused: A + fp32(p) = M - 2^-24 is an fp32 tie that goes to the even M, and the bf16
      tie then goes to the even 1 + 2^-6.
    All products here are exact in float64 (24 x 8 significant bits)."""
    target = 2.0 ** -8 - 2.0 ** -24
    ys, ws = [], []
    for yb in range(0x3F80, 0x4000):  # every bf16 in [1, 2)
        yv = float(oracle.bf16_to_f32(np.array([yb], np.uint16))[0])
        w0 = np.float32(target / yv)
        for d in range(-3, 4):
            wv = np.float32(w0)
            for _ in range(abs(d)):
                wv = np.nextafter(wv, np.float32(np.inf if d > 0 else 0))
            p = float(wv) * yv  # exact
            if p < target and float(np.float32(p)) == target:
                ys.append(yb)
                ws.append(wv)
    assert len(ys) >= 4, "construction found too few cases"
    n = len(ys)
    A = 0x3F81
    y = np.array([[A] * 8] + [[yb] * 8 for yb in ys], np.uint16)  # row 0 holds A, row i holds y_i
    pair_row = np.stack([np.zeros(n, np.int32), np.arange(1, n + 1, dtype=np.int32)], axis=1)
    w = np.stack([np.ones(n, np.float32), np.array(ws, np.float32)], axis=1)
    out = oracle.combine(y, w, pair_row)
    assert (out == A).all(), out[:, 0]  # the unfused fold would give 0x3F82
