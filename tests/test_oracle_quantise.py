"""Exact per-code pin of the oracle's fp8 quantiser (eplref_quantize_row_e4m3).

The definition: per 128-element block, a = max|x| (exact in fp32), s = fl32(a / 448), and every
element's code is E4M3(fl32(x / s)), both divisions IEEE fp32 round-to-nearest-even, E4M3
rounding to nearest with ties to the even code and saturation at 448; a block with a = 0 gets
s = 0 and all codes 0. The test recomputes that definition independently: numpy's float32
division (IEEE) for s and for each quotient, then the brute-force nearest-of-all-codes E4M3 search
of tests/test_oracle_formats.py for the code. Every code of every block must agree exactly.

The blocks are chosen so that plausible misreadings fail:
* random normal blocks at many scales;
* power-of-two amax (a = 448 * 2^m), where s is exact;
* blocks built from the exact-tie pairs of tests/golden/e4m3_quotient_cases.txt, where
  E4M3(x * 448 / a) taken exactly (no fp32 quotient) gives other codes, and so does a
  multiplication by the rounded reciprocal;
* subnormal-heavy blocks, whose quotients fall in the E4M3 subnormal range.
"""
import os

import numpy as np

import oracle
from paper_2607_06202_amd import workloads as W
from tests.test_oracle_formats import brute_e4m3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_quotient_cases.txt")


def definition_codes(xb):
    """Codes and scales of bf16 blocks [n, 128] by the definition, computed with numpy alone."""
    xf = oracle.bf16_to_f32(xb).reshape(-1, 128)
    a = np.abs(xf).max(axis=1)
    s = a / np.float32(448.0)
    with np.errstate(divide="ignore", invalid="ignore"):
        v = xf / s[:, None]
    codes = np.zeros(xf.shape, np.uint8)
    nz = a > 0
    if nz.any():
        codes[nz] = brute_e4m3(v[nz].astype(np.float64).ravel()).reshape(-1, 128)
    return codes, s


def golden_blocks():
    blocks, codes, scales = [], [], []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        tag, *vals = line.split()
        if tag == "x":
            blocks.append([int(v, 16) for v in vals])
        elif tag == "q":
            codes.append([int(v, 16) for v in vals])
        elif tag == "s":
            scales.append(int(vals[0], 16))
    return (np.array(blocks, np.uint16), np.array(codes, np.uint8),
            np.array(scales, np.uint32).view(np.float32))


def varied_blocks():
    rng = np.random.default_rng(77)
    out = []
    # random normal blocks over 2^-40 .. 2^40
    f = rng.standard_normal((512, 128)) * 2.0 ** rng.integers(-40, 40, (512, 1))
    out.append(W.f32_to_bf16_bits(f.astype(np.float32).ravel()).reshape(-1, 128))
    # power-of-two amax: s = 2^m exactly
    f = rng.standard_normal((128, 128)).astype(np.float32)
    m = rng.integers(-20, 20, 128)
    f = f / np.abs(f).max(axis=1, keepdims=True) * np.float32(400.0)
    f[:, 0] = 448.0
    f *= (2.0 ** m)[:, None].astype(np.float32)
    out.append(W.f32_to_bf16_bits(f.ravel()).reshape(-1, 128))
    # exact-tie pairs, rescaled by powers of two (the quotients are unchanged)
    gx, _, _ = golden_blocks()
    for e in (-12, -3, 0, 5, 17):
        f = oracle.bf16_to_f32(gx) * np.float32(2.0 ** e)
        out.append(W.f32_to_bf16_bits(f.ravel()).reshape(-1, 128))
    # subnormal-heavy: one large value and the rest 2^-12 .. 2^-20 of it, bf16 subnormals included
    f = rng.standard_normal((128, 128)) * 2.0 ** rng.integers(-20, -11, (128, 128))
    f[:, 0] = 1.0
    f[64:] *= 2.0 ** -120
    out.append(W.f32_to_bf16_bits(f.astype(np.float32).ravel()).reshape(-1, 128))
    # all-zero blocks of both signs
    out.append(np.array([[0] * 128, [0x8000] * 128], np.uint16))
    return np.concatenate(out)


def test_every_code_follows_the_fp32_quotient():
    xb = varied_blocks()
    row = xb.reshape(-1)
    H = row.size
    q, s = oracle.quantize_row_e4m3(row)
    want_q, want_s = definition_codes(xb)
    np.testing.assert_array_equal(s.view(np.uint32), want_s.view(np.uint32))
    bad = np.argwhere(q.reshape(-1, 128) != want_q)
    assert bad.size == 0, "codes differ at %s" % bad[:8].tolist()
    assert xb.shape[0] >= 800


def test_golden_tie_blocks():
    """The stored blocks: the oracle reproduces the stored codes, the numpy recomputation of the
    definition agrees, and in every block the exact quotient x * 448 / a (and the product with the
    rounded reciprocal) would give other codes."""
    gx, gq, gs = golden_blocks()
    assert gx.shape[0] >= 8
    q, s = oracle.quantize_row_e4m3(gx.reshape(-1))
    np.testing.assert_array_equal(q.reshape(-1, 128), gq)
    np.testing.assert_array_equal(s.view(np.uint32), gs.view(np.uint32))
    want_q, want_s = definition_codes(gx)
    np.testing.assert_array_equal(gq, want_q)
    np.testing.assert_array_equal(gs.view(np.uint32), want_s.view(np.uint32))
    xf = oracle.bf16_to_f32(gx).astype(np.float64)
    a = np.abs(xf).max(axis=1, keepdims=True)
    exact = brute_e4m3((xf * 448.0 / a).ravel()).reshape(gq.shape)
    recip = np.float32(1.0) / gs
    mult = brute_e4m3((oracle.bf16_to_f32(gx) * recip[:, None]).astype(np.float64).ravel()).reshape(gq.shape)
    for b in range(gq.shape[0]):
        assert (exact[b] != gq[b]).any(), "block %d does not tell the exact quotient apart" % b
    assert (mult != gq).any(), "no block tells the reciprocal product apart"
