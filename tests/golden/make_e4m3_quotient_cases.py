#!/usr/bin/env python3
"""Writes e4m3_quotient_cases.txt: fp8 quantiser blocks on which the order of the quotient step
decides codes.

The quantiser's definition (one fp32 scale s = fl32(a / 448) per 128-element block, a = max|x|,
then q = E4M3(fl32(x / s))) rounds twice in fp32 before the E4M3 rounding. A different reading,
q = E4M3(x * 448 / a) taken exactly, gives other codes wherever x * 448 / a is an exact E4M3 tie:
the fp32 quotient then lands one fp32 ulp off the tie and rounds away from the even code. This
script enumerates every pair of positive bf16 values (a in [1, 2), x <= a down to 2^-30), keeps the
pairs on which the two readings differ (found with numpy and the tests' brute-force E4M3 search),
builds blocks whose amax is a and which hold those x values (both signs), pads them with seeded
values below a, and stores each block with the codes and scale the oracle produces for it.

Only the oracle (oracle/) and numpy compute anything stored here. Run from the repository root:
    python tests/golden/make_e4m3_quotient_cases.py
"""
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)
import oracle  # noqa: E402
from tests.test_oracle_formats import brute_e4m3  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "e4m3_quotient_cases.txt")


def bf16_bits(f):
    return (np.asarray(f, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def discriminating_pairs():
    am = np.arange(128, 256)
    a = (am / 128.0).astype(np.float32)
    xm = np.arange(128, 256) / 128.0
    es = np.arange(-30, 1)
    X = (xm[None, :] * 2.0 ** es[:, None]).ravel().astype(np.float32)
    A = np.repeat(a, X.size)
    XX = np.tile(X, a.size)
    keep = XX <= A
    A, XX = A[keep], XX[keep]
    v = XX / (A / np.float32(448.0))  # the definition, in numpy fp32 (IEEE division)
    fp32_codes = oracle.f32_to_e4m3(v)
    exact = XX.astype(np.float64) * 448.0 / A.astype(np.float64)
    exact_codes = np.concatenate([brute_e4m3(exact[i:i + 100000]) for i in range(0, exact.size, 100000)])
    d = np.nonzero(fp32_codes != exact_codes)[0]
    return A[d], XX[d]


def main():
    A, X = discriminating_pairs()
    rng = np.random.default_rng(2607)
    lines = ["# fp8 E4M3 quantiser blocks on which fl32(x / fl32(a/448)) and the exact x*448/a round to",
             "# different codes (written by make_e4m3_quotient_cases.py from the oracle and numpy only).",
             "# Per block, three lines: 'x' and 128 bf16 inputs (hex), 'q' and the 128 codes the oracle",
             "# gives (hex), 's' and the block scale's fp32 bits (hex). Element 0 is the block's amax a.",
             "# %d discriminating (a, x) pairs were found among all positive bf16 pairs with a in [1, 2)." % len(A)]
    for a in np.unique(A):
        xs = X[A == a]
        blk = np.empty(128, np.float32)
        blk[0] = a
        vals = np.concatenate([xs, -xs])
        blk[1:1 + vals.size] = vals
        rest = 127 - vals.size
        pad = rng.standard_normal(rest).astype(np.float32) * np.float32(a) / 4
        pad = np.clip(pad, -np.float32(a) * 0.99, np.float32(a) * 0.99)
        blk[1 + vals.size:] = pad
        xb = bf16_bits(blk)
        q, s = oracle.quantize_row_e4m3(xb)
        lines.append("x " + " ".join("%04x" % v for v in xb))
        lines.append("q " + " ".join("%02x" % v for v in q))
        lines.append("s %08x" % int(s.view(np.uint32)[0]))
    open(OUT, "w").write("\n".join(lines) + "\n")
    print("wrote %s: %d blocks" % (OUT, len(np.unique(A))))


if __name__ == "__main__":
    main()
