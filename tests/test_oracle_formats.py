"""Pins for the oracle's number formats.

* E4M3 is checked against an independent brute force: the nearest of all finite codes, with
  ties going to the even mantissa and saturation at 448. The codes are decoded with the
  specification's formula.
* E4M3 is also checked against the OCP anchor table in tests/golden.
* bf16 rounding is checked against torch's float32 -> bfloat16 conversion, which is a library
  routine.
"""
import os

import numpy as np
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e4m3_ocp_anchors.txt")


def spec_e4m3_table():
    """code -> value from the OCP E4M3 formula; NaN codes map to nan."""
    vals = np.zeros(256)
    for c in range(256):
        s, e, m = c >> 7, (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            v = np.nan
        elif e == 0:
            v = (m / 8) * 2.0 ** (1 - 7)
        else:
            v = (1 + m / 8) * 2.0 ** (e - 7)
        vals[c] = -v if s else v
    return vals


def brute_e4m3(v):
    """Nearest finite E4M3 code by exhaustive search; ties to the even mantissa; |v| >= 448 -> 448."""
    v = np.asarray(v, np.float64)
    tab = spec_e4m3_table()
    pos = np.arange(0, 127)  # codes 0x00..0x7E: all finite non-negative values, ascending
    pv = tab[pos]
    a = np.abs(v)
    dist = np.abs(a[:, None] - pv[None, :])
    best = dist.min(axis=1, keepdims=True)
    cand = dist == best
    # among equally near codes prefer the even mantissa (code bit 0 clear)
    even = cand & ((pos[None, :] & 1) == 0)
    pick = np.where(even.any(axis=1), even.argmax(axis=1), cand.argmax(axis=1))
    code = pos[pick]
    code = np.where(a >= 448.0, 0x7E, code)
    return (code | np.where(np.signbit(v), 0x80, 0)).astype(np.uint8)


def test_e4m3_golden_anchors():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    for code_s, val_s in rows:
        code, val = int(code_s, 16), float(val_s)
        dec = float(oracle.lib().eplref_e4m3_to_f32(code))
        assert dec == val and np.signbit(dec) == np.signbit(val), (code_s, dec, val)
        assert int(oracle.lib().eplref_f32_to_e4m3(val)) == code
        assert spec_e4m3_table()[code] == val


def test_e4m3_decode_matches_spec_formula():
    tab = spec_e4m3_table()
    dec = oracle.e4m3_to_f32(np.arange(256, dtype=np.uint8)).astype(np.float64)
    fin = ~np.isnan(tab)
    np.testing.assert_array_equal(dec[fin], tab[fin])
    assert np.isnan(dec[~fin]).all() and (~fin).sum() == 2


def _e4m3_probe_inputs():
    tab = spec_e4m3_table()
    pv = np.sort(tab[0:127])
    mids = (pv[1:] + pv[:-1]) / 2  # exact ties (representable in fp32)
    f32 = lambda a: np.asarray(a, np.float64).astype(np.float32)
    ties = f32(mids)
    up = np.nextafter(ties, np.float32(np.inf))
    dn = np.nextafter(ties, np.float32(0))
    exact = f32(pv)
    rng = np.random.default_rng(5)
    bits = rng.integers(0, 2 ** 32, size=1 << 18, dtype=np.uint64).astype(np.uint32)
    rnd = bits.view(np.float32)
    rnd = rnd[np.isfinite(rnd) & (np.abs(rnd) < 2000)]
    wide = (rng.standard_normal(1 << 16) * 150).astype(np.float32)
    tiny = (rng.standard_normal(1 << 14) * 2.0 ** -9).astype(np.float32)
    bf = (np.arange(1 << 16, dtype=np.uint32) << 16).view(np.float32)
    bf = bf[np.isfinite(bf)]
    specials = np.array([0.0, -0.0, 448, 464, 464.0001, 479.99, 480, 1e30, -1e30, np.inf, -np.inf,
                         2.0 ** -10, -(2.0 ** -10), 2.0 ** -10 * 1.0000001, 2.0 ** -149, 1.5 * 2.0 ** -9],
                        np.float32)
    allv = np.concatenate([ties, -ties, up, -up, dn, -dn, exact, -exact, rnd, wide, tiny, bf, specials])
    return allv


def test_e4m3_round_vs_bruteforce():
    v = _e4m3_probe_inputs()
    got = oracle.f32_to_e4m3(v)
    for s in range(0, v.size, 1 << 14):
        want = brute_e4m3(v[s:s + (1 << 14)].astype(np.float64))
        bad = np.nonzero(got[s:s + (1 << 14)] != want)[0]
        assert bad.size == 0, (v[s + bad[:5]], got[s + bad[:5]], want[bad[:5]])


def test_e4m3_nan():
    assert oracle.lib().eplref_f32_to_e4m3(float("nan")) & 0x7F == 0x7F


def bf16_torch(v):
    return torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(
        np.uint16)


def test_bf16_round_vs_torch():
    rng = np.random.default_rng(11)
    bits = rng.integers(0, 2 ** 32, size=1 << 22, dtype=np.uint64).astype(np.uint32)
    hi = rng.integers(0, 1 << 16, size=1 << 18, dtype=np.uint32) << 16
    ties = np.concatenate([hi | 0x8000, hi | 0x7FFF, hi | 0x8001, hi, hi | 0xFFFF])
    edge = np.array([0x7F7F8000, 0x7F7F7FFF, 0x7F7FFFFF, 0x7F800000, 0xFF800000, 0x00000001, 0x80000001,
                     0x007FFFFF, 0x00008000, 0x00018000, 0x80008000, 0x00000000, 0x80000000], np.uint32)
    v = np.concatenate([bits, ties, edge]).view(np.float32)
    fin = ~np.isnan(v)
    got = oracle.f32_to_bf16(v)
    want = bf16_torch(v)
    bad = np.nonzero(fin & (got != want))[0]
    assert bad.size == 0, (v[bad[:5]], got[bad[:5]], want[bad[:5]])
    # NaN stays NaN (quiet bit set)
    nan_out = got[~fin]
    assert ((nan_out & 0x7F80) == 0x7F80).all() and ((nan_out & 0x7F) != 0).all()


def test_bf16_widen_exact():
    h = np.arange(1 << 16, dtype=np.uint16)
    f = oracle.bf16_to_f32(h)
    t = torch.from_numpy(h.view(np.int16)).view(torch.bfloat16).float().numpy()
    same = (f.view(np.uint32) == t.view(np.uint32)) | (np.isnan(f) & np.isnan(t))
    assert same.all()
    f2 = np.array([oracle.lib().eplref_bf16_to_f32(int(x)) for x in h[::97]], np.float32)
    assert ((f2.view(np.uint32) == f[::97].view(np.uint32)) | np.isnan(f2)).all()
