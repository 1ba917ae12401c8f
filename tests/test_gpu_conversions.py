"""The device number conversions against the oracle over every one of the 2^32 fp32 bit patterns:
fp32 -> E4M3 (round to nearest even, saturating to 448, sign kept on zero, NaN -> 0x7F | sign) and
fp32 -> bf16 (round to nearest even; NaN quieted). epl_debug_f32_to_* apply exactly the conversions
epl_dispatch and epl_combine use. The sweep runs in 16 chunks of 2^28 patterns; the oracle's
single-threaded C conversion is called on slices of each chunk from a thread pool."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2607_06202_amd import epl
from tests.gpu_util import device

pytestmark = pytest.mark.gpu

CHUNK = 1 << 28


def _oracle_slices(fn, v, dtype):
    parts = max(1, min(16, os.cpu_count() or 1))
    out = np.empty(v.size, dtype)
    edges = np.linspace(0, v.size, parts + 1).astype(np.int64)

    def work(i):
        out[edges[i]:edges[i + 1]] = fn(v[edges[i]:edges[i + 1]]).view(dtype)

    with ThreadPoolExecutor(parts) as ex:
        list(ex.map(work, range(parts)))
    return out


def _device_patterns(start, dev):
    bits = torch.arange(start, start + CHUNK, dtype=torch.int64, device=dev)
    bits = torch.where(bits >= 1 << 31, bits - (1 << 32), bits).to(torch.int32)
    return bits.view(torch.float32)


def _sweep(device_fn, oracle_fn, dtype, what):
    dev = device()
    for c in range((1 << 32) // CHUNK):
        start = c * CHUNK
        got = device_fn(_device_patterns(start, dev)).cpu().numpy().view(dtype)
        v = (np.arange(CHUNK, dtype=np.uint32) + np.uint32(start)).view(np.float32)
        want = _oracle_slices(oracle_fn, v, dtype)
        bad = np.flatnonzero(got != want)
        if bad.size:
            bits = v[bad[:8]].view(np.uint32)
            raise AssertionError("%s: %d of 2^28 patterns in chunk %d differ, e.g. %s: got %s, want %s" % (
                what, bad.size, c, [hex(b) for b in bits], [hex(g) for g in got[bad[:8]]],
                [hex(w) for w in want[bad[:8]]]))


def test_e4m3_every_fp32_pattern():
    _sweep(epl.debug_f32_to_e4m3, oracle.f32_to_e4m3, np.uint8, "fp32 -> e4m3")


def test_bf16_every_fp32_pattern():
    _sweep(epl.debug_f32_to_bf16, oracle.f32_to_bf16, np.uint16, "fp32 -> bf16")
