"""Seeded synthetic MoE routing workloads: inputs only, none of the method's arithmetic.

Both the GPU path and the CPU oracle consume the arrays built here. Nothing in this
module computes a layout, a dispatch or a combine.

Counter-based generator
-----------------------
Every random 64-bit word is a pure function of ``(seed, stream, index)``::

    mix64(z)   = SplitMix64 finaliser: z ^= z>>30; z *= 0xBF58476D1CE4E5B9;
                                       z ^= z>>27; z *= 0x94D049BB133111EB; z ^= z>>31
    key        = mix64((seed << 32) | stream)
    u64(i)     = mix64(key + (i + 1) * 0x9E3779B97F4A7C15)          (all mod 2^64)

so the result does not depend on chunking or thread count. Derived draws:

* ``unit(u)``    = ((u >> 11) + 0.5) / 2^53, a double in (0, 1).
* ``normal(u)``  = Box-Muller on the two 32-bit halves, a = u >> 32, b = u & 0xffffffff:
  sqrt(-2 ln((a+.5)/2^32)) * cos(2 pi (b+.5)/2^32), in float64; then float32 (RNE); then
  bfloat16 (RNE) for token payloads.
* ``below(u, n)`` = ((u >> 32) * n) >> 32, an integer in [0, n).

Streams: 1 token payload x, 2 routing draws, 3 gate logits, 4 hot-token coin,
5 expert popularity permutation, 6 group Gumbel keys, 7 expert Gumbel keys, 8 hot group,
9 expert-output rows y.

The five named workloads follow the paper's DeepSeek-V3/R1 shape (hidden 7168, 256 routed
experts, top-8; evaluation setup, model-configuration table) plus one tiny case; the paper's
own traffic comes from real models served by vLLM-Ascend, which these seeded inputs stand in
for.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

STREAM_X, STREAM_ROUTE, STREAM_LOGIT, STREAM_HOT = 1, 2, 3, 4
STREAM_PERM, STREAM_GROUP, STREAM_EXPERT, STREAM_HOTGROUP, STREAM_Y = 5, 6, 7, 8, 9

# Attempt budget reserved per token for rejection sampling; attempt a of token g uses
# counter g * _ATTEMPT_STRIDE + a, so extending the search never reuses a counter.
_ATTEMPT_STRIDE = 1 << 16


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def rand_u64(seed: int, stream: int, index) -> np.ndarray:
    """u64(seed, stream, index) for an array of non-negative counters."""
    with np.errstate(over="ignore"):
        key = _mix64(np.array([(int(seed) << 32) | int(stream)], dtype=np.uint64))[0]
        i = np.asarray(index, dtype=np.uint64)
        return _mix64(key + (i + np.uint64(1)) * _GAMMA)


def unit(u: np.ndarray) -> np.ndarray:
    return ((u >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)


def normal_f64(u: np.ndarray) -> np.ndarray:
    a = (u >> np.uint64(32)).astype(np.float64)
    b = (u & np.uint64(0xFFFFFFFF)).astype(np.float64)
    u1 = (a + 0.5) * (2.0 ** -32)
    u2 = (b + 0.5) * (2.0 ** -32)
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)


def below(u: np.ndarray, n: int) -> np.ndarray:
    return (((u >> np.uint64(32)) * np.uint64(n)) >> np.uint64(32)).astype(np.int64)


def f32_to_bf16_bits(v: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round-to-nearest-even, via torch's CPU conversion."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _normal_block(key: np.uint64, start: int, out_f32: np.ndarray) -> None:
    """normal(u64(start + i)) for i < len(out_f32), written as float32 (RNE). In-place
    arithmetic on small reused buffers; same values as normal_f64(rand_u64(...))."""
    n = out_f32.shape[0]
    z = np.arange(start + 1, start + 1 + n, dtype=np.uint64)
    tmp = np.empty(n, dtype=np.uint64)
    with np.errstate(over="ignore"):
        np.multiply(z, _GAMMA, out=z)
        np.add(z, key, out=z)
        for sh, mul in ((30, _M1), (27, _M2)):
            np.right_shift(z, np.uint64(sh), out=tmp)
            np.bitwise_xor(z, tmp, out=z)
            np.multiply(z, mul, out=z)
        np.right_shift(z, np.uint64(31), out=tmp)
        np.bitwise_xor(z, tmp, out=z)
    f1 = np.empty(n)
    f2 = np.empty(n)
    np.right_shift(z, np.uint64(32), out=tmp)
    f1[:] = tmp
    np.bitwise_and(z, np.uint64(0xFFFFFFFF), out=tmp)
    f2[:] = tmp
    f1 += 0.5
    f1 *= 2.0 ** -32
    f2 += 0.5
    f2 *= 2.0 ** -32
    f2 *= 2.0 * math.pi
    np.log(f1, out=f1)
    f1 *= -2.0
    np.sqrt(f1, out=f1)
    np.cos(f2, out=f2)
    f1 *= f2
    out_f32[:] = f1


def normal_bf16(seed: int, stream: int, n: int, offset: int = 0, threads: int | None = None) -> np.ndarray:
    """n bf16 bit patterns of N(0,1); element i uses counter offset + i."""
    with np.errstate(over="ignore"):
        key = _mix64(np.array([(int(seed) << 32) | int(stream)], dtype=np.uint64))[0]
    out = np.empty(n, dtype=np.uint16)
    chunk = 1 << 20
    starts = list(range(0, n, chunk))

    def work(s0: int) -> None:
        s1 = min(n, s0 + chunk)
        f = np.empty(s1 - s0, dtype=np.float32)
        for b0 in range(s0, s1, 1 << 16):
            b1 = min(s1, b0 + (1 << 16))
            _normal_block(key, offset + b0, f[b0 - s0 : b1 - s0])
        out[s0:s1] = f32_to_bf16_bits(f)

    nthr = threads or min(16, os.cpu_count() or 1)
    if len(starts) <= 1 or nthr <= 1:
        for s0 in starts:
            work(s0)
    else:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(work, starts))
    return out


# --------------------------------------------------------------------------- routing
def distinct_uniform(seed: int, tokens: np.ndarray, k: int, n: int, stream: int = STREAM_ROUTE) -> np.ndarray:
    """For each token id in ``tokens``: k distinct ids in [0, n), drawn uniformly by rejection
    (draw below(u, n), reject repeats), kept in draw order. Returns [len(tokens), k] int64."""
    if k > n:
        raise ValueError("cannot draw %d distinct ids out of %d" % (k, n))
    tokens = np.asarray(tokens, dtype=np.int64)
    m = tokens.shape[0]
    chosen = np.full((m, k), -1, dtype=np.int64)
    count = np.zeros(m, dtype=np.int64)
    col = np.arange(k)[None, :]
    attempt = 0
    batch = max(4 * k, 16)
    while True:
        todo = np.nonzero(count < k)[0]
        if todo.size == 0:
            break
        if attempt + batch > _ATTEMPT_STRIDE:
            raise RuntimeError("rejection sampling ran out of attempts")
        ctr = tokens[todo, None].astype(np.uint64) * np.uint64(_ATTEMPT_STRIDE) + np.arange(
            attempt, attempt + batch, dtype=np.uint64
        )[None, :]
        draws = below(rand_u64(seed, stream, ctr), n)
        ch = chosen[todo]
        cn = count[todo]
        for a in range(batch):
            cand = draws[:, a]
            dup = ((ch == cand[:, None]) & (col < cn[:, None])).any(axis=1)
            acc = (cn < k) & ~dup
            rows = np.nonzero(acc)[0]
            ch[rows, cn[rows]] = cand[rows]
            cn = cn + acc
        chosen[todo] = ch
        count[todo] = cn
        attempt += batch
    return chosen


def softmax_gate_weights(seed: int, T: int, k: int) -> np.ndarray:
    """Gate weights: float32 softmax over each token's k logits z ~ N(0,1) (stream 3,
    counter g*k + j): subtract the max, exp, sum in j order, divide."""
    z = normal_f64(rand_u64(seed, STREAM_LOGIT, np.arange(T * k, dtype=np.uint64))).astype(np.float32)
    z = z.reshape(T, k)
    m = z.max(axis=1, keepdims=True)
    ex = np.exp(z - m).astype(np.float32)
    s = np.zeros((T, 1), dtype=np.float32)
    for j in range(k):
        s = (s + ex[:, j : j + 1]).astype(np.float32)
    return (ex / s).astype(np.float32)


def gumbel(u: np.ndarray) -> np.ndarray:
    return -np.log(-np.log(unit(u)))


def zipf_group_limited(seed: int, T: int, E: int, R: int, k: int, zipf_s: float = 1.2,
                       n_groups: int = 8, groups_per_token: int = 4) -> np.ndarray:
    """Skewed routing: expert popularity p_e ~ (pi(e)+1)^-s for a seeded permutation pi;
    ranks are split into ``n_groups`` contiguous groups; each token first draws
    ``groups_per_token`` distinct groups without replacement with probability ~ group mass
    (Gumbel-top-k), then k distinct experts from those groups with probability ~ p_e
    (Gumbel-top-k). Ids are returned in descending key order."""
    if R % n_groups or E % R:
        raise ValueError("ranks must split evenly into groups")
    perm_keys = rand_u64(seed, STREAM_PERM, np.arange(E, dtype=np.uint64))
    order = np.argsort(perm_keys, kind="stable")
    pi = np.empty(E, dtype=np.int64)
    pi[order] = np.arange(E)
    p = (pi + 1.0) ** (-zipf_s)
    p = p / p.sum()
    el = E // R
    group_of = (np.arange(E) // el) // (R // n_groups)
    mass = np.bincount(group_of, weights=p, minlength=n_groups)
    gk = np.log(mass)[None, :] + gumbel(
        rand_u64(seed, STREAM_GROUP, np.arange(T * n_groups, dtype=np.uint64))).reshape(T, n_groups)
    top_g = np.argsort(-gk, axis=1, kind="stable")[:, :groups_per_token]
    allowed = np.zeros((T, n_groups), dtype=bool)
    np.put_along_axis(allowed, top_g, True, axis=1)
    out = np.empty((T, k), dtype=np.int64)
    step = 4096
    for t0 in range(0, T, step):
        t1 = min(T, t0 + step)
        ctr = np.arange(t0 * E, t1 * E, dtype=np.uint64)
        ek = np.log(p)[None, :] + gumbel(rand_u64(seed, STREAM_EXPERT, ctr)).reshape(t1 - t0, E)
        ek = np.where(allowed[t0:t1][:, group_of], ek, -np.inf)
        out[t0:t1] = np.argsort(-ek, axis=1, kind="stable")[:, :k]
    return out


def hot_group(seed: int, T: int, E: int, R: int, k: int, hot_frac: float = 0.2,
              n_groups: int = 16) -> np.ndarray:
    """Hot-spot routing: ranks form ``n_groups`` contiguous groups; one seeded group h is hot.
    Each token is hot with probability ``hot_frac`` (unit(u) < hot_frac); a hot token takes k
    distinct uniform experts of group h, any other token k distinct uniform experts of all E."""
    per_group = E // n_groups
    h = int(below(rand_u64(seed, STREAM_HOTGROUP, np.array([0], dtype=np.uint64)), n_groups)[0])
    hot = unit(rand_u64(seed, STREAM_HOT, np.arange(T, dtype=np.uint64))) < hot_frac
    out = np.empty((T, k), dtype=np.int64)
    toks = np.arange(T)
    hot_t = toks[hot]
    cold_t = toks[~hot]
    if hot_t.size:
        out[hot_t] = h * per_group + distinct_uniform(seed, hot_t, k, per_group)
    if cold_t.size:
        out[cold_t] = distinct_uniform(seed, cold_t, k, E)
    return out


def with_replacement(seed: int, T: int, k: int, lo: int, hi: int) -> np.ndarray:
    """Ids drawn independently and uniformly from [lo, hi) -- duplicates and, when the range
    leaves [0, E), invalid ids included. Used for edge-case tests."""
    u = rand_u64(seed, STREAM_ROUTE, np.arange(T * k, dtype=np.uint64))
    return (lo + below(u, hi - lo)).reshape(T, k)


# --------------------------------------------------------------------------- workloads
@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    R: int          # virtual EP ranks
    E: int          # routed experts (E % R == 0; rank d owns experts [d*E/R, (d+1)*E/R))
    k: int          # top-k
    Tr: int         # tokens per rank
    H: int          # hidden size
    payload: str    # "bf16" or "fp8"
    routing: str    # "uniform" | "zipf_group" | "hot_group"

    @property
    def T(self) -> int:
        return self.R * self.Tr


WORKLOADS = {
    "tiny": Workload("tiny", 4, 16, 2, 128, 256, "bf16", "uniform"),
    "decode_ep64": Workload("decode_ep64", 64, 256, 8, 128, 7168, "bf16", "uniform"),
    "prefill_ep32": Workload("prefill_ep32", 32, 256, 8, 4096, 7168, "bf16", "uniform"),
    "skewed_fp8_ep64": Workload("skewed_fp8_ep64", 64, 256, 8, 256, 7168, "fp8", "zipf_group"),
    "large_ep256": Workload("large_ep256", 256, 256, 8, 64, 7168, "bf16", "hot_group"),
}
WORKLOAD_ORDER = ["tiny", "decode_ep64", "prefill_ep32", "skewed_fp8_ep64", "large_ep256"]

# The paper's other evaluated model shapes (its model-configuration table: hidden size, routed
# experts, top-8) at decode batch sizes, and its default ablation setting (128 ranks, 64 tokens per
# rank, one expert per rank), all with uniform routing and bf16 payloads.
MODEL_WORKLOADS = {
    "qwen3_30b_ep16": Workload("qwen3_30b_ep16", 16, 128, 8, 128, 2048, "bf16", "uniform"),
    "glm47_ep32": Workload("glm47_ep32", 32, 160, 8, 128, 5120, "bf16", "uniform"),
    "deepseek_ep128_bs64": Workload("deepseek_ep128_bs64", 128, 128, 8, 64, 7168, "bf16", "uniform"),
}
MODEL_ORDER = list(MODEL_WORKLOADS)
WORKLOADS.update(MODEL_WORKLOADS)


def routing(w: Workload, seed: int = 0) -> np.ndarray:
    """[T, k] int32 expert ids for a named workload."""
    T = w.T
    if w.routing == "uniform":
        ids = distinct_uniform(seed, np.arange(T), w.k, w.E)
    elif w.routing == "zipf_group":
        ids = zipf_group_limited(seed, T, w.E, w.R, w.k)
    elif w.routing == "hot_group":
        ids = hot_group(seed, T, w.E, w.R, w.k)
    else:
        raise ValueError(w.routing)
    return np.ascontiguousarray(ids, dtype=np.int32)


def tokens_bf16(w: Workload, seed: int = 0) -> np.ndarray:
    """[T, H] token payload as bf16 bit patterns (uint16), N(0,1)."""
    return normal_bf16(seed, STREAM_X, w.T * w.H).reshape(w.T, w.H)


def gate_weights(w: Workload, seed: int = 0) -> np.ndarray:
    return softmax_gate_weights(seed, w.T, w.k)


def device_normal_bf16(shape, seed: int, device):
    """N(0,1) bf16 tensor drawn on the device with torch's seeded Philox generator (input
    data only; used where host generation of multi-GB payloads would be too slow)."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return torch.randn(*shape, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)


def node_hop_classes(R: int, ranks_per_node: int = 8) -> np.ndarray:
    """Hop class of every (source rank, destination rank) for R ranks placed ranks_per_node to a node
    (8 GPUs on one xGMI node): 0 within the source's node, 1 across nodes -> [R, R] int32. A topology
    input of the hierarchical schedule, not part of its arithmetic."""
    node = np.arange(R) // ranks_per_node
    return (node[:, None] != node[None, :]).astype(np.int32)
