"""Pins for the oracle's routing layout (counts, CalCumSum offsets, slots, dedup).

None of these checks re-derives the oracle's counting sort. Each one pins it to something
else:
* an independent brute force: a stable comparison sort of the pair list, and Python sets for
  each token's destination ranks;
* exhaustive enumeration of micro routing tables;
* closed forms for special cases;
* invariants that any correct layout must satisfy.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2607_06202_amd import workloads as W


def brute_layout(R, E, k, Tr, idx):
    """Independent brute force: sorted() (a stable comparison sort) over the valid pairs keyed by
    expert id; destination-rank sets via Python sets."""
    T = R * Tr
    El = E // R
    idx = np.asarray(idx).reshape(T, k)
    pairs = [(g, j, int(idx[g, j])) for g in range(T) for j in range(k)]
    valid = [(g, j, e) for (g, j, e) in pairs if 0 <= e < E]
    order = sorted(valid, key=lambda t: t[2])
    pair_row = np.full((T, k), -1, np.int64)
    recv_src = [g for (g, j, e) in order]
    recv_j = [j for (g, j, e) in order]
    for row, (g, j, e) in enumerate(order):
        pair_row[g, j] = row
    send_cnt = np.zeros((R, E), np.int64)
    for (g, j, e) in valid:
        send_cnt[g // Tr, e] += 1
    recv_cnt = send_cnt.sum(0)
    expert_off = np.concatenate([[0], np.cumsum(recv_cnt)])
    rank_off = np.array([expert_off[d * El] for d in range(R + 1)])
    seg_off = np.zeros((E, R), np.int64)
    for e in range(E):
        for s in range(R):
            seg_off[e, s] = sum(1 for (g, j, ee) in valid if ee < e or (ee == e and g // Tr < s))
    D = [set(e // El for (gg, j, e) in valid if gg == g) for g in range(T)]
    tok_nranks = np.array([len(D[g]) for g in range(T)])
    rank_cnt = np.zeros((R, R), np.int64)
    for g in range(T):
        for r in D[g]:
            rank_cnt[g // Tr, r] += 1
    pair_rslot = np.full((T, k), -1, np.int64)
    for (g, j, e) in valid:
        s, r = g // Tr, e // El
        pair_rslot[g, j] = sum(1 for g2 in range(s * Tr, g) if r in D[g2])
    return dict(send_cnt=send_cnt, rank_cnt=rank_cnt, expert_off=expert_off, rank_off=rank_off, seg_off=seg_off,
                tok_nranks=tok_nranks, pair_row=pair_row, pair_rslot=pair_rslot, recv_src=np.array(recv_src),
                recv_j=np.array(recv_j), num_invalid=len(pairs) - len(valid))


def assert_matches_brute(R, E, k, Tr, idx):
    ref = oracle.layout(R, E, k, Tr, idx)
    bf = brute_layout(R, E, k, Tr, idx)
    for name, want in bf.items():
        got = getattr(ref, name)
        if name == "num_invalid":
            assert got == want, name
        else:
            np.testing.assert_array_equal(np.asarray(got).reshape(np.shape(want)), want, err_msg=name)
    return ref


def check_invariants(R, E, k, Tr, idx, L):
    """I1-I7 for a layout."""
    T = R * Tr
    El = E // R
    idx = np.asarray(idx).reshape(T, k)
    valid = (idx >= 0) & (idx < E)
    P = int(valid.sum())
    # I1 counts sum to the routed pairs
    assert L.send_cnt.sum() == P == T * k - L.num_invalid
    assert L.P == P
    # I2 pair_row restricted to valid pairs is a bijection onto [0, P)
    rows = L.pair_row[valid]
    assert np.array_equal(np.sort(rows), np.arange(P))
    assert (L.pair_row[~valid] == -1).all()
    # I3 inverse maps
    g_of = np.repeat(np.arange(T), k).reshape(T, k)
    j_of = np.tile(np.arange(k), T).reshape(T, k)
    assert np.array_equal(L.recv_src[rows], g_of[valid])
    assert np.array_equal(L.recv_j[rows], j_of[valid])
    # I4 row keys (e, s, g, j) strictly increasing in row order
    e_r = idx[L.recv_src, L.recv_j].astype(np.int64)
    key = ((e_r * R + L.recv_src // Tr) * T + L.recv_src) * k + L.recv_j if P else np.zeros(0)
    assert (np.diff(key) > 0).all()
    # I5 dedup totals equal the number of distinct (token, rank) pairs
    d = np.where(valid, idx // El, -1)
    distinct = sum(len(set(d[g][valid[g]].tolist())) for g in range(T))
    assert L.rank_cnt.sum() == L.tok_nranks.sum() == distinct
    # I6 pair_rslot over tokens of s bound for r is a bijection onto [0, rank_cnt[s][r])
    for s in range(R):
        toks = range(s * Tr, (s + 1) * Tr)
        for r in range(R):
            slots = sorted({int(L.pair_rslot[g, j]) for g in toks for j in range(k) if valid[g, j] and d[g, j] == r})
            assert slots == list(range(L.rank_cnt[s, r]))
    # I7 rank_off spans each rank's experts
    recv_cnt = L.send_cnt.sum(0)
    for r in range(R):
        assert L.rank_off[r + 1] - L.rank_off[r] == recv_cnt[r * El:(r + 1) * El].sum()


# ------------------------------------------------------------------ exhaustive micro tables
@pytest.mark.parametrize("R,E,Tr,k,lo,hi", [
    (2, 4, 1, 2, -1, 5),   # 6^4 = 1296 tables, ids include -1 and E
    (2, 2, 2, 2, -1, 2),   # 3^8 = 6561 tables, one expert per rank
    (1, 3, 3, 1, -1, 3),   # 4^3 = 64 tables, single rank
    (3, 3, 1, 2, 0, 3),    # 3^6 = 729 tables, k=2 over 3 ranks
])
def test_layout_exhaustive_micro(R, E, Tr, k, lo, hi):
    T = R * Tr
    n = 0
    for tab in itertools.product(range(lo, hi), repeat=T * k):
        idx = np.array(tab, np.int32).reshape(T, k)
        assert_matches_brute(R, E, k, Tr, idx)
        n += 1
    assert n == (hi - lo) ** (T * k)


def brute_layout_batch(R, E, k, Tr, idx):
    """The brute force over a batch of routing tables idx [N, T, k], in numpy: each table's pair
    list stably sorted by expert id (argsort, kind="stable"), segment offsets counted as the pairs
    that sort before (e, s), and each token's destination ranks as a boolean membership row."""
    N, T, _ = idx.shape
    El = E // R
    e = idx.reshape(N, T * k).astype(np.int64)
    valid = (e >= 0) & (e < E)
    src = np.arange(T * k) // k // Tr
    send_cnt = (valid[..., None] & (e[..., None] == np.arange(E))).reshape(N, R, Tr * k, E).sum(2)
    expert_off = np.concatenate([np.zeros((N, 1), np.int64), np.cumsum(send_cnt.sum(1), 1)], 1)
    ee, ss = np.arange(E)[:, None], np.arange(R)[None, :]
    e4 = e[:, :, None, None]
    before = (e4 < ee) | ((e4 == ee) & (src[None, :, None, None] < ss))
    seg_off = (before & valid[:, :, None, None]).sum(1)
    pos = np.arange(T * k)
    order = np.argsort(np.where(valid, e, E), axis=1, kind="stable")
    P = valid.sum(1)[:, None]
    pair_row = np.empty((N, T * k), np.int64)
    np.put_along_axis(pair_row, order, np.broadcast_to(pos, (N, T * k)), 1)
    pair_row[~valid] = -1
    d = np.where(valid, e // El, -1).reshape(N, T, k)
    D = (d[..., None] == np.arange(R)).any(2)  # [N, T, R]: token g sends to rank r
    Dr = D.reshape(N, R, Tr, R)
    earlier = (np.cumsum(Dr, 2) - Dr).reshape(N, T, R)  # earlier tokens of the same source rank
    slot = np.take_along_axis(earlier, np.maximum(d, 0), 2)
    return dict(send_cnt=send_cnt, rank_cnt=Dr.sum(2), expert_off=expert_off, rank_off=expert_off[:, ::El],
                seg_off=seg_off, tok_nranks=D.sum(2), pair_row=pair_row.reshape(N, T, k),
                pair_rslot=np.where(d >= 0, slot, -1), recv_src=np.where(pos < P, order // k, -1),
                recv_j=np.where(pos < P, order % k, -1), num_invalid=(~valid).sum(1))


def test_layout_exhaustive_every_table():
    """Every routing table of 2 ranks x 2 tokens, top-2 over 4 experts (2 per rank), with ids in
    {-1, 0, 1, 2, 3}: 5^8 = 390,625 tables against the batched brute force."""
    R, E, Tr, k = 2, 4, 2, 2
    T = R * Tr
    idx = (np.indices((5,) * (T * k)).reshape(T * k, -1).T - 1).astype(np.int32).reshape(-1, T, k)
    N = idx.shape[0]
    assert N == 5 ** 8
    want = brute_layout_batch(R, E, k, Tr, idx)
    sample = np.random.default_rng(5).choice(N, 300, replace=False)
    for n in sample:  # the batched form agrees with the per-table brute force
        one = brute_layout(R, E, k, Tr, idx[n])
        for name, v in one.items():
            w = want[name][n]
            if name in ("recv_src", "recv_j"):
                w = w[:len(v)]
            np.testing.assert_array_equal(np.asarray(w).reshape(np.shape(v)), v, err_msg=name)
    got = {name: np.full(v.shape, -9, np.int64) for name, v in want.items()}
    for n in range(N):
        L = oracle.layout(R, E, k, Tr, idx[n])
        for name in ("send_cnt", "rank_cnt", "expert_off", "rank_off", "seg_off", "tok_nranks", "pair_row",
                     "pair_rslot"):
            got[name][n] = getattr(L, name)
        P = L.recv_src.size
        got["recv_src"][n, :P] = L.recv_src
        got["recv_j"][n, :P] = L.recv_j
        got["recv_src"][n, P:] = got["recv_j"][n, P:] = -1
        got["num_invalid"][n] = L.num_invalid
    for name, v in want.items():
        bad = np.flatnonzero((got[name] != v).reshape(N, -1).any(1))
        assert bad.size == 0, "%s differs on %d tables, e.g. %s" % (name, bad.size, idx[bad[0]].tolist())


# ------------------------------------------------------------------ randomised shapes
@pytest.mark.parametrize("seed", range(12))
def test_layout_random_vs_brute(seed):
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.integers(1, 6))
    El = int(rng.integers(1, 4))
    E = R * El
    k = int(rng.integers(1, 7))
    Tr = int(rng.integers(0, 9))
    T = R * Tr
    idx = rng.integers(-2, E + 2, size=(T, k)).astype(np.int32)
    L = assert_matches_brute(R, E, k, Tr, idx)
    check_invariants(R, E, k, Tr, idx, L)


def np_stable_layout(R, E, k, Tr, idx):
    """Vectorised second implementation for larger sizes: numpy's stable argsort by expert id."""
    T = R * Tr
    idx = np.asarray(idx).reshape(T, k)
    flat = idx.ravel()
    valid = (flat >= 0) & (flat < E)
    pid = np.nonzero(valid)[0]
    order = pid[np.argsort(flat[pid], kind="stable")]
    pair_row = np.full(T * k, -1, np.int64)
    pair_row[order] = np.arange(order.size)
    return pair_row.reshape(T, k), order // k, order % k


@pytest.mark.parametrize("R,El,k,Tr,seed", [(8, 4, 8, 64, 0), (16, 1, 8, 40, 1), (5, 3, 5, 33, 2),
                                            (1, 64, 6, 300, 3), (32, 2, 3, 17, 4)])
def test_layout_medium_vs_numpy_sort(R, El, k, Tr, seed):
    E = R * El
    idx = W.with_replacement(seed, R * Tr, k, -1, E + 1).astype(np.int32)
    L = oracle.layout(R, E, k, Tr, idx)
    pr, src, jj = np_stable_layout(R, E, k, Tr, idx)
    np.testing.assert_array_equal(L.pair_row, pr)
    np.testing.assert_array_equal(L.recv_src, src)
    np.testing.assert_array_equal(L.recv_j, jj)
    check_invariants(R, E, k, Tr, idx, L)


# ------------------------------------------------------------------ closed forms / special cases
def test_k1_single_rank_is_stable_counting_sort():
    rng = np.random.default_rng(7)
    E, T = 13, 500
    ids = rng.integers(0, E, size=T).astype(np.int32)
    L = oracle.layout(1, E, 1, T, ids.reshape(T, 1))
    perm = np.argsort(ids, kind="stable")
    np.testing.assert_array_equal(L.recv_src, perm)
    inv = np.empty(T, np.int64)
    inv[perm] = np.arange(T)
    np.testing.assert_array_equal(L.pair_row[:, 0], inv)
    np.testing.assert_array_equal(np.diff(L.expert_off), np.bincount(ids, minlength=E))


def test_one_expert_per_rank_dedup_equals_counts():
    w = W.WORKLOADS["large_ep256"]
    idx = W.routing(w)
    L = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    np.testing.assert_array_equal(L.rank_cnt, L.send_cnt)  # El = 1: ranks are experts
    np.testing.assert_array_equal(L.tok_nranks, [len(set(r)) for r in idx.tolist()])
    assert (L.tok_nranks == 8).all()  # distinct ids, one expert per rank -> exactly k ranks


def test_every_token_hits_every_expert():
    R, El, Tr = 4, 2, 9
    E = k = R * El
    rng = np.random.default_rng(3)
    idx = np.stack([rng.permutation(E) for _ in range(R * Tr)]).astype(np.int32)
    L = oracle.layout(R, E, k, Tr, idx)
    T = R * Tr
    np.testing.assert_array_equal(np.diff(L.expert_off), np.full(E, T))
    for e in range(E):
        np.testing.assert_array_equal(L.recv_src[L.expert_off[e]:L.expert_off[e + 1]], np.arange(T))
    assert (L.tok_nranks == R).all()
    np.testing.assert_array_equal(L.rank_cnt, np.full((R, R), Tr))


def test_identical_routing_closed_form():
    R, El, k, Tr = 6, 3, 5, 7
    E = R * El
    row = np.array([4, 17, 4, 0, 9], np.int32)  # duplicate id 4 on purpose
    idx = np.tile(row, (R * Tr, 1))
    L = oracle.layout(R, E, k, Tr, idx)
    m = np.bincount(row, minlength=E)
    for e in range(E):
        for s in range(R):
            assert L.seg_off[e, s] == L.expert_off[e] + s * Tr * m[e]
    # dedup: ranks of {4, 17, 0, 9} = {1, 5, 0, 3}; every token's pairs 0 and 2 share a slot
    assert (L.tok_nranks == 4).all()
    np.testing.assert_array_equal(L.pair_rslot[:, 0], L.pair_rslot[:, 2])
    np.testing.assert_array_equal(L.pair_rslot[:Tr, 0], np.arange(Tr))


def test_empty_and_all_invalid():
    L = oracle.layout(3, 6, 4, 0, np.zeros((0, 4), np.int32))
    assert L.P == 0 and L.num_invalid == 0 and (L.send_cnt == 0).all() and (L.seg_off == 0).all()
    idx = np.full((6, 2), -1, np.int32)
    idx[1, 1] = 6  # == E, also invalid
    L = oracle.layout(3, 6, 2, 2, idx)
    assert L.P == 0 and L.num_invalid == 12
    assert (L.pair_row == -1).all() and (L.pair_rslot == -1).all() and (L.tok_nranks == 0).all()


def test_bad_shapes_rejected():
    with pytest.raises(ValueError):
        oracle.layout(3, 7, 2, 1, np.zeros((3, 2), np.int32))  # E % R != 0


# ------------------------------------------------------------------ named workloads
@pytest.mark.parametrize("name", ["tiny", "decode_ep64", "skewed_fp8_ep64", "large_ep256"])
def test_named_workload_invariants(name):
    w = W.WORKLOADS[name]
    idx = W.routing(w)
    L = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    pr, src, jj = np_stable_layout(w.R, w.E, w.k, w.Tr, idx)
    np.testing.assert_array_equal(L.pair_row, pr)
    if name == "tiny":
        check_invariants(w.R, w.E, w.k, w.Tr, idx, L)
    # statistical sanity (not parity): mean per-(rank, expert) count is Tr*k/E
    assert abs(L.send_cnt.mean() - w.Tr * w.k / w.E) < 1e-9
    assert L.num_invalid == 0 and L.P == w.T * w.k


def test_expected_distinct_ranks_uniform():
    """Mean |D(g)| under uniform routing without replacement is R*(1 - C(E-El,k)/C(E,k))."""
    from math import comb
    for name in ["tiny", "decode_ep64"]:
        w = W.WORKLOADS[name]
        L = oracle.layout(w.R, w.E, w.k, w.Tr, W.routing(w))
        El = w.E // w.R
        expect = w.R * (1 - comb(w.E - El, w.k) / comb(w.E, w.k))
        se = np.std(L.tok_nranks) / np.sqrt(w.T)
        assert abs(L.tok_nranks.mean() - expect) < 5 * se + 1e-9


def test_layout_deterministic():
    w = W.WORKLOADS["skewed_fp8_ep64"]
    idx = W.routing(w)
    a = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    b = oracle.layout(w.R, w.E, w.k, w.Tr, idx)
    for f in ["pair_row", "pair_rslot", "recv_src", "seg_off", "rank_cnt"]:
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
