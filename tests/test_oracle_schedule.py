"""Pins of the oracle's hierarchical token-level scheduling (Hierarchical Token-level Scheduling:
Latency Homogenization; Hardware-Accelerated Mapper, Expert Remapping via Logical Matrix
Transposition and Token-level Load Partition).

The remapped expert sequence is pinned against numpy's own transpose of the padded matrix, closed
forms (the divisible case, one row, more rows than experts) and a worked example derived by hand.
The schedule (equal slices of each source rank's pairs in that sequence, each slice's first expert
and offset, and its pairs per hop class) is pinned against
* a brute force over the materialised pair sequence, which assigns every position its owner from
  the inverse formula owner(p) = ceil((p+1)·n/m) − 1 (derived from the slice bounds, not retyped);
* Algorithm 1's lookup, via the separately pinned row location, on the remapped cumulative counts;
* conservation (every class's pairs land in exactly one slice), slice sizes that differ by at most
  one, and the empty cases (a rank with no pairs, more workers than pairs);
* the per-hop bound v_{j,h} <= ceil(V_h / n) in a closed-form case that meets it exactly.
"""
import itertools

import numpy as np
import pytest

import oracle


def _numpy_transpose_order(E, rows):
    c = -(-E // rows)
    cells = np.full(rows * c, -1, np.int64)
    cells[:E] = np.arange(E)
    seq = cells.reshape(rows, c).T.ravel()
    return seq[seq >= 0]


@pytest.mark.parametrize("E,rows", [(E, r) for E in (1, 2, 7, 10, 16, 64, 160, 256, 1024)
                                    for r in (1, 2, 3, 4, 5, 8, 16, 48, 64, 256, 2000)])
def test_transposed_order_is_the_matrix_read_by_columns(E, rows):
    got = oracle.transposed_order(E, rows)
    np.testing.assert_array_equal(got, _numpy_transpose_order(E, rows))
    assert sorted(got.tolist()) == list(range(E))  # a permutation


def test_transposed_order_closed_forms_and_worked_example():
    # divisible: position i holds expert (i mod rows)*(E/rows) + i div rows
    for E, rows in ((256, 4), (256, 16), (128, 8), (160, 32), (12, 3)):
        i = np.arange(E)
        np.testing.assert_array_equal(oracle.transposed_order(E, rows), (i % rows) * (E // rows) + i // rows)
    # one row, or at least as many rows as experts: the natural order
    for E in (1, 5, 256):
        np.testing.assert_array_equal(oracle.transposed_order(E, 1), np.arange(E))
        np.testing.assert_array_equal(oracle.transposed_order(E, E), np.arange(E))
        np.testing.assert_array_equal(oracle.transposed_order(E, E + 9), np.arange(E))
    # 10 experts on 3 rows of 4 columns: rows [0 1 2 3], [4 5 6 7], [8 9]; columns read top down
    assert oracle.transposed_order(10, 3).tolist() == [0, 4, 8, 1, 5, 9, 2, 6, 3, 7]


def _brute_schedule(send_cnt, order, hop, n, NH):
    R, E = send_cnt.shape
    El = E // R
    se = np.full((R, n), -1, np.int64)
    so = np.full((R, n), -1, np.int64)
    cnt = np.zeros((R, n, NH), np.int64)
    for s in range(R):
        seq = np.repeat(order, send_cnt[s, order])  # the expert of every position
        m = len(seq)
        if m == 0:
            continue
        p = np.arange(m)
        owner = -(-(p + 1) * n // m) - 1  # ceil((p+1)·n/m) − 1
        assert owner.min() >= 0 and owner.max() < n and np.all(np.diff(owner) >= 0)
        run_start = {}
        for q in range(m):
            run_start.setdefault(int(seq[q]), q)
        cls = hop[s, seq // El]
        for j in range(n):
            mine = np.nonzero(owner == j)[0]
            if mine.size == 0:
                continue
            first = int(mine[0])
            se[s, j] = seq[first]
            so[s, j] = first - run_start[int(seq[first])]
            ok = (cls[mine] >= 0) & (cls[mine] < NH)
            cnt[s, j] = np.bincount(cls[mine][ok], minlength=NH)[:NH]
    return se, so, cnt


def _random_case(rng, R, El, NH, max_cnt, zero_frac=0.3):
    E = R * El
    send = rng.integers(0, max_cnt + 1, size=(R, E)).astype(np.int32)
    send[rng.random((R, E)) < zero_frac] = 0
    hop = rng.integers(0, NH, size=(R, R)).astype(np.int32)
    return send, hop


@pytest.mark.parametrize("R,El,NH,n,max_cnt,rows", [
    (2, 2, 1, 3, 3, 3), (4, 4, 2, 5, 4, 5), (4, 4, 2, 40, 2, 40), (8, 2, 3, 7, 6, 2),
    (3, 5, 2, 4, 9, 0), (16, 4, 2, 12, 3, 12), (6, 1, 4, 1, 5, 1), (5, 3, 2, 16, 1, 4),
])
def test_schedule_against_brute_force(R, El, NH, n, max_cnt, rows):
    rng = np.random.default_rng(R * 1000 + n)
    for trial in range(4):
        send, hop = _random_case(rng, R, El, NH, max_cnt)
        E = R * El
        order = oracle.transposed_order(E, rows) if rows else rng.permutation(E).astype(np.int32)
        got = oracle.hop_schedule(send, order, hop, n, NH)
        want = _brute_schedule(send, order, hop, n, NH)
        for g, w, name in zip(got, want, ("start_expert", "start_offset", "counts")):
            np.testing.assert_array_equal(g, w, err_msg="%s trial %d" % (name, trial))


def test_schedule_conservation_and_equal_slices():
    rng = np.random.default_rng(7)
    R, El, NH = 16, 16, 3
    E = R * El
    for n in (1, 5, 48, 300):
        send, hop = _random_case(rng, R, El, NH, 6)
        order = oracle.transposed_order(E, n)
        se, so, cnt = oracle.hop_schedule(send, order, hop, n, NH)
        El_of = np.arange(E) // El
        for s in range(R):
            V = np.bincount(hop[s, El_of], weights=send[s], minlength=NH)  # pairs per class
            np.testing.assert_array_equal(cnt[s].sum(axis=0), V)
            sizes = cnt[s].sum(axis=1)
            m = int(send[s].sum())
            assert sizes.sum() == m and sizes.max() - sizes.min() <= 1
            assert set(np.unique(sizes)) <= {m // n, -(-m // n)}
            # an empty slice has no start; a non-empty one starts on an expert with pairs left
            empty = sizes == 0
            assert np.all(se[s][empty] == -1) and np.all(so[s][empty] == -1)
            assert np.all(so[s][~empty] >= 0) and np.all(so[s][~empty] < send[s, se[s][~empty]])


def test_schedule_starts_follow_algorithm_1():
    """Each slice's start is Algorithm 1's lookup of the slice's first position over the cumulative
    counts of the remapped sequence (the oracle's row location, pinned on its own)."""
    rng = np.random.default_rng(11)
    R, El, NH, n = 8, 32, 2, 48
    E = R * El
    send, hop = _random_case(rng, R, El, NH, 5, zero_frac=0.5)
    order = oracle.transposed_order(E, n)
    se, so, _ = oracle.hop_schedule(send, order, hop, n, NH)
    for s in range(R):
        m = int(send[s].sum())
        off = np.concatenate([[0], np.cumsum(send[s, order])]).astype(np.int32)
        lo = (np.arange(n, dtype=np.int64) * m) // n
        hi = (np.arange(1, n + 1, dtype=np.int64) * m) // n
        pos, off_in = oracle.locate_rows(off, lo.astype(np.int32))
        live = hi > lo
        np.testing.assert_array_equal(se[s][live], order[pos[live]])
        np.testing.assert_array_equal(so[s][live], off_in[live])


def test_schedule_empty_cases():
    R, El, NH = 4, 2, 2
    E = R * El
    send = np.zeros((R, E), np.int32)
    send[1, 3] = 2  # rank 1 sends two pairs; the others none
    hop = np.zeros((R, R), np.int32)
    hop[1, 1] = 1
    se, so, cnt = oracle.hop_schedule(send, np.arange(E, dtype=np.int32), hop, 5, NH)
    assert np.all(se[[0, 2, 3]] == -1) and np.all(cnt[[0, 2, 3]] == 0)
    # m = 2 over 5 workers: owner(p) = ceil((p+1)*5/2) - 1 gives positions 0, 1 to workers 2 and 4
    assert se[1].tolist() == [-1, -1, 3, -1, 3] and so[1].tolist() == [-1, -1, 0, -1, 1]
    assert cnt[1, :, 1].tolist() == [0, 0, 1, 0, 1]
    # a class outside [0, NH) is counted nowhere
    hop[1, 1] = 7
    _, _, cnt = oracle.hop_schedule(send, np.arange(E, dtype=np.int32), hop, 5, NH)
    assert not cnt.any()


def test_per_hop_bound_met_exactly_by_the_transposition():
    """256 experts on 64 ranks in 4 nodes of 16 ranks; a source's class-0 experts are its own
    node's 64. Every expert gets u pairs from every source, and 16 workers read a 4-row matrix:
    the sequence takes one expert from each node in turn, a slice is 32 pairs = 4 whole turns, so
    every slice holds exactly V_h / n pairs of each class: the bound ceil(V_h / n) with equality.
    In the natural order a slice lies inside one node, and the own node's slices hold 4 times the
    bound."""
    R, E, u, n = 64, 256, 2, 16
    node = np.arange(R) // 16
    hop = (node[:, None] != node[None, :]).astype(np.int32)
    send = np.full((R, E), u, np.int32)
    V = np.array([64 * u, 192 * u])
    _, _, cnt = oracle.hop_schedule(send, oracle.transposed_order(E, 4), hop, n, 2)
    assert np.all(cnt == V // n)
    _, _, nat = oracle.hop_schedule(send, np.arange(E, dtype=np.int32), hop, n, 2)
    assert nat[:, :, 0].max() == 4 * (V[0] // n)
    assert np.all(nat.sum(axis=2) == E * u // n)


def test_small_exhaustive_orders():
    """Every expert order of 4 experts on 2 ranks, every count vector in {0,1,2}^4, 3 workers."""
    R, E, n, NH = 2, 4, 3, 2
    hop = np.array([[0, 1], [1, 0]], np.int32)
    for perm in itertools.permutations(range(E)):
        order = np.array(perm, np.int32)
        for counts in itertools.product(range(3), repeat=E):
            send = np.array([counts, counts[::-1]], np.int32)
            got = oracle.hop_schedule(send, order, hop, n, NH)
            want = _brute_schedule(send, order, hop, n, NH)
            for g, w in zip(got, want):
                np.testing.assert_array_equal(g, w)


def test_transposition_evens_out_the_hop_mix_of_the_decode_layout():
    """The decode workload's own counts (64 ranks in 8 nodes of 8, 256 experts, 32 workers): the
    variance of each hop class's load across workers, summed over the classes (tr of the covariance,
    the paper's objective), falls under the transposition, and most with one matrix row per node,
    where every slice draws experts from all nodes."""
    from paper_2607_06202_amd import workloads as W

    w = W.WORKLOADS["decode_ep64"]
    ref = oracle.layout(w.R, w.E, w.k, w.Tr, W.routing(w))
    send = ref.send_cnt.reshape(w.R, w.E)
    hop = W.node_hop_classes(w.R)
    n = 32

    def tr_sigma(order):
        _, _, cnt = oracle.hop_schedule(send, order, hop, n, 2)
        np.testing.assert_array_equal(cnt.sum(axis=(1, 2)), send.sum(axis=1))  # every pair counted once
        return cnt.astype(np.float64).var(axis=1).sum(axis=1).mean()

    natural = tr_sigma(np.arange(w.E, dtype=np.int32))
    per_worker = tr_sigma(oracle.transposed_order(w.E, n))
    per_node = tr_sigma(oracle.transposed_order(w.E, w.R // 8))
    assert per_node < per_worker < natural
    assert natural > 10 * per_node
