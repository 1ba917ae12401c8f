"""Pins of the oracle's row location (Token-level Load Partition; Algorithm 1, Quaternary Search).

The paper states the lookup on the reordered expert list itself: the count of list entries
below a pivot expert (its VectorCount) is the cumulative token count at that pivot, the expert
of a target position is the window's left end once the search converges, and the offset is the
target minus the count below that expert. These tests pin the oracle, which reads the answer
off the exclusive prefix expert_off by a linear scan, against:
* that list formulation by brute force, exhaustively over small count vectors with empty experts;
* the closed form for equal counts;
* a four-way interval search of this test's own (window invariant off[lo] <= t < off[hi],
  three cut points per step, at most ceil(log4 E) steps), on random lists with empty experts;
and show why a window of one expert needs an explicit stop (Algorithm 1's termination reading).
"""
import itertools

import numpy as np
import pytest

import oracle


def _expert_list(counts):
    """The reordered expert list: expert e repeated counts[e] times, experts ascending."""
    return np.repeat(np.arange(len(counts), dtype=np.int32), counts)


def _offsets(counts):
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


def _vector_count(lst, p):
    return int(np.count_nonzero(lst < p))


def _four_way_locate(off, t):
    """A four-way interval search over experts, written for this test from Algorithm 1's idea:
    the window [lo, hi) of experts always satisfies off[lo] <= t < off[hi]; each step cuts it
    into four parts of ceil(width / 4) experts (the last part possibly shorter) and keeps the
    part whose cumulative range holds t, reading three cut points of the prefix. It stops once
    one expert is left. Returns (expert, offset, steps)."""
    lo, hi = 0, len(off) - 1
    assert off[lo] <= t < off[hi]
    steps = 0
    while hi - lo > 1:
        width = -(-(hi - lo) // 4)
        cuts = [min(lo + i * width, hi) for i in (1, 2, 3)]
        part = sum(1 for c in cuts if off[c] <= t)  # cut points at or below the target
        bounds = [lo] + cuts + [hi]
        lo, hi = bounds[part], bounds[part + 1]
        assert off[lo] <= t < off[hi], (lo, hi, t)
        steps += 1
    return lo, t - int(off[lo]), steps


def test_exhaustive_small_lists_against_the_list_formulation():
    """Every count vector over up to 4 experts with 0..3 tokens each, every target in [-1, P]:
    the expert is the list entry at the target, the offset the number of entries before the
    first entry of that expert; outside [0, P) both are -1."""
    cases = 0
    for E in range(1, 5):
        for counts in itertools.product(range(4), repeat=E):
            lst = _expert_list(counts)
            P = lst.size
            rows = np.arange(-1, P + 1, dtype=np.int32)
            e, o = oracle.locate_rows(_offsets(counts), rows)
            for r, ge, go in zip(rows, e, o):
                if 0 <= r < P:
                    assert ge == lst[r] and go == r - _vector_count(lst, lst[r]), (counts, r)
                else:
                    assert ge == -1 and go == -1, (counts, r)
            cases += 1
    assert cases == 4 + 16 + 64 + 256


def test_dense_rows_equal_counts_closed_form():
    """c tokens per expert: the packed row r belongs to expert r // c at offset r % c."""
    for E, c in [(1, 7), (16, 1), (256, 5), (1024, 3)]:
        e, o = oracle.locate_rows(_offsets([c] * E), n=E * c + 2)
        r = np.arange(E * c)
        np.testing.assert_array_equal(e[:E * c], r // c)
        np.testing.assert_array_equal(o[:E * c], r % c)
        assert (e[E * c:] == -1).all() and (o[E * c:] == -1).all()


@pytest.mark.parametrize("seed", range(6))
def test_four_way_search_agrees(seed):
    """Random per-expert counts with about 40% of the experts empty: the four-way search keeps
    its window invariant, returns the oracle's expert and offset for every target, and needs at
    most ceil(log4(E)) steps."""
    rng = np.random.default_rng(seed)
    E = int(rng.choice([1, 2, 3, 5, 16, 63, 160, 256, 300]))
    counts = rng.integers(0, 4, E) * (rng.random(E) < 0.6)
    counts[rng.integers(0, E)] += 1  # at least one token
    off = _offsets(counts)
    P = int(off[-1])
    e, o = oracle.locate_rows(off, n=P)
    bound = int(np.ceil(np.log(E) / np.log(4) - 1e-12)) if E > 1 else 0
    for t in range(P):
        qe, qo, steps = _four_way_locate(off, t)
        assert (qe, qo) == (e[t], o[t]), (seed, t)
        assert steps <= bound, (seed, t, steps, bound)


def test_one_expert_window_needs_an_explicit_stop():
    """Algorithm 1's update recomputes its pivot spacing as ceil(width / 4) and stops only when
    the window is empty or that spacing is zero. Once the window spans one expert the spacing is
    ceil(1/4) = 1, so neither test holds and the window is mapped to itself: the reading stops the
    search at width one instead. Shown on the four-way step above, with the stop removed: from a
    one-expert window it returns the same window."""
    off = _offsets([2, 0, 3, 1])
    for lo in range(4):
        if off[lo + 1] == off[lo]:
            continue
        t = int(off[lo])
        width = -(-1 // 4)
        assert width == 1
        cuts = [min(lo + i * width, lo + 1) for i in (1, 2, 3)]
        part = sum(1 for c in cuts if off[c] <= t)
        bounds = [lo] + cuts + [lo + 1]
        assert (bounds[part], bounds[part + 1]) == (lo, lo + 1)
