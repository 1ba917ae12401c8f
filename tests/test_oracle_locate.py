"""Pins of the oracle's row location (Token-level Load Partition; Algorithm 1, Quaternary Search).

The paper states the lookup on the reordered expert list itself: the count of list entries
below a pivot expert (its VectorCount) is the cumulative token count at that pivot, the expert
of a target position is the window's left end once the search converges, and the offset is the
target minus the count below that expert. These tests pin the oracle, which reads the answer
off the exclusive prefix expert_off by a linear scan, against:
* that list formulation by brute force, exhaustively over small count vectors with empty experts;
* the closed form for equal counts;
* the paper's quaternary search written out step by step (three pivots per step, with the
  termination reading), on random lists with empty experts;
and show that the printed loop, taken literally, never leaves a window of one expert.
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


def _quaternary_search(lst, t, n_exp, fixed=True, max_steps=64):
    """The paper's Algorithm 1: window [L, R] over experts, pivots L + i*Gap for i = 1..3, counts
    by VectorCount, narrow to the first quadrant whose right count exceeds the target. With
    fixed=True the loop runs while the window spans more than one expert."""
    L, R, c_left = 0, n_exp, 0
    gap = -(-(R - L) // 4)
    steps = 0
    while gap >= 1 and (not fixed or R - L > 1):
        steps += 1
        if steps > max_steps:
            raise RuntimeError("window stuck at [%d, %d]" % (L, R))
        pivots = [L + i * gap for i in (1, 2, 3)]
        counts = [_vector_count(lst, p) for p in pivots]
        q = next((i for i in (1, 2, 3) if t < counts[i - 1]), 4)
        bounds = [L] + pivots + [R]
        lefts = [c_left] + counts
        L, R, c_left = bounds[q - 1], bounds[q], lefts[q - 1]
        gap = -(-(R - L) // 4)
        if R <= L or gap == 0:
            break
    return L, t - _vector_count(lst, L), steps


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
def test_paper_quaternary_search_agrees(seed):
    """Random per-expert counts with about 40% of the experts empty:
    the quaternary search, run to a one-expert window, returns the oracle's expert and offset
    for every target, in at most ceil(log4(E)) + 1 steps."""
    rng = np.random.default_rng(seed)
    E = int(rng.choice([1, 2, 3, 5, 16, 63, 160, 256, 300]))
    counts = rng.integers(0, 4, E) * (rng.random(E) < 0.6)
    counts[rng.integers(0, E)] += 1  # at least one token
    lst = _expert_list(counts)
    e, o = oracle.locate_rows(_offsets(counts), n=lst.size)
    bound = int(np.ceil(np.log(max(E, 2)) / np.log(4))) + 1
    for t in range(lst.size):
        qe, qo, steps = _quaternary_search(lst, t, E)
        assert (qe, qo) == (e[t], o[t]), (seed, t)
        assert steps <= bound


def test_printed_loop_does_not_leave_a_one_expert_window():
    """Taken literally, the loop recomputes Gap = ceil(1/4) = 1 once R - L = 1, picks the same
    quadrant again and never meets its break condition; the reading stops at R - L = 1."""
    counts = [2, 0, 3, 1]
    lst = _expert_list(counts)
    e, o = oracle.locate_rows(_offsets(counts), n=lst.size)
    for t in range(lst.size):
        with pytest.raises(RuntimeError, match="stuck"):
            _quaternary_search(lst, t, len(counts), fixed=False)
        assert _quaternary_search(lst, t, len(counts))[:2] == (e[t], o[t])
