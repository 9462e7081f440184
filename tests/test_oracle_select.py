"""Pins for the oracle's budgeted unit selection: a hand-worked plan, the unit-FIFO special case,
budget extremes, and a property checker that characterises the plan without sorting."""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import BudgetError, TagError


def _units_from_lens(lens):
    first, last, s = [], [], 0
    for n in lens:
        first.append(s if n > 0 else 10 ** 6)
        last.append(s + n - 1 if n > 0 else -1)
        s += n
    return np.array(first), np.array(last)


def test_hand_worked_example(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "select_worked_example.json")))
    score, keep, kept = oracle.select_units(g["wsum"], g["len"], g["first"], g["last"], g["flags"],
                                            g["budget"], g["recent"])
    assert score.tolist() == g["expected_score"]
    assert keep.tolist() == g["expected_keep"]
    assert kept == g["expected_kept_tokens"]


def _fifo(lens, sys_mask, budget):
    """Unit-level FIFO (the paper's `basic` baseline): protect system units, evict the oldest
    complete units until the rest fits."""
    t_sys = sum(n for n, s in zip(lens, sys_mask) if s)
    keep = [1 if s and n > 0 else 0 for n, s in zip(lens, sys_mask)]
    others = [u for u in range(len(lens)) if not sys_mask[u] and lens[u] > 0]
    # drop from the oldest until what remains fits
    i = 0
    while sum(lens[u] for u in others[i:]) > budget - t_sys:
        i += 1
    for u in others[i:]:
        keep[u] = 1
    return keep


@pytest.mark.parametrize("seed", range(20))
def test_equal_scores_reduce_to_unit_fifo(seed):
    rng = np.random.default_rng(seed)
    U = int(rng.integers(1, 40))
    lens = rng.integers(1, 60, size=U).tolist()
    sys_mask = [False] * U
    if seed % 3 == 0:
        sys_mask[0] = True
    if seed % 5 == 0:
        lens[int(rng.integers(U))] = 0          # an empty unit id
    first, last = _units_from_lens(lens)
    wsum = [7 * n for n in lens]                # every score is 7
    flags = [1 if s else 0 for s in sys_mask]
    t_sys = sum(n for n, s in zip(lens, sys_mask) if s)
    budget = t_sys + int(rng.integers(0, sum(lens) + 1))
    recent = int(rng.integers(0, 200))
    score, keep, kept = oracle.select_units(wsum, lens, first, last, flags, budget, recent)
    assert keep.tolist() == _fifo(lens, sys_mask, budget)
    assert kept == sum(n for n, k in zip(lens, keep) if k)


def test_full_budget_keeps_everything():
    lens = [5, 0, 9, 3, 12]
    first, last = _units_from_lens(lens)
    _, keep, kept = oracle.select_units([50, 0, 10, 99, 1], lens, first, last, [0] * 5, 29, 4)
    assert keep.tolist() == [1, 0, 1, 1, 1] and kept == 29


def test_system_over_budget_raises():
    lens = [10, 5]
    first, last = _units_from_lens(lens)
    with pytest.raises(BudgetError):
        oracle.select_units([0, 0], lens, first, last, [1, 0], 9, 4)


def test_ties_go_to_the_newer_unit():
    lens = [4, 6, 6, 2]
    first, last = _units_from_lens(lens)
    # units 1 and 2 tie on score; budget fits the recent unit (3) and one of them
    _, keep, _ = oracle.select_units([0, 600, 600, 2], lens, first, last, [0] * 4, 8, 2)
    assert keep.tolist() == [0, 0, 1, 1]


@pytest.mark.parametrize("case", ["gap_inside", "out_of_order"])
def test_structure_errors(case):
    lens = [3, 3]
    if case == "gap_inside":
        first, last = [0, 3], [3, 5]            # unit 0 spans 4 slots with 3 live
    else:
        first, last = [5, 0], [7, 2]            # unit 1 lies before unit 0
    with pytest.raises(TagError):
        oracle.select_units([1, 1], lens, first, last, [0, 0], 100, 1)


def _check_plan(lens, sys_mask, score, keep, budget, recent):
    """The plan's defining properties, checked pairwise (no sorting, no walk)."""
    U = len(lens)
    live = [n > 0 for n in lens]
    t_sys = sum(lens[u] for u in range(U) if sys_mask[u] and live[u])
    assert all(keep[u] for u in range(U) if sys_mask[u] and live[u])
    assert not any(keep[u] for u in range(U) if not live[u])
    kept = sum(lens[u] for u in range(U) if keep[u])
    assert kept <= budget
    # recent group: the newest non-system live units whose suffix sum fits min(R, B - T_sys)
    cap = min(recent, budget - t_sys)
    rec = set()
    for u in range(U):
        if live[u] and not sys_mask[u]:
            suffix = sum(lens[v] for v in range(u, U) if live[v] and not sys_mask[v])
            if suffix <= cap:
                rec.add(u)
    assert all(keep[u] for u in rec)
    cands = [u for u in range(U) if live[u] and not sys_mask[u] and u not in rec]

    def outranks(a, b):
        return score[a] > score[b] or (score[a] == score[b] and a > b)
    chosen = [u for u in cands if keep[u]]
    dropped = [u for u in cands if not keep[u]]
    for a in chosen:
        for b in dropped:
            assert outranks(a, b)
    if dropped:
        best = [b for b in dropped if all(outranks(b, c) for c in dropped if c != b)][0]
        assert kept + lens[best] > budget


@pytest.mark.parametrize("seed", range(30))
def test_plan_properties_random(seed):
    rng = np.random.default_rng(100 + seed)
    U = int(rng.integers(1, 60))
    lens = rng.integers(0, 50, size=U).tolist()
    sys_mask = (rng.random(U) < 0.08).tolist()
    first, last = _units_from_lens(lens)
    # many ties: few distinct score levels
    wsum = [int(n) * int(rng.integers(0, 6)) * 1000 + int(rng.integers(0, max(n, 1)))
            for n in lens]
    flags = [1 if s else 0 for s in sys_mask]
    t_sys = sum(n for n, s in zip(lens, sys_mask) if s)
    budget = t_sys + int(rng.integers(0, sum(lens) + 1))
    recent = int(rng.integers(0, 120))
    score, keep, kept = oracle.select_units(wsum, lens, first, last, flags, budget, recent)
    for u in range(U):
        assert score[u] == (wsum[u] // lens[u] if lens[u] else 0)
    _check_plan(lens, sys_mask, score.tolist(), keep.tolist(), budget, recent)
    assert kept == sum(n for n, k in zip(lens, keep) if k)
