"""Pins of the span-plan oracle (recent units whole, sink prefixes, shared text budget, oldest-first
partial-first trimming) and of compaction with partially retained units."""
import json
import os

import numpy as np
import pytest

import oracle
import streamgen as sg

SYS, VIDEO, AUDIO, TEXT = 0, 1, 2, 3


def layout_of(modality, length):
    """Contiguous unit runs in order: slot tags, first and last slot per unit."""
    length = np.asarray(length, np.int64)
    first = np.concatenate([[0], np.cumsum(length)[:-1]])
    last = first + length - 1
    unit_id = np.repeat(np.arange(len(length)), length)
    mod = np.repeat(np.asarray(modality, np.int64), length)
    return unit_id, mod, first, last


def plan(modality, length, high, low, recent, sv, sa, tb, flags=None):
    unit_id, mod, first, last = layout_of(modality, length)
    if flags is None:
        flags = (np.asarray(modality) == SYS).astype(np.int64)
    um = oracle.unit_modality(mod, first, length)
    return oracle.plan_spans(length, first, last, flags, um, low, high, recent, sv, sa, tb)


@pytest.fixture(scope="module")
def golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "span_plan_worked_example.json")))


def test_worked_examples(golden):
    for c in golden["cases"]:
        kl, kept = plan(c["modality"], c["length"], c["high"], c["low"], c["recent"],
                        c["sink_video"], c["sink_audio"], c["text_budget"])
        assert kl.tolist() == c["expected_keep_len"], c["name"]
        assert kept == c["expected_kept"], c["name"]


def test_unit_modality_is_first_token():
    mod = np.array([2, 1, 1, 3, 3, 0])
    length = np.array([1, 2, 0, 3])
    first = np.array([0, 1, 6, 3])
    assert oracle.unit_modality(mod, first, length).tolist() == [2, 1, -1, 3]


def test_compaction_of_partial_units(golden):
    g = golden["compaction"]
    n = len(g["unit_id"])
    k = np.arange(n * 2 * 4, dtype=np.float32).reshape(n, 2, 4)
    kc = -np.arange(2 * 2 * 4, dtype=np.float32).reshape(2, 2, 4) - 1
    cp = oracle.compact_kv(k, k + 0.5, g["unit_id"], g["modality"], g["pos"], None, g["n_units"],
                           kc, kc - 0.5, g["chunk_modality"], g["chunk_unit"], 100,
                           g["page_size"], keep_len=g["keep_len"])
    assert cp["src_of_dst"].tolist() == g["expected_src_of_dst"]
    assert cp["unit_id"].tolist() == g["expected_unit_id"]
    assert cp["modality"].tolist() == g["expected_modality"]
    assert cp["pos"].tolist() == g["expected_pos"]
    assert cp["unit_remap"].tolist() == g["expected_unit_remap"]
    assert cp["n_ctx"] == g["expected_n_ctx"] and cp["n_pages"] == g["expected_n_pages"]
    assert np.array_equal(cp["k"][:5], k[[0, 4, 5, 9, 10]])
    assert np.array_equal(cp["v"][:5], k[[0, 4, 5, 9, 10]] + 0.5)


def test_reduces_to_unit_fifo():
    """No sinks, no text budget and a recent window covering everything: the plan is the paper's
    unit-level FIFO -- the newest whole units whose total fits the low watermark (at least the
    newest one)."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        U = int(rng.integers(1, 12))
        length = rng.integers(1, 30, U)
        mod = rng.integers(1, 4, U)
        low = int(rng.integers(0, length.sum() + 5))
        kl, kept = plan(mod, length, 0, low, 10 ** 9, 0, 0, 0)
        suffix = np.cumsum(length[::-1])[::-1]          # tokens of u and every newer unit
        want = np.where(suffix <= low, length, 0)
        want[-1] = length[-1]
        assert kl.tolist() == want.tolist()
        assert kept == want.sum()


def test_no_op_cases():
    rng = np.random.default_rng(6)
    for _ in range(100):
        U = int(rng.integers(1, 10))
        length = rng.integers(1, 40, U)
        mod = rng.integers(0, 4, U)
        total = int(length.sum())
        # at or below the high watermark
        kl, kept = plan(mod, length, total, 0, 0, 0, 0, 0)
        assert kl.tolist() == length.tolist() and kept == total
        # above it, but sinks and text budget hold everything and the target is not exceeded
        kl, kept = plan(mod, length, total - 1, total, 0, 10 ** 6, 10 ** 6, 10 ** 6)
        assert kl.tolist() == length.tolist() and kept == total


def brute_plan(modality, length, high, low, recent, sv, sa, tb):
    """The same policy from its outcome: the candidate plans are the untrimmed plan with the
    first d units of the drop order removed, d = 0, 1, ...; the answer is the smallest d that
    meets the target, leaves one unit, or exhausts the order."""
    U = len(length)
    total = int(sum(length))
    if total <= high:
        return list(map(int, length)), total
    sys_ = [modality[u] == SYS for u in range(U)]
    base = [0] * U
    for u in range(U):
        if sys_[u]:
            base[u] = int(length[u])
    acc, rec = 0, set()
    for u in reversed(range(U)):
        if sys_[u]:
            continue
        if acc + length[u] > recent:
            break
        acc += int(length[u])
        rec.add(u)
    left = tb
    for u in range(U):
        if sys_[u]:
            continue
        if u in rec:
            base[u] = int(length[u])
        elif modality[u] == VIDEO:
            base[u] = min(int(length[u]), sv)
        elif modality[u] == AUDIO:
            base[u] = min(int(length[u]), sa)
        else:
            base[u] = min(int(length[u]), left)
            left -= base[u]
    order = ([u for u in range(U) if 0 < base[u] < length[u]] +
             [u for u in range(U) if not sys_[u] and base[u] == length[u]])
    for d in range(len(order) + 1):
        cand = list(base)
        for u in order[:d]:
            cand[u] = 0
        n_ret = sum(1 for x in cand if x > 0)
        if sum(cand) <= low or n_ret <= 1 or d == len(order):
            return cand, sum(cand)
    raise AssertionError


def test_matches_outcome_search_on_small_streams():
    rng = np.random.default_rng(7)
    for _ in range(400):
        U = int(rng.integers(1, 9))
        length = rng.integers(1, 25, U)
        mod = rng.choice([SYS, VIDEO, AUDIO, TEXT], U, p=[0.1, 0.4, 0.3, 0.2])
        total = int(length.sum())
        high = int(rng.integers(0, total + 3))
        low = int(rng.integers(0, high + 1))
        args = (high, low, int(rng.integers(0, 40)), int(rng.integers(0, 12)),
                int(rng.integers(0, 6)), int(rng.integers(0, 30)))
        kl, kept = plan(mod, length, *args)
        want, wkept = brute_plan(mod.tolist(), length.tolist(), *args)
        assert kl.tolist() == want and kept == wkept


def test_plan_invariants_on_the_80k_history():
    cfg = sg.CONFIG_BY_NAME["history_80k"]
    lay = sg.make_stream(cfg).layout
    uid = np.asarray(lay.unit_id)
    U = lay.n_units
    length = np.bincount(uid[uid >= 0], minlength=U)
    first = np.full(U, lay.n_slots)
    for s in range(lay.n_slots - 1, -1, -1):
        if uid[s] >= 0:
            first[uid[s]] = s
    last = np.full(U, -1)
    for s in range(lay.n_slots):
        if uid[s] >= 0:
            last[uid[s]] = s
    flags = np.zeros(U, np.int64)
    um = oracle.unit_modality(lay.modality, np.minimum(first, lay.n_slots - 1), length)
    kl, kept = oracle.plan_spans(length, first, last, flags, um, cfg.budget, cfg.budget,
                                 cfg.recent, 256, 16, 1024)
    assert kept == kl.sum() and kept <= cfg.budget
    assert np.all((kl >= 0) & (kl <= length))
    # some units are shortened to their sink prefix, some dropped, the newest kept whole
    part = (kl > 0) & (kl < length)
    assert part.any() and (kl[length > 0] == 0).any()
    live = np.nonzero(length > 0)[0]
    assert kl[live[-1]] == length[live[-1]]
    assert set(kl[part & (um == VIDEO)].tolist()) <= {256}
    assert set(kl[part & (um == AUDIO)].tolist()) <= {16}
    # the trimming loop ran: every dropped unit is older than every shortened one
    dropped = np.nonzero((length > 0) & (kl == 0))[0]
    assert dropped.max() < np.nonzero(part)[0].min()
