"""Pins of the span-plan oracle (recent units whole, boundary tokens and sink prefixes of each
image and audio span, shared text budget, oldest-first partial-first trimming) and of compaction
with partially retained units (kept prefixes and per-slot masks)."""
import json
import os

import numpy as np
import pytest

import oracle
import streamgen as sg

SYS, VIDEO, AUDIO, TEXT, MARK = 0, 1, 2, 3, 4


def layout_of(modality, length):
    """Contiguous unit runs in order: slot tags, first and last slot per unit."""
    length = np.asarray(length, np.int64)
    first = np.concatenate([[0], np.cumsum(length)[:-1]])
    last = first + length - 1
    unit_id = np.repeat(np.arange(len(length)), length)
    mod = np.repeat(np.asarray(modality, np.int64), length)
    return unit_id, mod, first, last


def plan(modality, length, high, low, recent, sv, sa, tb, flags=None):
    """Plan of single-modality units; returns (keep_len, kept) and checks that the slot mask
    keeps a prefix of each unit's slots of that length."""
    unit_id, mod, first, last = layout_of(modality, length)
    if flags is None:
        flags = (np.asarray(modality) == SYS).astype(np.int64)
    kl, mask, kept = oracle.plan_spans(mod, length, first, last, flags, low, high, recent, sv,
                                       sa, tb)
    for u in range(len(length)):
        want = np.zeros(int(length[u]), np.uint8)
        want[:kl[u]] = 1
        assert mask[first[u]:first[u] + length[u]].tolist() == want.tolist()
    return kl, kept


def mixed_layout(units):
    """Units given token by token, as contiguous runs in order."""
    codes = [np.asarray(sg.unit_codes(u), np.int64) for u in units]
    length = np.array([len(c) for c in codes], np.int64)
    first = np.concatenate([[0], np.cumsum(length)[:-1]]).astype(np.int64)
    mod = np.concatenate(codes) if codes else np.zeros(0, np.int64)
    flags = np.array([int((c == SYS).any()) for c in codes], np.int64)
    return mod, length, first, first + length - 1, flags


@pytest.fixture(scope="module")
def golden(golden_dir):
    return json.load(open(os.path.join(golden_dir, "span_plan_worked_example.json")))


def test_worked_examples(golden):
    for c in golden["cases"]:
        kl, kept = plan(c["modality"], c["length"], c["high"], c["low"], c["recent"],
                        c["sink_video"], c["sink_audio"], c["text_budget"])
        assert kl.tolist() == c["expected_keep_len"], c["name"]
        assert kept == c["expected_kept"], c["name"]


def test_mixed_worked_examples(golden):
    for c in golden["mixed_cases"]:
        mod, length, first, last, flags = mixed_layout([sg.MixedUnit(tuple(u))
                                                        for u in c["units"]])
        kl, mask, kept = oracle.plan_spans(mod, length, first, last, flags, c["low"], c["high"],
                                           c["recent"], c["sink_video"], c["sink_audio"],
                                           c["text_budget"])
        assert kl.tolist() == c["expected_keep_len"], c["name"]
        assert kept == c["expected_kept"], c["name"]
        assert mask.tolist() == c["expected_keep_slot"], c["name"]


def test_mask_compaction(golden):
    g = golden["mask_compaction"]
    n = len(g["unit_id"])
    k = np.arange(n * 2 * 4, dtype=np.float32).reshape(n, 2, 4)
    kc = -np.arange(2 * 2 * 4, dtype=np.float32).reshape(2, 2, 4) - 1
    cp = oracle.compact_kv(k, k + 0.5, g["unit_id"], g["modality"], g["pos"], None, g["n_units"],
                           kc, kc - 0.5, g["chunk_modality"], g["chunk_unit"], 100,
                           g["page_size"], keep_slot=g["keep_slot"])
    assert cp["src_of_dst"].tolist() == g["expected_src_of_dst"]
    assert cp["unit_id"].tolist() == g["expected_unit_id"]
    assert cp["modality"].tolist() == g["expected_modality"]
    assert cp["pos"].tolist() == g["expected_pos"]
    assert cp["unit_remap"].tolist() == g["expected_unit_remap"]
    assert cp["n_ctx"] == g["expected_n_ctx"] and cp["n_pages"] == g["expected_n_pages"]
    assert np.array_equal(cp["k"][:3], k[[0, 1, 9]])


def test_mask_of_prefixes_equals_kept_prefixes():
    """A mask that keeps the first keep_len slots of every unit compacts exactly like keep_len."""
    rng = np.random.default_rng(11)
    for _ in range(50):
        units = sg.random_mixed_units(rng, int(rng.integers(1, 12)), hi=20)
        lay = sg.build_layout(units, [(AUDIO, 3)], set(rng.choice(len(units), len(units) // 4,
                                                                   replace=False).tolist()))
        uid = lay.unit_id.astype(np.int64)
        U = lay.n_units
        length = np.bincount(uid[uid >= 0], minlength=U)
        kl = np.array([int(rng.integers(0, n + 1)) for n in length])
        mask = np.zeros(lay.n_slots, np.uint8)
        seen = np.zeros(U, np.int64)
        for s in range(lay.n_slots):
            if uid[s] >= 0:
                mask[s] = seen[uid[s]] < kl[uid[s]]
                seen[uid[s]] += 1
        k = rng.standard_normal((lay.n_slots, 1, 4)).astype(np.float32)
        kc = np.zeros((3, 1, 4), np.float32)
        args = (k, k, lay.unit_id, lay.modality, lay.pos, None, U, kc, kc, lay.chunk_modality,
                lay.chunk_unit, 10 ** 6, 8)
        a = oracle.compact_kv(*args, keep_len=kl)
        b = oracle.compact_kv(*args, keep_slot=mask)
        for key in ("src_of_dst", "unit_id", "modality", "pos", "unit_remap"):
            assert a[key].tolist() == b[key].tolist(), key
        assert a["n_ctx"] == b["n_ctx"]


def older_selection(mod, length, first, flags, recent, sv, sa, tb):
    """The sink-phase selection of every older unit, written as prefix operations over slots
    (independent of the oracle's per-unit walk): a slot starts a span where its unit starts or
    its tag changes; its place in the span is its distance from the latest start; text slots of
    older units are ranked by an exclusive running count."""
    n = len(mod)
    U = len(length)
    uid = np.full(n, -1)
    for u in range(U):
        uid[first[u]:first[u] + length[u]] = u
    live = length > 0
    is_sys = live & (flags & 1 != 0)
    elig = np.where(live & ~is_sys, length, 0)
    suffix = np.cumsum(elig[::-1])[::-1]           # eligible tokens of u and every newer unit
    recent_u = live & ~is_sys & (suffix <= recent)
    older_u = live & ~is_sys & ~recent_u
    idx = np.arange(n)
    starts = np.ones(n, bool)
    starts[1:] = (mod[1:] != mod[:-1]) | (uid[1:] != uid[:-1])
    run_pos = idx - np.maximum.accumulate(np.where(starts, idx, 0)) + 1
    older_slot = (uid >= 0) & older_u[np.maximum(uid, 0)]
    older_text = older_slot & (mod == TEXT)
    rank = np.cumsum(older_text) - older_text
    keep = older_slot & ((mod == MARK) | ((mod == VIDEO) & (run_pos <= sv)) |
                         ((mod == AUDIO) & (run_pos <= sa)) | (older_text & (rank < tb)))
    return uid, is_sys, recent_u, older_u, keep


def test_mixed_plan_matches_outcome_search():
    """Random mixed streams: the sink-phase selection from prefix operations, then the trimming
    rule from its outcome (the smallest number of drops along the drop order that meets the
    target, leaves one unit, or exhausts the order), equal the oracle's plan and mask."""
    rng = np.random.default_rng(12)
    for _ in range(300):
        units = sg.random_mixed_units(rng, int(rng.integers(1, 9)), hi=16,
                                      sys_prefix=int(rng.integers(0, 2)) * 5)
        mod, length, first, last, flags = mixed_layout(units)
        total = int(length.sum())
        high = int(rng.integers(0, total + 3))
        low = int(rng.integers(0, high + 1))
        recent, sv, sa, tb = (int(rng.integers(0, 40)), int(rng.integers(0, 6)),
                              int(rng.integers(0, 4)), int(rng.integers(0, 20)))
        kl, mask, kept = oracle.plan_spans(mod, length, first, last, flags, low, high, recent,
                                           sv, sa, tb)
        if total <= high:
            assert kl.tolist() == length.tolist() and mask.all() and kept == total
            continue
        uid, is_sys, recent_u, older_u, sel = older_selection(mod, length, first, flags, recent,
                                                             sv, sa, tb)
        base = np.where(is_sys | recent_u, length, 0)
        for u in np.nonzero(older_u)[0]:
            base[u] = sel[uid == u].sum()
        order = ([u for u in range(len(length)) if 0 < base[u] < length[u]] +
                 [u for u in range(len(length)) if length[u] > 0 and not is_sys[u]
                  and base[u] == length[u]])
        for d in range(len(order) + 1):
            cand = base.copy()
            cand[order[:d]] = 0
            if cand.sum() <= low or (cand > 0).sum() <= 1 or d == len(order):
                break
        assert kl.tolist() == cand.tolist() and kept == cand.sum()
        whole = (uid >= 0) & (is_sys | recent_u)[np.maximum(uid, 0)]
        want = ((whole | sel) & (uid >= 0) & (cand[np.maximum(uid, 0)] > 0)).astype(np.uint8)
        assert mask.tolist() == want.tolist()


def test_mixed_plan_on_the_grammar_80k_history():
    """The 80K history with each second as one grammar unit: every surviving partial unit keeps
    all its markers, at most 256 tokens of its image span and 16 of its audio span."""
    cfg = sg.CONFIG_BY_NAME["history_80k"]
    lay = sg.make_stream(cfg, grammar=True).layout
    uid = lay.unit_id.astype(np.int64)
    mod = lay.modality.astype(np.int64)
    U = lay.n_units
    length = np.bincount(uid[uid >= 0], minlength=U)
    first = np.array([np.nonzero(uid == u)[0][0] for u in range(U)])
    last = first + length - 1
    kl, mask, kept = oracle.plan_spans(mod, length, first, last, np.zeros(U, np.int64),
                                       cfg.budget, cfg.budget, cfg.recent, 256, 16, 1024)
    assert kept == kl.sum() == mask.sum() and kept <= cfg.budget
    part = np.nonzero((kl > 0) & (kl < length))[0]
    assert len(part) > 0 and (kl == 0).any()
    for u in part:
        m = mod[first[u]:last[u] + 1]
        k = mask[first[u]:last[u] + 1].astype(bool)
        assert k[m == MARK].all()
        assert 0 < k[m == VIDEO].sum() <= 256 or not (m == VIDEO).any()
        assert k[m == AUDIO].sum() == min(16, (m == AUDIO).sum())


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
    um = np.array([lay.modality[first[u]] if length[u] else -1 for u in range(U)])
    kl, _, kept = oracle.plan_spans(lay.modality, length, first, last, flags, cfg.budget,
                                    cfg.budget, cfg.recent, 256, 16, 1024)
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
