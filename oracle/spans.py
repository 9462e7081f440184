"""OmniPick span plan: recent units whole, sink prefixes of older units, a shared text budget and
the oldest-first trimming loop (oracle).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

Paper passages followed (Structure-aware retention planning, and Applying the retention plan):
  * Retention starts once the history exceeds the high watermark; the low watermark is the
    trimming target.  The system prefix stays protected throughout.
  * The most recent units are kept in full.
  * Older units are visited from oldest to newest; each keeps its boundary tokens and a short
    prefix of its image span and of its audio span (candidate sinks), with separate prefix
    lengths for image and audio; the rest of its modality tokens is discarded.  Text is kept
    from oldest to newest until a shared text budget is used up.
  * If the plan still exceeds the low watermark, units are dropped oldest first, partially
    retained units before complete ones, until the target is met or only one unit remains (so
    the target is not a strict bound).
  * A partially retained unit keeps its identity with a shorter length; its kept tokens move up
    by the deleted tokens before them (compaction, ``omnipage.compact_kv(keep_len=...)``).

Readings where the paper is silent:
  * Units are contiguous slot runs (as in the whole-unit plan).  A unit's retention class is the
    modality of its first token: the tag format carries no boundary-marker tokens, and the
    synthetic streams encode each second as one video unit and one audio unit, so a unit's
    sink prefix (its first tokens) is where its unit-start and modality-boundary tokens sit.
    A partially kept unit therefore keeps a prefix of its slots.
  * Protected: units holding a system token (never dropped, never shortened).
  * Recent window: walking live non-system units from newest to oldest, add whole units while
    the window stays within ``recent_tokens``; stop at the first that does not fit.
  * Older video units keep min(len, sink_video) tokens, audio units min(len, sink_audio); text
    units take min(len, what is left of text_budget) in oldest-first order, so the budget is
    used up to the token and the last text unit it reaches may be cut to a prefix.
  * Partially retained: 0 < kept < len.  Complete: kept == len (recent units, fully kept text,
    units shorter than their sink prefix), never protected ones.  The trimming loop drops all
    partially retained units (oldest first) before any complete unit (oldest first).
  * "Only one unit remains" counts every retained unit, protected ones included; the loop also
    ends when nothing droppable is left.
  * With the history at or below the high watermark nothing is removed.
"""
from __future__ import annotations

import numpy as np

from .omnipick import check_unit_structure

MOD_SYS, MOD_VIDEO, MOD_AUDIO, MOD_TEXT = 0, 1, 2, 3


def unit_modality(modality, first, length) -> np.ndarray:
    """Retention class of each live unit: the modality of its first slot (-1 without slots)."""
    modality = np.asarray(modality, np.int64)
    out = np.full(len(length), -1, np.int64)
    for u in range(len(length)):
        if length[u] > 0:
            out[u] = modality[first[u]]
    return out


def plan_spans(length, first, last, flags, unit_mod, low_watermark: int, high_watermark: int,
               recent_tokens: int, sink_video: int, sink_audio: int, text_budget: int):
    """Span retention plan of one segment.

    length, first, last, flags: per-unit structure (``score_units``); unit_mod: retention class
    per unit (``unit_modality``).  Returns (keep_len int64[U], kept_tokens int): the number of
    leading tokens of each unit that stay (0 = unit dropped, len = unit kept whole).
    Raises TagError for a broken unit structure.
    """
    length = np.asarray(length, np.int64)
    flags = np.asarray(flags, np.int64)
    U = len(length)
    check_unit_structure(length, first, last)
    live = length > 0
    keep_len = np.zeros(U, np.int64)

    total = int(length[live].sum())
    if total <= high_watermark:                      # below the high watermark: keep all
        keep_len[live] = length[live]
        return keep_len, total

    is_sys = live & ((flags & 1) != 0)
    keep_len[is_sys] = length[is_sys]                # system prefix, protected

    # recent units, kept in full
    is_recent = np.zeros(U, bool)
    t_rec = 0
    for u in range(U - 1, -1, -1):
        if not live[u] or is_sys[u]:
            continue
        if t_rec + length[u] > recent_tokens:
            break
        is_recent[u] = True
        t_rec += int(length[u])
        keep_len[u] = length[u]

    # older units, oldest to newest: sink prefixes per modality, text under a shared budget
    text_left = int(text_budget)
    for u in range(U):
        if not live[u] or is_sys[u] or is_recent[u]:
            continue
        m = unit_mod[u]
        if m == MOD_VIDEO:
            keep_len[u] = min(int(length[u]), int(sink_video))
        elif m == MOD_AUDIO:
            keep_len[u] = min(int(length[u]), int(sink_audio))
        elif m == MOD_TEXT:
            take = min(int(length[u]), text_left)
            keep_len[u] = take
            text_left -= take

    # trimming toward the low watermark
    kept = int(keep_len.sum())
    partial = [u for u in range(U) if 0 < keep_len[u] < length[u]]
    complete = [u for u in range(U) if live[u] and not is_sys[u] and keep_len[u] == length[u]]
    retained = int((keep_len > 0).sum())
    for u in partial + complete:
        if kept <= low_watermark or retained <= 1:
            break
        kept -= int(keep_len[u])
        keep_len[u] = 0
        retained -= 1
    return keep_len, kept
