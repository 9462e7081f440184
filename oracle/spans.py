"""OmniPick span plan: recent units whole, boundary tokens and sink prefixes of the image and
audio spans of older units, a shared text budget and the oldest-first trimming loop (oracle).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

Paper passages followed (Overview, key insight: the unit grammar; Structure-aware retention
planning; Applying the retention plan):
  * A unit is one streaming event: a start marker, an image span and an audio span each between
    their own open and close markers, text, and an end marker.
  * Retention starts once the history exceeds the high watermark; the low watermark is the
    trimming target.  The system prefix stays protected throughout.
  * The most recent units are kept in full.
  * Older units are visited from oldest to newest; each keeps its boundary tokens and a short
    prefix of its image span and of its audio span (candidate sinks), with separate prefix
    lengths for image and audio; the rest of its modality tokens is discarded.  Text (and
    earlier responses) is kept from oldest to newest until a shared text budget is used up.
  * If the plan still exceeds the low watermark, units are dropped oldest first, partially
    retained units before complete ones, until the target is met or only one unit remains (so
    the target is not a strict bound).
  * A partially retained unit keeps its identity with a shorter length, and its retained tokens
    move up by the deleted tokens before them (compaction, ``omnipage.compact_kv(keep_slot=...)``).

Readings where the paper is silent:
  * Tags: every token carries one modality tag; structural markers (the unit's start and end
    tokens, the open and close tokens of its image and audio spans) carry tag 4.  Units are
    contiguous slot runs in temporal order (as in the whole-unit plan).
  * A span is a maximal run of consecutive tokens of one unit with the same tag.  An older
    unit keeps every marker token, the first sink_video tokens of each video span, the first
    sink_audio tokens of each audio span, and its text tokens in slot order while the shared
    text budget lasts (used up to the token, so a text run may be cut).  A unit of one modality
    without markers is a single span, so it keeps a prefix of its slots.
  * Protected: units holding a system token (never dropped, never shortened).
  * Recent window: walking live non-system units from newest to oldest, add whole units while
    the window stays within ``recent_tokens``; stop at the first that does not fit.
  * Partially retained: 0 < kept < len.  Complete: kept == len (recent units, units whose every
    token survives the sink rules), never protected ones.  The trimming loop drops all partially
    retained units (oldest first) before any complete unit (oldest first).
  * "Only one unit remains" counts every retained unit, protected ones included; the loop also
    ends when nothing droppable is left.
  * With the history at or below the high watermark nothing is removed.
"""
from __future__ import annotations

import numpy as np

from .errors import TagError
from .omnipick import check_unit_structure

MOD_SYS, MOD_VIDEO, MOD_AUDIO, MOD_TEXT, MOD_MARK = 0, 1, 2, 3, 4


def plan_spans(modality, length, first, last, flags, low_watermark: int, high_watermark: int,
               recent_tokens: int, sink_video: int, sink_audio: int, text_budget: int):
    """Span retention plan of one segment.

    modality: per-slot tags; length, first, last, flags: per-unit structure (``score_units``).
    Returns (keep_len int64[U], keep_slot uint8[n_slots], kept_tokens int): the number of kept
    tokens of each unit (0 = unit dropped, len = unit kept whole) and which slots stay (0 for
    empty slots).  Raises TagError for a broken unit structure or a tag above 4.
    """
    modality = np.asarray(modality, np.int64)
    length = np.asarray(length, np.int64)
    first = np.asarray(first, np.int64)
    flags = np.asarray(flags, np.int64)
    n_slots = modality.shape[0]
    U = len(length)
    check_unit_structure(length, first, last)
    live = length > 0
    if np.any(live & ((first < 0) | (first + length > n_slots))):
        raise TagError("unit outside the pool")
    for u in range(U):
        if live[u] and np.any(modality[first[u]:first[u] + length[u]] > MOD_MARK):
            raise TagError(f"unit {u} holds a tag above 4")
    keep_slot = np.zeros(n_slots, np.uint8)

    def slots(u):
        return range(int(first[u]), int(first[u] + length[u]))

    total = int(length[live].sum())
    if total <= high_watermark:                      # below the high watermark: keep all
        for u in range(U):
            if live[u]:
                keep_slot[list(slots(u))] = 1
        return np.where(live, length, 0), keep_slot, total

    keep_len = np.zeros(U, np.int64)
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

    # older units, oldest to newest: boundary tokens, sink prefixes of each image and audio
    # span, text while the shared budget lasts
    kept_older = {}
    text_left = int(text_budget)
    for u in range(U):
        if not live[u] or is_sys[u] or is_recent[u]:
            continue
        chosen = []
        prev, run = -1, 0
        for s in slots(u):
            m = int(modality[s])
            run = run + 1 if m == prev else 1        # position inside the current span
            prev = m
            if m == MOD_MARK:
                chosen.append(s)
            elif m == MOD_VIDEO and run <= sink_video:
                chosen.append(s)
            elif m == MOD_AUDIO and run <= sink_audio:
                chosen.append(s)
            elif m == MOD_TEXT and text_left > 0:
                chosen.append(s)
                text_left -= 1
        kept_older[u] = chosen
        keep_len[u] = len(chosen)

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

    for u in range(U):
        if keep_len[u] == 0:
            continue
        if u in kept_older:
            keep_slot[kept_older[u]] = 1
        else:
            keep_slot[list(slots(u))] = 1
    return keep_len, keep_slot, kept
