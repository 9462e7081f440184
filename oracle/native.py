"""Logical-only (native) KV layout, ordered-suffix migration and attention over a holey span
(oracle).

Test infrastructure: used only by tests, the smoke check and the CPU baseline.

Paper passages followed:
  * Applying the retention plan: unselected ranges are deleted logically; each retained token's
    logical position drops by the number of deleted tokens before it; surviving KV entries stay
    in their physical slots (migration is a separate decision).
  * Fragmentation after logical eviction: deletion leaves holes between retained entries; the
    physical span is the range of KV slots presented to attention, and a tile can be skipped
    only when every entry in it is masked.
  * Selective and efficient KV migration, ordered-suffix mode: scanning back from the end of the
    cache, find a suffix whose packing shortens the page-rounded physical span by at least a
    configured number of pages; pack only the retained entries of that suffix, keeping their
    order and leaving everything before it untouched; if no suffix qualifies, nothing moves.
    Moved entries keep their logical positions.
  * Retention-aware, tile-aligned paging: pages are fixed groups of contiguous slots.

Readings where the paper is silent:
  * A unit keeps its first keep_len[u] tokens in position order (whole-unit plans: len or 0);
    kept units are renumbered 0.. in temporal order, evicted slots get unit id -1 and
    position -1 (their K/V bytes stay and are never read as keys).
  * The new chunk goes into the lowest run of L empty slots inside the pool's capacity (the
    free space past the span end counts), with positions kept + i and unit ids after the kept
    units.
  * Span = last occupied slot + 1.  Cut c of the suffix search is any slot in [0, span]; the
    packed span of cut c is c + (live entries at or after c) when that suffix holds entries,
    else the span of what precedes c; among the cuts that save at least `min_pages` pages the
    largest is taken (fewest entries moved).  min_pages >= 1.
  * Attention over a span: chunk query i (logical position q_pos0 + i) sees slot j < span iff
    the slot holds an entry (position >= 0) whose position is <= q_pos0 + i.
"""
from __future__ import annotations

import numpy as np

from .errors import CapacityError


def evict_logical(unit_id, pos, keep_len, n_units: int, k=None, rope=None):
    """Logical eviction in place (returns new arrays).

    unit_id, pos: per-slot tags (-1 = empty).  keep_len: per unit, leading tokens (in position
    order) that stay.  Returns dict(unit_id, pos, unit_remap, kept, n_kept_units).

    rope: optional dict(base, dims, style, dtype) with k ([cap, H_kv, d] storage values, encoded
    at the old positions): the result then also holds "k_f64", the keys as float64 with every
    kept slot re-rotated by its position change (new - old position, rope.shift_keys); other
    slots are unchanged (the paper: the runtime adjusts the cached keys to the shifted
    positions, while the entries stay in their slots).
    """
    unit_id = np.asarray(unit_id, np.int64).copy()
    pos_in = pos
    pos = np.asarray(pos, np.int64).copy()
    quota = np.asarray(keep_len, np.int64).copy()
    live = np.nonzero(unit_id >= 0)[0]
    order = live[np.argsort(pos[live], kind="stable")]     # temporal order
    has_kept = np.zeros(n_units, bool)
    deleted = 0
    new_pos = {}
    for s in order:
        u = unit_id[s]
        if quota[u] > 0:
            quota[u] -= 1
            has_kept[u] = True
            new_pos[s] = pos[s] - deleted
        else:
            deleted += 1
    remap = np.full(n_units, -1, np.int64)
    nxt = 0
    for u in range(n_units):
        if has_kept[u]:
            remap[u] = nxt
            nxt += 1
    for s in live:
        if s in new_pos:
            unit_id[s] = remap[unit_id[s]]
            pos[s] = new_pos[s]
        else:
            unit_id[s] = -1
            pos[s] = -1
    out = {"unit_id": unit_id, "pos": pos, "unit_remap": remap, "kept": len(new_pos),
           "n_kept_units": nxt}
    if rope is not None:
        from .omnipick import to_f64
        from .rope import shift_keys
        old = np.asarray(pos_in, np.int64)
        shift = np.where(unit_id >= 0, pos - old, 0)
        out["k_f64"] = shift_keys(to_f64(k, rope["dtype"]), shift, rope["base"], rope["dims"],
                                  rope["style"])
    return out


def place_chunk(unit_id, chunk_len: int, cap: int) -> int:
    """Lowest slot s with [s, s + L) empty and inside [0, cap).  Raises CapacityError."""
    unit_id = np.asarray(unit_id)
    occupied = np.zeros(cap, bool)
    occupied[:len(unit_id)] = unit_id[:cap] >= 0
    run = 0
    for s in range(cap):
        run = 0 if occupied[s] else run + 1
        if run >= chunk_len:
            return s - chunk_len + 1
    if chunk_len == 0:
        return 0
    raise CapacityError(f"no run of {chunk_len} empty slots within capacity {cap}")


def span_of(unit_id) -> int:
    """Last occupied slot + 1 (0 for an empty pool)."""
    occ = np.nonzero(np.asarray(unit_id) >= 0)[0]
    return int(occ[-1]) + 1 if len(occ) else 0


def active_pages(unit_id, page_size: int) -> int:
    """Pages of `page_size` slots that hold at least one entry."""
    occ = np.nonzero(np.asarray(unit_id) >= 0)[0]
    return len(np.unique(occ // page_size))


def packed_span(live, c: int) -> int:
    """Span after packing the entries at or after slot c down to c (order kept)."""
    live = np.asarray(live, bool)
    n_suffix = int(live[c:].sum())
    if n_suffix > 0:
        return c + n_suffix
    before = np.nonzero(live[:c])[0]
    return int(before[-1]) + 1 if len(before) else 0


def plan_suffix(live, page_size: int, min_pages: int):
    """Largest cut c whose packing saves >= min_pages pages of span; (c, new span) or
    (-1, span) when no cut qualifies."""
    if min_pages < 1:
        raise ValueError("min_pages must be at least 1")
    live = np.asarray(live, bool)
    span = span_of(np.where(live, 0, -1))
    pages = lambda n: -(-n // page_size)  # noqa: E731
    for c in range(span, -1, -1):                         # scanning back from the end
        ns = packed_span(live, c)
        if pages(span) - pages(ns) >= min_pages:
            return c, ns
    return -1, span


def pack_suffix(k, v, unit_id, modality, pos, c: int):
    """Move the entries at or after slot c down to c + rank, in order; vacated slots become
    empty (K/V bytes of vacated slots are left as they were).  Returns dict(k, v, unit_id,
    modality, pos, moved) with moved = number of entries whose slot changed."""
    k = np.array(k, copy=True)
    v = np.array(v, copy=True)
    unit_id = np.array(unit_id, np.int64, copy=True)
    modality = np.array(modality, copy=True)
    pos = np.array(pos, np.int64, copy=True)
    src = [s for s in range(c, len(unit_id)) if unit_id[s] >= 0]
    rows_k = k[src].copy()
    rows_v = v[src].copy()
    tags = (unit_id[src].copy(), modality[src].copy(), pos[src].copy())
    moved = 0
    for r, s in enumerate(src):
        if c + r != s:
            moved += 1
    unit_id[c:] = -1
    pos[c:] = -1
    n = len(src)
    k[c:c + n] = rows_k
    v[c:c + n] = rows_v
    unit_id[c:c + n], modality[c:c + n], pos[c:c + n] = tags
    return {"k": k, "v": v, "unit_id": unit_id, "modality": modality, "pos": pos, "moved": moved}


def span_attention(q, k, v, key_pos, span: int, q_pos0: int, scale: float) -> np.ndarray:
    """Chunk attention over the slots [0, span) of a pool with holes, float64.

    q: [L, H_q, d]; k, v: [>= span, H_kv, d]; key_pos: per-slot logical position (-1 = empty).
    Query i sees slot j < span iff 0 <= key_pos[j] <= q_pos0 + i.  Every query must see a key.
    The K/V contents of empty slots do not enter the result.
    """
    q = np.asarray(q, np.float64)
    kp = np.asarray(key_pos, np.int64)[:span]
    empty = (kp < 0)[:, None, None]
    k = np.where(empty, 0.0, np.asarray(k, np.float64)[:span])
    v = np.where(empty, 0.0, np.asarray(v, np.float64)[:span])
    L, Hq, d = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    visible = (kp[None, :] >= 0) & (kp[None, :] <= (q_pos0 + np.arange(L))[:, None])
    if not np.all(visible.any(axis=1)):
        raise ValueError("a query sees no key")
    out = np.empty((L, Hq, d), np.float64)
    for h in range(Hq):
        g = h // group
        s = scale * (q[:, h, :] @ k[:, g, :].T)
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out
