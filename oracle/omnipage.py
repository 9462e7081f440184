"""OmniPage physical compaction of the retained history (oracle).

Paper passages followed:
  * Applying the retention plan: unselected ranges are deleted and each retained token's logical
    position is shifted down by the number of deleted tokens before it; unit records are
    updated, modality labels preserved.
  * Compaction-movement trade-off: eager compaction packs all retained KV entries into a
    contiguous prefix after an eviction.
  * Selective migration, ordered-suffix mode: packing preserves the order of the moved entries;
    with the cut point at the start of the cache it is the eager packing above.
  * Executing accepted moves: one source-to-destination map; moved entries keep their logical
    position, sequence and class.
  * Retention-aware, tile-aligned paging: pages are fixed groups of contiguous slots; the physical
    span presented to attention is rounded to whole pages.

Readings where the paper is silent:
  * Out of place: the destination is a separate pool; destination row r holds the r-th retained
    live slot in slot order; the new chunk is appended directly after, with no page padding.
  * Kept units are renumbered 0.. in temporal order; dropped units map to -1; the chunk's units
    follow the kept ones.
  * Positions: history rows take pos - (number of deleted live slots before them); chunk row i
    takes kept + i.
  * ``src_of_dst`` is the source slot of each destination row, -1 for chunk rows.
"""
from __future__ import annotations

import numpy as np

from .errors import CapacityError, TagError


def n_pages(n_ctx: int, page_size: int) -> int:
    """Pages covering n_ctx contiguous slots."""
    return -(-int(n_ctx) // int(page_size))


def page_span(n_ctx: int, page_size: int) -> int:
    """Physical span in slots: n_ctx rounded up to whole pages."""
    return n_pages(n_ctx, page_size) * int(page_size)


def compact_kv(k_src, v_src, unit_id, modality, pos, keep, n_units: int,
               k_chunk, v_chunk, chunk_modality, chunk_unit, cap_dst: int, page_size: int,
               rope=None, keep_len=None, keep_slot=None):
    """Order-preserving out-of-place packing of the kept units' rows, then the chunk.

    keep: per unit, nonzero = kept whole.  keep_len (instead of keep, which is then ignored):
    per unit, the number of its leading live slots (in slot order) that stay -- the span plan's
    partially retained units of one modality.  keep_slot (instead of both): per slot, nonzero =
    the slot's entry stays -- the span plan's retained spans inside units; a unit survives if
    any of its slots does.

    k_src/v_src: [n_slots, H_kv, d] (any dtype; rows are copied verbatim).
    Returns a dict: k, v ([n_ctx, H_kv, d]), unit_id, modality, pos, src_of_dst (per destination
    row), unit_remap [n_units], n_ctx, n_pages.

    rope: optional dict(base, dims, style, dtype) -- the keys are rotary-encoded at their
    positions; the result then also holds "k_f64": the destination keys as float64 with every
    history row re-rotated by its position shift (new - old position, see rope.shift_keys) and
    the chunk rows unchanged (they are encoded at their new positions by the caller).
    """
    unit_id = np.asarray(unit_id, np.int64)
    n_slots = unit_id.shape[0]
    if np.any(unit_id < -1) or np.any(unit_id >= n_units):
        raise TagError("unit id out of range")
    L = len(chunk_modality)

    has_rows = np.zeros(n_units, bool)
    if keep_slot is not None:
        stay = (unit_id >= 0) & (np.asarray(keep_slot) != 0)
        has_rows[unit_id[stay]] = True
        kept_unit = has_rows
    else:
        has_rows[unit_id[unit_id >= 0]] = True
        if keep_len is not None:
            quota = np.asarray(keep_len, np.int64).copy()
        else:
            quota = np.where(np.asarray(keep) != 0, np.iinfo(np.int64).max, 0)
        kept_unit = (quota > 0) & has_rows
    unit_remap = np.full(n_units, -1, np.int64)
    nxt = 0
    for u in range(n_units):
        if kept_unit[u]:
            unit_remap[u] = nxt
            nxt += 1
    n_kept_units = nxt

    rows = []
    new_pos = []
    deleted = 0
    for s in range(n_slots):
        u = unit_id[s]
        if u < 0:
            continue
        if keep_slot is not None:
            stays = bool(stay[s])
        else:
            stays = quota[u] > 0
            quota[u] -= 1 if stays else 0
        if stays:
            rows.append(s)
            new_pos.append(int(pos[s]) - deleted)
        else:
            deleted += 1
    kept = len(rows)
    n_ctx = kept + L
    if n_ctx > cap_dst:
        raise CapacityError(f"{n_ctx} rows do not fit capacity {cap_dst}")

    rows = np.array(rows, np.int64)
    k = np.concatenate([np.asarray(k_src)[rows], np.asarray(k_chunk)], axis=0)
    v = np.concatenate([np.asarray(v_src)[rows], np.asarray(v_chunk)], axis=0)
    uid = np.concatenate([unit_remap[unit_id[rows]],
                          n_kept_units + np.asarray(chunk_unit, np.int64)])
    mod = np.concatenate([np.asarray(modality, np.int64)[rows],
                          np.asarray(chunk_modality, np.int64)])
    p = np.concatenate([np.array(new_pos, np.int64), kept + np.arange(L, dtype=np.int64)])
    src = np.concatenate([rows, np.full(L, -1, np.int64)])
    out = {"k": k, "v": v, "unit_id": uid, "modality": mod, "pos": p, "src_of_dst": src,
           "unit_remap": unit_remap, "n_ctx": n_ctx, "n_pages": n_pages(n_ctx, page_size),
           "kept": kept, "n_kept_units": n_kept_units}
    if rope is not None:
        from .omnipick import to_f64
        from .rope import shift_keys
        shift = np.zeros(n_ctx, np.int64)
        shift[:kept] = p[:kept] - np.asarray(pos, np.int64)[rows]
        out["k_f64"] = shift_keys(to_f64(k, rope["dtype"]), shift, rope["base"], rope["dims"],
                                  rope["style"])
    return out
