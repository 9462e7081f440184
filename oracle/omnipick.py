"""OmniPick logical retention: unit scoring and budgeted unit selection (oracle).

Paper passages followed:
  * Overview, key insight and workflow: the unit (one streaming event's tokens with their
    modality content and structural markers) is the granularity of retention; the history is
    split into must-keep (system prefix), recent-context and selected-history groups.
  * Structure-aware retention planning: retention starts when the history exceeds the high
    watermark and trims toward the low watermark; the most recent units are kept whole;
    older units are visited and kept until a budget is used up.
  * Modality-asymmetric attention: retention priority depends on modality (separate budgets).
  * Introduction, OmniPick paragraph: after the system prefix and the recent window, the
    remaining budget is allocated by modality importance.

Readings where the paper is silent (the paper's planner is metadata-only and prints no formula):
  * Unit importance (score): the modality-weighted mean fixed-point magnitude of the unit's
    cached keys.  Per element q(x) = floor(min(|x|, 32) * 2^16) with NaN and +-Inf counted as
    32; per slot a_s = sum of q over its H_kv * d key elements; per unit
    W_u = sum over live slots of w[modality] * a_s with w in units of 1/256;
    score_u = floor(W_u / len_u).  All integer, so the result does not depend on summation order.
  * Weights: video 1.0, audio 1.5, text 2.0 (system 2.0, irrelevant because protected).
  * The budget B is a hard cap on retained history tokens (high watermark = low watermark = B).
  * Protected: units containing a system token.  If they alone exceed B: BudgetError.
  * Recent window: walking live non-system units from newest to oldest, add whole units while the
    window stays within min(R, B - T_sys); stop at the first unit that does not fit.
  * Selected history: the remaining live units ranked by (score descending, unit id descending:
    ties go to the newer unit), kept in rank order while they fit into what is left of B; stop
    at the first that does not fit.
  * Units are whole: a unit is kept entirely or not at all.
  * Structural markers (modality tag 4: a unit's start and end tokens and the open and close
    tokens of its image and audio spans, as in the paper's unit grammar) are special tokens of
    the language model's text vocabulary, so the score weighs them as text.
"""
from __future__ import annotations

import numpy as np

from .errors import BudgetError, TagError

MOD_SYS = 0
MOD_TEXT = 3
MOD_MARK = 4
N_MODALITIES = 4          # weights: system, video, audio, text
N_TAGS = 5                # modality tags: the four modalities and the structural marker
Q_CLAMP = 32.0
Q_SCALE = 65536.0


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage values as float64: bfloat16 bits (uint16) or float32."""
    if dtype == "bf16":
        bits = np.asarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def quantize_magnitude(x: np.ndarray) -> np.ndarray:
    """q(x) = floor(min(|x|, 32) * 2^16) as int64; NaN and +-Inf give 32 * 2^16."""
    return np.floor(np.fmin(np.abs(x), Q_CLAMP) * Q_SCALE).astype(np.int64)


def weights_q88(weights) -> np.ndarray:
    """Modality weights as integers in units of 1/256; each must be exact and in (0, 4]."""
    out = []
    for w in weights:
        q = float(w) * 256.0
        if q != int(q) or not (0 < q <= 1024):
            raise ValueError(f"weight {w} is not an exact multiple of 1/256 in (0, 4]")
        out.append(int(q))
    if len(out) != N_MODALITIES:
        raise ValueError("need one weight per modality")
    return np.array(out, dtype=np.int64)


def check_slot_tags(unit_id: np.ndarray, modality: np.ndarray, n_units: int) -> None:
    if np.any(unit_id < -1) or np.any(unit_id >= n_units):
        raise TagError("unit id out of range")
    if np.any(modality < 0) or np.any(modality >= N_TAGS):
        raise TagError("modality out of range")


def weight_index(m: int) -> int:
    """Weight slot of a modality tag: structural markers take the text weight."""
    return MOD_TEXT if m == MOD_MARK else int(m)


def score_units(k: np.ndarray, dtype: str, unit_id: np.ndarray, modality: np.ndarray,
                weights, n_units: int):
    """Per-unit weighted magnitude sums and structure of one segment.

    k: [n_slots, H_kv, d] storage values.  Returns a dict of per-unit arrays:
      wsum  int64  W_u
      len   int64  number of live slots of u
      first int64  smallest slot of u (n_slots if u has none)
      last  int64  largest slot of u (-1 if u has none)
      flags int64  bit 0: u holds a system token
    """
    n_slots = k.shape[0]
    unit_id = np.asarray(unit_id, np.int64)
    modality = np.asarray(modality, np.int64)
    check_slot_tags(unit_id, modality, n_units)
    wq = weights_q88(weights)
    x = to_f64(k, dtype).reshape(n_slots, -1)
    a = quantize_magnitude(x).sum(axis=1)           # per-slot magnitude sum, exact int64

    wsum = np.zeros(n_units, np.int64)
    length = np.zeros(n_units, np.int64)
    first = np.full(n_units, n_slots, np.int64)
    last = np.full(n_units, -1, np.int64)
    flags = np.zeros(n_units, np.int64)
    for s in range(n_slots):                         # one pass in slot order
        u = unit_id[s]
        if u < 0:
            continue
        wsum[u] += wq[weight_index(modality[s])] * a[s]
        length[u] += 1
        first[u] = min(first[u], s)
        last[u] = max(last[u], s)
        if modality[s] == MOD_SYS:
            flags[u] |= 1
    return {"wsum": wsum, "len": length, "first": first, "last": last, "flags": flags}


def check_unit_structure(length, first, last) -> None:
    """Each live unit is one contiguous slot run and live units appear in id (temporal) order."""
    prev_last = -1
    for u in range(len(length)):
        if length[u] <= 0:
            continue
        if last[u] - first[u] + 1 != length[u] or first[u] <= prev_last:
            raise TagError(f"unit {u} is not a contiguous run in temporal order")
        prev_last = last[u]


def select_units(wsum, length, first, last, flags, budget: int, recent: int):
    """Budgeted whole-unit retention plan of one segment.

    Returns (score int64[U], keep uint8[U], kept_tokens int).  Raises TagError or BudgetError.
    """
    length = np.asarray(length, np.int64)
    wsum = np.asarray(wsum, np.int64)
    flags = np.asarray(flags, np.int64)
    U = len(length)
    check_unit_structure(length, first, last)

    live = length > 0
    score = np.zeros(U, np.int64)
    score[live] = wsum[live] // length[live]
    is_sys = live & ((flags & 1) != 0)

    # must-keep group: the protected system units
    t_sys = int(length[is_sys].sum())
    if t_sys > budget:
        raise BudgetError(f"system tokens {t_sys} exceed budget {budget}")

    # recent-context group: newest whole units within the recent window
    cap_rec = min(recent, budget - t_sys)
    is_recent = np.zeros(U, bool)
    t_rec = 0
    for u in range(U - 1, -1, -1):
        if not live[u] or is_sys[u]:
            continue
        if t_rec + length[u] > cap_rec:
            break
        is_recent[u] = True
        t_rec += int(length[u])

    # selected-history group: remaining units by modality-weighted importance
    cands = [u for u in range(U) if live[u] and not is_sys[u] and not is_recent[u]]
    cands.sort(key=lambda u: (-int(score[u]), -u))
    cap_sel = budget - t_sys - t_rec
    chosen = np.zeros(U, bool)
    t_sel = 0
    for u in cands:
        if t_sel + length[u] > cap_sel:
            break
        chosen[u] = True
        t_sel += int(length[u])

    keep = (is_sys | is_recent | chosen).astype(np.uint8)
    return score, keep, t_sys + t_rec + t_sel
