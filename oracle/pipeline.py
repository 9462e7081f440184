"""One stream step in the oracle: score -> select -> compact -> attend (float64 attention).

Paper: Overview, workflow (retention fires when the history crosses the threshold, OmniPick
updates the logical cache, OmniPage lays it out, the next input is prefilled over it).  The step
order here trims first and then attends the new chunk over the trimmed history, which is the
paper's steady state (the input after a retention round sees the trimmed history).
"""
from __future__ import annotations

import numpy as np

from .attention import chunk_attention
from .omnipage import compact_kv
from .omnipick import score_units, select_units, to_f64


def stream_step(k_hist, v_hist, dtype, unit_id, modality, pos, n_units, weights, budget, recent,
                k_chunk, v_chunk, chunk_modality, chunk_unit, q, scale, cap_dst, page_size,
                attend: bool = True):
    """Storage arrays in (bf16 as uint16 bits, or float32); returns every stage's outputs."""
    sc = score_units(k_hist, dtype, unit_id, modality, weights, n_units)
    score, keep, kept_tokens = select_units(sc["wsum"], sc["len"], sc["first"], sc["last"],
                                            sc["flags"], budget, recent)
    cp = compact_kv(k_hist, v_hist, unit_id, modality, pos, keep, n_units, k_chunk, v_chunk,
                    chunk_modality, chunk_unit, cap_dst, page_size)
    out = None
    if attend:
        out = chunk_attention(to_f64(q, dtype), to_f64(cp["k"], dtype), to_f64(cp["v"], dtype),
                              scale)
    return {"score": sc, "unit_score": score, "keep": keep, "kept_tokens": kept_tokens,
            "compact": cp, "out": out}
