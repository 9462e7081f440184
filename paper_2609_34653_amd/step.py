"""Per-chunk stream step driver: owns the device buffers and issues the four C-ABI calls.

score -> select -> compact -> attend, all on one HIP stream with no host synchronisation inside
the step (kept_tokens and n_ctx stay on the device).  torch provides the device memory and the
stream; every computation is one of the library's kernels.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import omnitide as ot


class StreamStep:
    """Buffers for one configuration of the step.

    Pools are [n_seg, n_slots, H_kv, d]; the destination pool holds ``cap_dst`` rows
    (default budget + chunk_len, the most a step can retain).
    """

    def __init__(self, *, n_seg: int, n_slots: int, n_units: int, n_q_heads: int,
                 n_kv_heads: int, head_dim: int, chunk_len: int, budget: int, recent: int,
                 page_size: int, weights: Sequence[float], kv_dtype=torch.bfloat16,
                 cap_dst: Optional[int] = None, device="cuda"):
        self.n_seg, self.n_slots, self.n_units = n_seg, n_slots, n_units
        self.n_q_heads, self.n_kv_heads, self.head_dim = n_q_heads, n_kv_heads, head_dim
        self.chunk_len, self.budget, self.recent = chunk_len, budget, recent
        self.page_size, self.weights = page_size, tuple(weights)
        self.kv_dtype = kv_dtype
        self.cap_dst = cap_dst if cap_dst is not None else budget + chunk_len
        dev = torch.device(device)
        self.device = dev
        nu = n_seg * n_units
        i32 = dict(dtype=torch.int32, device=dev)
        self.unit_wsum = torch.zeros(nu, dtype=torch.int64, device=dev)
        self.unit_len = torch.zeros(nu, **i32)
        self.unit_first = torch.zeros(nu, **i32)
        self.unit_last = torch.zeros(nu, **i32)
        self.unit_flags = torch.zeros(nu, **i32)
        self.unit_score = torch.zeros(nu, dtype=torch.int64, device=dev)
        self.keep = torch.zeros(nu, dtype=torch.uint8, device=dev)
        self.keep_len = torch.zeros(nu, **i32)
        self.keep_slot = torch.zeros(n_seg * n_slots, dtype=torch.uint8, device=dev)
        self.span_ws = torch.zeros(max(1, ot.omnitide_plan_spans_workspace_bytes(n_seg, n_slots,
                                                                                 n_units)),
                                   dtype=torch.uint8, device=dev)
        self.kept_tokens = torch.zeros(n_seg, **i32)
        cap = self.cap_dst
        self.k_dst = torch.zeros(n_seg, cap, n_kv_heads, head_dim, dtype=kv_dtype, device=dev)
        self.v_dst = torch.zeros_like(self.k_dst)
        self.unit_id_dst = torch.zeros(n_seg * cap, **i32)
        self.modality_dst = torch.zeros(n_seg * cap, dtype=torch.uint8, device=dev)
        self.pos_dst = torch.zeros(n_seg * cap, **i32)
        self.src_of_dst = torch.zeros(n_seg * cap, **i32)
        self.unit_remap = torch.zeros(nu, **i32)
        self.n_ctx = torch.zeros(n_seg, **i32)
        self.n_pages = torch.zeros(n_seg, **i32)
        self.compact_ws = torch.zeros(max(1, ot.omnitide_compact_workspace_bytes(n_seg, n_units, cap)),
                                      dtype=torch.uint8, device=dev)
        aw = ot.omnitide_attn_workspace_bytes(
            n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim,
            dtype=ot.F32 if kv_dtype == torch.float32 else ot.BF16)
        self.attn_ws = torch.zeros(aw, dtype=torch.uint8, device=dev) if aw else None
        self.out = torch.zeros(n_seg, chunk_len, n_q_heads, head_dim, dtype=torch.float32,
                               device=dev)
        self.d_status = torch.zeros(1, **i32)

    # -- the four calls --------------------------------------------------------------------
    def score(self, k_hist, unit_id, modality, stream=None):
        ot.omnitide_score_units(k_hist, unit_id, modality, self.weights, self.n_units,
                                self.unit_wsum, self.unit_len, self.unit_first, self.unit_last,
                                self.unit_flags, self.d_status, stream)

    def select(self, stream=None):
        ot.omnitide_select_units(self.unit_wsum, self.unit_len, self.unit_first, self.unit_last,
                                 self.unit_flags, self.n_seg, self.n_units, self.budget,
                                 self.recent, self.unit_score, self.keep, self.kept_tokens,
                                 self.d_status, stream)

    def plan_spans(self, unit_id, modality, low, high, recent, sink_video, sink_audio,
                   text_budget, stream=None):
        """Span plan (recent units whole, boundary tokens and span sinks, text budget,
        trimming) into keep_len (per unit) and keep_slot (per slot); kept_tokens receives its
        total."""
        ot.omnitide_plan_spans(self.unit_len, self.unit_first, self.unit_last, self.unit_flags,
                               unit_id, modality, self.n_seg, self.n_slots, self.n_units, low,
                               high, recent, sink_video, sink_audio, text_budget, self.keep_len,
                               self.keep_slot, self.kept_tokens, self.span_ws, self.d_status,
                               stream)

    def compact_spans(self, k_hist, v_hist, unit_id, modality, pos, k_chunk, v_chunk,
                      chunk_modality, chunk_unit, stream=None, keep_slot=None, rope=None):
        """Compaction of the span plan's kept slots; rope as in ``compact``."""
        base, dims, style = rope if rope is not None else (0.0, 0, ot.ROPE_HALF)
        ot.omnitide_compact_kv_spans(
            k_hist, v_hist, self.page_size, unit_id, modality, pos,
            self.keep_slot if keep_slot is None else keep_slot, self.unit_len, self.unit_first,
            self.n_units, k_chunk, v_chunk, chunk_modality, chunk_unit, self.k_dst, self.v_dst,
            self.unit_id_dst, self.modality_dst, self.pos_dst, self.src_of_dst,
            self.unit_remap, self.n_ctx, self.n_pages, self.compact_ws, base, dims, style,
            d_status=self.d_status, stream=stream)

    def compact(self, k_hist, v_hist, unit_id, modality, pos, k_chunk, v_chunk, chunk_modality,
                chunk_unit, stream=None, keep=None, rope=None):
        """rope: optional (base, rotary dims, pairing) -- re-encode the moved keys."""
        args = (k_hist, v_hist, self.page_size, unit_id, modality, pos,
                self.keep if keep is None else keep, self.unit_len, self.unit_first, self.n_units,
                k_chunk, v_chunk, chunk_modality, chunk_unit, self.k_dst, self.v_dst,
                self.unit_id_dst, self.modality_dst, self.pos_dst, self.src_of_dst,
                self.unit_remap, self.n_ctx, self.n_pages, self.compact_ws)
        if rope is None:
            ot.omnitide_compact_kv(*args, self.d_status, stream)
        else:
            ot.omnitide_compact_kv_rope(*args, *rope, d_status=self.d_status, stream=stream)

    def attend(self, q, scale, k=None, v=None, stream=None):
        ot.omnitide_chunk_attn(q, self.k_dst if k is None else k, self.v_dst if v is None else v,
                               self.n_ctx, scale, self.out, self.attn_ws, self.d_status, stream)

    def run(self, k_hist, v_hist, unit_id, modality, pos, k_chunk, v_chunk, chunk_modality,
            chunk_unit, q, scale, stream=None):
        """One full step; asynchronous on ``stream``."""
        self.score(k_hist, unit_id, modality, stream)
        self.select(stream)
        self.compact(k_hist, v_hist, unit_id, modality, pos, k_chunk, v_chunk, chunk_modality,
                     chunk_unit, stream)
        self.attend(q, scale, stream=stream)
