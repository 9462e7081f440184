"""Thin Python binding of libomnitide.so (argument marshalling only).

Each function has the name of the C entry point it calls, takes torch tensors where the C
function takes device pointers, checks dtype / device / contiguity / shape, passes the current
HIP stream, and raises ``OmnitideError`` with the library's status code on failure.  Every step
of the computation runs in the HIP kernels; nothing here computes.  If the library has not been
built the first call raises (there is no fallback).

Tensor dtypes: unsigned 64-bit outputs (unit_wsum, unit_score) are held in torch.int64 tensors
and unsigned 32-bit flags in torch.int32 tensors (same bits; all values fit the signed range).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libomnitide.so")

OK, E_NULL, E_SHAPE, E_DTYPE, E_WEIGHT, E_CAPACITY, E_WORKSPACE, E_ALIAS, E_HIP, E_SCRATCH = \
    0, -1, -2, -3, -4, -5, -6, -7, -8, -9
NOALLOC_SCRATCH_BYTES = 64 << 20
E_BUDGET, E_TAGS, E_RANGE = -16, -17, -18
BF16, F32 = 0, 1
ROPE_HALF, ROPE_INTERLEAVED = 0, 1

EXPORTS = ("omnitide_score_units", "omnitide_select_units", "omnitide_compact_kv",
           "omnitide_compact_kv_rope", "omnitide_plan_spans",
           "omnitide_plan_spans_workspace_bytes", "omnitide_compact_kv_spans",
           "omnitide_compact_workspace_bytes", "omnitide_chunk_attn",
           "omnitide_chunk_attn_noalloc",
           "omnitide_attn_workspace_bytes", "omnitide_span_attn", "omnitide_evict_native",
           "omnitide_evict_native_workspace_bytes", "omnitide_evict_native_rope",
           "omnitide_evict_native_rope_workspace_bytes", "omnitide_pack_suffix",
           "omnitide_pack_suffix_workspace_bytes", "omnitide_place_chunk",
           "omnitide_place_chunk_workspace_bytes",
           "omnitide_span_attn_workspace_bytes", "omnitide_decode_attn",
           "omnitide_decode_workspace_bytes", "omnitide_decode_span_attn",
           "omnitide_decode_span_workspace_bytes", "omnitide_status_string", "omnitide_version")


class OmnitideError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} (status {code})")


_lib = None

_P = ctypes.c_void_p
_I = ctypes.c_int
_SZ = ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_34653_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        L.omnitide_score_units.argtypes = [_P, _I, _I, _I, _I, _I, _P, _P, _P, _I, _P, _P, _P,
                                           _P, _P, _P, _P]
        L.omnitide_select_units.argtypes = [_P, _P, _P, _P, _P, _I, _I, _I, _I, _P, _P, _P, _P,
                                            _P]
        L.omnitide_compact_kv.argtypes = [_P, _P, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P,
                                          _I, _P, _P, _P, _P, _I, _P, _P, _I, _P, _P, _P, _P, _P,
                                          _P, _P, _P, _SZ, _P, _P]
        L.omnitide_compact_kv_rope.argtypes = (L.omnitide_compact_kv.argtypes[:-2] +
                                               [ctypes.c_double, _I, _I, _P, _P])
        L.omnitide_compact_kv_spans.argtypes = L.omnitide_compact_kv_rope.argtypes
        L.omnitide_plan_spans.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I,
                                          _I, _I, _P, _P, _P, _P, _SZ, _P, _P]
        L.omnitide_plan_spans_workspace_bytes.argtypes = [_I, _I, _I]
        L.omnitide_plan_spans_workspace_bytes.restype = _SZ
        L.omnitide_compact_workspace_bytes.argtypes = [_I, _I, _I]
        L.omnitide_compact_workspace_bytes.restype = _SZ
        L.omnitide_chunk_attn.argtypes = [_P, _P, _P, _I, _P, _I, _I, _I, _I, _I, _I,
                                          ctypes.c_float, _P, _I, _P, _SZ, _P, _P]
        L.omnitide_chunk_attn_noalloc.argtypes = [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                                  ctypes.c_float, _P, _I, _P, _P]
        L.omnitide_attn_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I, _I]
        L.omnitide_attn_workspace_bytes.restype = _SZ
        L.omnitide_span_attn.argtypes = [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                         ctypes.c_float, _I, _P, _P, _SZ, _P, _P]
        L.omnitide_span_attn_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I]
        L.omnitide_span_attn_workspace_bytes.restype = _SZ
        L.omnitide_evict_native.argtypes = [_I, _I, _P, _P, _P, _P, _P, _I, _P, _P, _P, _P, _P,
                                            _SZ, _P, _P]
        L.omnitide_evict_native_workspace_bytes.argtypes = [_I, _I]
        L.omnitide_evict_native_workspace_bytes.restype = _SZ
        L.omnitide_evict_native_rope.argtypes = [_I, _I, _P, _P, _P, _P, _P, _I, _P, _I, _I, _I,
                                                 ctypes.c_double, _I, _I, _P, _P, _P, _P, _P,
                                                 _SZ, _P, _P]
        L.omnitide_evict_native_rope_workspace_bytes.argtypes = [_I, _I, _I]
        L.omnitide_evict_native_rope_workspace_bytes.restype = _SZ
        L.omnitide_pack_suffix.argtypes = [_P, _P, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P, _P,
                                           _P, _P, _P, _SZ, _P]
        L.omnitide_pack_suffix_workspace_bytes.argtypes = [_I, _I, _I, _I, _I]
        L.omnitide_pack_suffix_workspace_bytes.restype = _SZ
        L.omnitide_place_chunk.argtypes = [_P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P,
                                           _P, _I, _P, _P, _P, _P, _P, _SZ, _P, _P]
        L.omnitide_place_chunk_workspace_bytes.argtypes = [_I, _I]
        L.omnitide_place_chunk_workspace_bytes.restype = _SZ
        L.omnitide_decode_attn.argtypes = [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I,
                                           ctypes.c_float, _P, _P, _SZ, _P, _P]
        L.omnitide_decode_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I]
        L.omnitide_decode_workspace_bytes.restype = _SZ
        L.omnitide_decode_span_attn.argtypes = L.omnitide_span_attn.argtypes
        L.omnitide_decode_span_workspace_bytes.argtypes = [_I, _I, _I, _I, _I, _I]
        L.omnitide_decode_span_workspace_bytes.restype = _SZ
        L.omnitide_status_string.argtypes = [_I]
        L.omnitide_status_string.restype = ctypes.c_char_p
        L.omnitide_version.restype = ctypes.c_char_p
        for name in ("omnitide_score_units", "omnitide_select_units", "omnitide_compact_kv",
                     "omnitide_compact_kv_rope", "omnitide_compact_kv_spans",
                     "omnitide_plan_spans", "omnitide_chunk_attn",
                     "omnitide_chunk_attn_noalloc", "omnitide_span_attn",
                     "omnitide_evict_native", "omnitide_evict_native_rope",
                     "omnitide_pack_suffix", "omnitide_place_chunk",
                     "omnitide_decode_attn", "omnitide_decode_span_attn"):
            getattr(L, name).restype = _I
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().omnitide_status_string(int(code)).decode()


def version() -> str:
    return lib().omnitide_version().decode()


# ----------------------------------------------------------------------------- marshalling

def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _need(t: torch.Tensor, name: str, dtypes: Sequence[torch.dtype], numel: Optional[int] = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {list(dtypes)}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name}: expected {numel} elements, got {t.numel()}")


def _check(code: int, where: str):
    if code != OK:
        raise OmnitideError(code, where)


def _pool_dims(t: torch.Tensor, name: str):
    """[n_seg, n_slots, H, d] (or [n_slots, H, d] = one segment)."""
    if t.dim() == 3:
        return 1, t.shape[0], t.shape[1], t.shape[2]
    if t.dim() == 4:
        return tuple(t.shape)
    raise ValueError(f"{name} must be [n_seg, n_slots, H, d] or [n_slots, H, d]")


def _kv_dtype(t: torch.Tensor) -> int:
    return BF16 if t.dtype == torch.bfloat16 else F32


I64, I32, U8 = (torch.int64,), (torch.int32,), (torch.uint8,)


def omnitide_score_units(k, unit_id, modality, weights, n_units, unit_wsum, unit_len,
                         unit_first_slot, unit_last_slot, unit_flags, d_status=None, stream=None):
    n_seg, n_slots, H, d = _pool_dims(k, "k")
    _need(k, "k", (torch.bfloat16, torch.float32))
    _need(unit_id, "unit_id", I32, n_seg * n_slots)
    _need(modality, "modality", U8, n_seg * n_slots)
    nu = n_seg * n_units
    _need(unit_wsum, "unit_wsum", I64, nu)
    for t, nm in ((unit_len, "unit_len"), (unit_first_slot, "unit_first_slot"),
                  (unit_last_slot, "unit_last_slot"), (unit_flags, "unit_flags")):
        _need(t, nm, I32, nu)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    w = (ctypes.c_float * 4)(*[float(x) for x in weights])
    _check(lib().omnitide_score_units(_ptr(k), _kv_dtype(k), n_seg, n_slots, H, d,
                                      _ptr(unit_id), _ptr(modality), ctypes.cast(w, _P), n_units,
                                      _ptr(unit_wsum), _ptr(unit_len), _ptr(unit_first_slot),
                                      _ptr(unit_last_slot), _ptr(unit_flags), _ptr(d_status),
                                      _stream(stream)), "omnitide_score_units")


def omnitide_select_units(unit_wsum, unit_len, unit_first_slot, unit_last_slot, unit_flags,
                          n_seg, n_units, budget_tokens, recent_tokens, unit_score, keep,
                          kept_tokens, d_status=None, stream=None):
    nu = n_seg * n_units
    _need(unit_wsum, "unit_wsum", I64, nu)
    for t, nm in ((unit_len, "unit_len"), (unit_first_slot, "unit_first_slot"),
                  (unit_last_slot, "unit_last_slot"), (unit_flags, "unit_flags")):
        _need(t, nm, I32, nu)
    _need(unit_score, "unit_score", I64, nu)
    _need(keep, "keep", U8, nu)
    _need(kept_tokens, "kept_tokens", I32, n_seg)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_select_units(_ptr(unit_wsum), _ptr(unit_len), _ptr(unit_first_slot),
                                       _ptr(unit_last_slot), _ptr(unit_flags), n_seg, n_units,
                                       budget_tokens, recent_tokens, _ptr(unit_score), _ptr(keep),
                                       _ptr(kept_tokens), _ptr(d_status), _stream(stream)),
           "omnitide_select_units")


def omnitide_plan_spans_workspace_bytes(n_seg, n_slots, n_units) -> int:
    return int(lib().omnitide_plan_spans_workspace_bytes(n_seg, n_slots, n_units))


def omnitide_plan_spans(unit_len, unit_first_slot, unit_last_slot, unit_flags, unit_id, modality,
                        n_seg, n_slots, n_units, low_watermark, high_watermark, recent_tokens,
                        sink_video, sink_audio, text_budget, keep_len, keep_slot, kept_tokens,
                        workspace, d_status=None, stream=None):
    nu = n_seg * n_units
    for t, nm in ((unit_len, "unit_len"), (unit_first_slot, "unit_first_slot"),
                  (unit_last_slot, "unit_last_slot"), (unit_flags, "unit_flags"),
                  (keep_len, "keep_len")):
        _need(t, nm, I32, nu)
    _need(unit_id, "unit_id", I32, n_seg * n_slots)
    _need(modality, "modality", U8, n_seg * n_slots)
    _need(keep_slot, "keep_slot", U8, n_seg * n_slots)
    _need(kept_tokens, "kept_tokens", I32, n_seg)
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_plan_spans(_ptr(unit_len), _ptr(unit_first_slot), _ptr(unit_last_slot),
                                     _ptr(unit_flags), _ptr(unit_id), _ptr(modality), n_seg,
                                     n_slots, n_units, low_watermark, high_watermark,
                                     recent_tokens, sink_video, sink_audio, text_budget,
                                     _ptr(keep_len), _ptr(keep_slot), _ptr(kept_tokens),
                                     _ptr(workspace), workspace.numel(), _ptr(d_status),
                                     _stream(stream)),
           "omnitide_plan_spans")


def omnitide_compact_workspace_bytes(n_seg, n_units, cap_dst) -> int:
    return int(lib().omnitide_compact_workspace_bytes(n_seg, n_units, cap_dst))


def _compact_call_args(k_src, v_src, page_size, unit_id_src, modality_src, pos_src, keep,
                       unit_len, unit_first_slot, n_units, k_chunk, v_chunk, chunk_modality,
                       chunk_unit, k_dst, v_dst, unit_id_dst, modality_dst, pos_dst, src_of_dst,
                       unit_remap, n_ctx, n_pages, workspace, d_status, per_slot=False):
    """Checked C arguments shared by the compaction entry points (all but the rotary arguments
    and the stream).  `keep` is the uint8 keep flags per unit, or (per_slot) the span plan's
    uint8 keep mask per slot."""
    n_seg, n_slots, H, d = _pool_dims(k_src, "k_src")
    dt = (k_src.dtype,)
    _need(k_src, "k_src", (torch.bfloat16, torch.float32))
    _need(v_src, "v_src", dt, k_src.numel())
    ns = n_seg * n_slots
    _need(unit_id_src, "unit_id_src", I32, ns)
    _need(modality_src, "modality_src", U8, ns)
    _need(pos_src, "pos_src", I32, ns)
    nu = n_seg * n_units
    _need(keep, "keep_slot" if per_slot else "keep", U8, ns if per_slot else nu)
    _need(unit_len, "unit_len", I32, nu)
    _need(unit_first_slot, "unit_first_slot", I32, nu)
    L = 0 if chunk_modality is None else chunk_modality.numel()
    if L:
        _need(k_chunk, "k_chunk", dt, n_seg * L * H * d)
        _need(v_chunk, "v_chunk", dt, n_seg * L * H * d)
        _need(chunk_modality, "chunk_modality", U8, L)
        _need(chunk_unit, "chunk_unit", I32, L)
    ds, cap, Hd, dd = _pool_dims(k_dst, "k_dst")
    if ds != n_seg or Hd != H or dd != d:
        raise ValueError("k_dst shape does not match k_src")
    _need(k_dst, "k_dst", dt)
    _need(v_dst, "v_dst", dt, k_dst.numel())
    nd = n_seg * cap
    _need(unit_id_dst, "unit_id_dst", I32, nd)
    _need(modality_dst, "modality_dst", U8, nd)
    _need(pos_dst, "pos_dst", I32, nd)
    _need(src_of_dst, "src_of_dst", I32, nd)
    _need(unit_remap, "unit_remap", I32, nu)
    _need(n_ctx, "n_ctx", I32, n_seg)
    _need(n_pages, "n_pages", I32, n_seg)
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    return (_ptr(k_src), _ptr(v_src), _kv_dtype(k_src), n_seg, n_slots, H, d, page_size,
            _ptr(unit_id_src), _ptr(modality_src), _ptr(pos_src), _ptr(keep), _ptr(unit_len),
            _ptr(unit_first_slot), n_units, _ptr(k_chunk), _ptr(v_chunk), _ptr(chunk_modality),
            _ptr(chunk_unit), L, _ptr(k_dst), _ptr(v_dst), cap, _ptr(unit_id_dst),
            _ptr(modality_dst), _ptr(pos_dst), _ptr(src_of_dst), _ptr(unit_remap), _ptr(n_ctx),
            _ptr(n_pages), _ptr(workspace), workspace.numel())


def omnitide_compact_kv(k_src, v_src, page_size, unit_id_src, modality_src, pos_src, keep,
                        unit_len, unit_first_slot, n_units, k_chunk, v_chunk, chunk_modality,
                        chunk_unit, k_dst, v_dst, unit_id_dst, modality_dst, pos_dst, src_of_dst,
                        unit_remap, n_ctx, n_pages, workspace, d_status=None, stream=None):
    args = _compact_call_args(k_src, v_src, page_size, unit_id_src, modality_src, pos_src, keep,
                              unit_len, unit_first_slot, n_units, k_chunk, v_chunk,
                              chunk_modality, chunk_unit, k_dst, v_dst, unit_id_dst,
                              modality_dst, pos_dst, src_of_dst, unit_remap, n_ctx, n_pages,
                              workspace, d_status)
    _check(lib().omnitide_compact_kv(*args, _ptr(d_status), _stream(stream)),
           "omnitide_compact_kv")


def omnitide_compact_kv_rope(k_src, v_src, page_size, unit_id_src, modality_src, pos_src, keep,
                             unit_len, unit_first_slot, n_units, k_chunk, v_chunk,
                             chunk_modality, chunk_unit, k_dst, v_dst, unit_id_dst,
                             modality_dst, pos_dst, src_of_dst, unit_remap, n_ctx, n_pages,
                             workspace, rope_base, rope_dims, rope_style=ROPE_HALF,
                             d_status=None, stream=None):
    args = _compact_call_args(k_src, v_src, page_size, unit_id_src, modality_src, pos_src, keep,
                              unit_len, unit_first_slot, n_units, k_chunk, v_chunk,
                              chunk_modality, chunk_unit, k_dst, v_dst, unit_id_dst,
                              modality_dst, pos_dst, src_of_dst, unit_remap, n_ctx, n_pages,
                              workspace, d_status)
    _check(lib().omnitide_compact_kv_rope(*args, float(rope_base), int(rope_dims),
                                          int(rope_style), _ptr(d_status), _stream(stream)),
           "omnitide_compact_kv_rope")


def omnitide_compact_kv_spans(k_src, v_src, page_size, unit_id_src, modality_src, pos_src,
                              keep_slot, unit_len, unit_first_slot, n_units, k_chunk, v_chunk,
                              chunk_modality, chunk_unit, k_dst, v_dst, unit_id_dst,
                              modality_dst, pos_dst, src_of_dst, unit_remap, n_ctx, n_pages,
                              workspace, rope_base=0.0, rope_dims=0, rope_style=ROPE_HALF,
                              d_status=None, stream=None):
    args = _compact_call_args(k_src, v_src, page_size, unit_id_src, modality_src, pos_src,
                              keep_slot, unit_len, unit_first_slot, n_units, k_chunk, v_chunk,
                              chunk_modality, chunk_unit, k_dst, v_dst, unit_id_dst,
                              modality_dst, pos_dst, src_of_dst, unit_remap, n_ctx, n_pages,
                              workspace, d_status, per_slot=True)
    _check(lib().omnitide_compact_kv_spans(*args, float(rope_base), int(rope_dims),
                                           int(rope_style), _ptr(d_status), _stream(stream)),
           "omnitide_compact_kv_spans")


def omnitide_attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim,
                                  dtype=BF16) -> int:
    return int(lib().omnitide_attn_workspace_bytes(dtype, n_seg, cap, chunk_len, n_q_heads,
                                                   n_kv_heads, head_dim))


def omnitide_chunk_attn(q, k, v, n_ctx, scale, out, workspace=None, d_status=None, stream=None):
    """q/k/v bf16 or float32 (all the same); out float32 or bf16 (its dtype selects)."""
    if q.dim() == 3:
        n_seg, (L, Hq, d) = 1, q.shape
    else:
        n_seg, L, Hq, d = q.shape
    ds, cap, Hkv, dd = _pool_dims(k, "k")
    if ds != n_seg or dd != d:
        raise ValueError("k shape does not match q")
    _need(q, "q", (torch.bfloat16, torch.float32))
    _need(k, "k", (q.dtype,))
    _need(v, "v", (q.dtype,), k.numel())
    _need(n_ctx, "n_ctx", I32, n_seg)
    _need(out, "out", (torch.float32, torch.bfloat16), q.numel())
    if workspace is not None:
        _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_chunk_attn(_ptr(q), _ptr(k), _ptr(v), _kv_dtype(q), _ptr(n_ctx), n_seg,
                                     cap, L, Hq, Hkv, d, float(scale), _ptr(out), _kv_dtype(out),
                                     _ptr(workspace),
                                     0 if workspace is None else workspace.numel(),
                                     _ptr(d_status), _stream(stream)), "omnitide_chunk_attn")


def omnitide_chunk_attn_noalloc(q, k, v, n_ctx, scale, out, d_status=None, stream=None):
    """omnitide_chunk_attn with the library's fixed scratch (allocates nothing)."""
    if q.dim() == 3:
        n_seg, (L, Hq, d) = 1, q.shape
    else:
        n_seg, L, Hq, d = q.shape
    ds, cap, Hkv, dd = _pool_dims(k, "k")
    if ds != n_seg or dd != d:
        raise ValueError("k shape does not match q")
    _need(q, "q", (torch.bfloat16,))
    _need(k, "k", (torch.bfloat16,))
    _need(v, "v", (torch.bfloat16,), k.numel())
    _need(n_ctx, "n_ctx", I32, n_seg)
    _need(out, "out", (torch.float32, torch.bfloat16), q.numel())
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_chunk_attn_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(n_ctx), n_seg, cap,
                                             L, Hq, Hkv, d, float(scale), _ptr(out),
                                             _kv_dtype(out), _ptr(d_status), _stream(stream)),
           "omnitide_chunk_attn_noalloc")

def omnitide_span_attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads,
                                       head_dim) -> int:
    return int(lib().omnitide_span_attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads,
                                                        n_kv_heads, head_dim))


def omnitide_span_attn(q, k, v, key_pos, span, q_pos0, scale, out, workspace, d_status=None,
                       stream=None, skip_empty_tiles=True, position_order=False):
    """q [n_seg, L, Hq, d] bf16; k/v [n_seg, cap, Hkv, d] bf16; key_pos int32 [n_seg * cap]
    (-1 = empty slot); span, q_pos0 int32 [n_seg] (device); out float32 like q.
    Traversal: position_order (the entries gathered in position order; they must hold the
    positions 0 .. q_pos0 + L - 1 once each), else tile skipping if skip_empty_tiles, else the
    full span."""
    if q.dim() == 3:
        n_seg, (L, Hq, d) = 1, q.shape
    else:
        n_seg, L, Hq, d = q.shape
    ds, cap, Hkv, dd = _pool_dims(k, "k")
    if ds != n_seg or dd != d:
        raise ValueError("k shape does not match q")
    _need(q, "q", (torch.bfloat16,))
    _need(k, "k", (torch.bfloat16,))
    _need(v, "v", (torch.bfloat16,), k.numel())
    _need(key_pos, "key_pos", I32, n_seg * cap)
    _need(span, "span", I32, n_seg)
    _need(q_pos0, "q_pos0", I32, n_seg)
    _need(out, "out", (torch.float32,), q.numel())
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_span_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(key_pos), _ptr(span),
                                    _ptr(q_pos0), n_seg, cap, L, Hq, Hkv, d, float(scale),
                                    2 if position_order else 1 if skip_empty_tiles else 0,
                                    _ptr(out), _ptr(workspace),
                                    workspace.numel(),
                                    _ptr(d_status), _stream(stream)), "omnitide_span_attn")


def omnitide_decode_span_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads,
                                         head_dim) -> int:
    return int(lib().omnitide_decode_span_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads,
                                                          head_dim))


def omnitide_decode_span_attn(q, k, v, key_pos, span, q_pos0, scale, out, workspace,
                              d_status=None, stream=None, skip_empty_tiles=True,
                              position_order=False):
    """Decode attention of n_q tokens over a pool with holes: q [n_seg, n_q, Hq, d] bf16;
    k/v [n_seg, cap, Hkv, d] bf16; key_pos int32 [n_seg * cap] (-1 = empty slot); span, q_pos0
    int32 [n_seg] (device); out float32 like q.  Traversal as omnitide_span_attn."""
    if q.dim() == 3:
        n_seg, (nq, Hq, d) = 1, q.shape
    else:
        n_seg, nq, Hq, d = q.shape
    ds, cap, Hkv, dd = _pool_dims(k, "k")
    if ds != n_seg or dd != d:
        raise ValueError("k shape does not match q")
    _need(q, "q", (torch.bfloat16,))
    _need(k, "k", (torch.bfloat16,))
    _need(v, "v", (torch.bfloat16,), k.numel())
    _need(key_pos, "key_pos", I32, n_seg * cap)
    _need(span, "span", I32, n_seg)
    _need(q_pos0, "q_pos0", I32, n_seg)
    _need(out, "out", (torch.float32,), q.numel())
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_decode_span_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(key_pos), _ptr(span),
                                           _ptr(q_pos0), n_seg, cap, nq, Hq, Hkv, d,
                                           float(scale),
                                           2 if position_order else 1 if skip_empty_tiles else 0,
                                           _ptr(out),
                                           _ptr(workspace), workspace.numel(), _ptr(d_status),
                                           _stream(stream)), "omnitide_decode_span_attn")


def omnitide_evict_native_workspace_bytes(n_seg, n_units) -> int:
    return int(lib().omnitide_evict_native_workspace_bytes(n_seg, n_units))


def omnitide_evict_native(unit_id, pos, n_seg, n_units, unit_len, unit_remap, kept_tokens,
                          n_kept_units, span, workspace, keep=None, keep_len=None,
                          d_status=None, stream=None):
    """Logical eviction in place of the tags unit_id / pos ([n_seg * cap] int32)."""
    cap = unit_id.numel() // n_seg
    nu = n_seg * n_units
    _need(unit_id, "unit_id", I32, n_seg * cap)
    _need(pos, "pos", I32, n_seg * cap)
    if keep_len is not None:
        _need(keep_len, "keep_len", I32, nu)
    else:
        _need(keep, "keep", U8, nu)
    for t, nm in ((unit_len, "unit_len"), (unit_remap, "unit_remap")):
        _need(t, nm, I32, nu)
    for t, nm in ((kept_tokens, "kept_tokens"), (n_kept_units, "n_kept_units"), (span, "span")):
        _need(t, nm, I32, n_seg)
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_evict_native(n_seg, cap, _ptr(unit_id), _ptr(pos),
                                       _ptr(keep) if keep_len is None else None, _ptr(keep_len),
                                       _ptr(unit_len), n_units, _ptr(unit_remap),
                                       _ptr(kept_tokens), _ptr(n_kept_units), _ptr(span),
                                       _ptr(workspace), workspace.numel(), _ptr(d_status),
                                       _stream(stream)), "omnitide_evict_native")



def omnitide_evict_native_rope_workspace_bytes(n_seg, n_units, cap) -> int:
    return int(lib().omnitide_evict_native_rope_workspace_bytes(n_seg, n_units, cap))


def omnitide_evict_native_rope(unit_id, pos, k, n_seg, n_units, unit_len, unit_remap,
                               kept_tokens, n_kept_units, span, workspace, rope_base, rope_dims,
                               rope_style=ROPE_HALF, keep=None, keep_len=None, d_status=None,
                               stream=None):
    """Logical eviction in place plus the rotary adjustment, in place, of the keys k
    ([n_seg, cap, H, d] bf16 or float32) whose positions shift."""
    cap = unit_id.numel() // n_seg
    nu = n_seg * n_units
    ds, kcap, H, d = _pool_dims(k, "k")
    if ds != n_seg or kcap != cap:
        raise ValueError("k shape does not match the tags")
    _need(k, "k", (torch.bfloat16, torch.float32))
    _need(unit_id, "unit_id", I32, n_seg * cap)
    _need(pos, "pos", I32, n_seg * cap)
    if keep_len is not None:
        _need(keep_len, "keep_len", I32, nu)
    else:
        _need(keep, "keep", U8, nu)
    for t, nm in ((unit_len, "unit_len"), (unit_remap, "unit_remap")):
        _need(t, nm, I32, nu)
    for t, nm in ((kept_tokens, "kept_tokens"), (n_kept_units, "n_kept_units"), (span, "span")):
        _need(t, nm, I32, n_seg)
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_evict_native_rope(n_seg, cap, _ptr(unit_id), _ptr(pos),
                                            _ptr(keep) if keep_len is None else None,
                                            _ptr(keep_len), _ptr(unit_len), n_units, _ptr(k),
                                            _kv_dtype(k), H, d, float(rope_base), int(rope_dims),
                                            int(rope_style), _ptr(unit_remap), _ptr(kept_tokens),
                                            _ptr(n_kept_units), _ptr(span), _ptr(workspace),
                                            workspace.numel(), _ptr(d_status), _stream(stream)),
           "omnitide_evict_native_rope")

def omnitide_pack_suffix_workspace_bytes(dtype, n_seg, cap, n_kv_heads, head_dim) -> int:
    return int(lib().omnitide_pack_suffix_workspace_bytes(dtype, n_seg, cap, n_kv_heads,
                                                          head_dim))


def omnitide_pack_suffix(k, v, page_size, min_pages, unit_id, modality, pos, span, cut, moved,
                         workspace, stream=None):
    """Ordered-suffix packing in place of pools k/v [n_seg, cap, H, d] and their tags."""
    n_seg, cap, H, d = _pool_dims(k, "k")
    _need(k, "k", (torch.bfloat16, torch.float32))
    _need(v, "v", (k.dtype,), k.numel())
    _need(unit_id, "unit_id", I32, n_seg * cap)
    _need(modality, "modality", U8, n_seg * cap)
    _need(pos, "pos", I32, n_seg * cap)
    for t, nm in ((span, "span"), (cut, "cut"), (moved, "moved")):
        _need(t, nm, I32, n_seg)
    _need(workspace, "workspace", U8)
    _check(lib().omnitide_pack_suffix(_ptr(k), _ptr(v), _kv_dtype(k), n_seg, cap, H, d,
                                      page_size, min_pages, _ptr(unit_id), _ptr(modality),
                                      _ptr(pos), _ptr(span), _ptr(cut), _ptr(moved),
                                      _ptr(workspace), workspace.numel(), _stream(stream)),
           "omnitide_pack_suffix")


def omnitide_place_chunk_workspace_bytes(n_seg, cap) -> int:
    return int(lib().omnitide_place_chunk_workspace_bytes(n_seg, cap))


def omnitide_place_chunk(k, v, unit_id, modality, pos, k_chunk, v_chunk, chunk_modality,
                         chunk_unit, kept_tokens, n_kept_units, chunk_slot, span, workspace,
                         d_status=None, stream=None):
    """The chunk into the lowest run of empty slots of pools k/v [n_seg, cap, H, d]."""
    n_seg, cap, H, d = _pool_dims(k, "k")
    L = chunk_modality.numel()
    _need(k, "k", (torch.bfloat16, torch.float32))
    _need(v, "v", (k.dtype,), k.numel())
    _need(unit_id, "unit_id", I32, n_seg * cap)
    _need(modality, "modality", U8, n_seg * cap)
    _need(pos, "pos", I32, n_seg * cap)
    _need(k_chunk, "k_chunk", (k.dtype,), n_seg * L * H * d)
    _need(v_chunk, "v_chunk", (k.dtype,), n_seg * L * H * d)
    _need(chunk_modality, "chunk_modality", U8, L)
    _need(chunk_unit, "chunk_unit", I32, L)
    for t, nm in ((kept_tokens, "kept_tokens"), (n_kept_units, "n_kept_units"),
                  (chunk_slot, "chunk_slot"), (span, "span")):
        _need(t, nm, I32, n_seg)
    _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_place_chunk(_ptr(k), _ptr(v), _kv_dtype(k), n_seg, cap, H, d,
                                      _ptr(unit_id), _ptr(modality), _ptr(pos), _ptr(k_chunk),
                                      _ptr(v_chunk), _ptr(chunk_modality), _ptr(chunk_unit), L,
                                      _ptr(kept_tokens), _ptr(n_kept_units), _ptr(chunk_slot),
                                      _ptr(span), _ptr(workspace), workspace.numel(),
                                      _ptr(d_status), _stream(stream)),
           "omnitide_place_chunk")


def omnitide_decode_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads, head_dim) -> int:
    return int(lib().omnitide_decode_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads,
                                                     head_dim))


def omnitide_decode_attn(q, k, v, n_ctx, scale, out, workspace=None, d_status=None,
                         stream=None):
    """q [n_seg, n_q, Hq, d] bf16 (the last n_q tokens), k/v [n_seg, cap, Hkv, d] bf16,
    n_ctx int32 [n_seg] (device), out float32 like q."""
    if q.dim() == 3:
        q = q.unsqueeze(0)
    n_seg, n_q, Hq, d = q.shape
    ns, cap, Hkv, dk = _pool_dims(k, "k")
    if ns != n_seg or dk != d:
        raise ValueError("k does not match q")
    _need(q, "q", (torch.bfloat16,))
    _need(k, "k", (torch.bfloat16,))
    _need(v, "v", (torch.bfloat16,), k.numel())
    _need(n_ctx, "n_ctx", I32, n_seg)
    _need(out, "out", (torch.float32,), q.numel())
    if workspace is not None:
        _need(workspace, "workspace", U8)
    if d_status is not None:
        _need(d_status, "d_status", I32, 1)
    _check(lib().omnitide_decode_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(n_ctx), n_seg, cap, n_q,
                                      Hq, Hkv, d, float(scale), _ptr(out), _ptr(workspace),
                                      0 if workspace is None else workspace.numel(),
                                      _ptr(d_status), _stream(stream)), "omnitide_decode_attn")

