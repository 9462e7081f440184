"""Seeded synthetic omni-modal streams: the only module shared by the oracle and the HIP path.

It draws the structure of a stream (which units exist, their modality and length, which were
already evicted) and the random tensor values (keys, values, queries). It holds none of the
method's arithmetic: no score, no selection, no compaction, no attention.

Stream shapes follow the paper's description of its workloads (Background, Table of token counts:
640- or 2,304-token frames, 25 audio tokens per second, sparse text; Motivation: a 375-s video as
75 five-second chunks, about 80K tokens). The benchmark suites the paper evaluates on are not
used; these seeded streams stand in for them.

Draw order for one segment (layer), from ``numpy.random.default_rng(seed)``:
  1. structure draws (text lengths and seconds, frame sizes, evicted units), from the stream seed;
  2. per-unit scalar K offsets N(0, 0.5^2) for history units then chunk units,
     then per-unit V offsets in the same order;
  3. K history, V history, K chunk, V chunk as N(0, 1) float32 plus the unit's offset;
  4. Q as N(0, 1) float32.
Float32 draws are cast to bfloat16 with round-to-nearest-even (torch's CPU cast).
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Tuple

import numpy as np
import torch

MOD_SYS, MOD_VIDEO, MOD_AUDIO, MOD_TEXT, MOD_MARK = 0, 1, 2, 3, 4
MODALITY_NAMES = {MOD_SYS: "sys", MOD_VIDEO: "video", MOD_AUDIO: "audio", MOD_TEXT: "text",
                  MOD_MARK: "marker"}

# Modality importance weights (video 1.0, audio 1.5, text 2.0; system tokens are protected,
# their weight is irrelevant and set to 2.0).  Index = modality tag.
DEFAULT_WEIGHTS = (2.0, 1.0, 1.5, 2.0)


@dataclasses.dataclass(frozen=True)
class StreamConfig:
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                 # "f32" or "bf16": storage type of the KV pool
    page_size: int
    budget: int                # retained-history token budget B
    recent: int                # recent-window token cap R
    n_layers: int              # segments
    seed: int
    description: str
    weights: Tuple[float, float, float, float] = DEFAULT_WEIGHTS
    evict_frac: float = 0.0    # fraction of history units already evicted (holes)
    steps: int = 0             # stream-loop steps (loop config only)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


CONFIGS: List[StreamConfig] = [
    StreamConfig("tiny_1p6k_f32", 4, 1, 64, "f32", 64, 512, 89, 1, 0,
                 "18 s of [video 64 + audio 25] + text 32 = 1,634 tokens, chunk 89, budget 512"),
    StreamConfig("single_layer_8k", 32, 8, 128, "bf16", 64, 4096, 665, 1, 1,
                 "12 s of [video 640 + audio 25] + 212 text = 8,192 tokens, chunk 665, budget 4,096"),
    StreamConfig("hires_32k_36layer", 32, 8, 128, "bf16", 128, 8192, 2329, 36, 2,
                 "14 s of [video 2,304 + audio 25] + 162 text = 32,768 tokens x 36 layers, "
                 "chunk 2,329, budget 8,192"),
    StreamConfig("history_80k", 32, 8, 128, "bf16", 256, 16384, 665, 1, 3,
                 "375 s: 75 frames (61x640 + 14x2,304) + 375x25 audio + 1,249 text = 81,920 slots, "
                 "30% of units already evicted, chunk 665, budget 16,384", evict_frac=0.30),
    StreamConfig("stream_loop_64x665", 32, 8, 128, "bf16", 64, 16384, 665, 1, 4,
                 "prefill 16,384 (24 s of [video 640 + audio 25] + 424 text), then 64 steps of a "
                 "665-token chunk, budget 16,384", steps=64),
]
CONFIG_BY_NAME = {c.name: c for c in CONFIGS}


# ----------------------------------------------------------------------------- structure

def split_total(rng: np.random.Generator, total: int, lo: int = 16, hi: int = 64,
                n: Optional[int] = None) -> List[int]:
    """Seeded lengths in [lo, hi] that sum exactly to ``total`` (``n`` parts, else about 40 each)."""
    if n is None:
        n = max(math.ceil(total / hi), int(round(total / 40)))
    if n * lo > total or n * hi < total:
        raise ValueError(f"cannot split {total} into {n} parts in [{lo}, {hi}]")
    lens = [lo] * n
    rest = total - n * lo
    while rest > 0:
        open_idx = [i for i in range(n) if lens[i] < hi]
        i = open_idx[int(rng.integers(len(open_idx)))]
        lens[i] += 1
        rest -= 1
    return lens


def _with_text(rng, per_second: List[List[Tuple[int, int]]], text_total: int,
               n_text: Optional[int] = None):
    """Insert text units summing to ``text_total`` after the content of seeded seconds."""
    lens = split_total(rng, text_total, n=n_text)
    secs = np.sort(rng.choice(len(per_second), size=len(lens), replace=False))
    units = []
    ti = 0
    for t, content in enumerate(per_second):
        units.extend(content)
        while ti < len(lens) and secs[ti] == t:
            units.append((MOD_TEXT, lens[ti]))
            ti += 1
    return units


def stream_units(cfg: StreamConfig, rng: np.random.Generator):
    """History units [(modality, length)] in temporal order and the chunk's units."""
    if cfg.seed == 0:
        units = []
        for _ in range(18):
            units += [(MOD_VIDEO, 64), (MOD_AUDIO, 25)]
        units.append((MOD_TEXT, 32))
        chunk = [(MOD_VIDEO, 64), (MOD_AUDIO, 25)]
    elif cfg.seed == 1:
        units = _with_text(rng, [[(MOD_VIDEO, 640), (MOD_AUDIO, 25)] for _ in range(12)], 212, 4)
        chunk = [(MOD_VIDEO, 640), (MOD_AUDIO, 25)]
    elif cfg.seed == 2:
        units = _with_text(rng, [[(MOD_VIDEO, 2304), (MOD_AUDIO, 25)] for _ in range(14)], 162)
        chunk = [(MOD_VIDEO, 2304), (MOD_AUDIO, 25)]
    elif cfg.seed == 3:
        big = set(rng.choice(75, size=14, replace=False).tolist())
        per_second = []
        for t in range(375):
            content = []
            if t % 5 == 0:
                content.append((MOD_VIDEO, 2304 if (t // 5) in big else 640))
            content.append((MOD_AUDIO, 25))
            per_second.append(content)
        units = _with_text(rng, per_second, 1249)
        chunk = [(MOD_VIDEO, 640), (MOD_AUDIO, 25)]
    elif cfg.seed == 4:
        units = _with_text(rng, [[(MOD_VIDEO, 640), (MOD_AUDIO, 25)] for _ in range(24)], 424)
        chunk = [(MOD_VIDEO, 640), (MOD_AUDIO, 25)]
    else:
        raise ValueError(cfg.seed)
    return units, chunk


@dataclasses.dataclass(frozen=True)
class MixedUnit:
    """A unit given token by token: one modality tag per token (tag 4 = structural marker)."""
    codes: Tuple[int, ...]


def grammar_unit(n_video: int, n_audio: int, n_text: int) -> MixedUnit:
    """A unit in the paper's grammar (Overview, key insight): a start marker, the image span
    between its open and close markers, the audio span between its own markers, text, and an
    end marker.  An empty image or audio span is left out with its markers."""
    codes = [MOD_MARK]
    if n_video:
        codes += [MOD_MARK] + [MOD_VIDEO] * n_video + [MOD_MARK]
    if n_audio:
        codes += [MOD_MARK] + [MOD_AUDIO] * n_audio + [MOD_MARK]
    codes += [MOD_TEXT] * n_text + [MOD_MARK]
    return MixedUnit(tuple(codes))


def unit_codes(unit) -> np.ndarray:
    """Per-token modality tags of a unit given as (modality, length) or as a MixedUnit."""
    if isinstance(unit, MixedUnit):
        return np.asarray(unit.codes, np.uint8)
    m, n = unit
    return np.full(n, m, np.uint8)


def grammar_stream_units(cfg: StreamConfig, rng: np.random.Generator):
    """The history of ``cfg`` with each second's content as one grammar unit: the second's
    frame (if any), its audio and the text turns that follow it inside the same unit.  The
    chunk is one grammar unit too.  Same seeded structure draws as ``stream_units``."""
    units, chunk = stream_units(cfg, rng)
    out, cur = [], None
    for m, n in units:
        if m == MOD_TEXT and cur is not None:
            cur[2] += n
            continue
        if m == MOD_VIDEO or cur is None or (m == MOD_AUDIO and cur[1]):
            if cur is not None:
                out.append(grammar_unit(*cur))
            cur = [0, 0, 0]
        cur[0 if m == MOD_VIDEO else 1 if m == MOD_AUDIO else 2] += n
    if cur is not None:
        out.append(grammar_unit(*cur))
    nv = sum(n for m, n in chunk if m == MOD_VIDEO)
    na = sum(n for m, n in chunk if m == MOD_AUDIO)
    return out, [grammar_unit(nv, na, 0)]


@dataclasses.dataclass
class Layout:
    """Per-slot tags of a history pool: unit id (-1 = hole), modality, logical position."""
    unit_id: np.ndarray        # int32 [n_slots]
    modality: np.ndarray       # uint8 [n_slots]
    pos: np.ndarray            # int32 [n_slots]
    n_units: int               # live units, ids 0..n_units-1 in temporal order
    orig_unit: np.ndarray      # int32 [n_slots]: index into the original unit list (for offsets)
    n_orig_units: int
    chunk_modality: np.ndarray  # uint8 [L]
    chunk_unit: np.ndarray     # int32 [L], local unit index within the chunk
    n_chunk_units: int

    @property
    def n_slots(self) -> int:
        return int(self.unit_id.shape[0])

    @property
    def chunk_len(self) -> int:
        return int(self.chunk_modality.shape[0])


def build_layout(units, chunk, evicted: Optional[set] = None) -> Layout:
    """Units are (modality, length) pairs or MixedUnit token lists, in temporal order."""
    evicted = evicted or set()
    codes = [unit_codes(u) for u in units]
    n_slots = sum(len(c) for c in codes)
    unit_id = np.empty(n_slots, np.int32)
    modality = np.empty(n_slots, np.uint8)
    pos = np.empty(n_slots, np.int32)
    orig = np.empty(n_slots, np.int32)
    s = 0
    live_id = 0
    live_pos = 0
    for ui, c in enumerate(codes):
        n = len(c)
        modality[s:s + n] = c
        orig[s:s + n] = ui
        if ui in evicted:
            unit_id[s:s + n] = -1
            pos[s:s + n] = -1
        else:
            unit_id[s:s + n] = live_id
            pos[s:s + n] = np.arange(live_pos, live_pos + n, dtype=np.int32)
            live_id += 1
            live_pos += n
        s += n
    ccodes = [unit_codes(u) for u in chunk]
    cmod = np.concatenate([c for c in ccodes]) if ccodes else np.zeros(0, np.uint8)
    cunit = (np.concatenate([np.full(len(c), i, np.int32) for i, c in enumerate(ccodes)])
             if ccodes else np.zeros(0, np.int32))
    return Layout(unit_id, modality, pos, live_id, orig, len(units), cmod, cunit, len(chunk))


def choose_evicted(rng, units, frac: float, recent: int) -> set:
    """Seeded set of already-evicted history units: ``frac`` of the units outside the newest
    ``recent`` tokens (a native-layout history keeps its newest units whole)."""
    if frac <= 0:
        return set()
    tail = 0
    protected = set()
    for ui in range(len(units) - 1, -1, -1):
        n = len(unit_codes(units[ui]))
        if tail + n > recent:
            break
        tail += n
        protected.add(ui)
    pool = [ui for ui in range(len(units)) if ui not in protected]
    k = int(round(frac * len(units)))
    return set(rng.choice(pool, size=k, replace=False).tolist())


# ----------------------------------------------------------------------------- values

def to_storage(x: np.ndarray, dtype: str) -> torch.Tensor:
    t = torch.from_numpy(x)
    return t.to(torch.bfloat16) if dtype == "bf16" else t.clone()


@dataclasses.dataclass
class Segment:
    k_hist: torch.Tensor   # [n_slots, H_kv, d], storage dtype (CPU)
    v_hist: torch.Tensor
    k_chunk: torch.Tensor  # [L, H_kv, d]
    v_chunk: torch.Tensor
    q: torch.Tensor        # [L, H_q, d]; bf16 for bf16 pools, f32 for f32 pools


def draw_segment(cfg: StreamConfig, layout: Layout, seed: int) -> Segment:
    rng = np.random.default_rng(seed)
    H, d = cfg.n_kv_heads, cfg.head_dim
    n_hist_units = layout.n_orig_units
    n_chunk_units = layout.n_chunk_units
    off_k = rng.normal(0.0, 0.5, size=n_hist_units + n_chunk_units).astype(np.float32)
    off_v = rng.normal(0.0, 0.5, size=n_hist_units + n_chunk_units).astype(np.float32)
    n, L = layout.n_slots, layout.chunk_len
    k_hist = rng.standard_normal((n, H, d), dtype=np.float32)
    k_hist += off_k[layout.orig_unit][:, None, None]
    v_hist = rng.standard_normal((n, H, d), dtype=np.float32)
    v_hist += off_v[layout.orig_unit][:, None, None]
    cu = n_hist_units + layout.chunk_unit
    k_chunk = rng.standard_normal((L, H, d), dtype=np.float32)
    k_chunk += off_k[cu][:, None, None]
    v_chunk = rng.standard_normal((L, H, d), dtype=np.float32)
    v_chunk += off_v[cu][:, None, None]
    q = rng.standard_normal((L, cfg.n_q_heads, d), dtype=np.float32)
    return Segment(to_storage(k_hist, cfg.dtype), to_storage(v_hist, cfg.dtype),
                   to_storage(k_chunk, cfg.dtype), to_storage(v_chunk, cfg.dtype),
                   to_storage(q, cfg.dtype))


@dataclasses.dataclass
class Stream:
    cfg: StreamConfig
    layout: Layout

    def segment_seed(self, layer: int) -> int:
        return self.cfg.seed if self.cfg.n_layers == 1 else self.cfg.seed * 1000 + layer

    def segment(self, layer: int = 0) -> Segment:
        return draw_segment(self.cfg, self.layout, self.segment_seed(layer))


def make_stream(cfg: StreamConfig, grammar: bool = False) -> Stream:
    """The workload's stream; ``grammar`` groups each second into one mixed grammar unit."""
    rng = np.random.default_rng(cfg.seed)
    units, chunk = (grammar_stream_units if grammar else stream_units)(cfg, rng)
    evicted = choose_evicted(rng, units, cfg.evict_frac, cfg.recent)
    return Stream(cfg, build_layout(units, chunk, evicted))


def loop_chunk(cfg: StreamConfig, step: int) -> Tuple[Layout, Segment]:
    """Chunk of stream-loop step ``step`` (seed 1000*seed + step): a layout with no history."""
    _, chunk = stream_units(cfg, np.random.default_rng(cfg.seed))
    lay = build_layout([], chunk)
    return lay, draw_segment(cfg, lay, cfg.seed * 1000 + step)


# ----------------------------------------------------------------------------- small cases

def custom_stream(units, chunk, *, n_q_heads=4, n_kv_heads=1, head_dim=64, dtype="bf16",
                  page_size=64, budget=256, recent=32, seed=123, evicted=None,
                  weights=DEFAULT_WEIGHTS) -> Tuple[StreamConfig, Layout, Segment]:
    """A hand-specified stream for edge cases (tests): explicit units and chunk."""
    cfg = StreamConfig("custom", n_q_heads, n_kv_heads, head_dim, dtype, page_size, budget,
                       recent, 1, seed, "custom", weights=tuple(weights))
    lay = build_layout(units, chunk, set(evicted or ()))
    return cfg, lay, draw_segment(cfg, lay, seed)


def random_units(rng: np.random.Generator, n_units: int, lo: int = 1, hi: int = 40,
                 sys_prefix: int = 0):
    """Random single-modality unit list (tests)."""
    units = []
    if sys_prefix:
        units.append((MOD_SYS, sys_prefix))
    for _ in range(n_units):
        units.append((int(rng.integers(1, 4)), int(rng.integers(lo, hi + 1))))
    return units


def random_mixed_units(rng: np.random.Generator, n_units: int, hi: int = 40,
                       sys_prefix: int = 0):
    """Random units of mixed modality (tests): grammar units with random span lengths (empty
    spans included), units of one modality, and free token sequences with several spans of a
    modality, with or without markers between them."""
    units = []
    if sys_prefix:
        units.append((MOD_SYS, sys_prefix))
    for _ in range(n_units):
        kind = int(rng.integers(3))
        if kind == 0:
            units.append(grammar_unit(int(rng.integers(0, hi + 1)), int(rng.integers(0, hi // 2 + 1)),
                                      int(rng.integers(0, hi // 2 + 1))))
        elif kind == 1:
            units.append((int(rng.integers(1, 4)), int(rng.integers(1, hi + 1))))
        else:
            codes = []
            for _ in range(int(rng.integers(1, 6))):
                codes += [int(rng.integers(1, 5))] * int(rng.integers(1, hi // 2 + 1))
            units.append(MixedUnit(tuple(codes)))
    return units
