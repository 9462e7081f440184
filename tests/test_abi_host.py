"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every entry point
the header declares, and rejects misuse with the documented status code before touching the
device."""
import ctypes
import os
import re

import pytest

from paper_2609_34653_amd import omnitide as ot

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "omnitide.h")


@pytest.fixture(scope="module")
def L():
    return ot.lib()


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|size_t|const char\*)\s+(omnitide_\w+)\(", text, re.M)))


def test_exports_every_declared_symbol(L):
    names = header_functions()
    assert len(names) == 27
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(ot.EXPORTS)


def test_header_codes_match_binding():
    text = open(HEADER).read()
    codes = dict((k, int(v)) for k, v in re.findall(r"OMNITIDE_(E_\w+|OK)\s*=\s*(-?\d+)", text))
    assert codes["OK"] == ot.OK and codes["E_TAGS"] == ot.E_TAGS
    assert codes["E_BUDGET"] == ot.E_BUDGET and codes["E_CAPACITY"] == ot.E_CAPACITY
    assert codes["E_ALIAS"] == ot.E_ALIAS and codes["E_WORKSPACE"] == ot.E_WORKSPACE
    assert codes["E_RANGE"] == ot.E_RANGE and codes["E_SCRATCH"] == ot.E_SCRATCH
    assert len(set(codes.values())) == len(codes)


def test_status_strings_and_version():
    assert ot.status_string(0) == "ok"
    assert "budget" in ot.status_string(-16)
    assert "tags" in ot.status_string(-17)
    assert "2^51" in ot.status_string(ot.E_RANGE)
    assert ot.status_string(12345) == "unknown status"
    assert "gfx950" in ot.version()


P = ctypes.c_void_p
W_OK = (ctypes.c_float * 4)(2.0, 1.0, 1.5, 2.0)


def fake(i):
    """A distinct, never-dereferenced device address."""
    return P(0x10_0000_0000 + i * 0x1_0000_0000)


def score(L, **kw):
    a = dict(k=fake(0), dtype=0, n_seg=1, n_slots=1000, H=8, d=128, uid=fake(1), mod=fake(2),
             w=ctypes.cast(W_OK, P), U=10, wsum=fake(3), ln=fake(4), fs=fake(5), ls=fake(6),
             fl=fake(7), st=fake(8))
    a.update(kw)
    return L.omnitide_score_units(a["k"], a["dtype"], a["n_seg"], a["n_slots"], a["H"], a["d"],
                                  a["uid"], a["mod"], a["w"], a["U"], a["wsum"], a["ln"],
                                  a["fs"], a["ls"], a["fl"], a["st"], None)


def test_score_validation(L):
    assert score(L, k=None) == ot.E_NULL
    assert score(L, wsum=None) == ot.E_NULL
    assert score(L, w=None) == ot.E_NULL
    assert score(L, dtype=7) == ot.E_DTYPE
    assert score(L, d=96) == ot.E_SHAPE
    assert score(L, H=64) == ot.E_SHAPE            # 64 x 128 > 4096 elements per row
    assert score(L, U=0) == ot.E_SHAPE
    assert score(L, U=8193) == ot.E_SHAPE
    assert score(L, n_seg=0) == ot.E_SHAPE
    assert score(L, n_slots=-1) == ot.E_SHAPE
    for bad in ((2.0, 1.0, 1.0 / 3.0, 2.0), (0.0, 1.0, 1.0, 1.0), (5.0, 1, 1, 1),
                (float("nan"), 1, 1, 1)):
        w = (ctypes.c_float * 4)(*bad)
        assert score(L, w=ctypes.cast(w, P)) == ot.E_WEIGHT
    # an output overlapping the key pool
    assert score(L, wsum=P(fake(0).value + 64)) == ot.E_ALIAS
    assert score(L, ln=fake(3)) == ot.E_ALIAS      # two outputs at one address


def select(L, **kw):
    a = dict(ws=fake(0), ln=fake(1), fs=fake(2), ls=fake(3), fl=fake(4), n_seg=1, U=10, B=100,
             R=10, sc=fake(5), keep=fake(6), kt=fake(7), st=fake(8))
    a.update(kw)
    return L.omnitide_select_units(a["ws"], a["ln"], a["fs"], a["ls"], a["fl"], a["n_seg"],
                                   a["U"], a["B"], a["R"], a["sc"], a["keep"], a["kt"], a["st"],
                                   None)


def test_select_validation(L):
    assert select(L, keep=None) == ot.E_NULL
    assert select(L, U=9000) == ot.E_SHAPE
    assert select(L, B=-1) == ot.E_SHAPE
    assert select(L, R=-5) == ot.E_SHAPE
    assert select(L, keep=fake(1)) == ot.E_ALIAS


def compact(L, **kw):
    a = dict(ks=fake(0), vs=fake(1), dtype=0, n_seg=1, n=1000, H=8, d=128, P=64, uid=fake(2),
             mod=fake(3), pos=fake(4), keep=fake(5), ln=fake(6), fs=fake(7), U=10, kc=fake(8),
             vc=fake(9), cm=fake(10), cu=fake(11), Lc=16, kd=fake(12), vd=fake(13), cap=600,
             uidd=fake(14), modd=fake(15), posd=fake(16), src=fake(17), rm=fake(18), nctx=fake(19),
             npg=fake(20), ws=fake(21), wsb=1 << 20, st=fake(22))
    a.update(kw)
    return L.omnitide_compact_kv(a["ks"], a["vs"], a["dtype"], a["n_seg"], a["n"], a["H"], a["d"],
                                 a["P"], a["uid"], a["mod"], a["pos"], a["keep"], a["ln"],
                                 a["fs"], a["U"], a["kc"], a["vc"], a["cm"], a["cu"], a["Lc"],
                                 a["kd"], a["vd"], a["cap"], a["uidd"], a["modd"], a["posd"],
                                 a["src"], a["rm"], a["nctx"], a["npg"], a["ws"], a["wsb"],
                                 a["st"], None)


def compact_rope(L, base=10000.0, rdims=128, style=0, **kw):
    a = dict(ks=fake(0), vs=fake(1), dtype=0, n_seg=1, n=1000, H=8, d=128, P=64, uid=fake(2),
             mod=fake(3), pos=fake(4), keep=fake(5), ln=fake(6), fs=fake(7), U=10, kc=fake(8),
             vc=fake(9), cm=fake(10), cu=fake(11), Lc=16, kd=fake(12), vd=fake(13), cap=600,
             uidd=fake(14), modd=fake(15), posd=fake(16), src=fake(17), rm=fake(18), nctx=fake(19),
             npg=fake(20), ws=None, wsb=1 << 20, st=fake(22))
    a.update(kw)
    return L.omnitide_compact_kv_rope(a["ks"], a["vs"], a["dtype"], a["n_seg"], a["n"], a["H"],
                                      a["d"], a["P"], a["uid"], a["mod"], a["pos"], a["keep"],
                                      a["ln"], a["fs"], a["U"], a["kc"], a["vc"], a["cm"],
                                      a["cu"], a["Lc"], a["kd"], a["vd"], a["cap"], a["uidd"],
                                      a["modd"], a["posd"], a["src"], a["rm"], a["nctx"],
                                      a["npg"], a["ws"], a["wsb"], base, rdims, style, a["st"],
                                      None)


def test_compact_rope_validation(L):
    # valid rotary arguments get past their check (the missing workspace is reported next)
    assert compact_rope(L) == ot.E_WORKSPACE
    assert compact_rope(L, rdims=64, style=1) == ot.E_WORKSPACE
    assert compact_rope(L, rdims=24, style=1) == ot.E_WORKSPACE   # interleaved: any even width
    assert compact_rope(L, rdims=24, style=0, dtype=1) == ot.E_WORKSPACE   # f32 chunks: 4 dims
    for bad in (dict(rdims=0), dict(rdims=7), dict(rdims=130), dict(rdims=24, style=0),
                dict(style=2), dict(base=1.0), dict(base=float("inf")), dict(base=float("nan"))):
        assert compact_rope(L, **bad) == ot.E_SHAPE, bad
    # pointer and dtype errors come first
    assert compact_rope(L, rdims=7, kd=None) == ot.E_NULL
    assert compact_rope(L, rdims=7, dtype=3) == ot.E_DTYPE


def plan_spans(L, **kw):
    a = dict(ln=fake(0), fs=fake(1), ls=fake(2), fl=fake(3), uid=fake(8), mod=fake(4), n_seg=1,
             n_slots=1000, U=10, low=100, high=120, R=10, sv=4, sa=2, tb=16, kl=fake(5),
             ks=fake(9), kt=fake(6), ws=fake(10),
             wsb=ot.omnitide_plan_spans_workspace_bytes(1, 1000, 10), st=fake(7))
    a.update(kw)
    return L.omnitide_plan_spans(a["ln"], a["fs"], a["ls"], a["fl"], a["uid"], a["mod"],
                                 a["n_seg"], a["n_slots"], a["U"], a["low"], a["high"], a["R"],
                                 a["sv"], a["sa"], a["tb"], a["kl"], a["ks"], a["kt"], a["ws"],
                                 a["wsb"], a["st"], None)


def test_plan_spans_validation(L):
    assert plan_spans(L, kl=None) == ot.E_NULL
    assert plan_spans(L, mod=None) == ot.E_NULL
    assert plan_spans(L, uid=None) == ot.E_NULL
    assert plan_spans(L, ks=None) == ot.E_NULL
    assert plan_spans(L, ws=None) == ot.E_WORKSPACE
    assert plan_spans(L, wsb=ot.omnitide_plan_spans_workspace_bytes(1, 1000, 10) - 1) == \
        ot.E_WORKSPACE
    assert ot.omnitide_plan_spans_workspace_bytes(1, 1000, 10) >= 1000 * 4 + 10 * 12
    assert ot.omnitide_plan_spans_workspace_bytes(3, 1000, 10) == \
        3 * ot.omnitide_plan_spans_workspace_bytes(1, 1000, 10)
    assert plan_spans(L, ks=P(fake(8).value + 100)) == ot.E_ALIAS   # mask over the unit ids
    assert plan_spans(L, ws=P(fake(6).value)) == ot.E_ALIAS         # workspace over an output
    assert plan_spans(L, high=99) == ot.E_SHAPE          # high watermark below the low one
    assert plan_spans(L, low=-1) == ot.E_SHAPE
    for k in ("R", "sv", "sa", "tb"):
        assert plan_spans(L, **{k: -1}) == ot.E_SHAPE, k
    assert plan_spans(L, U=0) == ot.E_SHAPE
    assert plan_spans(L, U=8193) == ot.E_SHAPE
    assert plan_spans(L, n_slots=-1) == ot.E_SHAPE
    assert plan_spans(L, kl=fake(0)) == ot.E_ALIAS        # output over an input
    assert plan_spans(L, kt=P(fake(5).value + 8)) == ot.E_ALIAS   # two outputs overlap


def compact_spans(L, base=0.0, rdims=0, style=0, **kw):
    a = dict(ks=fake(0), vs=fake(1), dtype=0, n_seg=1, n=1000, H=8, d=128, P=64, uid=fake(2),
             mod=fake(3), pos=fake(4), ks_=fake(5), ln=fake(6), fs=fake(7), U=10, kc=fake(8),
             vc=fake(9), cm=fake(10), cu=fake(11), Lc=16, kd=fake(12), vd=fake(13), cap=600,
             uidd=fake(14), modd=fake(15), posd=fake(16), src=fake(17), rm=fake(18), nctx=fake(19),
             npg=fake(20), ws=None, wsb=1 << 20, st=fake(22))
    a.update(kw)
    return L.omnitide_compact_kv_spans(a["ks"], a["vs"], a["dtype"], a["n_seg"], a["n"], a["H"],
                                       a["d"], a["P"], a["uid"], a["mod"], a["pos"], a["ks_"],
                                       a["ln"], a["fs"], a["U"], a["kc"], a["vc"], a["cm"],
                                       a["cu"], a["Lc"], a["kd"], a["vd"], a["cap"], a["uidd"],
                                       a["modd"], a["posd"], a["src"], a["rm"], a["nctx"],
                                       a["npg"], a["ws"], a["wsb"], base, rdims, style, a["st"],
                                       None)


def test_compact_spans_validation(L):
    assert compact_spans(L) == ot.E_WORKSPACE           # valid: only the workspace is missing
    assert compact_spans(L, base=1e6, rdims=128) == ot.E_WORKSPACE
    assert compact_spans(L, ks_=None) == ot.E_NULL
    assert compact_spans(L, ks_=None, n=0) == ot.E_WORKSPACE  # no slots: the mask may be NULL
    assert compact_spans(L, rdims=-2) == ot.E_SHAPE
    assert compact_spans(L, base=1.0, rdims=64) == ot.E_SHAPE
    assert compact_spans(L, cap=15) == ot.E_CAPACITY
    assert compact_spans(L, ws=fake(21), kd=P(fake(5).value + 999)) == ot.E_ALIAS  # over the mask


def test_compact_validation(L):
    assert compact(L, kd=None) == ot.E_NULL
    assert compact(L, kc=None) == ot.E_NULL                  # chunk_len > 0 needs the chunk
    assert compact(L, P=48) == ot.E_SHAPE
    assert compact(L, dtype=3) == ot.E_DTYPE
    assert compact(L, cap=15) == ot.E_CAPACITY              # smaller than the chunk
    assert compact(L, ws=None) == ot.E_WORKSPACE
    assert compact(L, wsb=16) == ot.E_WORKSPACE
    assert compact(L, kd=P(fake(0).value + 4096)) == ot.E_ALIAS   # destination inside source
    assert ot.omnitide_compact_workspace_bytes(1, 10, 600) > 0


def attn(L, **kw):
    a = dict(q=fake(0), k=fake(1), v=fake(2), dt=0, nctx=fake(3), n_seg=1, cap=17049, Lc=665,
             Hq=32, Hkv=8, d=128, scale=0.0884, out=fake(4), odt=1, ws=fake(5), wsb=1 << 30,
             st=fake(6))
    a.update(kw)
    return L.omnitide_chunk_attn(a["q"], a["k"], a["v"], a["dt"], a["nctx"], a["n_seg"],
                                 a["cap"], a["Lc"], a["Hq"], a["Hkv"], a["d"], a["scale"],
                                 a["out"], a["odt"], a["ws"], a["wsb"], a["st"], None)


def test_attention_validation(L):
    assert attn(L, q=None) == ot.E_NULL
    assert attn(L, Hq=30) == ot.E_SHAPE
    assert attn(L, d=80) == ot.E_SHAPE
    assert attn(L, Lc=0) == ot.E_SHAPE
    assert attn(L, scale=float("inf")) == ot.E_SHAPE
    assert attn(L, cap=100) == ot.E_CAPACITY
    assert attn(L, ws=None) == ot.E_WORKSPACE
    assert attn(L, out=fake(1)) == ot.E_ALIAS
    assert attn(L, dt=2) == ot.E_DTYPE and attn(L, odt=5) == ot.E_DTYPE
    need = ot.omnitide_attn_workspace_bytes(1, 17049, 665, 32, 8, 128)
    assert need > 0 and attn(L, wsb=need - 1) == ot.E_WORKSPACE
    # split count: 21 row tiles x 8 KV heads -> 3 splits on the 80K-history shape
    assert need == 3 * 665 * 32 * 130 * 4
    # float32 inputs: the bf16 copies of q, k and v follow the partials
    need32 = ot.omnitide_attn_workspace_bytes(1, 17049, 665, 32, 8, 128, dtype=ot.F32)
    copies = 665 * 32 * 128 * 2 + 2 * 17049 * 8 * 128 * 2
    assert copies <= need32 - need <= copies + 4 * 256
    assert attn(L, dt=1, wsb=need32 - 1) == ot.E_WORKSPACE
    # a float32 output (4 bytes an element) ending inside q aliases it
    assert attn(L, out=P(fake(0).value - 665 * 32 * 128 * 3)) == ot.E_ALIAS


def attn_noalloc(L, **kw):
    a = dict(q=fake(0), k=fake(1), v=fake(2), nctx=fake(3), n_seg=1, cap=17049, Lc=665, Hq=32,
             Hkv=8, d=128, scale=0.0884, out=fake(4), st=fake(6))
    a.update(kw)
    return L.omnitide_chunk_attn_noalloc(a["q"], a["k"], a["v"], a["nctx"], a["n_seg"], a["cap"],
                                         a["Lc"], a["Hq"], a["Hkv"], a["d"], a["scale"],
                                         a["out"], a.get("odt", 1), a["st"], None)


def test_attention_noalloc_validation(L):
    """The same host checks as the workspace entry point (nothing launched here)."""
    assert attn_noalloc(L, q=None) == ot.E_NULL
    assert attn_noalloc(L, out=None) == ot.E_NULL
    assert attn_noalloc(L, Hq=30) == ot.E_SHAPE
    assert attn_noalloc(L, d=80) == ot.E_SHAPE
    assert attn_noalloc(L, scale=float("nan")) == ot.E_SHAPE
    assert attn_noalloc(L, cap=100) == ot.E_CAPACITY
    assert attn_noalloc(L, out=fake(1)) == ot.E_ALIAS
    assert attn_noalloc(L, st=P(fake(4).value + 8)) == ot.E_ALIAS
    assert "scratch" in ot.status_string(ot.E_SCRATCH)


def test_noalloc_scratch_covers_every_shape():
    """Splits times row-tile workgroups stay within 512, so the partials of any shape fit the
    fixed 64 MiB array (the E_SCRATCH check is a guard, not a reachable limit today)."""
    worst = 0
    for n_seg in (1, 2, 3, 8, 36):
        for Lc in (1, 32, 89, 128, 665, 1000, 2329, 8192):
            for Hq, Hkv in ((4, 1), (8, 8), (32, 8), (64, 4), (128, 1)):
                for d in (64, 128):
                    for cap in (Lc, 4096, 17049, 131072):
                        if cap < Lc:
                            continue
                        worst = max(worst, ot.omnitide_attn_workspace_bytes(n_seg, cap, Lc, Hq,
                                                                            Hkv, d))
    assert 0 < worst <= 512 * 128 * 130 * 4 <= ot.NOALLOC_SCRATCH_BYTES


def span_attn(L, **kw):
    a = dict(q=fake(0), k=fake(1), v=fake(2), kp=fake(3), span=fake(4), qp=fake(5), n_seg=1,
             cap=81920, Lc=665, Hq=32, Hkv=8, d=128, scale=0.0884, out=fake(6), ws=fake(7),
             wsb=1 << 30, st=fake(8), trav=1)
    a.update(kw)
    return L.omnitide_span_attn(a["q"], a["k"], a["v"], a["kp"], a["span"], a["qp"], a["n_seg"],
                                a["cap"], a["Lc"], a["Hq"], a["Hkv"], a["d"], a["scale"],
                                a["trav"], a["out"], a["ws"], a["wsb"], a["st"], None)


def test_span_attention_validation(L):
    for k in ("q", "kp", "span", "qp", "out"):
        assert span_attn(L, **{k: None}) == ot.E_NULL, k
    assert span_attn(L, Hq=30) == ot.E_SHAPE
    assert span_attn(L, cap=600) == ot.E_CAPACITY            # smaller than the chunk
    assert span_attn(L, cap=(1 << 21) + 1) == ot.E_CAPACITY  # over the tile-table limit
    assert span_attn(L, ws=None) == ot.E_WORKSPACE
    need = ot.omnitide_span_attn_workspace_bytes(1, 81920, 665, 32, 8, 128)
    assert need > ot.omnitide_attn_workspace_bytes(1, 81920, 665, 32, 8, 128)
    assert span_attn(L, wsb=need - 1) == ot.E_WORKSPACE
    assert span_attn(L, out=P(fake(3).value + 256)) == ot.E_ALIAS   # output over key_pos
    # chunk_attn keeps its own (smaller) workspace and needs no positions
    assert ot.omnitide_span_attn_workspace_bytes(1, 81920, 665, 30, 8, 128) == 0
    # traversals: 0 full span, 1 tile skipping, 2 position order; nothing else
    for trav in (-1, 3, 7):
        assert span_attn(L, trav=trav) == ot.E_SHAPE, trav
    # position order: 32-bit row offsets within a segment's pool, and room for the index
    assert span_attn(L, trav=2, cap=1 << 21) == ot.E_SHAPE        # 2^21 rows of 2 KB = 4 GiB
    assert span_attn(L, trav=2, cap=1 << 21, Hkv=4, ws=None) == ot.E_WORKSPACE
    part = ot.omnitide_attn_workspace_bytes(1, 81920, 665, 32, 8, 128)
    assert need >= -(-part // 256) * 256 + (81920 + 1) * 4


def evict(L, **kw):
    a = dict(n_seg=1, cap=1000, uid=fake(0), pos=fake(1), keep=fake(2), kl=None, ln=fake(3), U=10,
             rm=fake(4), kt=fake(5), nk=fake(6), span=fake(7), ws=fake(8), wsb=1 << 20,
             st=fake(9))
    a.update(kw)
    return L.omnitide_evict_native(a["n_seg"], a["cap"], a["uid"], a["pos"], a["keep"], a["kl"],
                                   a["ln"], a["U"], a["rm"], a["kt"], a["nk"], a["span"],
                                   a["ws"], a["wsb"], a["st"], None)


def test_evict_native_validation(L):
    assert evict(L, keep=None) == ot.E_NULL               # neither keep nor keep_len
    assert evict(L, span=None) == ot.E_NULL
    assert evict(L, cap=131073) == ot.E_SHAPE
    assert evict(L, U=8193) == ot.E_SHAPE
    assert evict(L, ws=None) == ot.E_WORKSPACE
    assert evict(L, wsb=16) == ot.E_WORKSPACE
    assert evict(L, rm=fake(3)) == ot.E_ALIAS              # output over unit_len
    assert evict(L, pos=P(fake(0).value + 8)) == ot.E_ALIAS   # in-place tags overlap
    assert ot.omnitide_evict_native_workspace_bytes(1, 10) == 160


def pack(L, **kw):
    a = dict(k=fake(0), v=fake(1), dtype=0, n_seg=1, cap=1000, H=8, d=128, P=256, T=1,
             uid=fake(2), mod=fake(3), pos=fake(4), span=fake(5), cut=fake(6), mv=fake(7),
             ws=fake(8), wsb=1 << 30)
    a.update(kw)
    return L.omnitide_pack_suffix(a["k"], a["v"], a["dtype"], a["n_seg"], a["cap"], a["H"],
                                  a["d"], a["P"], a["T"], a["uid"], a["mod"], a["pos"],
                                  a["span"], a["cut"], a["mv"], a["ws"], a["wsb"], None)


def test_pack_suffix_validation(L):
    assert pack(L, cut=None) == ot.E_NULL
    assert pack(L, dtype=2) == ot.E_DTYPE
    assert pack(L, T=0) == ot.E_SHAPE
    assert pack(L, P=0) == ot.E_SHAPE
    assert pack(L, cap=131073) == ot.E_SHAPE
    assert pack(L, ws=None) == ot.E_WORKSPACE
    need = ot.omnitide_pack_suffix_workspace_bytes(0, 1, 1000, 8, 128)
    assert need >= 1000 * 2 * 2048 and pack(L, wsb=need - 1) == ot.E_WORKSPACE
    assert pack(L, v=P(fake(0).value + 4096)) == ot.E_ALIAS


def place(L, **kw):
    a = dict(k=fake(0), v=fake(1), dtype=0, n_seg=1, cap=1000, H=8, d=128, uid=fake(2),
             mod=fake(3), pos=fake(4), kc=fake(5), vc=fake(6), cm=fake(7), cu=fake(8), Lc=16,
             kt=fake(9), nk=fake(10), slot=fake(11), span=fake(12), ws=fake(14), wsb=1 << 20,
             st=fake(13))
    a.update(kw)
    return L.omnitide_place_chunk(a["k"], a["v"], a["dtype"], a["n_seg"], a["cap"], a["H"],
                                  a["d"], a["uid"], a["mod"], a["pos"], a["kc"], a["vc"],
                                  a["cm"], a["cu"], a["Lc"], a["kt"], a["nk"], a["slot"],
                                  a["span"], a["ws"], a["wsb"], a["st"], None)


def test_place_chunk_validation(L):
    assert place(L, kc=None) == ot.E_NULL
    assert place(L, dtype=5) == ot.E_DTYPE
    assert place(L, Lc=0) == ot.E_SHAPE
    assert place(L, Lc=1001) == ot.E_CAPACITY
    assert place(L, slot=fake(9)) == ot.E_ALIAS            # output over kept_tokens
    assert place(L, ws=None) == ot.E_WORKSPACE
    assert place(L, wsb=8) == ot.E_WORKSPACE
    assert ot.omnitide_place_chunk_workspace_bytes(1, 1000) >= 125


def decode(L, **kw):
    a = dict(q=fake(0), k=fake(1), v=fake(2), n_ctx=fake(3), n_seg=1, cap=1000, nq=1, Hq=32,
             Hkv=8, d=128, scale=0.088, out=fake(4), ws=fake(5), wsb=1 << 24, st=fake(6))
    a.update(kw)
    return L.omnitide_decode_attn(a["q"], a["k"], a["v"], a["n_ctx"], a["n_seg"], a["cap"],
                                  a["nq"], a["Hq"], a["Hkv"], a["d"], a["scale"], a["out"],
                                  a["ws"], a["wsb"], a["st"], None)


def test_decode_validation(L):
    assert decode(L, q=None) == ot.E_NULL
    assert decode(L, nq=3) == ot.E_SHAPE          # 3 tokens x 4 heads > 8 query vectors
    assert decode(L, Hq=30) == ot.E_SHAPE         # not a multiple of the KV heads
    assert decode(L, d=96) == ot.E_SHAPE
    assert decode(L, scale=float("nan")) == ot.E_SHAPE
    assert decode(L, cap=0) == ot.E_CAPACITY
    assert decode(L, ws=None) == ot.E_WORKSPACE
    assert decode(L, out=P(fake(1).value + 64)) == ot.E_ALIAS
    assert ot.omnitide_decode_workspace_bytes(1, 1000, 1, 32, 8, 128) > 0
    assert ot.omnitide_decode_workspace_bytes(1, 1000, 1, 30, 8, 128) == 0



def decode_span(L, **kw):
    a = dict(q=fake(0), k=fake(1), v=fake(2), kp=fake(3), span=fake(4), qp=fake(5), n_seg=1,
             cap=81920, nq=1, Hq=32, Hkv=8, d=128, scale=0.088, trav=1, out=fake(6), ws=fake(7),
             wsb=1 << 30, st=fake(8))
    a.update(kw)
    return L.omnitide_decode_span_attn(a["q"], a["k"], a["v"], a["kp"], a["span"], a["qp"],
                                       a["n_seg"], a["cap"], a["nq"], a["Hq"], a["Hkv"], a["d"],
                                       a["scale"], a["trav"], a["out"], a["ws"], a["wsb"],
                                       a["st"], None)


def test_decode_span_validation(L):
    for k in ("q", "kp", "span", "qp", "out"):
        assert decode_span(L, **{k: None}) == ot.E_NULL, k
    assert decode_span(L, nq=3) == ot.E_SHAPE
    assert decode_span(L, cap=(1 << 21) + 1) == ot.E_CAPACITY
    for trav in (-1, 3):
        assert decode_span(L, trav=trav) == ot.E_SHAPE, trav
    # position order: 32-bit row offsets within a segment's pool, and room for the index
    assert decode_span(L, trav=2, cap=1 << 21) == ot.E_SHAPE
    assert decode_span(L, trav=2, ws=None) == ot.E_WORKSPACE
    need = ot.omnitide_decode_span_workspace_bytes(1, 81920, 1, 32, 8, 128)
    part = ot.omnitide_decode_workspace_bytes(1, 81920, 1, 32, 8, 128)
    assert need >= -(-part // 256) * 256 + (81920 + 1) * 4
    assert decode_span(L, trav=2, wsb=need - 1) == ot.E_WORKSPACE
