/*
 * omnitide.h -- C ABI of the per-chunk stream step of OmniTide on AMD Instinct MI355X (gfx950).
 *
 * One step over a KV pool whose slots are tagged with a unit id and a modality:
 *   1. omnitide_score_units   per-unit modality-weighted key magnitude (OmniPick importance)
 *   2. omnitide_select_units  budgeted whole-unit retention plan (OmniPick planning)
 *   3. omnitide_compact_kv    order-preserving packing of the kept rows + chunk (OmniPage)
 *   4. omnitide_chunk_attn    GQA prefill attention of the chunk over [history || chunk]
 * plus omnitide_compact_kv_rope (compaction with rotary re-encoding of the moved keys),
 * omnitide_plan_spans + omnitide_compact_kv_spans (the span plan: recent units whole, boundary
 * tokens and sink prefixes of the image and audio spans of older units, a shared text budget,
 * oldest-first trimming, then compaction of the kept slots) and omnitide_decode_attn (decode
 * attention of the last few tokens over the compacted pool); omnitide_evict_native, omnitide_pack_suffix, omnitide_place_chunk and
 * omnitide_span_attn keep the native (logical-only) layout with holes instead.
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers into memory the caller allocated (hipMalloc or a
 *     framework allocator), 16-byte aligned, unless the argument is documented as host.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Every call is asynchronous: it
 *     validates its arguments on the host, enqueues kernels on `stream` and returns.  Inputs must
 *     stay alive and unmodified until the stream has executed the call.
 *   - No call allocates or frees memory, and the library keeps no mutable global state; calls on
 *     distinct streams with distinct buffers may run from several host threads.
 *   - A segment is one independent pool (one layer, or one stream): every per-segment array is
 *     laid out segment-major, segments back to back.
 *   - Return value: OMNITIDE_OK, or a negative code for host-detected misuse, in which case
 *     nothing was enqueued.  OMNITIDE_E_HIP reports a failed kernel launch.
 *   - Data-dependent errors are detected on the device and written to *d_status (an int32 device
 *     word, may be NULL) with "first error wins" semantics (atomic compare-and-swap from 0).  The
 *     caller zeroes it and reads it after synchronising.  When it is non-zero the outputs of the
 *     failing call are unspecified but every write stays inside the caller's buffers.
 *
 * KV layout: K and V pools are [n_seg][n_slots][n_kv_heads][head_dim] (token-major: one slot's
 * keys for all KV heads form one contiguous row).  Tags are int32 unit id (-1 = empty slot),
 * uint8 modality (0 system, 1 video, 2 audio, 3 text, 4 structural marker: a unit's start and
 * end tokens and the open and close tokens of its image and audio spans) and int32 logical
 * position per slot.  Units are numbered 0..n_units-1 in temporal order; each live unit
 * occupies one contiguous run of slots, and runs appear in unit order.  A unit may mix
 * modalities (paper: Overview, the unit grammar).
 */
#ifndef OMNITIDE_H
#define OMNITIDE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  OMNITIDE_OK = 0,
  OMNITIDE_E_NULL = -1,       /* a required pointer is NULL */
  OMNITIDE_E_SHAPE = -2,      /* a size is out of range or inconsistent */
  OMNITIDE_E_DTYPE = -3,      /* unsupported element type */
  OMNITIDE_E_WEIGHT = -4,     /* a modality weight is not an exact multiple of 1/256 in (0, 4] */
  OMNITIDE_E_CAPACITY = -5,   /* destination pool too small (host: static check; device: actual) */
  OMNITIDE_E_WORKSPACE = -6,  /* workspace pointer NULL or smaller than required */
  OMNITIDE_E_ALIAS = -7,      /* an output overlaps an input it must not overlap */
  OMNITIDE_E_HIP = -8,        /* a HIP launch failed */
  OMNITIDE_E_SCRATCH = -9,    /* the call needs more scratch than the fixed array holds
                                 (omnitide_chunk_attn_noalloc) */
  OMNITIDE_E_BUDGET = -16,    /* device: protected (system) tokens exceed the budget */
  OMNITIDE_E_TAGS = -17,      /* device: malformed tags (id or modality out of range, a unit
                                 not one contiguous run, runs out of unit order) */
  OMNITIDE_E_RANGE = -18      /* device: a unit score of 2^51 or more (select's ranking key) */
};

enum { OMNITIDE_BF16 = 0, OMNITIDE_F32 = 1 };
/* rotary dimension pairing for omnitide_compact_kv_rope */
enum { OMNITIDE_ROPE_HALF = 0,          /* pairs (j, j + rope_dims/2) */
       OMNITIDE_ROPE_INTERLEAVED = 1 }; /* pairs (2j, 2j + 1) */
enum { OMNITIDE_MOD_SYS = 0, OMNITIDE_MOD_VIDEO = 1, OMNITIDE_MOD_AUDIO = 2, OMNITIDE_MOD_TEXT = 3,
       OMNITIDE_MOD_MARK = 4 };
/* key traversal of omnitide_span_attn */
enum { OMNITIDE_SPAN_FULL = 0,            /* every 64-slot tile of the span, masked */
       OMNITIDE_SPAN_SKIP_EMPTY = 1,      /* tiles without an entry skipped */
       OMNITIDE_SPAN_POSITION_ORDER = 2 };/* entries gathered in position order */

/* Limits checked on the host. */
#define OMNITIDE_MAX_UNITS 8192       /* units per segment */
#define OMNITIDE_MAX_ROW_ELEMS 4096   /* n_kv_heads * head_dim */

/*
 * omnitide_score_units -- unit importance (paper: OmniPick; Introduction, OmniPick paragraph:
 * the budget beyond the protected prefix and recent window goes by modality importance;
 * Modality-asymmetric attention).  The paper's planner reads only metadata and prints no score;
 * this entry point computes this library's importance statistic:
 *   q(x)  = floor(min(|x|, 32) * 2^16)        (NaN and +-Inf count as 32)
 *   a_s   = sum of q over the n_kv_heads*head_dim key elements of slot s
 *   W_u   = sum over live slots s of unit u of w[modality(s)] * a_s, w in units of 1/256
 *           (marker tokens take the text weight: they are special text-vocabulary tokens)
 * Exact integer arithmetic: the result does not depend on the order of summation.
 *
 *   k          [n_seg][n_slots][n_kv_heads][head_dim], dtype OMNITIDE_BF16 or OMNITIDE_F32
 *   unit_id    int32 [n_seg][n_slots]; -1 marks an empty slot
 *   modality   uint8 [n_seg][n_slots]
 *   weights    HOST float[4]: system, video, audio, text; each an exact multiple of 1/256 in
 *              (0, 4]
 *   outputs, [n_seg][n_units] each, fully overwritten:
 *     unit_wsum        uint64  W_u
 *     unit_len         int32   live slots of u
 *     unit_first_slot  int32   first slot of u (n_slots if u has none)
 *     unit_last_slot   int32   last slot of u (-1 if u has none)
 *     unit_flags       uint32  bit 0: u holds a system-modality token
 *   d_status   device: OMNITIDE_E_TAGS for a unit id outside [-1, n_units) or a modality > 4
 *              (such a slot is then ignored).
 * Limits: n_seg >= 1, n_slots >= 0, 1 <= n_units <= 8192, head_dim in {64, 128},
 * n_kv_heads >= 1, n_kv_heads * head_dim <= 4096.
 */
int omnitide_score_units(const void* k, int dtype, int n_seg, int n_slots, int n_kv_heads,
                         int head_dim, const int32_t* unit_id, const uint8_t* modality,
                         const float* weights, int n_units, uint64_t* unit_wsum,
                         int32_t* unit_len, int32_t* unit_first_slot, int32_t* unit_last_slot,
                         uint32_t* unit_flags, int32_t* d_status, void* stream);

/*
 * omnitide_select_units -- whole-unit retention plan (paper: Structure-aware retention
 * planning: system prefix protected, most recent units kept whole, older history kept until a
 * budget is used up; Overview: must-keep / recent-context / selected-history groups).
 * Per segment, with len_u > 0 marking live units:
 *   T_sys  = tokens of units with flag bit 0 (protected); T_sys > budget -> OMNITIDE_E_BUDGET
 *   recent = newest live non-system units, walked newest to oldest, added while their total
 *            stays <= min(recent_tokens, budget - T_sys); the walk stops at the first misfit
 *   score_u = floor(W_u / len_u); the remaining live units are ranked by (score desc, unit id
 *            desc: ties go to the newer unit) and kept in rank order while they fit into
 *            budget - T_sys - T_recent; the walk stops at the first that does not fit.
 *   Inputs are omnitide_score_units' outputs ([n_seg][n_units] each).
 *   unit_score   uint64 [n_seg][n_units]   floor(W_u / len_u), 0 for units without slots
 *   keep         uint8  [n_seg][n_units]   1 = unit retained whole
 *   kept_tokens  int32  [n_seg]            retained history tokens (<= budget)
 *   d_status     OMNITIDE_E_TAGS if a live unit is not one contiguous slot run or runs are
 *                out of unit order; OMNITIDE_E_RANGE if a score reaches 2^51 (the ranking key
 *                holds 51 bits of score; omnitide_score_units' outputs stay below 2^43);
 *                OMNITIDE_E_BUDGET as above (first match in this order).  On any error the
 *                segment's keep is all 0 and kept_tokens 0.
 * Limits: 1 <= n_units <= 8192, budget_tokens >= 0, recent_tokens >= 0.  One workgroup per
 * segment; latency-bound.
 */
int omnitide_select_units(const uint64_t* unit_wsum, const int32_t* unit_len,
                          const int32_t* unit_first_slot, const int32_t* unit_last_slot,
                          const uint32_t* unit_flags, int n_seg, int n_units, int budget_tokens,
                          int recent_tokens, uint64_t* unit_score, uint8_t* keep,
                          int32_t* kept_tokens, int32_t* d_status, void* stream);

/*
 * omnitide_compact_kv -- eager, order-preserving, out-of-place packing (paper: OmniPage;
 * Compaction-movement trade-off: eager compaction packs every retained entry into a contiguous
 * prefix; Selective migration, ordered-suffix mode with the cut at slot 0; Executing accepted
 * moves: one source-to-destination map; Applying the retention plan: each retained token's
 * position drops by the number of deleted tokens before it).
 * Per segment: destination row r < kept holds the r-th slot, in slot order, of the units with
 * keep != 0; rows [kept, kept + chunk_len) hold the chunk.  K and V rows are copied verbatim.
 *   k_src, v_src      [n_seg][n_slots_src][n_kv_heads][head_dim], dtype
 *   unit_id_src, modality_src, pos_src   per-slot tags [n_seg][n_slots_src]
 *   keep, unit_len, unit_first_slot      [n_seg][n_units] (select's and score's outputs)
 *   k_chunk, v_chunk  [n_seg][chunk_len][n_kv_heads][head_dim] (may be NULL iff chunk_len == 0)
 *   chunk_modality    uint8 [chunk_len], chunk_unit int32 [chunk_len]: the chunk's modality
 *                     and unit index (0.. in order), shared by all segments
 *   k_dst, v_dst      [n_seg][cap_dst][n_kv_heads][head_dim]; rows >= n_ctx untouched
 *   unit_id_dst       int32 [n_seg][cap_dst]: kept units renumbered 0.. in order, chunk units
 *                     after them; rows >= n_ctx are set to -1 (empty), so the destination is a
 *                     complete pool that can be the source of the next step (n_slots = cap_dst)
 *   modality_dst      uint8 [n_seg][cap_dst] (0 for rows >= n_ctx)
 *   pos_dst           int32 [n_seg][cap_dst]: pos_src - (deleted live slots before the source
 *                     slot); chunk row i gets kept + i; -1 for rows >= n_ctx
 *   src_of_dst        int32 [n_seg][cap_dst]: source slot of each row, -1 for chunk rows and
 *                     rows >= n_ctx
 *   unit_remap        int32 [n_seg][n_units]: new id of each unit, -1 if dropped
 *   n_ctx, n_pages    int32 [n_seg]: kept + chunk_len, ceil(n_ctx / page_size)
 *   workspace         device scratch of omnitide_compact_workspace_bytes() bytes
 *   d_status          OMNITIDE_E_CAPACITY if kept + chunk_len > cap_dst (n_ctx and n_pages
 *                     are then 0, no K/V row is written and every tag row is empty)
 * The source and destination pools (and tag arrays) must not overlap (OMNITIDE_E_ALIAS).
 * Limits: page_size in {32, 64, 128, 256}; cap_dst >= chunk_len; others as for score.
 */
int omnitide_compact_kv(const void* k_src, const void* v_src, int dtype, int n_seg,
                        int n_slots_src, int n_kv_heads, int head_dim, int page_size,
                        const int32_t* unit_id_src, const uint8_t* modality_src,
                        const int32_t* pos_src, const uint8_t* keep, const int32_t* unit_len,
                        const int32_t* unit_first_slot, int n_units, const void* k_chunk,
                        const void* v_chunk, const uint8_t* chunk_modality,
                        const int32_t* chunk_unit, int chunk_len, void* k_dst, void* v_dst,
                        int cap_dst, int32_t* unit_id_dst, uint8_t* modality_dst,
                        int32_t* pos_dst, int32_t* src_of_dst, int32_t* unit_remap,
                        int32_t* n_ctx, int32_t* n_pages, void* workspace,
                        size_t workspace_bytes, int32_t* d_status, void* stream);

/*
 * omnitide_compact_kv_rope -- omnitide_compact_kv plus the rotary re-encoding of the moved keys
 * (paper: section 5.2, Applying the retention plan).  Compaction lowers a kept token's position
 * by the deleted tokens before it; its cached key, rotated for the old position, is turned by
 * that (negative) shift so that it reads as rotated for the new one.  Same arguments, outputs
 * and errors as omnitide_compact_kv, except:
 *   k_dst   history row r (source slot s) holds K[s] with each pair (x, y) of its first
 *           rope_dims dimensions (per head) turned by shift * theta_j:
 *           (x cos - y sin, x sin + y cos), shift = pos_dst[r] - pos_src[s] (<= 0, minus the
 *           deleted live slots before s), theta_j = rope_base^(-2j / rope_dims),
 *           j < rope_dims / 2; the pairing is rope_style.  Chunk rows, dimensions >= rope_dims,
 *           rows with shift 0 and all of V are copied unchanged, bit for bit.
 *   rope_base    finite and > 1 (e.g. 10000 or 1e6)
 *   rope_dims    even, 2..head_dim; with OMNITIDE_ROPE_HALF a multiple of 16 (bf16) or 8 (f32)
 *   rope_style   OMNITIDE_ROPE_HALF or OMNITIDE_ROPE_INTERLEAVED
 * Precision: the angle shift * theta_j is reduced modulo 2 pi in double precision, its sine and
 * cosine and the rotation are computed in float, and the result is rounded to the storage type
 * (round to nearest even): within half a unit in the last place of the exactly rotated value
 * plus 2^-21 of the length of the rotated pair.
 * Invalid rope arguments return OMNITIDE_E_SHAPE (checked after null pointers and dtype).
 */
int omnitide_compact_kv_rope(const void* k_src, const void* v_src, int dtype, int n_seg,
                             int n_slots_src, int n_kv_heads, int head_dim, int page_size,
                             const int32_t* unit_id_src, const uint8_t* modality_src,
                             const int32_t* pos_src, const uint8_t* keep,
                             const int32_t* unit_len, const int32_t* unit_first_slot,
                             int n_units, const void* k_chunk, const void* v_chunk,
                             const uint8_t* chunk_modality, const int32_t* chunk_unit,
                             int chunk_len, void* k_dst, void* v_dst, int cap_dst,
                             int32_t* unit_id_dst, uint8_t* modality_dst, int32_t* pos_dst,
                             int32_t* src_of_dst, int32_t* unit_remap, int32_t* n_ctx,
                             int32_t* n_pages, void* workspace, size_t workspace_bytes,
                             double rope_base, int rope_dims, int rope_style,
                             int32_t* d_status, void* stream);

size_t omnitide_compact_workspace_bytes(int n_seg, int n_units, int cap_dst);

/*
 * omnitide_plan_spans -- span retention plan (paper: Overview, the unit grammar; Structure-aware
 * retention planning: retention starts above the high watermark and trims toward the low
 * watermark; the system prefix is protected; recent units are kept in full; older units,
 * oldest to newest, keep their boundary tokens and short prefixes of their image and audio
 * spans as sinks, with separate lengths per modality; text is kept oldest to newest until a
 * shared budget is used up; then units are dropped oldest first, partially retained ones
 * before complete ones, until the target is met or one unit remains).
 * Per segment, with len_u > 0 marking live units.  A span is a maximal run of consecutive
 * slots of one unit with the same modality tag.
 *   sum len_u <= high_watermark  -> every live slot stays (keep_len = len)
 *   otherwise:
 *     a unit holding a system token (flag bit 0) stays whole and is never dropped
 *     recent units stay whole: newest live non-system units walked newest to oldest while their
 *       total <= recent_tokens, stopping at the first misfit
 *     an older unit keeps its marker tokens (tag 4), the first sink_video slots of each video
 *       span, the first sink_audio slots of each audio span, and its first
 *       clamp(text_budget - T, 0, text_u) text slots, T = text slots of older units before it
 *       (the budget is used up to the token)
 *   then, while sum keep_len > low_watermark and more than one unit has keep_len > 0, the next
 *   unit of the drop order gets keep_len 0: partially retained units (0 < keep_len < len) by
 *   id, then complete non-system units by id.  The low watermark is a target, not a bound.
 *   Inputs: omnitide_score_units' unit_len, unit_first_slot, unit_last_slot, unit_flags
 *   ([n_seg][n_units]) for the slot tags unit_id (int32) and modality (uint8) [n_seg][n_slots].
 *   keep_len     int32 [n_seg][n_units]   kept slots of each unit (0: dropped, len: whole)
 *   keep_slot    uint8 [n_seg][n_slots]   1: the slot's entry stays; 0: deleted or empty slot
 *   kept_tokens  int32 [n_seg]            sum of keep_len
 *   workspace    device scratch of omnitide_plan_spans_workspace_bytes() bytes
 *   d_status     OMNITIDE_E_TAGS if a live unit is not one contiguous slot run inside
 *                [0, n_slots), runs are out of unit order, or a unit holds a modality > 4;
 *                the segment's keep_len and keep_slot are then all 0 and kept_tokens 0.
 * Limits: 1 <= n_units <= 8192, n_slots >= 0, 0 <= low_watermark <= high_watermark, and
 * recent_tokens, sink_video, sink_audio, text_budget >= 0.  Three kernels: a census of each
 * unit's spans (one wave per unit), the plan (one workgroup per segment), the slot mask.
 */
int omnitide_plan_spans(const int32_t* unit_len, const int32_t* unit_first_slot,
                        const int32_t* unit_last_slot, const uint32_t* unit_flags,
                        const int32_t* unit_id, const uint8_t* modality, int n_seg, int n_slots,
                        int n_units, int low_watermark, int high_watermark, int recent_tokens,
                        int sink_video, int sink_audio, int text_budget, int32_t* keep_len,
                        uint8_t* keep_slot, int32_t* kept_tokens, void* workspace,
                        size_t workspace_bytes, int32_t* d_status, void* stream);

size_t omnitide_plan_spans_workspace_bytes(int n_seg, int n_slots, int n_units);

/*
 * omnitide_compact_kv_spans -- compaction of a span plan (paper: Applying the retention plan --
 * unselected ranges are deleted, every retained token moves down by the deleted tokens before
 * it, a partially retained unit keeps its identity with its new length).  Same arguments,
 * outputs and errors as omnitide_compact_kv_rope with `keep` replaced by
 *   keep_slot  uint8 [n_seg][n_slots_src]: a live slot stays iff its byte is non-zero
 *              (omnitide_plan_spans' output; bytes of empty slots are ignored); a unit with no
 *              remaining slot is dropped and renumbered -1, the others keep their order and are
 *              renumbered densely.  Destination rows keep slot order; each moves down by the
 *              deleted live slots before its source slot.
 * and rope_dims == 0 meaning no rotary re-encoding (keys copied verbatim, rope_base and
 * rope_style ignored); otherwise the rope arguments are as for omnitide_compact_kv_rope.
 * d_status additionally reports OMNITIDE_E_TAGS for a live unit whose slot range
 * (unit_first_slot, unit_len) leaves the pool; such a unit keeps nothing.
 */
int omnitide_compact_kv_spans(const void* k_src, const void* v_src, int dtype, int n_seg,
                              int n_slots_src, int n_kv_heads, int head_dim, int page_size,
                              const int32_t* unit_id_src, const uint8_t* modality_src,
                              const int32_t* pos_src, const uint8_t* keep_slot,
                              const int32_t* unit_len, const int32_t* unit_first_slot,
                              int n_units, const void* k_chunk, const void* v_chunk,
                              const uint8_t* chunk_modality, const int32_t* chunk_unit,
                              int chunk_len, void* k_dst, void* v_dst, int cap_dst,
                              int32_t* unit_id_dst, uint8_t* modality_dst, int32_t* pos_dst,
                              int32_t* src_of_dst, int32_t* unit_remap, int32_t* n_ctx,
                              int32_t* n_pages, void* workspace, size_t workspace_bytes,
                              double rope_base, int rope_dims, int rope_style,
                              int32_t* d_status, void* stream);

/*
 * omnitide_chunk_attn -- grouped-query prefill attention of the new chunk over the compacted
 * history plus the chunk (paper: Background, prefill appends the new input's KV and attends over
 * the cache; Retention-aware paging: after packing, attention traverses the contiguous rows
 * [0, n_ctx)).  For query position i in [0, chunk_len) and query head h:
 *   out[i][h] = sum_j softmax_j(scale * <q[i][h], k[j][g]>) v[j][g],  g = h / (n_q_heads/n_kv_heads)
 *   over keys j <= n_ctx - chunk_len + i (causal, anchored bottom-right).
 *   q      [n_seg][chunk_len][n_q_heads][head_dim] of `dtype`
 *   k, v   [n_seg][cap][n_kv_heads][head_dim] of `dtype`: the pools written by
 *          omnitide_compact_kv (the chunk's own keys are the last chunk_len rows before n_ctx)
 *   dtype  OMNITIDE_BF16, or OMNITIDE_F32: q, k and v are then rounded to bf16 (nearest even)
 *          into the workspace first (all cap rows of k and v), and the bf16 kernels run on
 *          the copies
 *   n_ctx  int32 [n_seg], device: rows in use; chunk_len <= n_ctx <= cap is required (device
 *          check: OMNITIDE_E_CAPACITY, the segment's output is then not written)
 *   out    [n_seg][chunk_len][n_q_heads][head_dim] of `out_dtype`: OMNITIDE_F32, or
 *          OMNITIDE_BF16 (the float result rounded to nearest even)
 *   workspace  device scratch of omnitide_attn_workspace_bytes(dtype, ...) bytes (split-KV
 *          partials, and the bf16 copies for float32 inputs; may be NULL when that is 0)
 * Numerics: bf16 inputs, bf16 matrix-core products with fp32 accumulation, fp32 softmax.
 * Limits: head_dim in {64, 128}; n_q_heads % n_kv_heads == 0; chunk_len >= 1; cap >= chunk_len.
 */
int omnitide_chunk_attn(const void* q, const void* k, const void* v, int dtype,
                        const int32_t* n_ctx, int n_seg, int cap, int chunk_len, int n_q_heads,
                        int n_kv_heads, int head_dim, float scale, void* out, int out_dtype,
                        void* workspace, size_t workspace_bytes, int32_t* d_status,
                        void* stream);

size_t omnitide_attn_workspace_bytes(int dtype, int n_seg, int cap, int chunk_len,
                                     int n_q_heads, int n_kv_heads, int head_dim);

/*
 * omnitide_chunk_attn_noalloc -- omnitide_chunk_attn for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels, with the split-KV partials in a fixed array inside the library instead of
 * a caller workspace.  Same arguments, results and errors as omnitide_chunk_attn with bf16
 * inputs (no dtype argument) and without workspace / workspace_bytes; the output is bitwise
 * equal to omnitide_chunk_attn's.
 *   - The array holds OMNITIDE_NOALLOC_SCRATCH_BYTES bytes per device (allocated when the
 *     library's code is loaded on a device, kept until the process ends).  A shape whose
 *     omnitide_attn_workspace_bytes() exceeds it returns OMNITIDE_E_SCRATCH (host check,
 *     nothing enqueued); the 80K-history call (665 queries, 32/8 heads, d 128) needs ~33 MB.
 *   - No allocation or free of any kind.  The array's device address is looked up once per
 *     device (hipGetSymbolAddress, on the first call that runs on that device) and cached.
 *   - Every call on one device shares that device's array: calls that overlap in time on one
 *     device (different streams without ordering between them) race on it and give undefined
 *     results.  Calls ordered on one stream are safe; no call expects the array zeroed.
 */
#define OMNITIDE_NOALLOC_SCRATCH_BYTES (64u << 20)
int omnitide_chunk_attn_noalloc(const void* q, const void* k, const void* v,
                                const int32_t* n_ctx, int n_seg, int cap, int chunk_len,
                                int n_q_heads, int n_kv_heads, int head_dim, float scale,
                                void* out, int out_dtype, int32_t* d_status, void* stream);

/*
 * Native (logical-only) layout: the retained entries stay in their slots after eviction, the
 * new chunk fills the lowest run of empty slots, and attention runs over the physical span
 * (omnitide_span_attn).  Paper: Applying the retention plan (logical deletion, positions shift
 * down, entries stay in place); Fragmentation after logical eviction (holes, physical span);
 * Selective and efficient KV migration, ordered-suffix mode.
 *
 * Preconditions on the tags of a native pool ([n_seg][cap], cap <= 131,072): live entries carry
 * the logical positions 0..n-1 of their segment, each unit's tokens hold consecutive positions
 * and units follow each other in id (temporal) order; slots may be in any physical order.
 *
 * omnitide_evict_native -- logical eviction in place.  Unit u keeps its first keep_len[u] tokens
 * in position order (keep_len NULL: keep[u] != 0 keeps the whole unit).  Kept entries get the
 * unit's new id (kept units renumbered 0.. in order, unit_remap[u], -1 when dropped) and their
 * position minus the tokens deleted before them; evicted slots get unit id -1 and position -1
 * (their K/V bytes stay).  Outputs per segment: kept_tokens, n_kept_units, span (last occupied
 * slot + 1).  unit_len is omnitide_score_units' output.  d_status: OMNITIDE_E_TAGS for an entry
 * whose position lies outside its unit's range (tags then partly rewritten).
 */
int omnitide_evict_native(int n_seg, int cap, int32_t* unit_id, int32_t* pos,
                          const uint8_t* keep, const int32_t* keep_len, const int32_t* unit_len,
                          int n_units, int32_t* unit_remap, int32_t* kept_tokens,
                          int32_t* n_kept_units, int32_t* span, void* workspace,
                          size_t workspace_bytes, int32_t* d_status, void* stream);
size_t omnitide_evict_native_workspace_bytes(int n_seg, int n_units);

/*
 * omnitide_evict_native_rope -- omnitide_evict_native plus the rotary adjustment of the cached
 * keys that stay in place (paper: Applying the retention plan -- a retained token's position
 * drops by the deleted tokens before it and its cached key is re-rotated to match).  Same
 * arguments, outputs and errors as omnitide_evict_native, and:
 *   k       [n_seg][cap][n_kv_heads][head_dim] of `dtype` (OMNITIDE_BF16 or OMNITIDE_F32),
 *           rotary-encoded at the entries' old positions, updated in place: every kept slot
 *           whose position changes by shift (< 0) has each pair (x, y) of its first rope_dims
 *           dimensions per head turned by shift * theta_j (as omnitide_compact_kv_rope, same
 *           precision); the rows of other slots and dimensions >= rope_dims keep their bits.
 *   rope_base, rope_dims, rope_style  as omnitide_compact_kv_rope (OMNITIDE_E_SHAPE if invalid)
 *   workspace  omnitide_evict_native_rope_workspace_bytes() bytes (the unit table and one
 *           shift per slot).
 * The V pool is not touched (values carry no position).
 */
int omnitide_evict_native_rope(int n_seg, int cap, int32_t* unit_id, int32_t* pos,
                               const uint8_t* keep, const int32_t* keep_len,
                               const int32_t* unit_len, int n_units, void* k, int dtype,
                               int n_kv_heads, int head_dim, double rope_base, int rope_dims,
                               int rope_style, int32_t* unit_remap, int32_t* kept_tokens,
                               int32_t* n_kept_units, int32_t* span, void* workspace,
                               size_t workspace_bytes, int32_t* d_status, void* stream);
size_t omnitide_evict_native_rope_workspace_bytes(int n_seg, int n_units, int cap);

/*
 * omnitide_pack_suffix -- ordered-suffix migration in place (paper: scanning back from the end
 * of the cache, the suffix whose packing shortens the page-rounded span by at least a threshold
 * of pages is packed, order kept, everything before it untouched; no qualifying suffix, no
 * move).  Per segment, with span = last occupied slot + 1 and P = page_size: the packed span of
 * cut c is c + (entries at or after c); the largest c < span whose packed span needs at least
 * min_pages fewer pages of P slots than span is taken.  The entries at or after c move to
 * c, c+1, ... in slot order with their tags (positions unchanged); vacated slots become empty.
 * Outputs per segment: cut (-1: nothing moved), moved (entries whose slot changed), span (after
 * packing).  Rows are staged through the workspace (a destination can be an earlier entry's
 * source).  Limits: page_size >= 1, min_pages >= 1, cap <= 131,072.
 */
int omnitide_pack_suffix(void* k, void* v, int dtype, int n_seg, int cap, int n_kv_heads,
                         int head_dim, int page_size, int min_pages, int32_t* unit_id,
                         uint8_t* modality, int32_t* pos, int32_t* span, int32_t* cut,
                         int32_t* moved, void* workspace, size_t workspace_bytes, void* stream);
size_t omnitide_pack_suffix_workspace_bytes(int dtype, int n_seg, int cap, int n_kv_heads,
                                            int head_dim);

/*
 * omnitide_place_chunk -- the new chunk into the lowest run of chunk_len empty slots of the
 * pool (the free space past the span counts).  Row i goes to slot chunk_slot + i with unit id
 * n_kept_units + chunk_unit[i], modality chunk_modality[i] and position kept_tokens + i
 * (kept_tokens, n_kept_units: omnitide_evict_native's outputs).  Outputs per segment:
 * chunk_slot and span (covering the chunk).  d_status: OMNITIDE_E_CAPACITY when no run fits
 * (chunk_slot = -1, nothing written).  workspace: omnitide_place_chunk_workspace_bytes() bytes
 * (an occupancy bitmap).
 */
int omnitide_place_chunk(void* k, void* v, int dtype, int n_seg, int cap, int n_kv_heads,
                         int head_dim, int32_t* unit_id, uint8_t* modality, int32_t* pos,
                         const void* k_chunk, const void* v_chunk,
                         const uint8_t* chunk_modality, const int32_t* chunk_unit,
                         int chunk_len, const int32_t* kept_tokens,
                         const int32_t* n_kept_units, int32_t* chunk_slot, int32_t* span,
                         void* workspace, size_t workspace_bytes, int32_t* d_status,
                         void* stream);
size_t omnitide_place_chunk_workspace_bytes(int n_seg, int cap);

/*
 * omnitide_span_attn -- chunk attention over a pool with holes (paper: Fragmentation after
 * logical eviction -- deletion leaves holes between retained entries, attention is presented
 * the physical span, and a tile can be skipped only when every entry in it is masked).
 * For query position i in [0, chunk_len) and query head h:
 *   out[i][h] = sum_j softmax_j(scale * <q[i][h], k[j][g]>) v[j][g],  g as omnitide_chunk_attn
 *   over slots j < span[seg] with 0 <= key_pos[j] <= q_pos0[seg] + i.
 *   key_pos  int32 [n_seg][cap], device: logical position of each slot's entry, -1 = empty.
 *            The chunk's own keys must be in the pool with positions q_pos0 + i.
 *   span     int32 [n_seg], device: slots presented to attention; chunk_len <= span <= cap
 *            (device check: OMNITIDE_E_CAPACITY, the segment's output is then not written)
 *   q_pos0   int32 [n_seg], device: logical position of chunk query 0
 *   q, k, v, out, scale: as omnitide_chunk_attn.  The K/V bytes of empty slots are never used
 *   (they may hold anything, NaN included).
 *   q, k, v are bf16 and out float32 (OMNITIDE_E_DTYPE is not used here).
 *   workspace  device scratch of omnitide_span_attn_workspace_bytes() bytes (always > 0).
 * traversal -- which slots the kernel visits (the result is the same up to summation order):
 *   OMNITIDE_SPAN_FULL        every 64-slot tile of the span, masked (a kernel presented the
 *                             physical span);
 *   OMNITIDE_SPAN_SKIP_EMPTY  64-slot tiles without an entry are skipped (tile skipping).  In
 *                             both, tiles whose entries are all visible to every query of a
 *                             workgroup run unmasked;
 *   OMNITIDE_SPAN_POSITION_ORDER  the entries are gathered in position order through a
 *                             position -> slot index built in the workspace, so the attention
 *                             visits n = q_pos0 + chunk_len keys in dense 64-key tiles, as
 *                             omnitide_chunk_attn over a compacted pool.  Requires the entries of
 *                             [0, span) to hold the positions 0 .. n - 1 once each (the layout
 *                             omnitide_evict_native and omnitide_place_chunk maintain); a position
 *                             >= n, one held twice, one missing, or q_pos0 outside
 *                             [0, span - chunk_len] is reported as OMNITIDE_E_TAGS on the device
 *                             (the output is then unspecified).  Host limit: cap * n_kv_heads *
 *                             head_dim * 2 < 2^32 (OMNITIDE_E_SHAPE).
 *   other values: OMNITIDE_E_SHAPE.
 * With key_pos[j] = j for j < span and q_pos0 = span - chunk_len this computes
 * omnitide_chunk_attn with n_ctx = span (up to summation order).
 * Limits: as omnitide_chunk_attn, and cap <= 2,097,152.
 */
int omnitide_span_attn(const void* q, const void* k, const void* v, const int32_t* key_pos,
                       const int32_t* span, const int32_t* q_pos0, int n_seg, int cap,
                       int chunk_len, int n_q_heads, int n_kv_heads, int head_dim, float scale,
                       int traversal, float* out, void* workspace, size_t workspace_bytes,
                       int32_t* d_status, void* stream);

size_t omnitide_span_attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads,
                                          int n_kv_heads, int head_dim);

/*
 * omnitide_decode_attn -- decode attention over the compacted pool (paper: Background, decode
 * generates one token at a time reusing the cached states; OmniPage ablation, decode attention
 * time over the native, OmniPage and eagerly compacted layouts).  The chunk attention above
 * with chunk_len = n_q small: for query token i in [0, n_q) (the segment's last n_q positions)
 * and query head h,
 *   out[i][h] = sum_j softmax_j(scale * <q[i][h], k[j][g]>) v[j][g],  g = h / (n_q_heads/n_kv_heads)
 *   over keys j <= n_ctx - n_q + i.
 *   q            bf16 [n_seg][n_q][n_q_heads][head_dim]
 *   k, v         bf16 [n_seg][cap][n_kv_heads][head_dim] (rows [0, n_ctx) are read)
 *   n_ctx        int32 [n_seg] device; n_q <= n_ctx <= cap, else OMNITIDE_E_CAPACITY on the
 *                device and that segment's output is not written
 *   out          float32 [n_seg][n_q][n_q_heads][head_dim]
 *   workspace    device scratch of omnitide_decode_workspace_bytes() bytes (may be NULL when
 *                that is 0): split partials
 * Arithmetic: bf16 inputs, float dot products, softmax and accumulation (probabilities are not
 * rounded).  Bandwidth-bound: each (key, KV head) row is read once per call.
 * Limits: n_q * (n_q_heads / n_kv_heads) <= 8, head_dim in {64, 128}, scale finite.
 */
int omnitide_decode_attn(const void* q, const void* k, const void* v, const int32_t* n_ctx,
                         int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                         int head_dim, float scale, float* out, void* workspace,
                         size_t workspace_bytes, int32_t* d_status, void* stream);

size_t omnitide_decode_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads,
                                       int n_kv_heads, int head_dim);

/*
 * omnitide_decode_span_attn -- decode attention over a pool with holes (paper: OmniPage
 * ablation, decode attention time over the native and OmniPage layouts; Fragmentation after
 * logical eviction: attention is presented the physical span).  For query token i in [0, n_q)
 * and query head h:
 *   out[i][h] = sum_j softmax_j(scale * <q[i][h], k[j][g]>) v[j][g],  g = h / (n_q_heads/n_kv_heads)
 *   over slots j < span[seg] with 0 <= key_pos[j] <= q_pos0[seg] + i.
 *   key_pos, span, q_pos0: as omnitide_span_attn (the query tokens' own keys are in the pool at
 *            positions q_pos0 + i); n_q <= span <= cap, else OMNITIDE_E_CAPACITY on the device
 *            and that segment's output is not written.  The K/V bytes of empty slots are never
 *            used (they may hold anything, NaN included).
 *   traversal  as omnitide_span_attn: OMNITIDE_SPAN_FULL (every tile of the span is read and
 *            masked, a kernel presented the physical span), OMNITIDE_SPAN_SKIP_EMPTY (64-slot
 *            tiles without an entry are not read) or OMNITIDE_SPAN_POSITION_ORDER (the entries
 *            read in position order through a position -> slot index; they must hold the
 *            positions 0 .. q_pos0 + n_q - 1 once each, else OMNITIDE_E_TAGS on the device and
 *            the output is unspecified; host limit cap * n_kv_heads * head_dim * 2 < 2^32);
 *            other values: OMNITIDE_E_SHAPE.
 *   q, k, v, out, scale, arithmetic and limits: as omnitide_decode_attn; cap <= 2,097,152.
 *   workspace  device scratch of omnitide_decode_span_workspace_bytes() bytes (always > 0).
 * With key_pos[j] = j for j < span and q_pos0 = span - n_q this computes omnitide_decode_attn
 * with n_ctx = span (up to summation order).
 */
int omnitide_decode_span_attn(const void* q, const void* k, const void* v,
                              const int32_t* key_pos, const int32_t* span,
                              const int32_t* q_pos0, int n_seg, int cap, int n_q,
                              int n_q_heads, int n_kv_heads, int head_dim, float scale,
                              int traversal, float* out, void* workspace,
                              size_t workspace_bytes, int32_t* d_status, void* stream);

size_t omnitide_decode_span_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads,
                                            int n_kv_heads, int head_dim);

/* Static description of a status code. */
const char* omnitide_status_string(int code);

/* Library version string. */
const char* omnitide_version(void);

#ifdef __cplusplus
}
#endif

#endif /* OMNITIDE_H */
