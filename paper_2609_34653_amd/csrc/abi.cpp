// C ABI of the OmniTide stream step: host-side validation, then kernel launches.
//
// Validation runs before any HIP runtime call, so a misuse error is returned without touching
// the device (and can be exercised on a machine with no GPU).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <initializer_list>

#include "kernels.h"
#include "omnitide.h"

namespace {

using omnitide::AttnArgs;
using omnitide::CompactArgs;
using omnitide::DecodeArgs;

struct Range {
  const void* p;
  size_t bytes;
};

bool overlaps(Range a, Range b) {
  if (a.p == nullptr || b.p == nullptr || a.bytes == 0 || b.bytes == 0) return false;
  const uintptr_t a0 = reinterpret_cast<uintptr_t>(a.p), b0 = reinterpret_cast<uintptr_t>(b.p);
  return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

// Every output range must be disjoint from every input range and from every other output.
bool any_alias(std::initializer_list<Range> outs, std::initializer_list<Range> ins) {
  for (auto o = outs.begin(); o != outs.end(); ++o) {
    for (const Range& i : ins)
      if (overlaps(*o, i)) return true;
    for (auto o2 = o + 1; o2 != outs.end(); ++o2)
      if (overlaps(*o, *o2)) return true;
  }
  return false;
}

bool all_set(std::initializer_list<const void*> ptrs) {
  for (const void* p : ptrs)
    if (p == nullptr) return false;
  return true;
}

int elt_bytes(int dtype) { return dtype == OMNITIDE_BF16 ? 2 : dtype == OMNITIDE_F32 ? 4 : 0; }

bool row_ok(int n_kv_heads, int head_dim) {
  return (head_dim == 64 || head_dim == 128) && n_kv_heads >= 1 &&
         static_cast<long>(n_kv_heads) * head_dim <= OMNITIDE_MAX_ROW_ELEMS;
}

constexpr int kMaxGridY = 65535;

int hip_status(hipError_t e) { return e == hipSuccess ? OMNITIDE_OK : OMNITIDE_E_HIP; }

}  // namespace

extern "C" {

int omnitide_score_units(const void* k, int dtype, int n_seg, int n_slots, int n_kv_heads,
                         int head_dim, const int32_t* unit_id, const uint8_t* modality,
                         const float* weights, int n_units, uint64_t* unit_wsum,
                         int32_t* unit_len, int32_t* unit_first_slot, int32_t* unit_last_slot,
                         uint32_t* unit_flags, int32_t* d_status, void* stream) {
  if (!all_set({unit_wsum, unit_len, unit_first_slot, unit_last_slot, unit_flags, weights}))
    return OMNITIDE_E_NULL;
  if (n_slots > 0 && !all_set({k, unit_id, modality})) return OMNITIDE_E_NULL;
  const int eb = elt_bytes(dtype);
  if (eb == 0) return OMNITIDE_E_DTYPE;
  if (n_seg < 1 || n_seg > kMaxGridY || n_slots < 0 || n_units < 1 ||
      n_units > OMNITIDE_MAX_UNITS || !row_ok(n_kv_heads, head_dim) ||
      static_cast<long>(n_seg) * n_units > INT32_MAX)
    return OMNITIDE_E_SHAPE;
  uint32_t wq[4];
  for (int i = 0; i < 4; ++i) {
    const double w = static_cast<double>(weights[i]) * 256.0;
    if (!(w >= 1.0 && w <= 1024.0) || std::floor(w) != w) return OMNITIDE_E_WEIGHT;
    wq[i] = static_cast<uint32_t>(w);
  }
  const size_t slots = static_cast<size_t>(n_seg) * n_slots;
  const size_t units = static_cast<size_t>(n_seg) * n_units;
  const int row_elems = n_kv_heads * head_dim;
  if (any_alias({{unit_wsum, units * 8}, {unit_len, units * 4}, {unit_first_slot, units * 4},
                 {unit_last_slot, units * 4}, {unit_flags, units * 4}, {d_status, 4}},
                {{k, slots * row_elems * eb}, {unit_id, slots * 4}, {modality, slots}}))
    return OMNITIDE_E_ALIAS;
  return hip_status(omnitide::launch_score(
      k, dtype, n_seg, n_slots, row_elems, unit_id, modality, wq, n_units, unit_wsum, unit_len,
      unit_first_slot, unit_last_slot, unit_flags, d_status, static_cast<hipStream_t>(stream)));
}

int omnitide_select_units(const uint64_t* unit_wsum, const int32_t* unit_len,
                          const int32_t* unit_first_slot, const int32_t* unit_last_slot,
                          const uint32_t* unit_flags, int n_seg, int n_units, int budget_tokens,
                          int recent_tokens, uint64_t* unit_score, uint8_t* keep,
                          int32_t* kept_tokens, int32_t* d_status, void* stream) {
  if (!all_set({unit_wsum, unit_len, unit_first_slot, unit_last_slot, unit_flags, unit_score,
                keep, kept_tokens}))
    return OMNITIDE_E_NULL;
  if (n_seg < 1 || n_units < 1 || n_units > OMNITIDE_MAX_UNITS || budget_tokens < 0 ||
      recent_tokens < 0 || static_cast<long>(n_seg) * n_units > INT32_MAX)
    return OMNITIDE_E_SHAPE;
  const size_t units = static_cast<size_t>(n_seg) * n_units;
  if (any_alias({{unit_score, units * 8}, {keep, units}, {kept_tokens, n_seg * 4ull},
                 {d_status, 4}},
                {{unit_wsum, units * 8}, {unit_len, units * 4}, {unit_first_slot, units * 4},
                 {unit_last_slot, units * 4}, {unit_flags, units * 4}}))
    return OMNITIDE_E_ALIAS;
  return hip_status(omnitide::launch_select(unit_wsum, unit_len, unit_first_slot,
                                            unit_last_slot, unit_flags, n_seg, n_units,
                                            budget_tokens, recent_tokens, unit_score, keep,
                                            kept_tokens, d_status,
                                            static_cast<hipStream_t>(stream)));
}

size_t omnitide_compact_workspace_bytes(int n_seg, int n_units, int cap_dst) {
  if (n_seg < 1 || n_units < 1 || cap_dst < 0) return 0;
  return omnitide::compact_workspace_bytes(n_seg, n_units, cap_dst);
}

namespace {

int compact_impl(const void* k_src, const void* v_src, int dtype, int n_seg, int n_slots_src,
                 int n_kv_heads, int head_dim, int page_size, const int32_t* unit_id_src,
                 const uint8_t* modality_src, const int32_t* pos_src, const uint8_t* keep,
                 const int32_t* keep_len, const uint8_t* keep_slot, bool use_mask,
                 const int32_t* unit_len, const int32_t* unit_first_slot, int n_units,
                 const void* k_chunk, const void* v_chunk, const uint8_t* chunk_modality,
                 const int32_t* chunk_unit, int chunk_len, void* k_dst, void* v_dst, int cap_dst,
                 int32_t* unit_id_dst, uint8_t* modality_dst, int32_t* pos_dst,
                 int32_t* src_of_dst, int32_t* unit_remap, int32_t* n_ctx, int32_t* n_pages,
                 void* workspace, size_t workspace_bytes, bool rope, double rope_base,
                 int rope_dims, int rope_style, int32_t* d_status, void* stream) {
  // the plan: per-unit keep flags or kept prefixes, or (use_mask) a per-slot mask, which may
  // be NULL only for a pool without slots
  const void* plan = use_mask ? static_cast<const void*>(unit_len)
                     : keep != nullptr ? static_cast<const void*>(keep)
                                       : static_cast<const void*>(keep_len);
  if (!all_set({plan, unit_len, unit_first_slot, k_dst, v_dst, unit_id_dst, modality_dst,
                pos_dst, src_of_dst, unit_remap, n_ctx, n_pages}))
    return OMNITIDE_E_NULL;
  if (n_slots_src > 0 && !all_set({k_src, v_src, unit_id_src, modality_src, pos_src}))
    return OMNITIDE_E_NULL;
  if (use_mask && n_slots_src > 0 && keep_slot == nullptr) return OMNITIDE_E_NULL;
  if (chunk_len > 0 && !all_set({k_chunk, v_chunk, chunk_modality, chunk_unit}))
    return OMNITIDE_E_NULL;
  const int eb = elt_bytes(dtype);
  if (eb == 0) return OMNITIDE_E_DTYPE;
  if (rope) {
    const int chunk_elems = 16 / eb;
    if (!(rope_style == OMNITIDE_ROPE_HALF || rope_style == OMNITIDE_ROPE_INTERLEAVED) ||
        rope_dims < 2 || rope_dims % 2 != 0 || rope_dims > head_dim ||
        (rope_style == OMNITIDE_ROPE_HALF && (rope_dims / 2) % chunk_elems != 0) ||
        !(std::isfinite(rope_base) && rope_base > 1.0))
      return OMNITIDE_E_SHAPE;
  }
  if (n_seg < 1 || n_seg > kMaxGridY || n_slots_src < 0 || n_units < 1 ||
      n_units > OMNITIDE_MAX_UNITS || !row_ok(n_kv_heads, head_dim) || chunk_len < 0 ||
      !(page_size == 32 || page_size == 64 || page_size == 128 || page_size == 256) ||
      static_cast<long>(n_seg) * n_units > INT32_MAX)
    return OMNITIDE_E_SHAPE;
  if (cap_dst < chunk_len || cap_dst < 1) return OMNITIDE_E_CAPACITY;
  const size_t need = omnitide::compact_workspace_bytes(n_seg, n_units, cap_dst);
  if (workspace == nullptr || workspace_bytes < need) return OMNITIDE_E_WORKSPACE;
  const size_t row = static_cast<size_t>(n_kv_heads) * head_dim * eb;
  const size_t src_slots = static_cast<size_t>(n_seg) * n_slots_src;
  const size_t dst_slots = static_cast<size_t>(n_seg) * cap_dst;
  const size_t units = static_cast<size_t>(n_seg) * n_units;
  const size_t chunk_rows = static_cast<size_t>(n_seg) * chunk_len;
  if (any_alias({{k_dst, dst_slots * row}, {v_dst, dst_slots * row}, {unit_id_dst, dst_slots * 4},
                 {modality_dst, dst_slots}, {pos_dst, dst_slots * 4}, {src_of_dst, dst_slots * 4},
                 {unit_remap, units * 4}, {n_ctx, n_seg * 4ull}, {n_pages, n_seg * 4ull},
                 {workspace, need}, {d_status, 4}},
                {{k_src, src_slots * row}, {v_src, src_slots * row}, {unit_id_src, src_slots * 4},
                 {modality_src, src_slots}, {pos_src, src_slots * 4}, {keep, units},
                 {keep_len, units * 4}, {keep_slot, src_slots},
                 {unit_len, units * 4}, {unit_first_slot, units * 4},
                 {k_chunk, chunk_rows * row}, {v_chunk, chunk_rows * row},
                 {chunk_modality, static_cast<size_t>(chunk_len)},
                 {chunk_unit, static_cast<size_t>(chunk_len) * 4}}))
    return OMNITIDE_E_ALIAS;
  CompactArgs a;
  a.k_src = k_src;
  a.v_src = v_src;
  a.n_seg = n_seg;
  a.n_slots_src = n_slots_src;
  a.row_bytes = static_cast<int>(row);
  a.page_size = page_size;
  a.unit_id_src = unit_id_src;
  a.modality_src = modality_src;
  a.pos_src = pos_src;
  a.keep = keep;
  a.keep_len = keep_len;
  a.keep_slot = keep_slot;
  a.use_mask = use_mask;
  a.unit_len = unit_len;
  a.unit_first = unit_first_slot;
  a.n_units = n_units;
  a.k_chunk = k_chunk;
  a.v_chunk = v_chunk;
  a.chunk_modality = chunk_modality;
  a.chunk_unit = chunk_unit;
  a.chunk_len = chunk_len;
  a.k_dst = k_dst;
  a.v_dst = v_dst;
  a.cap_dst = cap_dst;
  a.unit_id_dst = unit_id_dst;
  a.modality_dst = modality_dst;
  a.pos_dst = pos_dst;
  a.src_of_dst = src_of_dst;
  a.unit_remap = unit_remap;
  a.n_ctx = n_ctx;
  a.n_pages = n_pages;
  a.workspace = workspace;
  a.d_status = d_status;
  a.n_kv_heads = n_kv_heads;
  a.head_dim = head_dim;
  a.rope_base = rope_base;
  a.rope_dims = rope ? rope_dims : 0;
  a.rope_half = rope_style == OMNITIDE_ROPE_HALF;
  return hip_status(omnitide::launch_compact(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

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
                        size_t workspace_bytes, int32_t* d_status, void* stream) {
  return compact_impl(k_src, v_src, dtype, n_seg, n_slots_src, n_kv_heads, head_dim, page_size,
                      unit_id_src, modality_src, pos_src, keep, nullptr, nullptr, false,
                      unit_len, unit_first_slot,
                      n_units, k_chunk, v_chunk, chunk_modality, chunk_unit, chunk_len, k_dst,
                      v_dst, cap_dst, unit_id_dst, modality_dst, pos_dst, src_of_dst,
                      unit_remap, n_ctx, n_pages, workspace, workspace_bytes, false, 0.0, 0, 0,
                      d_status, stream);
}

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
                             int32_t* d_status, void* stream) {
  return compact_impl(k_src, v_src, dtype, n_seg, n_slots_src, n_kv_heads, head_dim, page_size,
                      unit_id_src, modality_src, pos_src, keep, nullptr, nullptr, false,
                      unit_len, unit_first_slot,
                      n_units, k_chunk, v_chunk, chunk_modality, chunk_unit, chunk_len, k_dst,
                      v_dst, cap_dst, unit_id_dst, modality_dst, pos_dst, src_of_dst,
                      unit_remap, n_ctx, n_pages, workspace, workspace_bytes, true, rope_base,
                      rope_dims, rope_style, d_status, stream);
}

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
                              int32_t* d_status, void* stream) {
  return compact_impl(k_src, v_src, dtype, n_seg, n_slots_src, n_kv_heads, head_dim, page_size,
                      unit_id_src, modality_src, pos_src, nullptr, nullptr, keep_slot, true,
                      unit_len,
                      unit_first_slot, n_units, k_chunk, v_chunk, chunk_modality, chunk_unit,
                      chunk_len, k_dst, v_dst, cap_dst, unit_id_dst, modality_dst, pos_dst,
                      src_of_dst, unit_remap, n_ctx, n_pages, workspace, workspace_bytes,
                      rope_dims != 0, rope_base, rope_dims, rope_style, d_status, stream);
}

size_t omnitide_plan_spans_workspace_bytes(int n_seg, int n_slots, int n_units) {
  if (n_seg < 1 || n_slots < 0 || n_units < 1) return 0;
  return omnitide::span_plan_workspace_bytes(n_seg, n_slots, n_units);
}

int omnitide_plan_spans(const int32_t* unit_len, const int32_t* unit_first_slot,
                        const int32_t* unit_last_slot, const uint32_t* unit_flags,
                        const int32_t* unit_id, const uint8_t* modality, int n_seg, int n_slots,
                        int n_units, int low_watermark, int high_watermark, int recent_tokens,
                        int sink_video, int sink_audio, int text_budget, int32_t* keep_len,
                        uint8_t* keep_slot, int32_t* kept_tokens, void* workspace,
                        size_t workspace_bytes, int32_t* d_status, void* stream) {
  if (!all_set({unit_len, unit_first_slot, unit_last_slot, unit_flags, keep_len, kept_tokens}))
    return OMNITIDE_E_NULL;
  if (n_slots > 0 && !all_set({unit_id, modality, keep_slot})) return OMNITIDE_E_NULL;
  if (n_seg < 1 || n_seg > kMaxGridY || n_slots < 0 || n_units < 1 ||
      n_units > OMNITIDE_MAX_UNITS || low_watermark < 0 || high_watermark < low_watermark ||
      recent_tokens < 0 || sink_video < 0 || sink_audio < 0 || text_budget < 0 ||
      static_cast<long>(n_seg) * n_units > INT32_MAX ||
      static_cast<long>(n_seg) * n_slots > INT32_MAX)
    return OMNITIDE_E_SHAPE;
  const size_t need = omnitide::span_plan_workspace_bytes(n_seg, n_slots, n_units);
  if (workspace == nullptr || workspace_bytes < need) return OMNITIDE_E_WORKSPACE;
  const size_t units = static_cast<size_t>(n_seg) * n_units;
  const size_t slots = static_cast<size_t>(n_seg) * n_slots;
  if (any_alias({{keep_len, units * 4}, {keep_slot, slots}, {kept_tokens, n_seg * 4ull},
                 {workspace, need}, {d_status, 4}},
                {{unit_len, units * 4}, {unit_first_slot, units * 4}, {unit_last_slot, units * 4},
                 {unit_flags, units * 4}, {unit_id, slots * 4}, {modality, slots}}))
    return OMNITIDE_E_ALIAS;
  omnitide::SpanPlanArgs a;
  a.unit_len = unit_len;
  a.unit_first = unit_first_slot;
  a.unit_last = unit_last_slot;
  a.unit_flags = unit_flags;
  a.unit_id = unit_id;
  a.modality = modality;
  a.n_seg = n_seg;
  a.n_slots = n_slots;
  a.n_units = n_units;
  a.low = low_watermark;
  a.high = high_watermark;
  a.recent = recent_tokens;
  a.sink_video = sink_video;
  a.sink_audio = sink_audio;
  a.text_budget = text_budget;
  a.keep_len = keep_len;
  a.keep_slot = keep_slot;
  a.kept_tokens = kept_tokens;
  a.workspace = workspace;
  a.d_status = d_status;
  return hip_status(omnitide::launch_plan_spans(a, static_cast<hipStream_t>(stream)));
}

size_t omnitide_attn_workspace_bytes(int dtype, int n_seg, int cap, int chunk_len,
                                     int n_q_heads, int n_kv_heads, int head_dim) {
  if (elt_bytes(dtype) == 0 || n_seg < 1 || cap < 1 || chunk_len < 1 || n_kv_heads < 1 ||
      n_q_heads < n_kv_heads || n_q_heads % n_kv_heads != 0 ||
      !(head_dim == 64 || head_dim == 128))
    return 0;
  const size_t part =
      omnitide::attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim);
  if (dtype == OMNITIDE_BF16) return part;
  return omnitide::align256(part) +
         omnitide::attn_cast_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim);
}

namespace {

// Chunk attention over contiguous rows (key_pos == nullptr) or over a span with holes.
// dtype: of q, k, v (float32 only for contiguous rows: cast to bf16 in the workspace);
// out_dtype: of out (bf16 only for contiguous rows).
int attn_impl(const void* q, const void* k, const void* v, int dtype, const int32_t* n_ctx,
              const int32_t* key_pos, const int32_t* q_pos0, int n_seg, int cap, int chunk_len,
              int n_q_heads, int n_kv_heads, int head_dim, float scale, void* out,
              int out_dtype, void* workspace, size_t workspace_bytes, int32_t* d_status,
              void* stream, bool skip_empty = true, bool noalloc = false,
              bool pos_order = false) {
  const bool span = key_pos != nullptr || q_pos0 != nullptr;
  if (!all_set({q, k, v, n_ctx, out})) return OMNITIDE_E_NULL;
  if (span && !all_set({key_pos, q_pos0})) return OMNITIDE_E_NULL;
  const int eb = elt_bytes(dtype), ob = elt_bytes(out_dtype);
  if (eb == 0 || ob == 0 || ((span || noalloc) && (dtype != OMNITIDE_BF16)) ||
      (span && out_dtype != OMNITIDE_F32))
    return OMNITIDE_E_DTYPE;
  if (n_seg < 1 || n_seg > kMaxGridY || chunk_len < 1 || n_kv_heads < 1 ||
      n_q_heads < n_kv_heads || n_q_heads % n_kv_heads != 0 ||
      !(head_dim == 64 || head_dim == 128) || !std::isfinite(scale) ||
      static_cast<long>(chunk_len) * (n_q_heads / n_kv_heads) > (1L << 30))
    return OMNITIDE_E_SHAPE;
  if (cap < chunk_len || (span && cap > omnitide::span_attn_max_cap()))
    return OMNITIDE_E_CAPACITY;
  // position order gathers rows by 32-bit byte offsets from the segment's base
  if (pos_order && static_cast<size_t>(cap) * n_kv_heads * head_dim * 2 > 0xffffffffull)
    return OMNITIDE_E_SHAPE;
  size_t need =
      span ? omnitide::span_attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads,
                                                 head_dim)
           : omnitide::attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads,
                                            head_dim);
  if (dtype == OMNITIDE_F32)
    need = omnitide::align256(need) + omnitide::attn_cast_bytes(n_seg, cap, chunk_len,
                                                                n_q_heads, n_kv_heads, head_dim);
  if (noalloc) {
    if (need > OMNITIDE_NOALLOC_SCRATCH_BYTES) return OMNITIDE_E_SCRATCH;
  } else if (need > 0 && (workspace == nullptr || workspace_bytes < need)) {
    return OMNITIDE_E_WORKSPACE;
  }
  const size_t qrows = static_cast<size_t>(n_seg) * chunk_len * n_q_heads;
  const size_t kv = static_cast<size_t>(n_seg) * cap * n_kv_heads * head_dim * eb;
  if (any_alias({{out, qrows * head_dim * ob}, {noalloc ? nullptr : workspace, need},
                 {d_status, 4}},
                {{q, qrows * head_dim * eb}, {k, kv}, {v, kv}, {n_ctx, n_seg * 4ull},
                 {key_pos, static_cast<size_t>(n_seg) * cap * 4}, {q_pos0, n_seg * 4ull}}))
    return OMNITIDE_E_ALIAS;
  AttnArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.n_ctx = n_ctx;
  a.n_seg = n_seg;
  a.cap = cap;
  a.chunk_len = chunk_len;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.head_dim = head_dim;
  a.scale = scale;
  a.out = out;
  a.out_bf16 = out_dtype == OMNITIDE_BF16;
  a.in_f32 = dtype == OMNITIDE_F32;
  a.workspace = need > 0 ? workspace : nullptr;
  a.d_status = d_status;
  a.key_pos = key_pos;
  a.q_pos0 = q_pos0;
  a.skip_empty = skip_empty;
  a.pos_order = pos_order;
  if (noalloc) return hip_status(omnitide::launch_attn_noalloc(a, static_cast<hipStream_t>(stream)));
  return hip_status(omnitide::launch_attn(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

int omnitide_chunk_attn(const void* q, const void* k, const void* v, int dtype,
                        const int32_t* n_ctx, int n_seg, int cap, int chunk_len, int n_q_heads,
                        int n_kv_heads, int head_dim, float scale, void* out, int out_dtype,
                        void* workspace, size_t workspace_bytes, int32_t* d_status,
                        void* stream) {
  return attn_impl(q, k, v, dtype, n_ctx, nullptr, nullptr, n_seg, cap, chunk_len, n_q_heads,
                   n_kv_heads, head_dim, scale, out, out_dtype, workspace, workspace_bytes,
                   d_status, stream);
}

int omnitide_chunk_attn_noalloc(const void* q, const void* k, const void* v,
                                const int32_t* n_ctx, int n_seg, int cap, int chunk_len,
                                int n_q_heads, int n_kv_heads, int head_dim, float scale,
                                void* out, int out_dtype, int32_t* d_status, void* stream) {
  return attn_impl(q, k, v, OMNITIDE_BF16, n_ctx, nullptr, nullptr, n_seg, cap, chunk_len,
                   n_q_heads, n_kv_heads, head_dim, scale, out, out_dtype, nullptr, 0, d_status,
                   stream, true, true);
}

size_t omnitide_span_attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads,
                                          int n_kv_heads, int head_dim) {
  if (n_seg < 1 || cap < 1 || chunk_len < 1 || n_kv_heads < 1 || n_q_heads < n_kv_heads ||
      n_q_heads % n_kv_heads != 0 || !(head_dim == 64 || head_dim == 128))
    return 0;
  return omnitide::span_attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads,
                                             head_dim);
}

int omnitide_span_attn(const void* q, const void* k, const void* v, const int32_t* key_pos,
                       const int32_t* span, const int32_t* q_pos0, int n_seg, int cap,
                       int chunk_len, int n_q_heads, int n_kv_heads, int head_dim, float scale,
                       int traversal, float* out, void* workspace,
                       size_t workspace_bytes, int32_t* d_status, void* stream) {
  if (key_pos == nullptr || q_pos0 == nullptr) return OMNITIDE_E_NULL;
  if (traversal != OMNITIDE_SPAN_FULL && traversal != OMNITIDE_SPAN_SKIP_EMPTY &&
      traversal != OMNITIDE_SPAN_POSITION_ORDER)
    return OMNITIDE_E_SHAPE;
  return attn_impl(q, k, v, OMNITIDE_BF16, span, key_pos, q_pos0, n_seg, cap, chunk_len,
                   n_q_heads, n_kv_heads, head_dim, scale, out, OMNITIDE_F32, workspace,
                   workspace_bytes, d_status, stream, traversal != OMNITIDE_SPAN_FULL, false,
                   traversal == OMNITIDE_SPAN_POSITION_ORDER);
}

size_t omnitide_evict_native_workspace_bytes(int n_seg, int n_units) {
  if (n_seg < 1 || n_units < 1 || n_units > OMNITIDE_MAX_UNITS) return 0;
  return omnitide::evict_workspace_bytes(n_seg, n_units);
}

namespace {

int evict_impl(int n_seg, int cap, int32_t* unit_id, int32_t* pos, const uint8_t* keep,
               const int32_t* keep_len, const int32_t* unit_len, int n_units, void* k, int dtype,
               int n_kv_heads, int head_dim, bool rope, double rope_base, int rope_dims,
               int rope_style, int32_t* unit_remap, int32_t* kept_tokens, int32_t* n_kept_units,
               int32_t* span, void* workspace, size_t workspace_bytes, int32_t* d_status,
               void* stream) {
  if (!all_set({unit_len, unit_remap, kept_tokens, n_kept_units, span}) ||
      (keep == nullptr && keep_len == nullptr))
    return OMNITIDE_E_NULL;
  if (cap > 0 && !all_set({unit_id, pos})) return OMNITIDE_E_NULL;
  if (rope && cap > 0 && k == nullptr) return OMNITIDE_E_NULL;
  const int eb = rope ? elt_bytes(dtype) : 2;
  if (eb == 0) return OMNITIDE_E_DTYPE;
  if (rope && (!row_ok(n_kv_heads, head_dim) ||
               !(rope_style == OMNITIDE_ROPE_HALF || rope_style == OMNITIDE_ROPE_INTERLEAVED) ||
               rope_dims < 2 || rope_dims % 2 != 0 || rope_dims > head_dim ||
               (rope_style == OMNITIDE_ROPE_HALF && (rope_dims / 2) % (16 / eb) != 0) ||
               !(std::isfinite(rope_base) && rope_base > 1.0)))
    return OMNITIDE_E_SHAPE;
  if (n_seg < 1 || n_seg > kMaxGridY || cap < 0 || cap > omnitide::native_max_cap() ||
      n_units < 1 || n_units > OMNITIDE_MAX_UNITS)
    return OMNITIDE_E_SHAPE;
  const size_t need = rope ? omnitide::evict_rope_workspace_bytes(n_seg, n_units, cap)
                           : omnitide::evict_workspace_bytes(n_seg, n_units);
  if (workspace == nullptr || workspace_bytes < need) return OMNITIDE_E_WORKSPACE;
  const size_t slots = static_cast<size_t>(n_seg) * cap;
  const size_t units = static_cast<size_t>(n_seg) * n_units;
  const size_t kbytes = rope ? slots * n_kv_heads * head_dim * eb : 0;
  if (any_alias({{unit_id, slots * 4}, {pos, slots * 4}, {unit_remap, units * 4},
                 {kept_tokens, n_seg * 4ull}, {n_kept_units, n_seg * 4ull}, {span, n_seg * 4ull},
                 {workspace, need}, {d_status, 4}, {k, kbytes}},
                {{keep, keep_len ? 0 : units}, {keep_len, units * 4}, {unit_len, units * 4}}))
    return OMNITIDE_E_ALIAS;
  omnitide::EvictArgs a;
  a.n_seg = n_seg;
  a.cap = cap;
  a.n_units = n_units;
  a.unit_id = unit_id;
  a.pos = pos;
  a.keep = keep;
  a.keep_len = keep_len;
  a.unit_len = unit_len;
  a.unit_remap = unit_remap;
  a.kept_tokens = kept_tokens;
  a.n_kept_units = n_kept_units;
  a.span = span;
  a.workspace = workspace;
  a.d_status = d_status;
  if (rope) {
    a.k = k;
    a.dtype = dtype;
    a.n_kv_heads = n_kv_heads;
    a.head_dim = head_dim;
    a.rope_base = rope_base;
    a.rope_dims = rope_dims;
    a.rope_half = rope_style == OMNITIDE_ROPE_HALF;
  }
  return hip_status(omnitide::launch_evict(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

int omnitide_evict_native(int n_seg, int cap, int32_t* unit_id, int32_t* pos,
                          const uint8_t* keep, const int32_t* keep_len, const int32_t* unit_len,
                          int n_units, int32_t* unit_remap, int32_t* kept_tokens,
                          int32_t* n_kept_units, int32_t* span, void* workspace,
                          size_t workspace_bytes, int32_t* d_status, void* stream) {
  return evict_impl(n_seg, cap, unit_id, pos, keep, keep_len, unit_len, n_units, nullptr, 0, 0, 0,
                    false, 0.0, 0, 0, unit_remap, kept_tokens, n_kept_units, span, workspace,
                    workspace_bytes, d_status, stream);
}

size_t omnitide_evict_native_rope_workspace_bytes(int n_seg, int n_units, int cap) {
  if (n_seg < 1 || n_units < 1 || cap < 0) return 0;
  return omnitide::evict_rope_workspace_bytes(n_seg, n_units, cap);
}

int omnitide_evict_native_rope(int n_seg, int cap, int32_t* unit_id, int32_t* pos,
                               const uint8_t* keep, const int32_t* keep_len,
                               const int32_t* unit_len, int n_units, void* k, int dtype,
                               int n_kv_heads, int head_dim, double rope_base, int rope_dims,
                               int rope_style, int32_t* unit_remap, int32_t* kept_tokens,
                               int32_t* n_kept_units, int32_t* span, void* workspace,
                               size_t workspace_bytes, int32_t* d_status, void* stream) {
  return evict_impl(n_seg, cap, unit_id, pos, keep, keep_len, unit_len, n_units, k, dtype,
                    n_kv_heads, head_dim, true, rope_base, rope_dims, rope_style, unit_remap,
                    kept_tokens, n_kept_units, span, workspace, workspace_bytes, d_status, stream);
}

size_t omnitide_pack_suffix_workspace_bytes(int dtype, int n_seg, int cap, int n_kv_heads,
                                            int head_dim) {
  const int eb = elt_bytes(dtype);
  if (eb == 0 || n_seg < 1 || cap < 1 || !row_ok(n_kv_heads, head_dim)) return 0;
  return omnitide::suffix_workspace_bytes(n_seg, cap, n_kv_heads * head_dim * eb);
}

int omnitide_pack_suffix(void* k, void* v, int dtype, int n_seg, int cap, int n_kv_heads,
                         int head_dim, int page_size, int min_pages, int32_t* unit_id,
                         uint8_t* modality, int32_t* pos, int32_t* span, int32_t* cut,
                         int32_t* moved, void* workspace, size_t workspace_bytes, void* stream) {
  if (!all_set({k, v, unit_id, modality, pos, span, cut, moved})) return OMNITIDE_E_NULL;
  const int eb = elt_bytes(dtype);
  if (eb == 0) return OMNITIDE_E_DTYPE;
  if (n_seg < 1 || n_seg > kMaxGridY || cap < 1 || cap > omnitide::native_max_cap() ||
      !row_ok(n_kv_heads, head_dim) || page_size < 1 || min_pages < 1)
    return OMNITIDE_E_SHAPE;
  const int row = n_kv_heads * head_dim * eb;
  const size_t need = omnitide::suffix_workspace_bytes(n_seg, cap, row);
  if (workspace == nullptr || workspace_bytes < need) return OMNITIDE_E_WORKSPACE;
  const size_t slots = static_cast<size_t>(n_seg) * cap;
  if (any_alias({{k, slots * row}, {v, slots * row}, {unit_id, slots * 4}, {modality, slots},
                 {pos, slots * 4}, {span, n_seg * 4ull}, {cut, n_seg * 4ull},
                 {moved, n_seg * 4ull}, {workspace, need}},
                {}))
    return OMNITIDE_E_ALIAS;
  omnitide::SuffixArgs a;
  a.n_seg = n_seg;
  a.cap = cap;
  a.row_bytes = row;
  a.page_size = page_size;
  a.min_pages = min_pages;
  a.k = k;
  a.v = v;
  a.unit_id = unit_id;
  a.modality = modality;
  a.pos = pos;
  a.span = span;
  a.cut = cut;
  a.moved = moved;
  a.workspace = workspace;
  return hip_status(omnitide::launch_pack_suffix(a, static_cast<hipStream_t>(stream)));
}

int omnitide_place_chunk(void* k, void* v, int dtype, int n_seg, int cap, int n_kv_heads,
                         int head_dim, int32_t* unit_id, uint8_t* modality, int32_t* pos,
                         const void* k_chunk, const void* v_chunk,
                         const uint8_t* chunk_modality, const int32_t* chunk_unit,
                         int chunk_len, const int32_t* kept_tokens,
                         const int32_t* n_kept_units, int32_t* chunk_slot, int32_t* span,
                         void* workspace, size_t workspace_bytes, int32_t* d_status,
                         void* stream) {
  if (!all_set({k, v, unit_id, modality, pos, k_chunk, v_chunk, chunk_modality, chunk_unit,
                kept_tokens, n_kept_units, chunk_slot, span}))
    return OMNITIDE_E_NULL;
  const int eb = elt_bytes(dtype);
  if (eb == 0) return OMNITIDE_E_DTYPE;
  if (n_seg < 1 || n_seg > kMaxGridY || cap < 1 || cap > omnitide::native_max_cap() ||
      !row_ok(n_kv_heads, head_dim) || chunk_len < 1)
    return OMNITIDE_E_SHAPE;
  if (chunk_len > cap) return OMNITIDE_E_CAPACITY;
  const size_t need = omnitide::place_workspace_bytes(n_seg, cap);
  if (workspace == nullptr || workspace_bytes < need) return OMNITIDE_E_WORKSPACE;
  const int row = n_kv_heads * head_dim * eb;
  const size_t slots = static_cast<size_t>(n_seg) * cap;
  const size_t crow = static_cast<size_t>(n_seg) * chunk_len;
  if (any_alias({{k, slots * row}, {v, slots * row}, {unit_id, slots * 4}, {modality, slots},
                 {pos, slots * 4}, {chunk_slot, n_seg * 4ull}, {span, n_seg * 4ull},
                 {workspace, need}, {d_status, 4}},
                {{k_chunk, crow * row}, {v_chunk, crow * row},
                 {chunk_modality, static_cast<size_t>(chunk_len)},
                 {chunk_unit, static_cast<size_t>(chunk_len) * 4}, {kept_tokens, n_seg * 4ull},
                 {n_kept_units, n_seg * 4ull}}))
    return OMNITIDE_E_ALIAS;
  omnitide::PlaceArgs a;
  a.n_seg = n_seg;
  a.cap = cap;
  a.row_bytes = row;
  a.chunk_len = chunk_len;
  a.k = k;
  a.v = v;
  a.unit_id = unit_id;
  a.modality = modality;
  a.pos = pos;
  a.k_chunk = k_chunk;
  a.v_chunk = v_chunk;
  a.chunk_modality = chunk_modality;
  a.chunk_unit = chunk_unit;
  a.kept_tokens = kept_tokens;
  a.n_kept_units = n_kept_units;
  a.chunk_slot = chunk_slot;
  a.span = span;
  a.workspace = workspace;
  a.d_status = d_status;
  return hip_status(omnitide::launch_place_chunk(a, static_cast<hipStream_t>(stream)));
}

size_t omnitide_place_chunk_workspace_bytes(int n_seg, int cap) {
  if (n_seg < 1 || cap < 1) return 0;
  return omnitide::place_workspace_bytes(n_seg, cap);
}

size_t omnitide_decode_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads,
                                       int n_kv_heads, int head_dim) {
  if (n_seg < 1 || cap < 1 || n_q < 1 || n_kv_heads < 1 || n_q_heads < n_kv_heads ||
      n_q_heads % n_kv_heads != 0 || !(head_dim == 64 || head_dim == 128))
    return 0;
  return omnitide::decode_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads, head_dim);
}

namespace {

// Decode attention over contiguous rows (key_pos == nullptr) or over a span with holes.
int decode_impl(const void* q, const void* k, const void* v, const int32_t* n_ctx,
                const int32_t* key_pos, const int32_t* q_pos0, int n_seg, int cap, int n_q,
                int n_q_heads, int n_kv_heads, int head_dim, float scale, bool skip_empty,
                float* out, void* workspace, size_t workspace_bytes, int32_t* d_status,
                void* stream, bool pos_order = false) {
  const bool span = key_pos != nullptr || q_pos0 != nullptr;
  if (!all_set({q, k, v, n_ctx, out})) return OMNITIDE_E_NULL;
  if (span && !all_set({key_pos, q_pos0})) return OMNITIDE_E_NULL;
  if (n_seg < 1 || n_seg > kMaxGridY || n_q < 1 || n_kv_heads < 1 ||
      n_q_heads < n_kv_heads || n_q_heads % n_kv_heads != 0 || n_kv_heads > kMaxGridY ||
      !(head_dim == 64 || head_dim == 128) || !std::isfinite(scale) ||
      static_cast<long>(n_q) * (n_q_heads / n_kv_heads) > omnitide::decode_max_query_vectors())
    return OMNITIDE_E_SHAPE;
  if (cap < n_q || (span && cap > omnitide::span_attn_max_cap())) return OMNITIDE_E_CAPACITY;
  // position order gathers V rows by 32-bit byte offsets from the segment's base
  if (pos_order && static_cast<size_t>(cap) * n_kv_heads * head_dim * 2 > 0xffffffffull)
    return OMNITIDE_E_SHAPE;
  const size_t need =
      span ? omnitide::decode_span_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads,
                                                   head_dim)
           : omnitide::decode_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads, head_dim);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need)) return OMNITIDE_E_WORKSPACE;
  const size_t qrows = static_cast<size_t>(n_seg) * n_q * n_q_heads;
  const size_t kv = static_cast<size_t>(n_seg) * cap * n_kv_heads * head_dim * 2;
  if (any_alias({{out, qrows * head_dim * 4}, {workspace, need}, {d_status, 4}},
                {{q, qrows * head_dim * 2}, {k, kv}, {v, kv}, {n_ctx, n_seg * 4ull},
                 {key_pos, static_cast<size_t>(n_seg) * cap * 4}, {q_pos0, n_seg * 4ull}}))
    return OMNITIDE_E_ALIAS;
  DecodeArgs a;
  a.q = q;
  a.k = k;
  a.v = v;
  a.n_ctx = n_ctx;
  a.n_seg = n_seg;
  a.cap = cap;
  a.n_q = n_q;
  a.n_q_heads = n_q_heads;
  a.n_kv_heads = n_kv_heads;
  a.head_dim = head_dim;
  a.scale = scale;
  a.out = out;
  a.workspace = need > 0 ? workspace : nullptr;
  a.d_status = d_status;
  a.key_pos = key_pos;
  a.q_pos0 = q_pos0;
  a.skip_empty = skip_empty;
  a.pos_order = pos_order;
  return hip_status(omnitide::launch_decode(a, static_cast<hipStream_t>(stream)));
}

}  // namespace

int omnitide_decode_attn(const void* q, const void* k, const void* v, const int32_t* n_ctx,
                         int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                         int head_dim, float scale, float* out, void* workspace,
                         size_t workspace_bytes, int32_t* d_status, void* stream) {
  return decode_impl(q, k, v, n_ctx, nullptr, nullptr, n_seg, cap, n_q, n_q_heads, n_kv_heads,
                     head_dim, scale, true, out, workspace, workspace_bytes, d_status, stream);
}

size_t omnitide_decode_span_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads,
                                            int n_kv_heads, int head_dim) {
  if (n_seg < 1 || cap < 1 || n_q < 1 || n_kv_heads < 1 || n_q_heads < n_kv_heads ||
      n_q_heads % n_kv_heads != 0 || !(head_dim == 64 || head_dim == 128))
    return 0;
  return omnitide::decode_span_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads,
                                               head_dim);
}

int omnitide_decode_span_attn(const void* q, const void* k, const void* v,
                              const int32_t* key_pos, const int32_t* span,
                              const int32_t* q_pos0, int n_seg, int cap, int n_q,
                              int n_q_heads, int n_kv_heads, int head_dim, float scale,
                              int traversal, float* out, void* workspace,
                              size_t workspace_bytes, int32_t* d_status, void* stream) {
  if (key_pos == nullptr || q_pos0 == nullptr) return OMNITIDE_E_NULL;
  if (traversal != OMNITIDE_SPAN_FULL && traversal != OMNITIDE_SPAN_SKIP_EMPTY &&
      traversal != OMNITIDE_SPAN_POSITION_ORDER)
    return OMNITIDE_E_SHAPE;
  return decode_impl(q, k, v, span, key_pos, q_pos0, n_seg, cap, n_q, n_q_heads, n_kv_heads,
                     head_dim, scale, traversal != OMNITIDE_SPAN_FULL, out, workspace,
                     workspace_bytes, d_status, stream,
                     traversal == OMNITIDE_SPAN_POSITION_ORDER);
}

const char* omnitide_status_string(int code) {
  switch (code) {
    case OMNITIDE_OK: return "ok";
    case OMNITIDE_E_NULL: return "a required pointer is NULL";
    case OMNITIDE_E_SHAPE: return "a size is out of range or inconsistent";
    case OMNITIDE_E_DTYPE: return "unsupported element type";
    case OMNITIDE_E_WEIGHT: return "modality weight is not an exact multiple of 1/256 in (0, 4]";
    case OMNITIDE_E_CAPACITY: return "destination pool too small";
    case OMNITIDE_E_WORKSPACE: return "workspace missing or too small";
    case OMNITIDE_E_ALIAS: return "an output overlaps an input or another output";
    case OMNITIDE_E_HIP: return "HIP kernel launch failed";
    case OMNITIDE_E_SCRATCH: return "the call needs more scratch than the library's fixed array";
    case OMNITIDE_E_BUDGET: return "protected tokens exceed the retention budget";
    case OMNITIDE_E_TAGS: return "malformed unit/modality tags";
    case OMNITIDE_E_RANGE: return "a unit score is outside the range the selection ranks (2^51)";
    default: return "unknown status";
  }
}

const char* omnitide_version(void) { return "omnitide-mi355x 0.1.0 (gfx950)"; }

}  // extern "C"
