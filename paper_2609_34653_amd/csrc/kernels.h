// Internal launchers of the OmniTide kernels (called by abi.cpp after host validation).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace omnitide {

// Byte counts rounded up to the 256-byte boundaries workspaces place their arrays on.
__host__ __device__ inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }

hipError_t launch_score(const void* k, int dtype, int n_seg, int n_slots, int row_elems,
                        const int32_t* unit_id, const uint8_t* modality, const uint32_t wq[4],
                        int n_units, uint64_t* unit_wsum, int32_t* unit_len, int32_t* unit_first,
                        int32_t* unit_last, uint32_t* unit_flags, int32_t* d_status,
                        hipStream_t stream);

hipError_t launch_select(const uint64_t* unit_wsum, const int32_t* unit_len,
                         const int32_t* unit_first, const int32_t* unit_last,
                         const uint32_t* unit_flags, int n_seg, int n_units, int budget,
                         int recent, uint64_t* unit_score, uint8_t* keep, int32_t* kept_tokens,
                         int32_t* d_status, hipStream_t stream);

struct CompactArgs {
  const void* k_src;
  const void* v_src;
  int n_seg, n_slots_src, row_bytes, page_size;
  const int32_t* unit_id_src;
  const uint8_t* modality_src;
  const int32_t* pos_src;
  const uint8_t* keep;
  const int32_t* keep_len = nullptr;   // kept leading tokens per unit; replaces keep when set
  const uint8_t* keep_slot = nullptr;  // per-slot keep mask, used when use_mask (replaces keep
  bool use_mask = false;               // and keep_len; may be null only without slots)
  const int32_t* unit_len;
  const int32_t* unit_first;
  int n_units;
  const void* k_chunk;
  const void* v_chunk;
  const uint8_t* chunk_modality;
  const int32_t* chunk_unit;
  int chunk_len;
  void* k_dst;
  void* v_dst;
  int cap_dst;
  int32_t* unit_id_dst;
  uint8_t* modality_dst;
  int32_t* pos_dst;
  int32_t* src_of_dst;
  int32_t* unit_remap;
  int32_t* n_ctx;
  int32_t* n_pages;
  void* workspace;
  int32_t* d_status;
  // rotary re-encoding of moved keys: off when rope_dims == 0
  int n_kv_heads = 0, head_dim = 0;
  double rope_base = 0.0;
  int rope_dims = 0;
  bool rope_half = true;
};

size_t compact_workspace_bytes(int n_seg, int n_units, int cap_dst);

struct SpanPlanArgs {
  const int32_t* unit_len;
  const int32_t* unit_first;
  const int32_t* unit_last;
  const uint32_t* unit_flags;
  const int32_t* unit_id;
  const uint8_t* modality;
  int n_seg, n_slots, n_units;
  int low, high, recent, sink_video, sink_audio, text_budget;
  int32_t* keep_len;
  uint8_t* keep_slot;
  int32_t* kept_tokens;
  void* workspace;
  int32_t* d_status;
};

// Span-plan workspace per segment: a per-slot code, then three per-unit arrays.
__host__ __device__ inline size_t span_ws_info_bytes(int n_slots) {
  return (static_cast<size_t>(n_slots) * 4 + 255) / 256 * 256;
}
__host__ __device__ inline size_t span_ws_seg_bytes(int n_slots, int n_units) {
  return span_ws_info_bytes(n_slots) + (static_cast<size_t>(n_units) * 12 + 255) / 256 * 256;
}
size_t span_plan_workspace_bytes(int n_seg, int n_slots, int n_units);
hipError_t launch_plan_spans(const SpanPlanArgs& a, hipStream_t stream);

// Native layout: logical eviction in place, ordered-suffix packing, chunk placement.
struct EvictArgs {
  int n_seg, cap, n_units;
  int32_t* unit_id;          // [n_seg][cap], in place
  int32_t* pos;              // [n_seg][cap], in place
  const uint8_t* keep;       // one of keep / keep_len
  const int32_t* keep_len;
  const int32_t* unit_len;
  int32_t* unit_remap;
  int32_t* kept_tokens;
  int32_t* n_kept_units;
  int32_t* span;
  void* workspace;
  int32_t* d_status;
  // rotary adjustment of the keys that stay (off when rope_dims == 0)
  void* k = nullptr;
  int dtype = 0, n_kv_heads = 0, head_dim = 0;
  double rope_base = 0.0;
  int rope_dims = 0;
  bool rope_half = true;
};
struct SuffixArgs {
  int n_seg, cap, row_bytes, page_size, min_pages;
  void* k;
  void* v;
  int32_t* unit_id;
  uint8_t* modality;
  int32_t* pos;
  int32_t* span;
  int32_t* cut;
  int32_t* moved;
  void* workspace;
};
struct PlaceArgs {
  int n_seg, cap, row_bytes, chunk_len;
  void* k;
  void* v;
  int32_t* unit_id;
  uint8_t* modality;
  int32_t* pos;
  const void* k_chunk;
  const void* v_chunk;
  const uint8_t* chunk_modality;
  const int32_t* chunk_unit;
  const int32_t* kept_tokens;
  const int32_t* n_kept_units;
  int32_t* chunk_slot;
  int32_t* span;
  void* workspace;
  int32_t* d_status;
};
int native_max_cap();
size_t place_workspace_bytes(int n_seg, int cap);
size_t evict_workspace_bytes(int n_seg, int n_units);
size_t evict_rope_workspace_bytes(int n_seg, int n_units, int cap);
// Keys of the slots whose position changes (shift != 0) re-rotated in place by that change.
hipError_t launch_rope_in_place(void* k, int dtype, int n_seg, int cap, int n_kv_heads,
                                int head_dim, const int32_t* shift, double rope_base,
                                int rope_dims, bool rope_half, hipStream_t stream);
size_t suffix_workspace_bytes(int n_seg, int cap, int row_bytes);
hipError_t launch_evict(const EvictArgs& a, hipStream_t stream);
hipError_t launch_pack_suffix(const SuffixArgs& a, hipStream_t stream);
hipError_t launch_place_chunk(const PlaceArgs& a, hipStream_t stream);
hipError_t launch_compact(const CompactArgs& a, hipStream_t stream);

struct AttnArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* n_ctx;
  int n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim;
  float scale;
  void* out;
  bool out_bf16 = false;              // out is bf16 (rounded to nearest even), else float32
  bool in_f32 = false;                // q, k, v are float32: cast to bf16 in the workspace
  void* workspace;
  int32_t* d_status;
  // span mode (keys = the slots [0, span) of a pool with holes; n_ctx holds the span):
  const int32_t* key_pos = nullptr;   // [n_seg][cap] logical position, -1 = empty slot
  const int32_t* q_pos0 = nullptr;    // [n_seg] logical position of chunk query 0
  bool skip_empty = true;             // skip 64-slot tiles without an entry
  bool pos_order = false;             // keys in position order through a position index (the
                                      // entries hold positions 0 .. q_pos0 + chunk_len - 1)
};

int attn_num_splits(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                    int head_dim);

// Active 64-slot tiles of a span (a pool with holes), shared by the span chunk attention and the
// span decode: per tile its largest position, an empty-slot flag and 64 occupancy bits; the
// list of visited tiles (every tile of [0, span), or only tiles holding an entry) and its
// length per segment.  Segments whose span is outside [min_span, cap] get no tiles.
struct SpanTiles {
  int4* info;          // [n_seg][max_tiles]
  int32_t* list;       // [n_seg][max_tiles]
  int32_t* n_active;   // [n_seg]
  uint8_t* act;        // [n_seg][max_tiles]
};
SpanTiles span_tiles_at(void* buf, int n_seg, int cap);
// Key traversals of the chunk and decode attention kernels: the compacted pool's rows, a span's
// 64-slot tiles, or a span's entries in position order through a position -> slot index.
constexpr int kContig = 0, kSpanTiles = 1, kPosOrder = 2;
// Position -> slot index of n_seg spans whose entries hold the positions 0 .. q_pos0 + L - 1
// once each: int32 slot_of[n_seg][cap], then per segment pos_index_blocks(cap) entry counts
// (one per workgroup of the build).  The build reports a repeated or too-large position as
// OMNITIDE_E_TAGS; the attention kernels check that the counts add up to q_pos0 + L.
int pos_index_blocks(int cap);
size_t pos_index_bytes(int n_seg, int cap);
hipError_t launch_pos_index(const int32_t* key_pos, const int32_t* span, const int32_t* q_pos0,
                            int n_seg, int cap, int L, int32_t* slot_of, hipStream_t stream,
                            int32_t* d_status);
size_t span_tiles_bytes(int n_seg, int cap);
hipError_t launch_span_tiles(const int32_t* key_pos, const int32_t* span, int n_seg, int cap,
                             int min_span, bool skip_empty, void* buf, hipStream_t stream);
size_t attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                            int head_dim);
// bf16 copies of float32 q, k, v (placed after the 256-aligned partials)
size_t attn_cast_bytes(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                       int head_dim);
hipError_t launch_attn(const AttnArgs& a, hipStream_t stream);
// launch_attn with the split-KV partials in the library's fixed per-device scratch array (no
// allocation; the caller has checked attn_workspace_bytes <= OMNITIDE_NOALLOC_SCRATCH_BYTES).
hipError_t launch_attn_noalloc(const AttnArgs& a, hipStream_t stream);
size_t span_attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads,
                                 int n_kv_heads, int head_dim);
int span_attn_max_cap();

struct DecodeArgs {
  const void* q;
  const void* k;
  const void* v;
  const int32_t* n_ctx;
  int n_seg, cap, n_q, n_q_heads, n_kv_heads, head_dim;
  float scale;
  float* out;
  void* workspace;
  int32_t* d_status;
  // span mode (keys = the slots [0, span) of a pool with holes; n_ctx holds the span):
  const int32_t* key_pos = nullptr;   // [n_seg][cap] logical position, -1 = empty slot
  const int32_t* q_pos0 = nullptr;    // [n_seg] logical position of query token 0
  bool skip_empty = true;             // visit only 64-slot tiles holding an entry
  bool pos_order = false;             // keys in position order through a position index
};

int decode_num_splits(int n_seg, int cap, int n_kv_heads);
size_t decode_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                              int head_dim);
size_t decode_span_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                                   int head_dim);
int decode_max_query_vectors();
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);

}  // namespace omnitide
