// Eager, order-preserving, out-of-place compaction of the retained rows plus the chunk append.
// A unit keeps its first k live tokens: k = len for a unit kept whole (keep flag), or a
// kept-prefix length; or it keeps the slots a per-slot mask marks (the span plan's retained
// spans).  The deleted tokens of a partially kept unit count among the deleted tokens before
// every later token.
//
// Plan: exclusive scans over units give each kept unit its destination offset, its rank (= new
// unit id) and the number of deleted live tokens before it.  Up to 512 units every copy
// workgroup builds this table in LDS itself (wave 0, wave scans), so the compaction is a single
// kernel; beyond, a plan kernel (1024 threads) writes it to the workspace together with, for
// every destination tile, the rank of the unit holding the tile's first row.
// Mask: a count kernel (one wave per unit) gives each unit its kept count, the plan kernel
// scans those, and a map kernel (one wave per unit, one aligned 16-byte block of the mask per
// lane, an in-lane count plus one wave scan per 1,024 slots) writes each kept slot's
// destination row, its tags and its position shift.  Up to 512 units the map kernel builds the
// unit plan in LDS itself (as the copy workgroups do), so no plan kernel runs.
// Copy: one workgroup per destination tile of kTile rows.  The tile's rows are resolved to
// source slots (binary search over the LDS table, or a short forward walk from the workspace
// hint), then every thread moves 16-byte vectors of the K and V rows, and the rows' tags are
// written while the first rows are in flight.  Rows are whole 2 KB (bf16, 8 heads x 128) runs,
// so reads and writes are fully coalesced; source and destination never alias, so a single
// pass is safe (no scratch round trip).
#include "common.h"
#include "kernels.h"

namespace omnitide {
namespace {

constexpr int kPlanThreads = 1024;
constexpr int kPer = OMNITIDE_MAX_UNITS / kPlanThreads;
constexpr int kTile = 16;           // destination rows per copy workgroup
constexpr int kCopyThreads = 256;
// Buffer resource word 3 for raw (unformatted) data on this chip, and a byte offset past any
// buffer (accesses there read zero and write nothing).
constexpr int kBufFlags = 0x00020000;
constexpr int kOutOfBuf = 0x7ffffff0;

struct RankRec {
  int32_t off;     // destination row of the unit's first token
  int32_t first;   // source slot of the unit's first token
  int32_t del;     // deleted live tokens before the unit
  int32_t pad;
};

struct WsLayout {
  size_t rank_off, tile_off, meta_off, count_off, shift_off, seg_bytes;
};

__host__ __device__ inline WsLayout ws_layout(int n_units, int cap_dst) {
  WsLayout w;
  const size_t n_tiles = (static_cast<size_t>(cap_dst) + kTile - 1) / kTile;
  w.rank_off = 0;
  w.tile_off = (static_cast<size_t>(n_units) + 1) * sizeof(RankRec);
  w.meta_off = w.tile_off + ((n_tiles * 4 + 15) / 16) * 16;
  w.count_off = w.meta_off + 16;                                  // mask: kept count per unit
  w.shift_off = w.count_off + ((static_cast<size_t>(n_units) * 4 + 15) / 16) * 16;
  w.seg_bytes = ((w.shift_off + static_cast<size_t>(cap_dst) * 4 + 255) / 256) * 256;
  return w;
}

// Kept tokens per unit come from keep (whole units), keep_len (prefixes) or, when both are
// null, the mask count kernel's per-unit counts in the workspace.
__global__ __launch_bounds__(kPlanThreads) void compact_plan_kernel(
    const uint8_t* __restrict__ keep_g, const int32_t* __restrict__ keep_len_g,
    const int32_t* __restrict__ len_g, const int32_t* __restrict__ first_g, int n_units,
    int chunk_len, int cap_dst, int page_size,
    int32_t* __restrict__ remap_g, int32_t* __restrict__ n_ctx_g,
    int32_t* __restrict__ n_pages_g, uint8_t* __restrict__ ws, int32_t* __restrict__ status) {
  __shared__ int32_t scr[kPlanThreads / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = n_units;
  const int per = (U + kPlanThreads - 1) / kPlanThreads;
  const int u0 = tid * per;
  const size_t base = static_cast<size_t>(seg) * U;
  const WsLayout L = ws_layout(U, cap_dst);
  uint8_t* wseg = ws + static_cast<size_t>(seg) * L.seg_bytes;
  RankRec* rank = reinterpret_cast<RankRec*>(wseg + L.rank_off);
  int32_t* tile_hint = reinterpret_cast<int32_t*>(wseg + L.tile_off);
  int32_t* meta = reinterpret_cast<int32_t*>(wseg + L.meta_off);
  const int32_t* counts = reinterpret_cast<const int32_t*>(wseg + L.count_off);

  int kl[kPer], dl[kPer], fs[kPer];
  int my_k = 0, my_d = 0, my_n = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = u0 + i;
    kl[i] = dl[i] = fs[i] = 0;
    if (i < per && u < U) {
      const int n = max(len_g[base + u], 0);
      if (keep_len_g != nullptr) kl[i] = min(max(keep_len_g[base + u], 0), n);
      else if (keep_g != nullptr) kl[i] = keep_g[base + u] != 0 ? n : 0;
      else kl[i] = min(max(counts[u], 0), n);
      dl[i] = n - kl[i];
      fs[i] = first_g[base + u];
    }
    my_k += kl[i];
    my_d += dl[i];
    my_n += kl[i] > 0 ? 1 : 0;
  }
  int kept, dropped, n_kept;
  int off = block_exclusive_scan(my_k, scr, &kept);
  int del = block_exclusive_scan(my_d, scr, &dropped);
  int rk = block_exclusive_scan(my_n, scr, &n_kept);
  (void)dropped;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = u0 + i;
    if (i < per && u < U) {
      if (kl[i] > 0) {
        rank[rk] = RankRec{off, fs[i], del, 0};
        remap_g[base + u] = rk;
        // hints only for tiles inside the destination (kept may exceed it: capacity error)
        for (int t = (off + kTile - 1) / kTile; t * kTile < min(off + kl[i], cap_dst); ++t)
          tile_hint[t] = rk;
        ++rk;
      } else {
        remap_g[base + u] = -1;
      }
    }
    off += kl[i];
    del += dl[i];
  }
  if (tid == 0) {
    rank[n_kept] = RankRec{kept, 0, 0, 0};
    const int nctx = kept + chunk_len;
    meta[0] = kept;
    meta[1] = n_kept;
    if (nctx > cap_dst) {
      set_status(status, OMNITIDE_E_CAPACITY);
      n_ctx_g[seg] = 0;
      n_pages_g[seg] = 0;
    } else {
      n_ctx_g[seg] = nctx;
      n_pages_g[seg] = (nctx + page_size - 1) / page_size;
    }
  }
}

// Up to 512 units one wave plans (each lane owns 8 consecutive units, wave-level scans).
constexpr int kSmallUnits = 512;
constexpr int kSmallPer = kSmallUnits / kWave;

__device__ inline int wave_excl(int v, int* total) {
  const int inc = wave_inclusive_scan(v);
  *total = __shfl(inc, kWave - 1, kWave);
  return inc - v;
}

// Fused plan (U <= kSmallUnits): every copy workgroup has wave 0 scan the units into LDS (the
// tables compact_plan_kernel writes to the workspace), so the compaction is one kernel.
// Workgroup (0, seg) also writes unit_remap, n_ctx, n_pages and the capacity status.
template <bool FUSED>
struct TilePlan {};
template <>
struct TilePlan<true> {
  // by kept rank; entry kSmallUnits is a sink for the writes of units that keep nothing (roff
  // then takes the sentinel, written last)
  int32_t roff[kSmallUnits + 1];   // destination offset of each kept rank (+ sentinel)
  int32_t rfirst[kSmallUnits + 1]; // first source slot of each kept rank
  int32_t rdel[kSmallUnits + 1];   // deleted live tokens before each kept rank
  int32_t rank_of[kSmallUnits];    // kept rank of each unit, -1 if it keeps nothing
  int32_t kept, n_kept;
};

struct FusedPlanArgs {
  const uint8_t* keep;
  const int32_t* keep_len;
  const int32_t* len;
  const int32_t* first;
  int page_size;
  int32_t* remap;
  int32_t* n_ctx;
  int32_t* n_pages;
  int32_t* status;
  bool mapped;       // history rows were resolved by the mask map kernel
  const int32_t* counts = nullptr;   // kept count per unit (mask path), else keep / keep_len
};

__device__ inline void plan_in_lds(int seg, int n_units, int chunk_len, int cap_dst,
                                   const FusedPlanArgs& f, TilePlan<true>& P) {
  const bool writer = blockIdx.x == 0;
  if (threadIdx.x < kWave) {
    const int lane = threadIdx.x;
    const int U = n_units;
    const int u0 = lane * kSmallPer;
    const size_t base = static_cast<size_t>(seg) * U;
    int nl[kSmallPer], fs[kSmallPer], kq[kSmallPer];
    // all loads first, straight-line (the source of the kept counts is chosen once): one
    // memory round trip; keep flags become counts after every load is issued
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int u = min(u0 + i, U - 1);
      nl[i] = f.len[base + u];
      fs[i] = f.first[base + u];
    }
    const bool flags = f.counts == nullptr && f.keep_len == nullptr;
    if (f.counts != nullptr) {
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i) kq[i] = f.counts[min(u0 + i, U - 1)];
    } else if (f.keep_len != nullptr) {
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i) kq[i] = f.keep_len[base + min(u0 + i, U - 1)];
    } else {
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i) kq[i] = f.keep[base + min(u0 + i, U - 1)];
    }
    int kl[kSmallPer], dl[kSmallPer];
    int my_k = 0, my_d = 0, my_n = 0;
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int n = (u0 + i < U) ? max(nl[i], 0) : 0;
      kl[i] = flags ? (kq[i] != 0 ? n : 0) : min(max(kq[i], 0), n);
      dl[i] = n - kl[i];
      my_k += kl[i];
      my_d += dl[i];
      my_n += kl[i] > 0 ? 1 : 0;
    }
    int kept, dropped, n_kept;
    int off = wave_excl(my_k, &kept);
    int del = wave_excl(my_d, &dropped);
    int rk = wave_excl(my_n, &n_kept);
    (void)dropped;
    // branch-free: a unit that keeps nothing writes to the sink entry (units past U have
    // kl = 0); unit_remap through a buffer whose writes past U are dropped
    const __amdgpu_buffer_rsrc_t r_remap =
        __builtin_amdgcn_make_buffer_rsrc(f.remap + base, 0, 4 * U, kBufFlags);
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      const int u = u0 + i;
      const bool kk = kl[i] > 0;
      const int at = kk ? rk : kSmallUnits;
      P.roff[at] = off;
      P.rfirst[at] = fs[i];
      P.rdel[at] = del;
      P.rank_of[u] = kk ? rk : -1;
      if (writer)
        __builtin_amdgcn_raw_buffer_store_b32(kk ? rk : -1, r_remap, u < U ? 4 * u : kOutOfBuf,
                                              0, 0);
      rk += kk ? 1 : 0;
      off += kl[i];
      del += dl[i];
    }
    if (lane == 0) {
      P.roff[n_kept] = kept;
      P.kept = kept;
      P.n_kept = n_kept;
      if (writer) {
        const int nctx = kept + chunk_len;
        if (nctx > cap_dst) {
          set_status(f.status, OMNITIDE_E_CAPACITY);
          f.n_ctx[seg] = 0;
          f.n_pages[seg] = 0;
        } else {
          f.n_ctx[seg] = nctx;
          f.n_pages[seg] = (nctx + f.page_size - 1) / f.page_size;
        }
      }
    }
  }
  __syncthreads();
}

// Writes the tags of destination rows [r0, r0 + span) (span <= threads) and resolves them:
// src_row[i] is the source slot of row r0 + i, or -1 - c for chunk row c; shift_row[i] (if
// given) is the row's position change (minus the deleted live slots before it; 0 for chunk
// rows).  Rows [n_ctx, cap_dst) become empty slots, so the destination is a complete pool.
// Returns the number of rows to copy (0: none).  Ends with a workgroup barrier.
// With rank_row (and shift_row) given, the tags of the history and chunk rows are left to
// tile_tags: rank_row[i] receives the row's new unit id (history) or the kept unit count
// (chunk), so the caller can issue its row copies first and the tag reads overlap them.
__device__ inline int resolve_rows(int seg, int r0, int span, int nctx, int n_slots,
                                   int chunk_len, int cap_dst, int n_units,
                                   const uint8_t* __restrict__ mod_src,
                                   const int32_t* __restrict__ pos_src,
                                   const uint8_t* __restrict__ chunk_mod,
                                   const int32_t* __restrict__ chunk_unit,
                                   int32_t* __restrict__ uid_dst, uint8_t* __restrict__ mod_dst,
                                   int32_t* __restrict__ pos_dst,
                                   int32_t* __restrict__ src_of_dst,
                                   const uint8_t* __restrict__ ws, int32_t* src_row,
                                   int32_t* shift_row, const TilePlan<true>* plan, bool mapped,
                                   int32_t* rank_row) {
  const int tid = threadIdx.x;
  const size_t dst_tag = static_cast<size_t>(seg) * cap_dst;
  {
    const int r = r0 + tid;
    if (tid < span && r >= nctx && r < cap_dst) {
      uid_dst[dst_tag + r] = -1;
      mod_dst[dst_tag + r] = 0;
      pos_dst[dst_tag + r] = -1;
      src_of_dst[dst_tag + r] = -1;
    }
  }
  if (r0 >= nctx) return 0;
  const int nrows = min(span, nctx - r0);
  const int kept = nctx - chunk_len;
  const size_t src_tag = static_cast<size_t>(seg) * n_slots;

  if (tid < nrows) {
    const int r = r0 + tid;
    if (r < kept && mapped) {                     // the map kernel wrote the row's tags
      const WsLayout L = ws_layout(n_units, cap_dst);
      const int32_t* shift = reinterpret_cast<const int32_t*>(
          ws + static_cast<size_t>(seg) * L.seg_bytes + L.shift_off);
      src_row[tid] = src_of_dst[dst_tag + r];
      if (shift_row) shift_row[tid] = shift[r];
    } else if (r < kept) {
      int k;
      RankRec rec;
      if (plan != nullptr) {                      // largest kept rank k with roff[k] <= r
        int lo = 0, hi = plan->n_kept - 1;
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (plan->roff[mid] <= r) lo = mid; else hi = mid - 1;
        }
        k = lo;
        rec = RankRec{plan->roff[k], plan->rfirst[k], plan->rdel[k], 0};
      } else {
        const WsLayout L = ws_layout(n_units, cap_dst);
        const uint8_t* wseg = ws + static_cast<size_t>(seg) * L.seg_bytes;
        const RankRec* rank = reinterpret_cast<const RankRec*>(wseg + L.rank_off);
        const int32_t* tile_hint = reinterpret_cast<const int32_t*>(wseg + L.tile_off);
        k = tile_hint[r / kTile];
        while (rank[k + 1].off <= r) ++k;
        rec = rank[k];
      }
      const int s = rec.first + (r - rec.off);
      if (rank_row) {
        rank_row[tid] = k;
      } else {
        uid_dst[dst_tag + r] = k;
        mod_dst[dst_tag + r] = mod_src[src_tag + s];
        pos_dst[dst_tag + r] = pos_src[src_tag + s] - rec.del;
        src_of_dst[dst_tag + r] = s;
      }
      src_row[tid] = s;
      if (shift_row) shift_row[tid] = -rec.del;
    } else {
      const int i = r - kept;
      int n_kept_units;
      if (plan != nullptr) {
        n_kept_units = plan->n_kept;
      } else {
        const WsLayout L = ws_layout(n_units, cap_dst);
        const int32_t* meta = reinterpret_cast<const int32_t*>(
            ws + static_cast<size_t>(seg) * L.seg_bytes + L.meta_off);
        n_kept_units = meta[1];
      }
      if (rank_row) {
        rank_row[tid] = n_kept_units;
      } else {
        uid_dst[dst_tag + r] = n_kept_units + chunk_unit[i];
        mod_dst[dst_tag + r] = chunk_mod[i];
        pos_dst[dst_tag + r] = kept + i;
        src_of_dst[dst_tag + r] = -1;
      }
      src_row[tid] = -1 - i;
      if (shift_row) shift_row[tid] = 0;
    }
  }
  __syncthreads();
  return nrows;
}

// resolve_rows over destination tile t (kTile rows).
__device__ inline int resolve_tile(int seg, int t, int nctx, int n_slots, int chunk_len,
                                   int cap_dst, int n_units, const uint8_t* __restrict__ mod_src,
                                   const int32_t* __restrict__ pos_src,
                                   const uint8_t* __restrict__ chunk_mod,
                                   const int32_t* __restrict__ chunk_unit,
                                   int32_t* __restrict__ uid_dst, uint8_t* __restrict__ mod_dst,
                                   int32_t* __restrict__ pos_dst,
                                   int32_t* __restrict__ src_of_dst,
                                   const uint8_t* __restrict__ ws, int32_t* src_row,
                                   int32_t* shift_row, const TilePlan<true>* plan = nullptr,
                                   bool mapped = false, int32_t* rank_row = nullptr) {
  return resolve_rows(seg, t * kTile, kTile, nctx, n_slots, chunk_len, cap_dst, n_units,
                      mod_src, pos_src, chunk_mod, chunk_unit, uid_dst, mod_dst, pos_dst,
                      src_of_dst, ws, src_row, shift_row, plan, mapped, rank_row);
}

// The tag writes resolve_rows leaves to its caller when given rank_row: the history rows
// among destination rows [r0, r0 + nrows) (unless the mask map kernel wrote them) and the chunk
// rows.  One thread per row.
__device__ inline void tile_tags(int seg, int r0, int nrows, int nctx, int n_slots,
                                 int chunk_len, int cap_dst, const uint8_t* __restrict__ mod_src,
                                 const int32_t* __restrict__ pos_src,
                                 const uint8_t* __restrict__ chunk_mod,
                                 const int32_t* __restrict__ chunk_unit,
                                 int32_t* __restrict__ uid_dst, uint8_t* __restrict__ mod_dst,
                                 int32_t* __restrict__ pos_dst, int32_t* __restrict__ src_of_dst,
                                 const int32_t* src_row, const int32_t* shift_row,
                                 const int32_t* rank_row, bool mapped) {
  const int tid = threadIdx.x;
  if (tid >= nrows) return;
  const int r = r0 + tid;
  const int kept = nctx - chunk_len;
  const size_t d = static_cast<size_t>(seg) * cap_dst + r;
  if (r < kept) {
    if (mapped) return;
    const int s = src_row[tid];
    const size_t st = static_cast<size_t>(seg) * n_slots + s;
    uid_dst[d] = rank_row[tid];
    mod_dst[d] = mod_src[st];
    pos_dst[d] = pos_src[st] + shift_row[tid];
    src_of_dst[d] = s;
  } else {
    const int i = r - kept;
    uid_dst[d] = rank_row[tid] + chunk_unit[i];    // the chunk's tags are shared by segments
    mod_dst[d] = chunk_mod[i];
    pos_dst[d] = kept + i;
    src_of_dst[d] = -1;
  }
}

// The rows one copy workgroup moves: destination rows dst_row0 + [0, nrows), source slot (or
// chunk row) src_row[i]; per row a K run then a V run of row_vecs 16-byte vectors.
struct CopyRows {
  const uint8_t* k_src;
  const uint8_t* v_src;
  const uint8_t* k_chunk;
  const uint8_t* v_chunk;
  uint8_t* k_dst;
  uint8_t* v_dst;
  const int32_t* src_row;
  int row_bytes, row_vecs, vecs2;
  size_t src_base, chunk_base, dst_row0;
  int nrows;
};

// Loads rows [rb, rb + RB) into buf: thread tid takes vectors tid + 256 v of each row.
template <int RB, int VPT>
__device__ __forceinline__ void copy_load(const CopyRows& c, int rb, u32x4 (&buf)[RB][VPT]) {
  const int tid = threadIdx.x;
  // members into locals first: a select between two members' addresses would keep the struct
  // in memory
  const uint8_t *const ks = c.k_src, *const vs = c.v_src, *const kc = c.k_chunk,
                       *const vc = c.v_chunk;
#pragma unroll
  for (int j = 0; j < RB; ++j) {
    const int row = rb + j;
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const int f = tid + kCopyThreads * v;
      buf[j][v] = u32x4{0, 0, 0, 0};
      if (row < c.nrows && f < c.vecs2) {
        const int s = c.src_row[row];
        const bool is_v = f >= c.row_vecs;
        const int vec = is_v ? f - c.row_vecs : f;
        const uint8_t* src;
        if (s >= 0)
          src = (is_v ? vs : ks) + (c.src_base + s) * c.row_bytes;
        else
          src = (is_v ? vc : kc) + (c.chunk_base + (-1 - s)) * c.row_bytes;
        buf[j][v] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + vec);
      }
    }
  }
}

template <int RB, int VPT>
__device__ __forceinline__ void copy_store(const CopyRows& c, int rb,
                                           const u32x4 (&buf)[RB][VPT]) {
  const int tid = threadIdx.x;
  uint8_t *const kd = c.k_dst, *const vd = c.v_dst;
#pragma unroll
  for (int j = 0; j < RB; ++j) {
    const int row = rb + j;
#pragma unroll
    for (int v = 0; v < VPT; ++v) {
      const int f = tid + kCopyThreads * v;
      if (row < c.nrows && f < c.vecs2) {
        const bool is_v = f >= c.row_vecs;
        const int vec = is_v ? f - c.row_vecs : f;
        uint8_t* dst = (is_v ? vd : kd) + (c.dst_row0 + row) * c.row_bytes;
        __builtin_nontemporal_store(buf[j][v], reinterpret_cast<u32x4*>(dst) + vec);
      }
    }
  }
}

// Copy: one workgroup per TPW consecutive destination tiles.  Its rows are resolved at once;
// then batches of RB rows (RB x VPT x 4 KB of K and V) are software-pipelined through two
// register buffers, the loads of batch b+1 in flight while batch b is stored; the rows' tags
// are written while the first batch is in flight.
template <int VPT, bool FUSED, int TPW>
__global__ __launch_bounds__(kCopyThreads) void compact_copy_kernel(
    const uint8_t* __restrict__ k_src, const uint8_t* __restrict__ v_src, int n_slots,
    int row_bytes, const uint8_t* __restrict__ mod_src,
    const int32_t* __restrict__ pos_src, const uint8_t* __restrict__ k_chunk,
    const uint8_t* __restrict__ v_chunk, const uint8_t* __restrict__ chunk_mod,
    const int32_t* __restrict__ chunk_unit, int chunk_len, uint8_t* __restrict__ k_dst,
    uint8_t* __restrict__ v_dst, int cap_dst, int n_units, int32_t* __restrict__ uid_dst,
    uint8_t* __restrict__ mod_dst, int32_t* __restrict__ pos_dst,
    int32_t* __restrict__ src_of_dst, const int32_t* __restrict__ n_ctx_g,
    const uint8_t* __restrict__ ws, FusedPlanArgs fp) {
  constexpr int RB = VPT >= 16 ? 1 : 16 / VPT;     // rows per batch
  constexpr int SPAN = TPW * kTile;
  static_assert(SPAN <= kCopyThreads, "one resolving thread per row");
  __shared__ int32_t src_row[SPAN], shift_row[SPAN], rank_row[SPAN];
  __shared__ TilePlan<FUSED> plan;
  const int seg = blockIdx.y;
  const int r0 = blockIdx.x * SPAN;
  const int tid = threadIdx.x;
  int nctx;
  const TilePlan<true>* pp = nullptr;
  if constexpr (FUSED) {
    plan_in_lds(seg, n_units, chunk_len, cap_dst, fp, plan);
    nctx = plan.kept + chunk_len;
    if (nctx > cap_dst) nctx = 0;                 // capacity error: every row becomes empty
    pp = &plan;
  } else {
    nctx = n_ctx_g[seg];
  }
  const int nrows = resolve_rows(seg, r0, SPAN, nctx, n_slots, chunk_len, cap_dst, n_units,
                                 mod_src, pos_src, chunk_mod, chunk_unit, uid_dst, mod_dst,
                                 pos_dst, src_of_dst, ws, src_row, shift_row, pp, fp.mapped,
                                 rank_row);
  if (nrows == 0) return;

  const int row_vecs = row_bytes / 16;
  const int vecs2 = 2 * row_vecs;       // K row then V row
  const size_t src_base = static_cast<size_t>(seg) * n_slots;
  const size_t chunk_base = static_cast<size_t>(seg) * chunk_len;
  const size_t dst_base = static_cast<size_t>(seg) * cap_dst;
  const CopyRows cr{k_src, v_src, k_chunk, v_chunk, k_dst, v_dst, src_row, row_bytes,
                    row_vecs, vecs2, src_base, chunk_base, dst_base + r0, nrows};
  u32x4 bA[RB][VPT], bB[RB][VPT];
  copy_load<RB, VPT>(cr, 0, bA);
  tile_tags(seg, r0, nrows, nctx, n_slots, chunk_len, cap_dst, mod_src, pos_src, chunk_mod,
            chunk_unit, uid_dst, mod_dst, pos_dst, src_of_dst, src_row, shift_row, rank_row,
            fp.mapped);
  for (int rb = 0; rb < nrows; rb += 2 * RB) {
    if (rb + RB < nrows) copy_load<RB, VPT>(cr, rb + RB, bB);
    copy_store<RB, VPT>(cr, rb, bA);
    if (rb + RB < nrows) {
      if (rb + 2 * RB < nrows) copy_load<RB, VPT>(cr, rb + 2 * RB, bA);
      copy_store<RB, VPT>(cr, rb + RB, bB);
    }
  }
}

FusedPlanArgs fused_args(const CompactArgs& a) {
  return FusedPlanArgs{a.keep,      a.keep_len, a.unit_len, a.unit_first, a.page_size,
                       a.unit_remap, a.n_ctx,   a.n_pages,  a.d_status,   a.use_mask};
}

// Destination tiles per copy workgroup.  One: every workgroup of the grid is resident at once
// and the grid's reads and writes overlap across workgroups; two or four tiles per workgroup,
// pipelined, measured 7% and 25% slower on the 80K history.
constexpr int kCopyTiles = 1;

template <int VPT, bool FUSED>
hipError_t launch_copy(const CompactArgs& a, hipStream_t stream) {
  constexpr int span = kCopyTiles * kTile;
  const dim3 grid((a.cap_dst + span - 1) / span, a.n_seg);
  hipLaunchKernelGGL((compact_copy_kernel<VPT, FUSED, kCopyTiles>), grid, dim3(kCopyThreads), 0,
                     stream,
                     static_cast<const uint8_t*>(a.k_src), static_cast<const uint8_t*>(a.v_src),
                     a.n_slots_src, a.row_bytes, a.modality_src, a.pos_src,
                     static_cast<const uint8_t*>(a.k_chunk), static_cast<const uint8_t*>(a.v_chunk),
                     a.chunk_modality, a.chunk_unit, a.chunk_len, static_cast<uint8_t*>(a.k_dst),
                     static_cast<uint8_t*>(a.v_dst), a.cap_dst, a.n_units, a.unit_id_dst,
                     a.modality_dst, a.pos_dst, a.src_of_dst, a.n_ctx,
                     static_cast<const uint8_t*>(a.workspace), fused_args(a));
  return hipGetLastError();
}

// Copy with rotary re-encoding of the moved keys (paper: section 5.2, Applying the retention
// plan): a kept key rotated for its old position is turned by its position shift (the deleted
// tokens before it, negated).  A history row whose position changes by `shift` has each pair
// (x, y) of its first rot_dims key dimensions turned by shift * theta_j, theta_j =
// base^(-2j/rot_dims): (x cos - y sin, x sin + y cos).  Pairs are (j, j + rot_dims/2) (HALF) or
// (2j, 2j+1).  V rows, chunk rows and unshifted rows are copied unchanged.
// Angles: theta_j and the reduction of shift * theta_j modulo 2 pi in double precision, then a
// float sine/cosine of the reduced angle; the rotation itself in float, rounded to the storage
// type (round to nearest even).  One workgroup per 16-row tile; the tile's cos / sin table is
// built in LDS once and shared by all heads.
constexpr int kMaxHalfRot = 64;     // rot_dims <= head_dim <= 128
constexpr double kTwoPi = 6.283185307179586476925286766559;

// theta_j = base^(-2j / rot_dims) for j < rot_dims / 2, into LDS, by the workgroup's second wave
// (the first one builds the unit plan meanwhile).
__device__ inline void rope_thetas(double* theta, double rope_base, int rot_dims) {
  const int j = static_cast<int>(threadIdx.x) - kWave;
  if (j >= 0 && j < rot_dims / 2) theta[j] = pow(rope_base, -2.0 * j / rot_dims);
}

// cos / sin of shift * theta_j, one table row per run of equal shifts among the tile's rows (the
// rows of a unit share their shift, so a tile mostly needs one or two rows of angles);
// tab_of[r] = the run of row r.  The angle is reduced modulo 2 pi in double precision, then a
// float sine and cosine (shift 0: exactly (1, 0)).  Every thread finds the runs itself from
// shift_row, so filling the table needs no barrier of its own.
__device__ inline void rope_table(int nrows, int half, const int32_t* shift_row,
                                  const double* theta, float2 (*cs)[kMaxHalfRot],
                                  int32_t* tab_of) {
  uint32_t starts = 1u;
#pragma unroll
  for (int r = 1; r < kTile; ++r)
    starts |= (r < nrows && shift_row[r] != shift_row[r - 1]) ? (1u << r) : 0u;
  const int tid = threadIdx.x;
  if (tid < nrows) tab_of[tid] = __popc(starts & ((2u << tid) - 1u)) - 1;
  const int runs = __popc(starts);
  for (int idx = tid; idx < runs * half; idx += kCopyThreads) {
    const int k = idx / half, j = idx - k * half;
    const int sh = shift_row[nth_set_bit(starts, k)];
    float c = 1.f, sn = 0.f;
    if (sh != 0) {
      const double phi = static_cast<double>(sh) * theta[j];
      const double red = fma(-rint(phi * (1.0 / kTwoPi)), kTwoPi, phi);
      sincosf(static_cast<float>(red), &sn, &c);
    }
    cs[k][j] = make_float2(c, sn);
  }
}

// A tile's K work items in (row, head, item) order.  HALF: item it < pair_items of a head is the
// chunk pair (it, it + pair_items), which hold the two members of the same dimension pairs; the
// remaining items are the single chunks past rot_dims.  Otherwise every chunk is one item and
// turns its own dimension pairs below rot_dims.  Thread tid visits items tid, tid +
// kCopyThreads, ...; the cursor (row, head, item) steps by kCopyThreads items without a division.
template <int EB, bool HALF>
struct RopeItems {
  static constexpr int EPC = 16 / EB;             // elements per 16-byte chunk
  int n_kv_heads, rot_dims, chunks, pair_items, per_head;
  int s_it, s_hd, s_row;                          // one step of kCopyThreads items
  __device__ RopeItems(int n_kv_heads_, int head_dim, int rot_dims_)
      : n_kv_heads(n_kv_heads_), rot_dims(rot_dims_), chunks(head_dim / EPC),
        pair_items(HALF ? rot_dims_ / 2 / EPC : 0),
        per_head(HALF ? rot_dims_ / 2 / EPC + (head_dim - rot_dims_) / EPC : head_dim / EPC) {
    const int h = kCopyThreads / per_head;
    s_it = kCopyThreads - h * per_head;
    s_hd = h % n_kv_heads;
    s_row = h / n_kv_heads;
  }
  __device__ int count(int nrows) const { return nrows * n_kv_heads * per_head; }
  __device__ void start(int w, int& row, int& hd, int& it) const {
    row = w / (n_kv_heads * per_head);
    const int rem = w - row * n_kv_heads * per_head;
    hd = rem / per_head;
    it = rem - hd * per_head;
  }
  __device__ void step(int& row, int& hd, int& it) const {
    it += s_it;                                   // it, s_it < per_head: one carry at most
    const int c1 = it >= per_head ? 1 : 0;
    it -= c1 ? per_head : 0;
    hd += s_hd + c1;                              // hd, s_hd < n_kv_heads: likewise
    const int c2 = hd >= n_kv_heads ? 1 : 0;
    hd -= c2 ? n_kv_heads : 0;
    row += s_row + c2;
  }
  __device__ bool pair(int it) const { return HALF && it < pair_items; }
  // the item's (first) chunk, counted over its row
  __device__ int chunk(int hd, int it) const {
    return hd * chunks + (HALF && it >= pair_items ? it + pair_items : it);
  }
  // whether the item holds a dimension pair below rot_dims
  __device__ bool turns(int it) const { return HALF ? it < pair_items : it * EPC < rot_dims; }
};

template <int EB>
__device__ inline void unpack_chunk(const u32x4& v, float (&f)[16 / EB]) {
#pragma unroll
  for (int e = 0; e < 16 / EB; ++e) {
    const uint32_t w = v[e * EB / 4];
    if constexpr (EB == 2) f[e] = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    else f[e] = __uint_as_float(w);
  }
}

template <int EB>
__device__ inline u32x4 pack_chunk(const float (&f)[16 / EB]) {
  u32x4 v;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if constexpr (EB == 2) {
      const __bf16 lo = static_cast<__bf16>(f[2 * q]), hi = static_cast<__bf16>(f[2 * q + 1]);
      v[q] = static_cast<uint32_t>(__builtin_bit_cast(uint16_t, lo)) |
             (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, hi)) << 16);
    } else {
      v[q] = __float_as_uint(f[q]);
    }
  }
  return v;
}

// Turns the dimension pairs of item `it` by the table row tab: (x, y) -> (x cos - y sin,
// x sin + y cos) in float, rounded to the storage type.  A pair item's members are a and b.
template <int EB, bool HALF>
__device__ inline void turn_item(const RopeItems<EB, HALF>& g, int it, const float2* tab,
                                 u32x4& a, u32x4& b) {
  constexpr int EPC = 16 / EB;
  if constexpr (HALF) {
    float x[EPC], y[EPC];
    unpack_chunk<EB>(a, x);
    unpack_chunk<EB>(b, y);
#pragma unroll
    for (int e = 0; e < EPC; ++e) {
      const float2 r = tab[it * EPC + e];
      const float xe = x[e], ye = y[e];
      x[e] = fmaf(xe, r.x, -ye * r.y);
      y[e] = fmaf(xe, r.y, ye * r.x);
    }
    a = pack_chunk<EB>(x);
    b = pack_chunk<EB>(y);
  } else {
    float f[EPC];
    unpack_chunk<EB>(a, f);
#pragma unroll
    for (int m = 0; m < EPC / 2; ++m) {
      const int d0 = it * EPC + 2 * m;
      if (d0 < g.rot_dims) {
        const float2 r = tab[d0 / 2];
        const float x = f[2 * m], y = f[2 * m + 1];
        f[2 * m] = fmaf(x, r.x, -y * r.y);
        f[2 * m + 1] = fmaf(x, r.y, y * r.x);
      }
    }
    a = pack_chunk<EB>(f);
  }
}

constexpr int kRopeKB = 4;     // K items per thread per batch (a pair item is two vectors)
constexpr int kRopeVB = 8;     // V vectors per thread per batch

// A K item's row, head and item index in one register (row < 2^15, head < 2^8, item < 2^8);
// -1: nothing to do.
__device__ inline int pack_item(int row, int hd, int it) { return (row << 16) | (hd << 8) | it; }

// Copy with rotary re-encoding of the moved keys (paper: section 5.2, Applying the retention
// plan): V rows, chunk rows and unshifted rows are copied unchanged.  One workgroup per 16-row
// destination tile.  Each thread issues the loads of a batch of its V vectors and K items
// together; the first batch's loads are in flight while the tile's tags are written and its
// cos / sin table is built in LDS (one row per run of equal shifts, shared by all heads).
template <int EB, bool HALF, bool FUSED>
__global__ __launch_bounds__(kCopyThreads) void compact_copy_rope_kernel(
    const uint8_t* __restrict__ k_src, const uint8_t* __restrict__ v_src, int n_slots,
    int n_kv_heads, int head_dim, const uint8_t* __restrict__ mod_src,
    const int32_t* __restrict__ pos_src, const uint8_t* __restrict__ k_chunk,
    const uint8_t* __restrict__ v_chunk, const uint8_t* __restrict__ chunk_mod,
    const int32_t* __restrict__ chunk_unit, int chunk_len, uint8_t* __restrict__ k_dst,
    uint8_t* __restrict__ v_dst, int cap_dst, int n_units, int32_t* __restrict__ uid_dst,
    uint8_t* __restrict__ mod_dst, int32_t* __restrict__ pos_dst,
    int32_t* __restrict__ src_of_dst, const int32_t* __restrict__ n_ctx_g,
    const uint8_t* __restrict__ ws, double rope_base, int rot_dims, FusedPlanArgs fp) {
  __shared__ int32_t src_row[kTile], shift_row[kTile], rank_row[kTile], tab_of[kTile];
  __shared__ double theta[kMaxHalfRot];
  __shared__ float2 cs[kTile][kMaxHalfRot];
  __shared__ TilePlan<FUSED> plan;
  const int seg = blockIdx.y;
  const int t = blockIdx.x;
  const int tid = threadIdx.x;
  rope_thetas(theta, rope_base, rot_dims);
  int nctx;
  const TilePlan<true>* pp = nullptr;
  if constexpr (FUSED) {
    plan_in_lds(seg, n_units, chunk_len, cap_dst, fp, plan);
    nctx = plan.kept + chunk_len;
    if (nctx > cap_dst) nctx = 0;
    pp = &plan;
  } else {
    nctx = n_ctx_g[seg];
  }
  const int nrows = resolve_tile(seg, t, nctx, n_slots, chunk_len, cap_dst, n_units, mod_src,
                                 pos_src, chunk_mod, chunk_unit, uid_dst, mod_dst, pos_dst,
                                 src_of_dst, ws, src_row, shift_row, pp, fp.mapped, rank_row);
  if (nrows == 0) return;
  const int r0 = t * kTile;

  const int row_bytes = n_kv_heads * head_dim * EB;
  const int row_vecs = row_bytes / 16;
  const int nv = nrows * row_vecs;
  const size_t src_base = static_cast<size_t>(seg) * n_slots;
  const size_t chunk_base = static_cast<size_t>(seg) * chunk_len;
  // the tile's destination rows are contiguous: vector f of the tile is vector f of these
  u32x4* const kd = reinterpret_cast<u32x4*>(k_dst + (static_cast<size_t>(seg) * cap_dst + r0) *
                                                         row_bytes);
  u32x4* const vd = reinterpret_cast<u32x4*>(v_dst + (static_cast<size_t>(seg) * cap_dst + r0) *
                                                         row_bytes);
  auto row_src = [&](const uint8_t* pool, const uint8_t* chunk, int row) {
    const int s = src_row[row];
    return reinterpret_cast<const u32x4*>(s >= 0 ? pool + (src_base + s) * row_bytes
                                                 : chunk + (chunk_base + (-1 - s)) * row_bytes);
  };
  const RopeItems<EB, HALF> g(n_kv_heads, head_dim, rot_dims);
  int kr, kh, ki;
  g.start(tid, kr, kh, ki);
  const int s_vr = kCopyThreads / row_vecs, s_vv = kCopyThreads - s_vr * row_vecs;
  int vr = tid / row_vecs, vv = tid - vr * row_vecs;
  constexpr int kItemsPerBatch = kCopyThreads * kRopeKB, kVecsPerBatch = kCopyThreads * kRopeVB;
  const int n_batches = max((g.count(nrows) + kItemsPerBatch - 1) / kItemsPerBatch,
                            (nv + kVecsPerBatch - 1) / kVecsPerBatch);
  // one batch: the loads, then (first batch) the tags and the table, then the stores
  auto batch = [&](int b) {
    u32x4 va[kRopeVB], ka[kRopeKB], kb[kRopeKB];
    int kp[kRopeKB];
#pragma unroll
    for (int i = 0; i < kRopeVB; ++i) {
      if (vr < nrows) va[i] = __builtin_nontemporal_load(row_src(v_src, v_chunk, vr) + vv);
      vv += s_vv;
      const int c = vv >= row_vecs ? 1 : 0;
      vv -= c ? row_vecs : 0;
      vr += s_vr + c;
    }
#pragma unroll
    for (int i = 0; i < kRopeKB; ++i) {
      kp[i] = kr < nrows ? pack_item(kr, kh, ki) : -1;
      if (kr < nrows) {
        const u32x4* src = row_src(k_src, k_chunk, kr) + g.chunk(kh, ki);
        ka[i] = __builtin_nontemporal_load(src);
        if (g.pair(ki)) kb[i] = __builtin_nontemporal_load(src + g.pair_items);
      }
      g.step(kr, kh, ki);
    }
    if (b == 0) {
      tile_tags(seg, r0, nrows, nctx, n_slots, chunk_len, cap_dst, mod_src, pos_src, chunk_mod,
                chunk_unit, uid_dst, mod_dst, pos_dst, src_of_dst, src_row, shift_row, rank_row,
                fp.mapped);
      rope_table(nrows, rot_dims / 2, shift_row, theta, cs, tab_of);
      __syncthreads();
    }
    // every load of the batch has landed before the first store: the stores, each under its
    // own condition, then need no wait between them
    __builtin_amdgcn_s_waitcnt(kVmcntZero);
#pragma unroll
    for (int i = 0; i < kRopeVB; ++i) {
      const int f = tid + kCopyThreads * (b * kRopeVB + i);
      if (f < nv) __builtin_nontemporal_store(va[i], vd + f);
    }
#pragma unroll
    for (int i = 0; i < kRopeKB; ++i) {
      if (kp[i] < 0) continue;
      const int row = kp[i] >> 16, hd = (kp[i] >> 8) & 0xff, it = kp[i] & 0xff;
      if (shift_row[row] != 0 && g.turns(it))
        turn_item<EB, HALF>(g, it, cs[tab_of[row]], ka[i], kb[i]);
      u32x4* dst = kd + row * row_vecs + g.chunk(hd, it);
      __builtin_nontemporal_store(ka[i], dst);
      if (g.pair(it)) __builtin_nontemporal_store(kb[i], dst + g.pair_items);
    }
  };
  batch(0);                                      // the first batch on its own, so that no
  for (int b = 1; b < n_batches; ++b) batch(b);  // wait is placed for a later one's registers
}

// In-place rotary adjustment of the keys that stay in their slots while their position shifts
// (native eviction): one workgroup per 16-slot tile of the pool; shift_g holds each slot's
// position change (0: empty, evicted or unmoved; such rows are not touched, nor are the chunks
// past rot_dims).  Batches of a thread's K items as in the rotary copy.
template <int EB, bool HALF>
__global__ __launch_bounds__(kCopyThreads) void rope_in_place_kernel(
    uint8_t* __restrict__ k, int cap, int n_kv_heads, int head_dim,
    const int32_t* __restrict__ shift_g, double rope_base, int rot_dims) {
  __shared__ int32_t shift_row[kTile], tab_of[kTile];
  __shared__ double theta[kMaxHalfRot];
  __shared__ float2 cs[kTile][kMaxHalfRot];
  const int seg = blockIdx.y;
  const int r0 = blockIdx.x * kTile;
  const int nrows = min(kTile, cap - r0);
  const int tid = threadIdx.x;
  const int sh = tid < nrows ? shift_g[static_cast<size_t>(seg) * cap + r0 + tid] : 0;
  if (tid < kTile) shift_row[tid] = sh;
  rope_thetas(theta, rope_base, rot_dims);
  if (__syncthreads_or(sh != 0) == 0) return;     // nothing in this tile moves
  const int row_vecs = n_kv_heads * head_dim * EB / 16;
  u32x4* const base = reinterpret_cast<u32x4*>(
      k + (static_cast<size_t>(seg) * cap + r0) * n_kv_heads * head_dim * EB);
  const RopeItems<EB, HALF> g(n_kv_heads, head_dim, rot_dims);
  int kr, kh, ki;
  g.start(tid, kr, kh, ki);
  constexpr int kItemsPerBatch = kCopyThreads * kRopeKB;
  const int n_batches = (g.count(nrows) + kItemsPerBatch - 1) / kItemsPerBatch;
  auto batch = [&](int b) {
    u32x4 ka[kRopeKB], kb[kRopeKB];
    int kp[kRopeKB];
#pragma unroll
    for (int i = 0; i < kRopeKB; ++i) {
      const bool live = kr < nrows && shift_row[min(kr, kTile - 1)] != 0 && g.turns(ki);
      kp[i] = live ? pack_item(kr, kh, ki) : -1;
      if (live) {
        const u32x4* src = base + kr * row_vecs + g.chunk(kh, ki);
        ka[i] = __builtin_nontemporal_load(src);
        if (g.pair(ki)) kb[i] = __builtin_nontemporal_load(src + g.pair_items);
      }
      g.step(kr, kh, ki);
    }
    if (b == 0) {
      rope_table(nrows, rot_dims / 2, shift_row, theta, cs, tab_of);
      __syncthreads();
    }
    __builtin_amdgcn_s_waitcnt(kVmcntZero);
#pragma unroll
    for (int i = 0; i < kRopeKB; ++i) {
      if (kp[i] < 0) continue;
      const int row = kp[i] >> 16, hd = (kp[i] >> 8) & 0xff, it = kp[i] & 0xff;
      turn_item<EB, HALF>(g, it, cs[tab_of[row]], ka[i], kb[i]);
      u32x4* dst = base + row * row_vecs + g.chunk(hd, it);
      __builtin_nontemporal_store(ka[i], dst);
      if (g.pair(it)) __builtin_nontemporal_store(kb[i], dst + g.pair_items);
    }
  };
  batch(0);
  for (int b = 1; b < n_batches; ++b) batch(b);
}

template <int EB, bool HALF, bool FUSED>
hipError_t launch_copy_rope(const CompactArgs& a, hipStream_t stream) {
  const dim3 grid((a.cap_dst + kTile - 1) / kTile, a.n_seg);
  hipLaunchKernelGGL((compact_copy_rope_kernel<EB, HALF, FUSED>), grid, dim3(kCopyThreads), 0,
                     stream,
                     static_cast<const uint8_t*>(a.k_src), static_cast<const uint8_t*>(a.v_src),
                     a.n_slots_src, a.n_kv_heads, a.head_dim, a.modality_src, a.pos_src,
                     static_cast<const uint8_t*>(a.k_chunk), static_cast<const uint8_t*>(a.v_chunk),
                     a.chunk_modality, a.chunk_unit, a.chunk_len, static_cast<uint8_t*>(a.k_dst),
                     static_cast<uint8_t*>(a.v_dst), a.cap_dst, a.n_units, a.unit_id_dst,
                     a.modality_dst, a.pos_dst, a.src_of_dst, a.n_ctx,
                     static_cast<const uint8_t*>(a.workspace), a.rope_base, a.rope_dims,
                     fused_args(a));
  return hipGetLastError();
}

constexpr int kUnitWaves = 4;      // one wave per unit in the mask kernels

__device__ inline bool unit_in_pool(int n, int f, int n_slots) {
  return n > 0 && f >= 0 && f <= n_slots - n;
}

constexpr int kUnitPer = 16;       // consecutive slots per lane in one step of a unit walk

__global__ __launch_bounds__(kUnitWaves * kWave) void compact_mask_count_kernel(
    const uint8_t* __restrict__ mask_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ first_g, int n_slots, int n_units, int cap_dst,
    uint8_t* __restrict__ ws, int32_t* __restrict__ status) {
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int u = blockIdx.x * kUnitWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (u >= n_units) return;
  const WsLayout L = ws_layout(n_units, cap_dst);
  int32_t* cnt = reinterpret_cast<int32_t*>(ws + static_cast<size_t>(seg) * L.seg_bytes +
                                            L.count_off);
  const size_t ub = static_cast<size_t>(seg) * n_units;
  const int n = len_g[ub + u], f = first_g[ub + u];
  uint32_t c = 0;
  if (unit_in_pool(n, f, n_slots)) {
    const uint8_t* m = mask_g + static_cast<size_t>(seg) * n_slots;
    const uintptr_t end = reinterpret_cast<uintptr_t>(m + f + n);
    for (uintptr_t blk = block16_floor(m + f) + kUnitPer * static_cast<uintptr_t>(lane);
         blk < end; blk += kUnitPer * kWave) {
      const int s0 = static_cast<int>(static_cast<intptr_t>(blk) - reinterpret_cast<intptr_t>(m));
      uint8_t b[16];
      load_block16(blk, b);
#pragma unroll
      for (int j = 0; j < kUnitPer; ++j) c += (s0 + j >= f && s0 + j < f + n && b[j] != 0);
    }
    c = wave_sum_u32(c);
  } else if (n > 0 && lane == 0) {
    set_status(status, OMNITIDE_E_TAGS);          // a unit outside the pool keeps nothing
  }
  if (lane == 0) cnt[u] = static_cast<int32_t>(c);
}

// One wave maps the kept slots of one unit (slots [f, f + n), mask m of the segment): kept slot
// number `within` of the unit goes to destination row rec_off + within with the unit's new id
// rk, and its position drops by the deleted live slots before it (rec_del plus those of the
// unit).  The wave walks aligned 16-slot blocks, 16 per lane per step, with one wave scan of
// the kept counts per step.  Branch-free per slot: the tag reads and writes of slots that are
// not kept use an offset past their buffer, which the hardware turns into a zero read and a
// dropped write.
__device__ inline void map_unit_slots(const uint8_t* m, int f, int n, int rk, int rec_off,
                                      int rec_del, int lane, int seg, int n_slots, int cap_dst,
                                      const uint8_t* mod_src, const int32_t* pos_src,
                                      int32_t* uid_dst, uint8_t* mod_dst, int32_t* pos_dst,
                                      int32_t* src_of_dst, int32_t* shift) {
  constexpr int P = kUnitPer;
  const size_t sb = static_cast<size_t>(seg) * n_slots;
  const size_t db = static_cast<size_t>(seg) * cap_dst;
  const __amdgpu_buffer_rsrc_t r_mod_s =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(mod_src + sb), 0, n_slots, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_pos_s = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(pos_src + sb), 0, 4 * n_slots, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_src =
      __builtin_amdgcn_make_buffer_rsrc(src_of_dst + db, 0, 4 * cap_dst, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_uid =
      __builtin_amdgcn_make_buffer_rsrc(uid_dst + db, 0, 4 * cap_dst, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_mod =
      __builtin_amdgcn_make_buffer_rsrc(mod_dst + db, 0, cap_dst, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_pos =
      __builtin_amdgcn_make_buffer_rsrc(pos_dst + db, 0, 4 * cap_dst, kBufFlags);
  const __amdgpu_buffer_rsrc_t r_shift =
      __builtin_amdgcn_make_buffer_rsrc(shift, 0, 4 * cap_dst, kBufFlags);
  const uintptr_t end = reinterpret_cast<uintptr_t>(m + f + n);
  int carry = 0;                                  // kept slots of the unit before the step
  for (uintptr_t c = block16_floor(m + f); c < end; c += P * kWave) {
    const uintptr_t blk = c + P * static_cast<uintptr_t>(lane);
    const int s0 = static_cast<int>(static_cast<intptr_t>(blk) - reinterpret_cast<intptr_t>(m));
    bool keep[P];
    int nk = 0;
    {
      uint8_t b[16] = {};
      if (blk < end) load_block16(blk, b);
#pragma unroll
      for (int j = 0; j < P; ++j) keep[j] = (s0 + j >= f) & (s0 + j < f + n) & (b[j] != 0);
    }
#pragma unroll
    for (int j = 0; j < P; ++j) nk += keep[j] ? 1 : 0;
    const int incl = wave_inclusive_scan(nk);
    int within = carry + incl - nk;               // kept slots of the unit before s0
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int s = s0 + j;
      const int r = rec_off + within;
      const int delb = rec_del + (s - f) - within;   // deleted live slots before s
      const int so = keep[j] ? s : kOutOfBuf / 4;    // source slot, or past the buffers
      const int ro = keep[j] ? r : kOutOfBuf / 4;    // destination row, or past the buffers
      const int mod = __builtin_amdgcn_raw_buffer_load_b8(r_mod_s, so, 0, 0);
      const int pos = __builtin_amdgcn_raw_buffer_load_b32(r_pos_s, 4 * so, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(s, r_src, 4 * ro, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(rk, r_uid, 4 * ro, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b8(static_cast<uint8_t>(mod), r_mod, ro, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(pos - delb, r_pos, 4 * ro, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b32(-delb, r_shift, 4 * ro, 0, 0);
      within += keep[j] ? 1 : 0;
    }
    carry += __shfl(incl, kWave - 1, kWave);
  }
}

__global__ __launch_bounds__(kUnitWaves * kWave) void compact_mask_map_kernel(
    const uint8_t* __restrict__ mask_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ first_g, const uint8_t* __restrict__ mod_src,
    const int32_t* __restrict__ pos_src, int n_slots, int n_units, int cap_dst,
    const int32_t* __restrict__ remap_g, const int32_t* __restrict__ n_ctx_g,
    int32_t* __restrict__ uid_dst, uint8_t* __restrict__ mod_dst, int32_t* __restrict__ pos_dst,
    int32_t* __restrict__ src_of_dst, uint8_t* __restrict__ ws) {
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int u = blockIdx.x * kUnitWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (u >= n_units) return;
  if (n_ctx_g[seg] == 0) return;                  // capacity error: no history row is written
  const size_t ub = static_cast<size_t>(seg) * n_units;
  const int rk = remap_g[ub + u];
  if (rk < 0) return;                             // nothing kept (count 0 also for bad units)
  const int n = len_g[ub + u], f = first_g[ub + u];
  const WsLayout L = ws_layout(n_units, cap_dst);
  uint8_t* wseg = ws + static_cast<size_t>(seg) * L.seg_bytes;
  const RankRec rec = reinterpret_cast<const RankRec*>(wseg + L.rank_off)[rk];
  int32_t* shift = reinterpret_cast<int32_t*>(wseg + L.shift_off);
  const size_t sb = static_cast<size_t>(seg) * n_slots;
  map_unit_slots(mask_g + sb, f, n, rk, rec.off, rec.del, lane, seg, n_slots, cap_dst, mod_src,
                 pos_src, uid_dst, mod_dst, pos_dst, src_of_dst, shift);
}

// Up to kSmallUnits units: the plan over the count kernel's per-unit counts is built in LDS by
// every map workgroup (wave 0, as in the fused copy), so no plan kernel runs; workgroup 0 also
// writes unit_remap, n_ctx, n_pages, the kept totals and the capacity status.  Then one wave per
// unit maps its kept slots as compact_mask_map_kernel does.
__global__ __launch_bounds__(kUnitWaves * kWave) void compact_mask_map_fused_kernel(
    const uint8_t* __restrict__ mask_g, const uint8_t* __restrict__ mod_src,
    const int32_t* __restrict__ pos_src, int n_slots, int n_units, int chunk_len, int cap_dst,
    int32_t* __restrict__ uid_dst, uint8_t* __restrict__ mod_dst, int32_t* __restrict__ pos_dst,
    int32_t* __restrict__ src_of_dst, uint8_t* __restrict__ ws, FusedPlanArgs fp) {
  __shared__ TilePlan<true> plan;
  const int seg = blockIdx.y;
  const WsLayout L = ws_layout(n_units, cap_dst);
  uint8_t* wseg = ws + static_cast<size_t>(seg) * L.seg_bytes;
  fp.counts = reinterpret_cast<const int32_t*>(wseg + L.count_off);
  plan_in_lds(seg, n_units, chunk_len, cap_dst, fp, plan);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    int32_t* meta = reinterpret_cast<int32_t*>(wseg + L.meta_off);
    meta[0] = plan.kept;
    meta[1] = plan.n_kept;
  }
  if (plan.kept + chunk_len > cap_dst) return;    // capacity error: no history row is written
  const int lane = threadIdx.x & (kWave - 1);
  const int u = blockIdx.x * kUnitWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (u >= n_units) return;
  const int rk = plan.rank_of[u];
  if (rk < 0) return;                             // nothing kept (count 0 also for bad units)
  const size_t ub = static_cast<size_t>(seg) * n_units;
  const int n = fp.len[ub + u], f = fp.first[ub + u];
  const int rec_off = plan.roff[rk], rec_del = plan.rdel[rk];
  int32_t* shift = reinterpret_cast<int32_t*>(wseg + L.shift_off);
  const size_t sb = static_cast<size_t>(seg) * n_slots;
  map_unit_slots(mask_g + sb, f, n, rk, rec_off, rec_del, lane, seg, n_slots, cap_dst, mod_src,
                 pos_src, uid_dst, mod_dst, pos_dst, src_of_dst, shift);
}

}  // namespace

hipError_t launch_rope_in_place(void* k, int dtype, int n_seg, int cap, int n_kv_heads,
                                int head_dim, const int32_t* shift, double rope_base,
                                int rope_dims, bool rope_half, hipStream_t stream) {
  const dim3 grid((cap + kTile - 1) / kTile, n_seg);
  uint8_t* kp = static_cast<uint8_t*>(k);
#define OMNITIDE_ROPE_IP(EB, HALF)                                                          \
  hipLaunchKernelGGL((rope_in_place_kernel<EB, HALF>), grid, dim3(kCopyThreads), 0, stream, \
                     kp, cap, n_kv_heads, head_dim, shift, rope_base, rope_dims)
  if (dtype == OMNITIDE_BF16) {
    if (rope_half) OMNITIDE_ROPE_IP(2, true); else OMNITIDE_ROPE_IP(2, false);
  } else {
    if (rope_half) OMNITIDE_ROPE_IP(4, true); else OMNITIDE_ROPE_IP(4, false);
  }
#undef OMNITIDE_ROPE_IP
  return hipGetLastError();
}

size_t compact_workspace_bytes(int n_seg, int n_units, int cap_dst) {
  return ws_layout(n_units, cap_dst).seg_bytes * static_cast<size_t>(n_seg);
}

template <bool FUSED>
hipError_t launch_copies(const CompactArgs& a, hipStream_t stream) {
  if (a.rope_dims > 0) {
    const int eb = a.row_bytes / (a.n_kv_heads * a.head_dim);
    if (eb == 2) return a.rope_half ? launch_copy_rope<2, true, FUSED>(a, stream)
                                    : launch_copy_rope<2, false, FUSED>(a, stream);
    return a.rope_half ? launch_copy_rope<4, true, FUSED>(a, stream)
                       : launch_copy_rope<4, false, FUSED>(a, stream);
  }
  const int vecs2 = 2 * a.row_bytes / 16;
  const int vpt = (vecs2 + kCopyThreads - 1) / kCopyThreads;
  if (vpt <= 1) return launch_copy<1, FUSED>(a, stream);
  if (vpt <= 2) return launch_copy<2, FUSED>(a, stream);
  if (vpt <= 4) return launch_copy<4, FUSED>(a, stream);
  if (vpt <= 8) return launch_copy<8, FUSED>(a, stream);
  return hipErrorInvalidValue;
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t stream) {
  uint8_t* ws = static_cast<uint8_t*>(a.workspace);
  if (a.use_mask) {
    // Per-slot mask: kept counts per unit, the unit plan over them, then the row map.
    const dim3 ugrid((a.n_units + kUnitWaves - 1) / kUnitWaves, a.n_seg);
    hipLaunchKernelGGL(compact_mask_count_kernel, ugrid, dim3(kUnitWaves * kWave), 0, stream,
                       a.keep_slot, a.unit_len, a.unit_first, a.n_slots_src, a.n_units,
                       a.cap_dst, ws, a.d_status);
    if (a.n_units <= kSmallUnits) {
      // the map workgroups plan for themselves
      hipLaunchKernelGGL(compact_mask_map_fused_kernel, ugrid, dim3(kUnitWaves * kWave), 0,
                         stream, a.keep_slot, a.modality_src, a.pos_src, a.n_slots_src,
                         a.n_units, a.chunk_len, a.cap_dst, a.unit_id_dst, a.modality_dst,
                         a.pos_dst, a.src_of_dst, ws, fused_args(a));
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      return launch_copies<false>(a, stream);
    }
    const uint8_t* no_keep = nullptr;             // counts come from the workspace
    const int32_t* no_keep_len = nullptr;
    hipLaunchKernelGGL(compact_plan_kernel, dim3(a.n_seg), dim3(kPlanThreads), 0, stream,
                       no_keep, no_keep_len, a.unit_len, a.unit_first, a.n_units, a.chunk_len,
                       a.cap_dst, a.page_size, a.unit_remap, a.n_ctx, a.n_pages, ws,
                       a.d_status);
    hipLaunchKernelGGL(compact_mask_map_kernel, ugrid, dim3(kUnitWaves * kWave), 0, stream,
                       a.keep_slot, a.unit_len, a.unit_first, a.modality_src, a.pos_src,
                       a.n_slots_src, a.n_units, a.cap_dst, a.unit_remap, a.n_ctx,
                       a.unit_id_dst, a.modality_dst, a.pos_dst, a.src_of_dst, ws);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_copies<false>(a, stream);
  }
  // Up to 512 units every copy workgroup plans for itself (one kernel); beyond, a plan kernel
  // writes the rank table and tile hints to the workspace first.
  if (a.n_units <= kSmallUnits) return launch_copies<true>(a, stream);
  hipLaunchKernelGGL(compact_plan_kernel, dim3(a.n_seg), dim3(kPlanThreads), 0, stream, a.keep,
                     a.keep_len, a.unit_len, a.unit_first, a.n_units, a.chunk_len, a.cap_dst,
                     a.page_size, a.unit_remap, a.n_ctx, a.n_pages, ws, a.d_status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_copies<false>(a, stream);
}

}  // namespace omnitide
