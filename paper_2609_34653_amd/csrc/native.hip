// Native (logical-only) layout: logical eviction in place, ordered-suffix migration and chunk
// placement into the lowest run of empty slots.
//
//   evict_plan     one workgroup per segment: scans over units give each unit its first
//                  logical position (exclusive sum of lengths), kept length, deleted tokens
//                  before it and new id; the table goes to the workspace.
//   evict_apply    one thread per slot: rewrites the tags in place (kept: new id, position minus
//                  the deleted tokens before its unit; otherwise empty); the span (last occupied
//                  slot + 1) is a per-wave maximum published with one atomic per wave.
//   The single-workgroup scans below first pack the segment's occupancy into an LDS bitmap
//   (one bit per slot, all loads in flight at once), then work on bits: counts are popcounts
//   and "last occupied slot" is a bit scan.
//   suffix_plan    one workgroup per segment: the packed span of cut c is c + (entries at or
//                  after c), or the span of what precedes c when that suffix is empty; it never
//                  decreases with c, so the cuts that save >= min_pages pages form a prefix of
//                  [0, span) and the largest is a block-wide maximum.  Lists the suffix entries
//                  in slot order.
//   suffix_gather  suffix entries whose slot changes -> workspace (rows and tags), in order;
//   suffix_scatter workspace -> slots c + rank, vacated slots marked empty.  A destination can
//                  be the source of an earlier entry, hence the round trip through scratch.
//   place_plan     one workgroup per segment: the lowest slot s with [s, s + L) empty, from a
//                  running "last occupied slot" carried across threads (for L >= 32 decided
//                  per bitmap word, since such a run must contain a whole empty word).
//   chunk_write    the chunk's K/V rows and tags into [s, s + L).
#include "common.h"
#include "kernels.h"

namespace omnitide {
namespace {

constexpr int kNatThreads = 1024;
constexpr int kNatPer = OMNITIDE_MAX_UNITS / kNatThreads;
constexpr int kRowsPerBlock = 16;
constexpr int kNatBatch = 8;       // 16-byte vectors of K (and of V) per thread per copy batch
constexpr int kCopyThreads = 256;

struct UnitRec {
  int32_t pos0;   // logical position of the unit's first token
  int32_t kl;     // kept leading tokens
  int32_t del;    // deleted tokens of earlier units
  int32_t rank;   // new id, -1 when dropped
};

__global__ __launch_bounds__(kNatThreads) void evict_plan_kernel(
    const uint8_t* __restrict__ keep_g, const int32_t* __restrict__ keep_len_g,
    const int32_t* __restrict__ len_g, int n_units, UnitRec* __restrict__ table,
    int32_t* __restrict__ remap_g, int32_t* __restrict__ kept_g,
    int32_t* __restrict__ n_kept_units_g, int32_t* __restrict__ span_g) {
  __shared__ int32_t scr[kNatThreads / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = n_units;
  const int per = (U + kNatThreads - 1) / kNatThreads;
  const int u0 = tid * per;
  const size_t base = static_cast<size_t>(seg) * U;
  int ln[kNatPer], kl[kNatPer];
  int my_len = 0, my_kept = 0, my_del = 0, my_n = 0;
#pragma unroll
  for (int i = 0; i < kNatPer; ++i) {
    const int u = u0 + i;
    ln[i] = kl[i] = 0;
    if (i < per && u < U) {
      ln[i] = max(len_g[base + u], 0);
      kl[i] = keep_len_g != nullptr ? min(max(keep_len_g[base + u], 0), ln[i])
                                    : (keep_g[base + u] != 0 ? ln[i] : 0);
    }
    my_len += ln[i];
    my_kept += kl[i];
    my_del += ln[i] - kl[i];
    my_n += kl[i] > 0 ? 1 : 0;
  }
  int total_len, kept, dropped, n_kept;
  int pos0 = block_exclusive_scan(my_len, scr, &total_len);
  int del = block_exclusive_scan(my_del, scr, &dropped);
  int rk = block_exclusive_scan(my_n, scr, &n_kept);
  (void)block_exclusive_scan(my_kept, scr, &kept);
#pragma unroll
  for (int i = 0; i < kNatPer; ++i) {
    const int u = u0 + i;
    if (i < per && u < U) {
      const int r = kl[i] > 0 ? rk++ : -1;
      table[base + u] = UnitRec{pos0, kl[i], del, r};
      remap_g[base + u] = r;
    }
    pos0 += ln[i];
    del += ln[i] - kl[i];
  }
  if (tid == 0) {
    kept_g[seg] = kept;
    n_kept_units_g[seg] = n_kept;
    span_g[seg] = 0;                               // raised by evict_apply
  }
}

// Occupancy bitmap of one segment's slots [0, cap): bit j of word w is slot 32 w + j.  Built by
// a grid of waves (one coalesced 64-slot load and a ballot per wave), then loaded into LDS by
// the single-workgroup scans.
constexpr int kMaxNatWords = 4096;                 // 131,072 slots

__global__ __launch_bounds__(kCopyThreads) void occupancy_kernel(const int32_t* __restrict__ uid_g,
                                                                 int cap, int nwords,
                                                                 uint32_t* __restrict__ bits_g) {
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int ch = blockIdx.x * (kCopyThreads / kWave) + threadIdx.x / kWave;
  const int s = ch * kWave + lane;
  const bool occ = s < cap && uid_g[static_cast<size_t>(seg) * cap + s] >= 0;
  const uint64_t m = __ballot(occ);
  if (lane == 0 && 2 * ch < nwords) {
    bits_g[static_cast<size_t>(seg) * nwords + 2 * ch] = static_cast<uint32_t>(m);
    if (2 * ch + 1 < nwords)
      bits_g[static_cast<size_t>(seg) * nwords + 2 * ch + 1] = static_cast<uint32_t>(m >> 32);
  }
}

__device__ inline void load_bitmap(const uint32_t* __restrict__ bits_g, uint32_t* bits,
                                   int nwords) {
  constexpr int kIter = kMaxNatWords / kNatThreads;
  uint32_t w[kIter];
#pragma unroll
  for (int i = 0; i < kIter; ++i) {                // all loads in flight, then the LDS writes
    const int idx = threadIdx.x + i * kNatThreads;
    w[i] = idx < nwords ? bits_g[idx] : 0u;
  }
#pragma unroll
  for (int i = 0; i < kIter; ++i) {
    const int idx = threadIdx.x + i * kNatThreads;
    if (idx < nwords) bits[idx] = w[i];
  }
  __syncthreads();
}
// shift_g (optional, [n_seg][cap]): each slot's position change (0 for slots that are empty,
// evicted or keep their position), for the rotary adjustment of the keys that stay.
__global__ __launch_bounds__(kCopyThreads) void evict_apply_kernel(
    int32_t* __restrict__ uid_g, int32_t* __restrict__ pos_g, int cap, int n_units,
    const UnitRec* __restrict__ table, const int32_t* __restrict__ len_g,
    int32_t* __restrict__ span_g, int32_t* __restrict__ shift_g, int32_t* __restrict__ status) {
  const int seg = blockIdx.y;
  const int s = blockIdx.x * kCopyThreads + threadIdx.x;
  const size_t sb = static_cast<size_t>(seg) * cap;
  const size_t ub = static_cast<size_t>(seg) * n_units;
  int end = 0;                                    // slot + 1 if this slot stays occupied
  if (s < cap) {
    const int u = uid_g[sb + s];
    int shift = 0;
    if (u >= 0) {
      bool bad = u >= n_units;
      if (!bad) {
        const UnitRec rec = table[ub + u];
        const int p = pos_g[sb + s];
        const int r = p - rec.pos0;               // rank of the token inside its unit
        bad = r < 0 || r >= len_g[ub + u];
        if (!bad && r < rec.kl) {
          uid_g[sb + s] = rec.rank;
          pos_g[sb + s] = p - rec.del;
          shift = -rec.del;
          end = s + 1;
        } else if (!bad) {
          uid_g[sb + s] = -1;
          pos_g[sb + s] = -1;
        }
      }
      if (bad) set_status(status, OMNITIDE_E_TAGS);
    }
    if (shift_g != nullptr) shift_g[sb + s] = shift;
  }
  end = wave_max_i32(end);
  if ((threadIdx.x & (kWave - 1)) == 0 && end > 0) atomicMax(span_g + seg, end);
}

__global__ __launch_bounds__(kNatThreads) void suffix_plan_kernel(
    const uint32_t* __restrict__ bits_g, int cap, int page_size, int min_pages,
    int32_t* __restrict__ list, int32_t* __restrict__ meta, int32_t* __restrict__ span_g,
    int32_t* __restrict__ cut_g, int32_t* __restrict__ moved_g) {
  __shared__ uint32_t bits[kMaxNatWords];
  __shared__ int32_t scr[kNatThreads / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const size_t sb = static_cast<size_t>(seg) * cap;
  const int nwords = (cap + 31) / 32;
  load_bitmap(bits_g + static_cast<size_t>(seg) * nwords, bits, nwords);
  // thread t owns words [w0, w1), i.e. slots [32 w0, 32 w1)
  const int wpt = (nwords + kNatThreads - 1) / kNatThreads;
  const int w0 = min(tid * wpt, nwords), w1 = min(w0 + wpt, nwords);
  int my_live = 0, my_last = -1;
  for (int w = w0; w < w1; ++w) {
    my_live += __popc(bits[w]);
    if (bits[w]) my_last = 32 * w + 31 - __clz(bits[w]);
  }
  int total;
  const int live_before = block_exclusive_scan(my_live, scr, &total);
  int span_m1;
  const int last_before = block_exclusive_max(my_last, -1, scr, &span_m1);
  const int span = span_m1 + 1;
  const int pages_now = (span + page_size - 1) / page_size;
  // A cut c < span qualifies iff its packed span c + (entries at or after c) fits in
  // pages_now - min_pages pages, i.e. is at most `limit` slots.  Largest such c in this
  // thread's slots (the packed span never decreases with c).
  const long limit = static_cast<long>(pages_now - min_pages) * page_size;
  (void)last_before;
  // Per word: with e entries before slot 32w, slot 32w + j has packed span
  // (32w + total - e) + z(j), z(j) = empty slots of the word below j (non-decreasing), so the
  // largest qualifying j is the position of zero number K = limit - (32w + total - e) (or the
  // word's last slot below the span when it has at most K zeros below it).
  int best = -1;
  if (limit >= 0) {
    int live_lt = live_before;                      // entries before slot 32 w
    for (int w = w0; w < w1 && 32 * w < span; ++w) {
      const uint32_t word = bits[w];
      const int jmax = min(31, span - 1 - 32 * w);  // slots of the word below the span
      const long K = limit - (32L * w + total - live_lt);
      if (K >= 0) {
        const uint32_t valid = jmax == 31 ? ~0u : ((1u << (jmax + 1)) - 1u);
        const uint32_t zeros = ~word & valid;
        const int nz_below_max = __popc(zeros & ((1u << jmax) - 1u) & valid);
        best = 32 * w + (K >= nz_below_max ? jmax : nth_set_bit(zeros, static_cast<int>(K)));
      }
      live_lt += __popc(word);
    }
  }
  int c;
  (void)block_exclusive_max(best, -1, scr, &c);
  int n_suffix = 0, new_span = span, moved = 0;
  if (c >= 0) {
    // entries before c, counted by the thread whose range holds c
    int mine = 0;
    if (c >= 32 * w0 && c < 32 * w1) {
      mine = live_before;
      for (int w = w0; w < c / 32; ++w) mine += __popc(bits[w]);
      mine += __popc(bits[c / 32] & ((1u << (c % 32)) - 1u));
    }
    const int before_c = block_sum(mine, scr);
    n_suffix = total - before_c;
    new_span = c + n_suffix;
    int live_lt = live_before, moved_here = 0;
    for (int w = w0; w < w1 && 32 * w < span; ++w) {
      uint32_t word = bits[w];
      while (word) {
        const int j = __ffs(word) - 1;
        word &= word - 1;
        const int s = 32 * w + j;
        if (s >= c) {
          const int r = live_lt - before_c;
          list[sb + r] = s;
          moved_here += (c + r != s) ? 1 : 0;
        }
        ++live_lt;
      }
    }
    moved = block_sum(moved_here, scr);
  }
  if (tid == 0) {
    cut_g[seg] = c;
    moved_g[seg] = moved;
    span_g[seg] = new_span;
    meta[2 * seg] = n_suffix;
    meta[2 * seg + 1] = span;                       // span before packing
  }
}

// Rows and tags of the suffix entries whose slot changes: src -> scratch (SCATTER = false) or
// scratch -> c + rank (SCATTER = true, which also empties the vacated slots).
template <bool SCATTER>
__global__ __launch_bounds__(kCopyThreads) void suffix_copy_kernel(
    uint8_t* __restrict__ k, uint8_t* __restrict__ v, int cap, int row_bytes,
    int32_t* __restrict__ uid_g, uint8_t* __restrict__ mod_g, int32_t* __restrict__ pos_g,
    const int32_t* __restrict__ list, const int32_t* __restrict__ meta,
    const int32_t* __restrict__ cut_g, uint8_t* __restrict__ scr_rows,
    int32_t* __restrict__ scr_tags) {
  __shared__ int32_t src_row[kRowsPerBlock];
  const int seg = blockIdx.y;
  const int c = cut_g[seg];
  if (c < 0) return;
  const int n_suffix = meta[2 * seg];
  const int old_span = meta[2 * seg + 1];
  const size_t sb = static_cast<size_t>(seg) * cap;
  const int r0 = blockIdx.x * kRowsPerBlock;
  const int tid = threadIdx.x;
  if (SCATTER) {
    // vacated slots [c + n_suffix, old_span): this block's share
    for (int i = tid; i < kRowsPerBlock; i += kCopyThreads) {
      const int s = c + n_suffix + r0 + i;
      if (s < old_span) {
        uid_g[sb + s] = -1;
        pos_g[sb + s] = -1;
      }
    }
  }
  if (r0 >= n_suffix) return;
  const int nr = min(kRowsPerBlock, n_suffix - r0);
  if (tid < nr) {
    const int r = r0 + tid;
    const int s = list[sb + r];
    src_row[tid] = s != c + r ? s : -1;            // -1: already in place
    if (s != c + r) {
      int32_t* t = scr_tags + 3 * (sb + r);
      if (SCATTER) {
        uid_g[sb + c + r] = t[0];
        mod_g[sb + c + r] = static_cast<uint8_t>(t[1]);
        pos_g[sb + c + r] = t[2];
      } else {
        t[0] = uid_g[sb + s];
        t[1] = mod_g[sb + s];
        t[2] = pos_g[sb + s];
      }
    }
  }
  __syncthreads();
  const int vecs = row_bytes / 16;
  const int total = nr * vecs;
  // kNatBatch vectors of K and of V per thread in flight together, then the stores back to back
  for (int f0 = 0; f0 < total; f0 += kCopyThreads * kNatBatch) {
    u32x4 kb[kNatBatch], vb[kNatBatch];
#pragma unroll
    for (int j = 0; j < kNatBatch; ++j) {
      const int f = f0 + tid + kCopyThreads * j;
      const int i = f / vecs, e = f - i * vecs;
      const int s = f < total ? src_row[i] : -1;
      if (s < 0) continue;
      const int r = r0 + i;
      const size_t scr_off = ((sb + r) * 2) * static_cast<size_t>(row_bytes);
      const u32x4* ks = reinterpret_cast<const u32x4*>(
          SCATTER ? scr_rows + scr_off : k + (sb + s) * static_cast<size_t>(row_bytes));
      const u32x4* vs = reinterpret_cast<const u32x4*>(
          SCATTER ? scr_rows + scr_off + row_bytes
                  : v + (sb + s) * static_cast<size_t>(row_bytes));
      kb[j] = __builtin_nontemporal_load(ks + e);
      vb[j] = __builtin_nontemporal_load(vs + e);
    }
    __builtin_amdgcn_s_waitcnt(kVmcntZero);
#pragma unroll
    for (int j = 0; j < kNatBatch; ++j) {
      const int f = f0 + tid + kCopyThreads * j;
      const int i = f / vecs, e = f - i * vecs;
      const int s = f < total ? src_row[i] : -1;
      if (s < 0) continue;
      const int r = r0 + i;
      const size_t scr_off = ((sb + r) * 2) * static_cast<size_t>(row_bytes);
      u32x4* kd = reinterpret_cast<u32x4*>(
          SCATTER ? k + (sb + c + r) * static_cast<size_t>(row_bytes) : scr_rows + scr_off);
      u32x4* vd = reinterpret_cast<u32x4*>(
          SCATTER ? v + (sb + c + r) * static_cast<size_t>(row_bytes)
                  : scr_rows + scr_off + row_bytes);
      kd[e] = kb[j];
      vd[e] = vb[j];
    }
  }
}

__global__ __launch_bounds__(kNatThreads) void place_plan_kernel(
    const uint32_t* __restrict__ bits_g, int cap, int chunk_len, int32_t* __restrict__ slot_g,
    int32_t* __restrict__ span_g, int32_t* __restrict__ status) {
  __shared__ uint32_t bits[kMaxNatWords];
  __shared__ int32_t scr[kNatThreads / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int nwords = (cap + 31) / 32;
  load_bitmap(bits_g + static_cast<size_t>(seg) * nwords, bits, nwords);
  const int wpt = (nwords + kNatThreads - 1) / kNatThreads;
  const int w0 = min(tid * wpt, nwords), w1 = min(w0 + wpt, nwords);
  int my_last = -1;
  for (int w = w0; w < w1; ++w)
    if (bits[w]) my_last = 32 * w + 31 - __clz(bits[w]);
  int last_all;
  int last = block_exclusive_max(my_last, -1, scr, &last_all);
  // first slot s of this range where the empty run ending at s reaches chunk_len
  int cand = -1;
  for (int w = w0; w < w1 && cand < 0; ++w) {
    const uint32_t word = bits[w];
    const int end = min(32 * w + 32, cap);          // slots of this word: [32 w, end)
    if (chunk_len >= 32) {
      // A run of chunk_len >= 32 empty slots that ends inside this word ends before the
      // word's first occupied slot: O(1) per word.
      const int s = max(32 * w, last + chunk_len);  // first slot ending a long enough run
      const int first_set = word ? 32 * w + __ffs(word) - 1 : end;
      if (s < min(first_set, end)) {
        cand = s - chunk_len + 1;
        break;
      }
      if (word) last = 32 * w + 31 - __clz(word);
      continue;
    }
    if (word == 0u) {                               // all empty: the run only grows
      if (last + chunk_len < end) cand = last + 1;
      continue;
    }
    for (int s = 32 * w; s < end; ++s) {
      if ((word >> (s - 32 * w)) & 1u) {
        last = s;
      } else if (s - last >= chunk_len) {
        cand = s - chunk_len + 1;
        break;
      }
    }
  }
  // lowest candidate over all threads = -(largest of the negated candidates)
  int best;
  (void)block_exclusive_max(cand >= 0 ? -cand : -INT32_MAX, -INT32_MAX, scr, &best);
  if (tid == 0) {
    if (best == -INT32_MAX) {
      slot_g[seg] = -1;
      set_status(status, OMNITIDE_E_CAPACITY);
    } else {
      const int s = -best;
      slot_g[seg] = s;
      span_g[seg] = max(last_all + 1, s + chunk_len);
    }
  }
}

__global__ __launch_bounds__(kCopyThreads) void chunk_write_kernel(
    uint8_t* __restrict__ k, uint8_t* __restrict__ v, int cap, int row_bytes,
    int32_t* __restrict__ uid_g, uint8_t* __restrict__ mod_g, int32_t* __restrict__ pos_g,
    const uint8_t* __restrict__ k_chunk, const uint8_t* __restrict__ v_chunk,
    const uint8_t* __restrict__ chunk_mod, const int32_t* __restrict__ chunk_unit,
    int chunk_len, const int32_t* __restrict__ slot_g, const int32_t* __restrict__ kept_g,
    const int32_t* __restrict__ n_kept_units_g) {
  const int seg = blockIdx.y;
  const int s = slot_g[seg];
  if (s < 0) return;
  const size_t sb = static_cast<size_t>(seg) * cap;
  const size_t cb = static_cast<size_t>(seg) * chunk_len;
  const int r0 = blockIdx.x * kRowsPerBlock;
  const int nr = min(kRowsPerBlock, chunk_len - r0);
  const int tid = threadIdx.x;
  if (nr <= 0) return;
  if (tid < nr) {
    const int i = r0 + tid;
    uid_g[sb + s + i] = n_kept_units_g[seg] + chunk_unit[i];
    mod_g[sb + s + i] = chunk_mod[i];
    pos_g[sb + s + i] = kept_g[seg] + i;
  }
  const int vecs = row_bytes / 16;
  const int total = nr * vecs;
  // kNatBatch vectors of K and of V per thread in flight together, then the stores back to back
  for (int f0 = 0; f0 < total; f0 += kCopyThreads * kNatBatch) {
    u32x4 kb[kNatBatch], vb[kNatBatch];
#pragma unroll
    for (int j = 0; j < kNatBatch; ++j) {
      const int f = f0 + tid + kCopyThreads * j;
      if (f >= total) continue;
      const int i = r0 + f / vecs, e = f % vecs;
      kb[j] = reinterpret_cast<const u32x4*>(k_chunk + (cb + i) * row_bytes)[e];
      vb[j] = reinterpret_cast<const u32x4*>(v_chunk + (cb + i) * row_bytes)[e];
    }
    __builtin_amdgcn_s_waitcnt(kVmcntZero);
#pragma unroll
    for (int j = 0; j < kNatBatch; ++j) {
      const int f = f0 + tid + kCopyThreads * j;
      if (f >= total) continue;
      const int i = r0 + f / vecs, e = f % vecs;
      reinterpret_cast<u32x4*>(k + (sb + s + i) * static_cast<size_t>(row_bytes))[e] = kb[j];
      reinterpret_cast<u32x4*>(v + (sb + s + i) * static_cast<size_t>(row_bytes))[e] = vb[j];
    }
  }
}

}  // namespace

int native_max_cap() { return kMaxNatWords * 32; }

size_t evict_workspace_bytes(int n_seg, int n_units) {
  return static_cast<size_t>(n_seg) * n_units * sizeof(UnitRec);
}

size_t evict_rope_workspace_bytes(int n_seg, int n_units, int cap) {
  return align256(evict_workspace_bytes(n_seg, n_units)) +
         static_cast<size_t>(n_seg) * cap * sizeof(int32_t);
}

hipError_t launch_evict(const EvictArgs& a, hipStream_t stream) {
  UnitRec* table = static_cast<UnitRec*>(a.workspace);
  hipLaunchKernelGGL(evict_plan_kernel, dim3(a.n_seg), dim3(kNatThreads), 0, stream, a.keep,
                     a.keep_len, a.unit_len, a.n_units, table, a.unit_remap, a.kept_tokens,
                     a.n_kept_units, a.span);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.cap == 0) return hipSuccess;
  // with rotary adjustment: the slots' shifts go to the workspace after the unit table
  int32_t* shift = a.rope_dims > 0 ? reinterpret_cast<int32_t*>(
                                         static_cast<uint8_t*>(a.workspace) +
                                         align256(evict_workspace_bytes(a.n_seg, a.n_units)))
                                   : nullptr;
  const dim3 grid((a.cap + kCopyThreads - 1) / kCopyThreads, a.n_seg);
  hipLaunchKernelGGL(evict_apply_kernel, grid, dim3(kCopyThreads), 0, stream, a.unit_id, a.pos,
                     a.cap, a.n_units, table, a.unit_len, a.span, shift, a.d_status);
  e = hipGetLastError();
  if (e != hipSuccess || shift == nullptr) return e;
  return launch_rope_in_place(a.k, a.dtype, a.n_seg, a.cap, a.n_kv_heads, a.head_dim, shift,
                              a.rope_base, a.rope_dims, a.rope_half, stream);
}

static size_t bitmap_bytes(int n_seg, int cap) {
  return ((static_cast<size_t>(n_seg) * ((cap + 31) / 32) * 4 + 255) / 256) * 256;
}

static hipError_t launch_occupancy(const int32_t* uid, int n_seg, int cap, uint32_t* bits,
                                   hipStream_t stream) {
  const int nwords = (cap + 31) / 32;
  const int chunks = (cap + kWave - 1) / kWave;
  const int per_block = kCopyThreads / kWave;
  hipLaunchKernelGGL(occupancy_kernel, dim3((chunks + per_block - 1) / per_block, n_seg),
                     dim3(kCopyThreads), 0, stream, uid, cap, nwords, bits);
  return hipGetLastError();
}

size_t suffix_workspace_bytes(int n_seg, int cap, int row_bytes) {
  const size_t slots = static_cast<size_t>(n_seg) * cap;
  const size_t list = ((slots * 4 + 255) / 256) * 256;
  const size_t meta = 256 + ((static_cast<size_t>(n_seg) * 8 + 255) / 256) * 256;
  const size_t tags = ((slots * 12 + 255) / 256) * 256;
  return list + meta + tags + bitmap_bytes(n_seg, cap) +
         slots * 2 * static_cast<size_t>(row_bytes);
}

size_t place_workspace_bytes(int n_seg, int cap) { return bitmap_bytes(n_seg, cap); }

hipError_t launch_pack_suffix(const SuffixArgs& a, hipStream_t stream) {
  const size_t slots = static_cast<size_t>(a.n_seg) * a.cap;
  uint8_t* w = static_cast<uint8_t*>(a.workspace);
  int32_t* list = reinterpret_cast<int32_t*>(w);
  w += ((slots * 4 + 255) / 256) * 256;
  int32_t* meta = reinterpret_cast<int32_t*>(w);
  w += 256 + ((static_cast<size_t>(a.n_seg) * 8 + 255) / 256) * 256;
  int32_t* tags = reinterpret_cast<int32_t*>(w);
  w += ((slots * 12 + 255) / 256) * 256;
  uint32_t* bits = reinterpret_cast<uint32_t*>(w);
  w += bitmap_bytes(a.n_seg, a.cap);
  uint8_t* rows = w;
  hipError_t e = launch_occupancy(a.unit_id, a.n_seg, a.cap, bits, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(suffix_plan_kernel, dim3(a.n_seg), dim3(kNatThreads), 0, stream, bits,
                     a.cap, a.page_size, a.min_pages, list, meta, a.span, a.cut, a.moved);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid((a.cap + kRowsPerBlock - 1) / kRowsPerBlock, a.n_seg);
  uint8_t* k = static_cast<uint8_t*>(a.k);
  uint8_t* v = static_cast<uint8_t*>(a.v);
  hipLaunchKernelGGL(suffix_copy_kernel<false>, grid, dim3(kCopyThreads), 0, stream, k, v,
                     a.cap, a.row_bytes, a.unit_id, a.modality, a.pos, list, meta, a.cut, rows,
                     tags);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(suffix_copy_kernel<true>, grid, dim3(kCopyThreads), 0, stream, k, v,
                     a.cap, a.row_bytes, a.unit_id, a.modality, a.pos, list, meta, a.cut, rows,
                     tags);
  return hipGetLastError();
}

hipError_t launch_place_chunk(const PlaceArgs& a, hipStream_t stream) {
  uint32_t* bits = static_cast<uint32_t*>(a.workspace);
  hipError_t e = launch_occupancy(a.unit_id, a.n_seg, a.cap, bits, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(place_plan_kernel, dim3(a.n_seg), dim3(kNatThreads), 0, stream, bits, a.cap,
                     a.chunk_len, a.chunk_slot, a.span, a.d_status);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid((a.chunk_len + kRowsPerBlock - 1) / kRowsPerBlock, a.n_seg);
  hipLaunchKernelGGL(chunk_write_kernel, grid, dim3(kCopyThreads), 0, stream,
                     static_cast<uint8_t*>(a.k), static_cast<uint8_t*>(a.v), a.cap, a.row_bytes,
                     a.unit_id, a.modality, a.pos, static_cast<const uint8_t*>(a.k_chunk),
                     static_cast<const uint8_t*>(a.v_chunk), a.chunk_modality, a.chunk_unit,
                     a.chunk_len, a.chunk_slot, a.kept_tokens, a.n_kept_units);
  return hipGetLastError();
}

}  // namespace omnitide
