// OmniPick span plan in three kernels.
//
// 1. Census (one wave per unit).  The wave walks its unit's slots 1024 at a time (one aligned
//    16-byte block of tags per lane) and
//    finds where each span starts: at the unit's first slot and wherever the tag changes.  A
//    running maximum of the start slots (wave scan plus a carry across chunks) gives every
//    token its place in its span.  Each slot gets a code in the workspace: marker tokens and
//    the first sink_video / sink_audio tokens of each video / audio span are sinks (kept while
//    the unit is retained at all), text tokens get their rank among the unit's text tokens,
//    everything else is dropped from a partially kept unit.  Per unit: sinks, text tokens.
// 2. Plan (one workgroup per segment: one wave up to 512 units, 1024 threads beyond).  Each
//    thread owns up to 8 consecutive units.  Every step of the plan is a scan over units in id
//    (temporal) order, so the sequential walks of the planner become thresholds on prefix sums:
//      recent    newest live non-system units whose suffix total (own tokens included) is at
//                most R: lengths are positive, so the suffix grows monotonically and "stop at
//                the first misfit" is the set {u : suffix(u) <= R}
//      older     unit u keeps its sinks plus clamp(text_budget - T_u, 0, text_u) of its text
//                tokens, T_u = text tokens of older units before u
//      trimming  drop order = partially retained units by id, then complete non-system units
//                by id.  The i-th candidate is dropped iff, before it, the plan still exceeds
//                the low watermark and more than one unit is retained.  Both quantities only
//                decrease along the order, so each candidate decides from its exclusive prefix
//                (tokens and count of earlier candidates) alone.
// 3. Mark (one thread per slot): the slot stays if its unit is kept whole, or its unit is kept
//    in part and the slot is a sink or one of the unit's first text_keep text tokens.
#include "common.h"
#include "kernels.h"

namespace omnitide {

size_t span_plan_workspace_bytes(int n_seg, int n_slots, int n_units) {
  return span_ws_seg_bytes(n_slots, n_units) * static_cast<size_t>(n_seg);
}

namespace {

constexpr int kMaxPer = 8;
constexpr int kCensusWaves = 4;
constexpr int32_t kInfoSink = -1;   // marker, or inside the sink prefix of its span
constexpr int32_t kInfoDrop = -2;   // any other non-text token

struct SpanWs {
  int32_t* info;        // [n_slots] per-slot code: kInfoSink, kInfoDrop or text rank in unit
  int32_t* sinks;       // [U] sink tokens of the unit (-1: bad tag or slots outside the pool)
  int32_t* text;        // [U] text tokens of the unit
  int32_t* text_keep;   // [U] text tokens an older unit keeps
};

__device__ inline SpanWs span_ws(uint8_t* ws, int seg, int n_slots, int n_units) {
  uint8_t* b = ws + span_ws_seg_bytes(n_slots, n_units) * static_cast<size_t>(seg);
  const size_t info_bytes = span_ws_info_bytes(n_slots);
  const size_t ub = static_cast<size_t>(n_units) * 4;
  return SpanWs{reinterpret_cast<int32_t*>(b), reinterpret_cast<int32_t*>(b + info_bytes),
                reinterpret_cast<int32_t*>(b + info_bytes + ub),
                reinterpret_cast<int32_t*>(b + info_bytes + 2 * ub)};
}

constexpr int kCensusPer = 16;          // consecutive slots per lane in one census step
// Buffer resource word 3 for raw (unformatted) 32-bit data on this chip, and a byte offset past
// any buffer (accesses there read zero and write nothing).
constexpr int kBufferFlags = 0x00020000;
constexpr int kOutOfBuffer = 0x7fffffff;

__global__ __launch_bounds__(kCensusWaves * kWave) void span_census_kernel(
    const uint8_t* __restrict__ mod_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ first_g, int n_slots, int n_units, int sink_video,
    int sink_audio, uint8_t* __restrict__ ws, int32_t* __restrict__ status) {
  constexpr int P = kCensusPer;
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int u = blockIdx.x * kCensusWaves + __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  if (u >= n_units) return;
  const SpanWs W = span_ws(ws, seg, n_slots, n_units);
  const size_t ub = static_cast<size_t>(seg) * n_units;
  const int n = len_g[ub + u];
  const int f = first_g[ub + u];
  if (n <= 0 || f < 0 || f > n_slots - n) {     // no slots, or not inside the pool (the plan
    if (lane == 0) {                            // reports the latter as a tag error)
      W.sinks[u] = n <= 0 ? 0 : -1;
      W.text[u] = 0;
    }
    return;
  }
  // aligned 16-slot blocks of the segment's tag bytes (slot s at seg_tags + s)
  const uint8_t* seg_tags = mod_g + static_cast<size_t>(seg) * n_slots;
  const uintptr_t blk0 = block16_floor(seg_tags + f);
  const uintptr_t end = reinterpret_cast<uintptr_t>(seg_tags + f + n);
  const __amdgpu_buffer_rsrc_t info_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(W.info, 0, 4 * n_slots, kBufferFlags);
  int carry_tag = -1;      // tag of the slot before the step (-1 at the unit's start)
  int carry_start = f;     // first slot of the span that slot belongs to
  int carry_text = 0;      // the unit's text tokens before the step
  int sinks = 0;
  bool bad = false;
  for (uintptr_t c = blk0; c < end; c += P * kWave) {
    const uintptr_t b = c + P * static_cast<uintptr_t>(lane);   // this lane's block
    const int s0 = static_cast<int>(static_cast<intptr_t>(b) -
                                    reinterpret_cast<intptr_t>(seg_tags));
    int m[P];
    {
      uint8_t raw[16] = {};
      if (b < end) load_block16(b, raw);
#pragma unroll
      for (int j = 0; j < P; ++j) m[j] = ((s0 + j >= f) & (s0 + j < f + n)) ? raw[j] : -1;
    }
    int prev = __shfl_up(m[P - 1], 1, kWave);
    if (lane == 0) prev = carry_tag;
    int run = -1, nt = 0;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int pm = j == 0 ? prev : m[j - 1];
      if (m[j] >= 0 && m[j] != pm) run = s0 + j;   // a span starts here
      nt += m[j] == OMNITIDE_MOD_TEXT ? 1 : 0;
    }
    // running maximum of span starts, and over the lanes before this one
    const int inc = wave_scan_max_i32(run, -1);
    const int exc = dpp_move<kDppWaveShr1, 0xf>(-1, inc);
    int start = max(exc, carry_start);             // span start of the slot before s0
    const int incl = wave_inclusive_scan(nt);
    const int text_tot = __shfl(incl, kWave - 1, kWave);
    int text_rank = carry_text + incl - nt;        // the unit's text tokens before s0
    // Branch-free per slot (selects instead of divergent branches); the code of a slot outside
    // the unit goes to an offset past the buffer, which the hardware drops.
    int pm = prev;
#pragma unroll
    for (int j = 0; j < P; ++j) {
      const int s = s0 + j;
      // (bitwise & and | on the conditions: no short-circuit branches)
      const bool live = m[j] >= 0;
      start = (live & (m[j] != pm)) ? s : start;
      const int place = s - start + 1;             // 1-based place in its span
      const bool text = m[j] == OMNITIDE_MOD_TEXT;
      const bool sink = (m[j] == OMNITIDE_MOD_MARK) |
                        ((m[j] == OMNITIDE_MOD_VIDEO) & (place <= sink_video)) |
                        ((m[j] == OMNITIDE_MOD_AUDIO) & (place <= sink_audio));
      const int32_t code = text ? text_rank : (sink ? kInfoSink : kInfoDrop);
      text_rank += (live & text) ? 1 : 0;
      sinks += (live & !text & sink) ? 1 : 0;
      bad |= live & (m[j] > OMNITIDE_MOD_MARK);
      __builtin_amdgcn_raw_buffer_store_b32(code, info_rsrc, live ? 4 * s : kOutOfBuffer, 0, 0);
      pm = m[j];
    }
    carry_tag = __shfl(m[P - 1], kWave - 1, kWave);
    carry_start = max(carry_start, __shfl(inc, kWave - 1, kWave));
    carry_text += text_tot;
  }
  const uint32_t tot = wave_sum_u32(static_cast<uint32_t>(sinks));
  const bool any_bad = __any(bad);
  if (lane == 0) {
    W.sinks[u] = any_bad ? -1 : static_cast<int32_t>(tot);
    W.text[u] = carry_text;
    if (any_bad) set_status(status, OMNITIDE_E_TAGS);
  }
}

template <int T>
__global__ __launch_bounds__(T) void plan_spans_kernel(
    const int32_t* __restrict__ len_g, const int32_t* __restrict__ first_g,
    const int32_t* __restrict__ last_g, const uint32_t* __restrict__ flags_g, int n_slots,
    int n_units, int low, int high, int recent, int text_budget,
    int32_t* __restrict__ keep_len_g, int32_t* __restrict__ kept_g, uint8_t* __restrict__ ws,
    int32_t* __restrict__ status) {
  __shared__ int32_t scr[T / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = n_units;
  const int per = (U + T - 1) / T;
  const int u0 = tid * per;
  const size_t base = static_cast<size_t>(seg) * U;
  const SpanWs W = span_ws(ws, seg, n_slots, n_units);

  int ln[kMaxPer], fs[kMaxPer], ls[kMaxPer], sk[kMaxPer], tx[kMaxPer];
  uint32_t fl[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {        // all loads first: one memory round trip
    const int u = min(u0 + i, U - 1);
    ln[i] = len_g[base + u];
    fs[i] = first_g[base + u];
    ls[i] = last_g[base + u];
    fl[i] = flags_g[base + u];
    sk[i] = W.sinks[u];
    tx[i] = W.text[u];
  }
  bool bad = false;
  int my_max_first = -1;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (!(i < per && u0 + i < U) || ln[i] <= 0) ln[i] = 0;
    const bool live = ln[i] > 0;
    const bool in_range = live && fs[i] >= 0 && fs[i] <= n_slots - ln[i];
    bad |= live && (!in_range || ls[i] - fs[i] + 1 != ln[i] || sk[i] < 0);
    if (live) my_max_first = max(my_max_first, fs[i]);
  }
  // live units must appear in unit order
  int ignored;
  int run = block_exclusive_max(my_max_first, -1, scr, &ignored);
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (ln[i] > 0) {
      bad |= fs[i] <= run;
      run = max(run, fs[i]);
    }
  }
  const int n_bad = block_sum(bad ? 1 : 0, scr);
  auto write_out = [&](const int* kl) {
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i)
      if (i < per && u0 + i < U) keep_len_g[base + u0 + i] = kl[i];
  };
  int kl[kMaxPer];
  if (n_bad > 0) {
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) kl[i] = 0;
    write_out(kl);
    if (tid == 0) {
      kept_g[seg] = 0;
      set_status(status, OMNITIDE_E_TAGS);
    }
    return;
  }

  int my_len = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) my_len += ln[i];
  const int total = block_sum(my_len, scr);
  if (total <= high) {                         // at or below the high watermark: keep all
    write_out(ln);
    if (tid == 0) kept_g[seg] = total;
    return;
  }

  bool sys[kMaxPer];
  int my_elig = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    sys[i] = ln[i] > 0 && (fl[i] & 1u) != 0;
    my_elig += (ln[i] > 0 && !sys[i]) ? ln[i] : 0;
  }
  // recent window: suffix sums of eligible lengths
  int elig_total;
  const int elig_before = block_exclusive_scan(my_elig, scr, &elig_total);
  int suffix = elig_total - elig_before - my_elig;
  bool rec[kMaxPer];
#pragma unroll
  for (int i = kMaxPer - 1; i >= 0; --i) {
    rec[i] = false;
    if (ln[i] > 0 && !sys[i]) {
      suffix += ln[i];
      rec[i] = suffix <= recent;
    }
  }
  // older units: their sinks, and text tokens under the shared budget (oldest first)
  int my_text = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) my_text += (ln[i] > 0 && !sys[i] && !rec[i]) ? tx[i] : 0;
  int text_total;
  int text_before = block_exclusive_scan(my_text, scr, &text_total);
  int my_kept = 0, my_part = 0, my_part_n = 0, my_comp = 0, my_comp_n = 0, my_ret = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    int k = 0, tk = 0;
    if (ln[i] > 0) {
      if (sys[i] || rec[i]) {
        k = ln[i];
      } else {
        tk = min(tx[i], max(text_budget - text_before, 0));
        k = sk[i] + tk;
        text_before += tx[i];
      }
    }
    if (i < per && u0 + i < U) W.text_keep[u0 + i] = tk;
    kl[i] = k;
    my_kept += k;
    my_ret += k > 0 ? 1 : 0;
    if (k > 0 && k < ln[i]) {
      my_part += k;
      ++my_part_n;
    } else if (k > 0 && !sys[i]) {
      my_comp += k;
      ++my_comp_n;
    }
  }
  const int kept0 = block_sum(my_kept, scr);
  const int retained0 = block_sum(my_ret, scr);
  int part_tok, part_n, comp_tok, comp_n;
  int part_before = block_exclusive_scan(my_part, scr, &part_tok);
  int part_rank = block_exclusive_scan(my_part_n, scr, &part_n);
  int comp_before = block_exclusive_scan(my_comp, scr, &comp_tok);
  int comp_rank = block_exclusive_scan(my_comp_n, scr, &comp_n);
  (void)comp_tok;
  (void)comp_n;
  int my_final = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    const int k = kl[i];
    if (k > 0 && k < ln[i]) {
      // candidate number part_rank (0-based) of the drop order
      if (kept0 - part_before > low && retained0 - part_rank > 1) kl[i] = 0;
      part_before += k;
      ++part_rank;
    } else if (k > 0 && !sys[i]) {
      if (kept0 - part_tok - comp_before > low && retained0 - part_n - comp_rank > 1) kl[i] = 0;
      comp_before += k;
      ++comp_rank;
    }
    my_final += kl[i];
  }
  write_out(kl);
  const int kept = block_sum(my_final, scr);
  if (tid == 0) kept_g[seg] = kept;
}

}  // namespace

constexpr int kMarkThreads = 256;

__global__ __launch_bounds__(kMarkThreads) void span_mark_kernel(
    const int32_t* __restrict__ uid_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ keep_len_g, int n_slots, int n_units, uint8_t* __restrict__ ws,
    uint8_t* __restrict__ keep_slot_g) {
  const int seg = blockIdx.y;
  const int s = blockIdx.x * kMarkThreads + threadIdx.x;
  if (s >= n_slots) return;
  const size_t sb = static_cast<size_t>(seg) * n_slots;
  const size_t ub = static_cast<size_t>(seg) * n_units;
  const int u = uid_g[sb + s];
  uint8_t out = 0;
  if (u >= 0 && u < n_units) {
    const int kl = keep_len_g[ub + u];
    if (kl > 0) {
      if (kl >= len_g[ub + u]) {
        out = 1;
      } else {
        const SpanWs W = span_ws(ws, seg, n_slots, n_units);
        const int32_t code = W.info[s];
        out = (code == kInfoSink || (code >= 0 && code < W.text_keep[u])) ? 1 : 0;
      }
    }
  }
  keep_slot_g[sb + s] = out;
}

hipError_t launch_plan_spans(const SpanPlanArgs& a, hipStream_t stream) {
  uint8_t* ws = static_cast<uint8_t*>(a.workspace);
  const dim3 cgrid((a.n_units + kCensusWaves - 1) / kCensusWaves, a.n_seg);
  hipLaunchKernelGGL(span_census_kernel, cgrid, dim3(kCensusWaves * kWave), 0, stream,
                     a.modality, a.unit_len, a.unit_first, a.n_slots, a.n_units, a.sink_video,
                     a.sink_audio, ws, a.d_status);
  if (a.n_units <= 64 * kMaxPer)
    hipLaunchKernelGGL(plan_spans_kernel<64>, dim3(a.n_seg), dim3(64), 0, stream, a.unit_len,
                       a.unit_first, a.unit_last, a.unit_flags, a.n_slots, a.n_units, a.low,
                       a.high, a.recent, a.text_budget, a.keep_len, a.kept_tokens, ws,
                       a.d_status);
  else
    hipLaunchKernelGGL(plan_spans_kernel<1024>, dim3(a.n_seg), dim3(1024), 0, stream, a.unit_len,
                       a.unit_first, a.unit_last, a.unit_flags, a.n_slots, a.n_units, a.low,
                       a.high, a.recent, a.text_budget, a.keep_len, a.kept_tokens, ws,
                       a.d_status);
  if (a.n_slots > 0) {
    const dim3 mgrid((a.n_slots + kMarkThreads - 1) / kMarkThreads, a.n_seg);
    hipLaunchKernelGGL(span_mark_kernel, mgrid, dim3(kMarkThreads), 0, stream, a.unit_id,
                       a.unit_len, a.keep_len, a.n_slots, a.n_units, ws, a.keep_slot);
  }
  return hipGetLastError();
}

}  // namespace omnitide
