// OmniPick span plan, one workgroup per segment (one wave up to 512 units, 1024 threads beyond).
//
// Each thread owns up to 8 consecutive units.  Every step of the plan is a scan over units in
// id (temporal) order, so the sequential walks of the planner become thresholds on prefix sums:
//   recent    newest live non-system units whose suffix total (own tokens included) is at most
//             R: lengths are positive, so the suffix grows monotonically and "stop at the first
//             misfit" is the set {u : suffix(u) <= R}
//   sinks     older video / audio units keep min(len, sink_video / sink_audio) leading tokens
//   text      older text unit u keeps clamp(text_budget - (older text tokens before u), 0, len)
//   trimming  drop order = partially retained units by id, then complete non-system units by
//             id.  The i-th candidate is dropped iff, before it, the plan still exceeds the low
//             watermark and more than one unit is retained.  Both quantities only decrease along
//             the order, so each candidate decides from its exclusive prefix (tokens and count
//             of earlier candidates) alone.
#include "common.h"
#include "kernels.h"

namespace omnitide {
namespace {

constexpr int kMaxPer = 8;

template <int T>
__global__ __launch_bounds__(T) void plan_spans_kernel(
    const int32_t* __restrict__ len_g, const int32_t* __restrict__ first_g,
    const int32_t* __restrict__ last_g, const uint32_t* __restrict__ flags_g,
    const uint8_t* __restrict__ mod_g, int n_slots, int n_units, int low, int high, int recent,
    int sink_video, int sink_audio, int text_budget, int32_t* __restrict__ keep_len_g,
    int32_t* __restrict__ kept_g, int32_t* __restrict__ status) {
  __shared__ int32_t scr[T / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = n_units;
  const int per = (U + T - 1) / T;
  const int u0 = tid * per;
  const size_t base = static_cast<size_t>(seg) * U;
  const size_t sbase = static_cast<size_t>(seg) * n_slots;

  int ln[kMaxPer], fs[kMaxPer], ls[kMaxPer];
  uint32_t fl[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {        // all loads first: one memory round trip
    const int u = min(u0 + i, U - 1);
    ln[i] = len_g[base + u];
    fs[i] = first_g[base + u];
    ls[i] = last_g[base + u];
    fl[i] = flags_g[base + u];
  }
  bool bad = false;
  int my_max_first = -1;
  int md[kMaxPer];
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    if (!(i < per && u0 + i < U) || ln[i] <= 0) ln[i] = 0;
    const bool live = ln[i] > 0;
    const bool in_range = live && fs[i] >= 0 && fs[i] < n_slots;
    bad |= live && (!in_range || ls[i] - fs[i] + 1 != ln[i]);
    md[i] = in_range ? mod_g[sbase + fs[i]] : 0;
    bad |= live && md[i] > OMNITIDE_MOD_TEXT;
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
  // older units: sink prefixes and the shared text budget (oldest first)
  int my_text = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i)
    my_text += (ln[i] > 0 && !sys[i] && !rec[i] && md[i] == OMNITIDE_MOD_TEXT) ? ln[i] : 0;
  int text_total;
  int text_before = block_exclusive_scan(my_text, scr, &text_total);
  int my_kept = 0, my_part = 0, my_part_n = 0, my_comp = 0, my_comp_n = 0, my_ret = 0;
#pragma unroll
  for (int i = 0; i < kMaxPer; ++i) {
    int k = 0;
    if (ln[i] > 0) {
      if (sys[i] || rec[i]) {
        k = ln[i];
      } else if (md[i] == OMNITIDE_MOD_VIDEO) {
        k = min(ln[i], sink_video);
      } else if (md[i] == OMNITIDE_MOD_AUDIO) {
        k = min(ln[i], sink_audio);
      } else if (md[i] == OMNITIDE_MOD_TEXT) {
        k = min(ln[i], max(text_budget - text_before, 0));
        text_before += ln[i];
      }
    }
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

hipError_t launch_plan_spans(const SpanPlanArgs& a, hipStream_t stream) {
  if (a.n_units <= 64 * kMaxPer)
    hipLaunchKernelGGL(plan_spans_kernel<64>, dim3(a.n_seg), dim3(64), 0, stream, a.unit_len,
                       a.unit_first, a.unit_last, a.unit_flags, a.modality, a.n_slots,
                       a.n_units, a.low, a.high, a.recent, a.sink_video, a.sink_audio,
                       a.text_budget, a.keep_len, a.kept_tokens, a.d_status);
  else
    hipLaunchKernelGGL(plan_spans_kernel<1024>, dim3(a.n_seg), dim3(1024), 0, stream, a.unit_len,
                       a.unit_first, a.unit_last, a.unit_flags, a.modality, a.n_slots,
                       a.n_units, a.low, a.high, a.recent, a.sink_video, a.sink_audio,
                       a.text_budget, a.keep_len, a.kept_tokens, a.d_status);
  return hipGetLastError();
}

}  // namespace omnitide
