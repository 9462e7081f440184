// Budgeted whole-unit selection, one workgroup per segment.  Up to 512 units: a single wave
// (select_small_kernel); beyond: 1024 threads with all state in LDS (select_kernel).
//
// Groups (paper: must-keep, recent-context, selected-history):
//   protected  units holding a system token (all kept; over budget -> OMNITIDE_E_BUDGET)
//   recent     newest live non-system units whose suffix total fits min(R, B - T_sys); because
//              lengths are positive the suffix total grows monotonically, so "walk newest to
//              oldest and stop at the first misfit" is the set {u : suffix(u) <= cap}
//   selected   remaining live units sorted by the 64-bit key (score << 13 | id) descending
//              (bitonic sort in LDS), kept while the inclusive prefix of their lengths fits;
//              the prefix sum grows monotonically, so "stop at the first misfit" is again a
//              threshold on the prefix.
// Thread t owns the consecutive units [t*per, (t+1)*per), per = ceil(U / 1024) <= 8.
#include "common.h"
#include "kernels.h"

namespace omnitide {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kMaxUnits = OMNITIDE_MAX_UNITS;
constexpr int kPer = kMaxUnits / kSelThreads;
constexpr int kIdBits = 13;   // 2^13 = kMaxUnits
// Scores below 2^51 fit the 64-bit ranking key (score << kIdBits | id) with one bit to spare.
// omnitide_score_units never exceeds 2^43: a slot contributes at most 4,096 elements x 2^21 x
// a weight of 2^10.
constexpr int kScoreBits = 51;

// floor(n / d) for d >= 1.  Below 2^53 the dividend is exact in double: the correctly rounded
// quotient is at most one above the floor (when the true quotient lies just below an integer),
// which the remainder's sign corrects.  Larger dividends take the integer division.
__device__ inline uint64_t udiv64(uint64_t n, uint32_t d) {
  if (n < (1ull << 53)) {
    uint64_t q = static_cast<uint64_t>(static_cast<double>(n) / static_cast<double>(d));
    if (static_cast<int64_t>(n - q * d) < 0) --q;
    return q;
  }
  return n / d;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const uint64_t* __restrict__ wsum_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ first_g, const int32_t* __restrict__ last_g,
    const uint32_t* __restrict__ flags_g, int n_units, int budget, int recent,
    uint64_t* __restrict__ score_g, uint8_t* __restrict__ keep_g,
    int32_t* __restrict__ kept_tokens_g, int32_t* __restrict__ status) {
  __shared__ uint64_t keys[kMaxUnits];
  __shared__ int32_t lens[kMaxUnits];
  __shared__ uint8_t chosen[kMaxUnits];
  __shared__ int32_t scr_i[kSelThreads / kWave + 1];

  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int U = n_units;
  const int per = (U + kSelThreads - 1) / kSelThreads;
  const int u0 = tid * per;
  const size_t base = static_cast<size_t>(seg) * U;

  int ln[kPer], fs[kPer], ls[kPer];
  bool sys[kPer];
  uint64_t sc[kPer];
  bool bad = false, big = false;
  int my_max_first = -1;
  uint32_t fl[kPer];
  uint64_t ws[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {           // all loads first: one memory round trip
    const int u = min(u0 + i, U - 1);
    ln[i] = len_g[base + u];
    fs[i] = first_g[base + u];
    ls[i] = last_g[base + u];
    fl[i] = flags_g[base + u];
    ws[i] = wsum_g[base + u];
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = u0 + i;
    const bool mine = i < per && u < U;
    if (!mine || ln[i] <= 0) ln[i] = 0;
    const bool live = ln[i] > 0;
    sys[i] = live && (fl[i] & 1u) != 0;
    sc[i] = live ? udiv64(ws[i], static_cast<uint32_t>(ln[i])) : 0;
    bad |= live && (ls[i] - fs[i] + 1) != ln[i];
    big |= (sc[i] >> kScoreBits) != 0;          // the ranking key holds kScoreBits of score
    if (live) my_max_first = max(my_max_first, fs[i]);
    if (mine) {
      score_g[base + u] = sc[i];
      chosen[u] = 0;
      lens[u] = ln[i];
    }
  }
  // live units must appear in unit order: each first slot exceeds every earlier live unit's
  int ignored;
  int run = block_exclusive_max(my_max_first, -1, scr_i, &ignored);
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (ln[i] > 0) {
      bad |= fs[i] <= run;
      run = max(run, fs[i]);
    }
  }
  const int n_bad = block_sum(bad ? 1 : 0, scr_i);
  const int n_big = block_sum(big ? 1 : 0, scr_i);

  int my_sys = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) my_sys += sys[i] ? ln[i] : 0;
  const int t_sys = block_sum(my_sys, scr_i);

  if (n_bad > 0 || n_big > 0 || t_sys > budget) {
    for (int u = tid; u < U; u += kSelThreads) keep_g[base + u] = 0;
    if (tid == 0) {
      kept_tokens_g[seg] = 0;
      set_status(status, n_bad > 0   ? OMNITIDE_E_TAGS
                         : n_big > 0 ? OMNITIDE_E_RANGE
                                     : OMNITIDE_E_BUDGET);
    }
    return;
  }

  // recent window: suffix sums of eligible (live, non-system) lengths
  const int cap_rec = min(recent, budget - t_sys);
  int my_elig = 0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) my_elig += (ln[i] > 0 && !sys[i]) ? ln[i] : 0;
  int elig_total;
  const int elig_before = block_exclusive_scan(my_elig, scr_i, &elig_total);
  int suffix = elig_total - elig_before - my_elig;   // eligible tokens in later threads
  bool rec[kPer];
  int my_rec = 0;
#pragma unroll
  for (int i = kPer - 1; i >= 0; --i) {
    rec[i] = false;
    if (ln[i] > 0 && !sys[i]) {
      suffix += ln[i];
      rec[i] = suffix <= cap_rec;
      my_rec += rec[i] ? ln[i] : 0;
    }
  }
  const int t_rec = block_sum(my_rec, scr_i);
  const int cap_sel = budget - t_sys - t_rec;

  // candidates sorted by (score desc, id desc); key 0 = not a candidate (sorts last)
  int P = 1;
  while (P < U) P <<= 1;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = u0 + i;
    if (i < per && u < U) {
      const bool cand = ln[i] > 0 && !sys[i] && !rec[i];
      keys[u] = cand ? ((sc[i] << kIdBits) | static_cast<uint64_t>(u)) + 1 : 0;
    }
  }
  for (int u = U + tid; u < P; u += kSelThreads) keys[u] = 0;
  __syncthreads();
  for (int kk = 2; kk <= P; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += kSelThreads) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = keys[i], b = keys[ixj];
          const bool desc = (i & kk) == 0;
          if (desc ? (a < b) : (a > b)) {
            keys[i] = b;
            keys[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
  }

  // prefix of candidate lengths in rank order; thread t owns ranks [t*per2, (t+1)*per2)
  const int per2 = (P + kSelThreads - 1) / kSelThreads;
  const int r0 = tid * per2;
  int my_cand = 0;
  for (int i = 0; i < per2; ++i) {
    const int r = r0 + i;
    if (r < P && keys[r] != 0) my_cand += lens[(keys[r] - 1) & (kMaxUnits - 1)];
  }
  int ignored2;
  int pre = block_exclusive_scan(my_cand, scr_i, &ignored2);
  int my_sel = 0;
  for (int i = 0; i < per2; ++i) {
    const int r = r0 + i;
    if (r < P && keys[r] != 0) {
      const int u = static_cast<int>((keys[r] - 1) & (kMaxUnits - 1));
      pre += lens[u];
      if (pre <= cap_sel) {
        chosen[u] = 1;
        my_sel += lens[u];
      }
    }
  }
  const int t_sel = block_sum(my_sel, scr_i);   // contains a barrier: chosen[] is complete
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int u = u0 + i;
    if (i < per && u < U) keep_g[base + u] = (sys[i] || rec[i] || chosen[u]) ? 1 : 0;
  }
  if (tid == 0) kept_tokens_g[seg] = t_sys + t_rec + t_sel;
}


// Single-wave variant for U <= 512 (every lane owns 8 consecutive units): the same plan with
// wave-level scans (no workgroup barriers) and, instead of a full sort, an MSD radix select of
// the cut.  The walk "rank order, stop at the first misfit" keeps exactly the candidates whose
// key exceeds the first misfit's key; the misfit is found digit by digit: a histogram of
// candidate lengths over the next key bits (LDS atomics) and a scan in descending digit order
// locate the bucket where the running total first exceeds the cap; higher buckets are kept,
// lower ones dropped, and the search continues inside that bucket until it holds one key.
// Digits are 10 bits wide (1,024 buckets), so a 50-bit key takes five passes.
constexpr int kSmallUnits = 512;
constexpr int kSmallPer = kSmallUnits / kWave;
constexpr int kDigitBits = 10;                       // radix-select digit
constexpr int kBuckets = 1 << kDigitBits;
constexpr int kBucketsPerLane = kBuckets / kWave;


__device__ inline int wave_exclusive_sum(int v, int* total) {
  const int inc = wave_inclusive_scan(v);
  *total = __shfl(inc, kWave - 1, kWave);
  return inc - v;
}

__global__ __launch_bounds__(kWave) void select_small_kernel(
    const uint64_t* __restrict__ wsum_g, const int32_t* __restrict__ len_g,
    const int32_t* __restrict__ first_g, const int32_t* __restrict__ last_g,
    const uint32_t* __restrict__ flags_g, int n_units, int budget, int recent,
    uint64_t* __restrict__ score_g, uint8_t* __restrict__ keep_g,
    int32_t* __restrict__ kept_tokens_g, int32_t* __restrict__ status) {
  __shared__ __attribute__((aligned(16))) int32_t hist[kBuckets];
  const int seg = blockIdx.x;
  const int lane = threadIdx.x;
  const int U = n_units;
  const int u0 = lane * kSmallPer;
  const size_t base = static_cast<size_t>(seg) * U;

  int ln[kSmallPer], fs[kSmallPer], ls[kSmallPer];
  uint32_t fl[kSmallPer];
  uint64_t ws[kSmallPer];
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {      // all loads first: one memory round trip
    const int u = min(u0 + i, U - 1);
    ln[i] = len_g[base + u];
    fs[i] = first_g[base + u];
    ls[i] = last_g[base + u];
    fl[i] = flags_g[base + u];
    ws[i] = wsum_g[base + u];
  }
  bool sys[kSmallPer];
  uint64_t key[kSmallPer];
  bool bad = false, big = false;
  int my_max_first = -1;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    const int u = u0 + i;
    if (u >= U || ln[i] <= 0) ln[i] = 0;
    const bool live = ln[i] > 0;
    sys[i] = live && (fl[i] & 1u) != 0;
    const uint64_t sc = live ? udiv64(ws[i], static_cast<uint32_t>(ln[i])) : 0;
    bad |= live && (ls[i] - fs[i] + 1) != ln[i];
    big |= (sc >> kScoreBits) != 0;
    if (live) my_max_first = max(my_max_first, fs[i]);
    if (u < U) score_g[base + u] = sc;
    key[i] = (sc << kIdBits) | static_cast<uint64_t>(u);
  }
  // unit order: every live unit's first slot exceeds all earlier live units' first slots
  int run = wave_exclusive_max_i32(my_max_first, -1);
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    if (ln[i] > 0) {
      bad |= fs[i] <= run;
      run = max(run, fs[i]);
    }
  }
  int my_sys = 0, my_elig = 0;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    my_sys += sys[i] ? ln[i] : 0;
    my_elig += (ln[i] > 0 && !sys[i]) ? ln[i] : 0;
  }
  int t_sys, elig_total;
  wave_exclusive_sum(my_sys, &t_sys);
  const int elig_before = wave_exclusive_sum(my_elig, &elig_total);
  const bool any_bad = __any(bad);
  const bool any_big = __any(big);
  if (any_bad || any_big || t_sys > budget) {
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i)
      if (u0 + i < U) keep_g[base + u0 + i] = 0;
    if (lane == 0) {
      kept_tokens_g[seg] = 0;
      set_status(status, any_bad   ? OMNITIDE_E_TAGS
                         : any_big ? OMNITIDE_E_RANGE
                                   : OMNITIDE_E_BUDGET);
    }
    return;
  }
  // recent window: suffix sums of eligible lengths, newest unit first
  const int cap_rec = min(recent, budget - t_sys);
  int suffix = elig_total - elig_before - my_elig;
  bool rec[kSmallPer];
  int my_rec = 0;
#pragma unroll
  for (int i = kSmallPer - 1; i >= 0; --i) {
    rec[i] = false;
    if (ln[i] > 0 && !sys[i]) {
      suffix += ln[i];
      rec[i] = suffix <= cap_rec;
      my_rec += rec[i] ? ln[i] : 0;
    }
  }
  int t_rec;
  wave_exclusive_sum(my_rec, &t_rec);
  const int cap_sel = budget - t_sys - t_rec;

  // radix select of the first misfit among candidates (state: 1 active, 2 kept, 0 dropped)
  int state[kSmallPer];
  uint64_t kmax = 0;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    state[i] = (ln[i] > 0 && !sys[i] && !rec[i]) ? 1 : 0;
    if (state[i]) kmax = max(kmax, key[i]);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) kmax = max(kmax, __shfl_xor(kmax, off, kWave));
  int taken = 0;                                   // tokens already kept by the search
  int hi = 64 - __builtin_clzll(kmax | 1);         // key bits in use
  while (hi > 0) {
    const int lo = max(hi - kDigitBits, 0);
    const uint64_t mask = (1ull << (hi - lo)) - 1;
#pragma unroll
    for (int j = 0; j < kBucketsPerLane / 4; ++j)
      *reinterpret_cast<int4*>(&hist[kBucketsPerLane * lane + 4 * j]) = make_int4(0, 0, 0, 0);
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i)
      if (state[i] == 1) atomicAdd(&hist[(key[i] >> lo) & mask], ln[i]);
    __syncthreads();
    // descending digit order: lane owns digits kBuckets-1 - kBucketsPerLane*lane - j
    int hv[kBucketsPerLane], hsum = 0;
    {
      const int top = kBuckets - kBucketsPerLane * (lane + 1);   // lowest digit of the lane
#pragma unroll
      for (int j = 0; j < kBucketsPerLane / 4; ++j) {
        const int4 w = *reinterpret_cast<const int4*>(&hist[top + 4 * j]);
        hv[kBucketsPerLane - 1 - 4 * j] = w.x;
        hv[kBucketsPerLane - 2 - 4 * j] = w.y;
        hv[kBucketsPerLane - 3 - 4 * j] = w.z;
        hv[kBucketsPerLane - 4 - 4 * j] = w.w;
      }
#pragma unroll
      for (int j = 0; j < kBucketsPerLane; ++j) hsum += hv[j];
    }
    int tot;
    int acc = taken + wave_exclusive_sum(hsum, &tot);
    (void)tot;
    int cut = -1;                                  // first digit whose bucket overflows
#pragma unroll
    for (int j = 0; j < kBucketsPerLane; ++j) {
      if (cut < 0 && acc + hv[j] > cap_sel) cut = kBuckets - 1 - kBucketsPerLane * lane - j;
      acc += hv[j];
    }
    const uint64_t cut_lanes = __ballot(cut >= 0);
    if (cut_lanes == 0) {                          // every active candidate fits
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i)
        if (state[i] == 1) state[i] = 2;
      break;
    }
    const int d_cut = __shfl(cut, __builtin_ctzll(cut_lanes), kWave);
    int my_above = 0;
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) {
      if (state[i] == 1) {
        const int dg = static_cast<int>((key[i] >> lo) & mask);
        if (dg > d_cut) {
          state[i] = 2;
          my_above += ln[i];
        } else if (dg < d_cut) {
          state[i] = 0;
        }
      }
    }
    int above, my_left = 0, left;
#pragma unroll
    for (int i = 0; i < kSmallPer; ++i) my_left += state[i] == 1 ? 1 : 0;
    wave_exclusive_sum(my_above, &above);
    wave_exclusive_sum(my_left, &left);
    taken += above;
    hi = lo;
    __syncthreads();
    if (hi == 0 || left <= 1) {                    // one key left in the bucket: the misfit
#pragma unroll
      for (int i = 0; i < kSmallPer; ++i)
        if (state[i] == 1) state[i] = 0;
      break;
    }
  }
  int my_sel = 0;
#pragma unroll
  for (int i = 0; i < kSmallPer; ++i) {
    const int u = u0 + i;
    if (u < U) {
      const bool kp = sys[i] || rec[i] || state[i] == 2;
      keep_g[base + u] = kp ? 1 : 0;
      my_sel += state[i] == 2 ? ln[i] : 0;
    }
  }
  int t_sel;
  wave_exclusive_sum(my_sel, &t_sel);
  if (lane == 0) kept_tokens_g[seg] = t_sys + t_rec + t_sel;
}

}  // namespace

hipError_t launch_select(const uint64_t* wsum, const int32_t* len, const int32_t* first,
                         const int32_t* last, const uint32_t* flags, int n_seg, int n_units,
                         int budget, int recent, uint64_t* score, uint8_t* keep,
                         int32_t* kept_tokens, int32_t* status, hipStream_t stream) {
  if (n_units <= kSmallUnits)
    hipLaunchKernelGGL(select_small_kernel, dim3(n_seg), dim3(kWave), 0, stream, wsum, len,
                       first, last, flags, n_units, budget, recent, score, keep, kept_tokens,
                       status);
  else
    hipLaunchKernelGGL(select_kernel, dim3(n_seg), dim3(kSelThreads), 0, stream, wsum, len,
                       first, last, flags, n_units, budget, recent, score, keep, kept_tokens,
                       status);
  return hipGetLastError();
}

}  // namespace omnitide
