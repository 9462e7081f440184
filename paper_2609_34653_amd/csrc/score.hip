// Unit scoring: a bandwidth-bound segmented reduction over the key pool.
//
// Importance statistic (this library's reading; the paper's planner uses metadata only):
//   q(x) = floor(min(|x|, 32) * 2^16), a_s = sum_q over a slot's key row,
//   W_u  = sum over the unit's live slots of w[modality] * a_s (w in 1/256 units).
// Everything is integer, so the per-unit sums do not depend on the order in which waves add
// them, and repeated runs are bitwise identical.
//
// Work split: each wave owns RPW consecutive slots.  Tags are wave-uniform per row, so the
// segmentation by unit is scalar control flow: a lane keeps a 64-bit running sum of its share of
// the current unit and the wave reduces and publishes it (global atomics) only when the unit id
// changes or its slot range ends.  Rows of empty slots (unit id -1) are never read.
#include "common.h"
#include "kernels.h"

namespace omnitide {
namespace {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Sum of q(x) over eight bf16 values held in a 16-byte vector.
//   |x| bits -> packed 16-bit min against 32.0 (NaN/Inf bit patterns are larger, so they clamp)
//   -> +16 on the exponent (x * 2^16, exact; zero and subnormals stay below 1)
//   -> float to unsigned conversion truncates, which is floor for non-negative values.
__device__ inline uint32_t qsum_bf16x8(u32x4 v) {
  const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t a = w[i] & 0x7fff7fffu;
    u16x2 h = __builtin_bit_cast(u16x2, a);
    h = __builtin_elementwise_min(h, (u16x2){0x4200, 0x4200});
    a = __builtin_bit_cast(uint32_t, h) + 0x08000800u;   // no carry: each half <= 0x4A00
    s += static_cast<uint32_t>(__uint_as_float(a << 16));
    s += static_cast<uint32_t>(__uint_as_float(a & 0xffff0000u));
  }
  return s;
}

// Same for four float32 values.
__device__ inline uint32_t qsum_f32x4(u32x4 v) {
  const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
  uint32_t s = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t a = min(w[i] & 0x7fffffffu, 0x42000000u) + 0x08000000u;
    s += static_cast<uint32_t>(__uint_as_float(a));
  }
  return s;
}

__global__ void score_init_kernel(int total, int n_slots, uint64_t* __restrict__ wsum,
                                  int32_t* __restrict__ len, int32_t* __restrict__ first,
                                  int32_t* __restrict__ last, uint32_t* __restrict__ flags) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    wsum[i] = 0;
    len[i] = 0;
    first[i] = n_slots;
    last[i] = -1;
    flags[i] = 0;
  }
}

constexpr int kScoreWaves = 4;

template <int VPL>
struct ScoreShape {
  static constexpr int RB = VPL >= 16 ? 1 : 16 / VPL;   // rows whose loads are in flight together
  static constexpr int RPW = RB >= 16 ? RB : 16;        // rows owned by one wave
};

template <bool BF16, int VPL>
__global__ __launch_bounds__(kScoreWaves * kWave) void score_kernel(
    const u32x4* __restrict__ k, int n_slots, int row_vecs, const int32_t* __restrict__ unit_id,
    const uint8_t* __restrict__ modality, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
    int n_units, uint64_t* __restrict__ wsum, int32_t* __restrict__ len,
    int32_t* __restrict__ first, int32_t* __restrict__ last, uint32_t* __restrict__ flags,
    int32_t* __restrict__ status) {
  constexpr int RB = ScoreShape<VPL>::RB;
  constexpr int RPW = ScoreShape<VPL>::RPW;
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const long s0 = (static_cast<long>(blockIdx.x) * kScoreWaves + wave) * RPW;
  if (s0 >= n_slots) return;
  const int nrows = static_cast<int>(min(static_cast<long>(RPW), n_slots - s0));

  const size_t tag0 = static_cast<size_t>(seg) * n_slots + s0;
  int uid = -1, mod = 0;
  if (lane < nrows) {
    uid = unit_id[tag0 + lane];
    mod = modality[tag0 + lane];
  }
  const bool bad = lane < nrows && (uid < -1 || uid >= n_units || mod > 4);
  if (bad) {
    set_status(status, OMNITIDE_E_TAGS);
    uid = -1;
  }
  const uint32_t w = mod == 0 ? w0 : mod == 1 ? w1 : mod == 2 ? w2 : w3;
  const u32x4* rows = k + (static_cast<size_t>(seg) * n_slots + s0) * row_vecs;
  const size_t uo = static_cast<size_t>(seg) * n_units;

  uint64_t acc = 0;       // this lane's share of the current unit's weighted sum
  int cur = -1, cnt = 0, f = 0, l = 0;
  uint32_t sysf = 0;
  auto flush = [&]() {
    if (cur < 0) return;
    const uint64_t tot = wave_sum_u64(acc);
    if (lane == 0) {
      atomicAdd(reinterpret_cast<unsigned long long*>(wsum + uo + cur),
                static_cast<unsigned long long>(tot));
      atomicAdd(len + uo + cur, cnt);
      atomicMin(first + uo + cur, f);
      atomicMax(last + uo + cur, l);
      if (sysf) atomicOr(flags + uo + cur, 1u);
    }
  };

  for (int r0 = 0; r0 < nrows; r0 += RB) {
    u32x4 buf[RB][VPL];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int row = r0 + r;
      const int u = row < nrows ? readlane(uid, row) : -1;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int idx = lane + kWave * v;
        buf[r][v] = u32x4{0, 0, 0, 0};
        if (u >= 0 && idx < row_vecs)
          buf[r][v] = __builtin_nontemporal_load(rows + static_cast<size_t>(row) * row_vecs + idx);
      }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int row = r0 + r;
      if (row >= nrows) break;
      const int u = readlane(uid, row);
      if (u < 0) continue;
      if (u != cur) {
        flush();
        cur = u;
        acc = 0;
        cnt = 0;
        f = static_cast<int>(s0) + row;
        sysf = 0;
      }
      uint32_t part = 0;
#pragma unroll
      for (int v = 0; v < VPL; ++v) part += BF16 ? qsum_bf16x8(buf[r][v]) : qsum_f32x4(buf[r][v]);
      acc += static_cast<uint64_t>(part) * readlane(w, row);
      ++cnt;
      l = static_cast<int>(s0) + row;
      sysf |= readlane(mod, row) == 0 ? 1u : 0u;
    }
  }
  flush();
}

template <bool BF16, int VPL>
hipError_t launch_score_t(const void* k, int n_seg, int n_slots, int row_vecs,
                          const int32_t* unit_id, const uint8_t* modality, const uint32_t wq[4],
                          int n_units, uint64_t* wsum, int32_t* len, int32_t* first,
                          int32_t* last, uint32_t* flags, int32_t* status, hipStream_t stream) {
  constexpr int RPW = ScoreShape<VPL>::RPW;
  const long waves = (static_cast<long>(n_slots) + RPW - 1) / RPW;
  const dim3 grid(static_cast<unsigned>((waves + kScoreWaves - 1) / kScoreWaves),
                  static_cast<unsigned>(n_seg));
  hipLaunchKernelGGL((score_kernel<BF16, VPL>), grid, dim3(kScoreWaves * kWave), 0, stream,
                     static_cast<const u32x4*>(k), n_slots, row_vecs, unit_id, modality, wq[0],
                     wq[1], wq[2], wq[3], n_units, wsum, len, first, last, flags, status);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score(const void* k, int dtype, int n_seg, int n_slots, int row_elems,
                        const int32_t* unit_id, const uint8_t* modality, const uint32_t wq[4],
                        int n_units, uint64_t* wsum, int32_t* len, int32_t* first, int32_t* last,
                        uint32_t* flags, int32_t* status, hipStream_t stream) {
  const int total = n_seg * n_units;
  const int init_blocks = (total + 255) / 256;
  hipLaunchKernelGGL(score_init_kernel, dim3(init_blocks), dim3(256), 0, stream, total, n_slots,
                     wsum, len, first, last, flags);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_slots == 0) return e;
  const bool bf16 = dtype == OMNITIDE_BF16;
  const int row_vecs = row_elems * (bf16 ? 2 : 4) / 16;
  const int vpl = (row_vecs + kWave - 1) / kWave;
#define OMNITIDE_SCORE_CASE(V)                                                                  \
  if (vpl <= V)                                                                                 \
    return bf16 ? launch_score_t<true, V>(k, n_seg, n_slots, row_vecs, unit_id, modality, wq,  \
                                          n_units, wsum, len, first, last, flags, status,      \
                                          stream)                                               \
                : launch_score_t<false, V>(k, n_seg, n_slots, row_vecs, unit_id, modality, wq, \
                                           n_units, wsum, len, first, last, flags, status,     \
                                           stream);
  OMNITIDE_SCORE_CASE(1)
  OMNITIDE_SCORE_CASE(2)
  OMNITIDE_SCORE_CASE(4)
  OMNITIDE_SCORE_CASE(8)
  OMNITIDE_SCORE_CASE(16)
#undef OMNITIDE_SCORE_CASE
  return hipErrorInvalidValue;
}

}  // namespace omnitide
