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
// the current unit and the wave reduces it when the unit id changes or its slot range ends.  A
// wave's first and last runs are merged over the workgroup's four waves (64 consecutive slots,
// mostly one unit) before they are published with global atomics.  Rows of empty slots (unit
// id -1) are never read.
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
constexpr int kBufFlags = 0x00020000;     // buffer descriptor word 3 for raw 32-bit accesses
constexpr int kOutOfBuf = 0x7ffffff0;     // an offset past every buffer view used here
constexpr int kNontemporal = 2;           // cache policy of a buffer access: nontemporal

// The rows of one unit summed by one wave (or merged over a workgroup's waves).
struct UnitRun {
  uint64_t wsum;
  int unit, cnt, first, last;
  uint32_t sys;
};

// Adds a run into the unit's accumulators (order-independent integer atomics).
__device__ inline void publish_run(const UnitRun& r, uint64_t* wsum, int32_t* len,
                                   int32_t* first, int32_t* last, uint32_t* flags) {
  atomicAdd(reinterpret_cast<unsigned long long*>(wsum + r.unit),
            static_cast<unsigned long long>(r.wsum));
  atomicAdd(len + r.unit, r.cnt);
  atomicMin(first + r.unit, r.first);
  atomicMax(last + r.unit, r.last);
  if (r.sys) atomicOr(flags + r.unit, 1u);
}

// Rows per wave, and rows whose loads a wave issues as one batch before their arithmetic.  With
// the unconditional buffer loads the waits are graded (the compiler moves later rows' loads up
// past earlier rows' arithmetic).  When the grid holds enough waves to keep the memory system
// busy, small batches measured fastest (2 KB rows, 80K-slot pool, 5,120 waves: one row per batch
// 25.0 us per call, two 25.1, four 25.4, eight 26.2); a small pool needs the deep batches for
// enough loads in flight (8K-slot pool, 512 waves: 10.3 us with eight rows, 15.0 us with one).
template <int VPL, bool DEEP>
struct ScoreShape {
  static constexpr int RB = DEEP ? (VPL >= 16 ? 1 : 16 / VPL) : (VPL >= 2 ? 1 : 2);
  static constexpr int RPW = 16;
};
constexpr long kShallowMinWaves = 4096;   // four waves per SIMD of the whole chip

template <bool BF16, int VPL, bool DEEP>
__global__ __launch_bounds__(kScoreWaves * kWave) void score_kernel(
    const u32x4* __restrict__ k, int n_slots, int row_vecs, const int32_t* __restrict__ unit_id,
    const uint8_t* __restrict__ modality, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
    int n_units, uint64_t* __restrict__ wsum, int32_t* __restrict__ len,
    int32_t* __restrict__ first, int32_t* __restrict__ last, uint32_t* __restrict__ flags,
    int32_t* __restrict__ status) {
  constexpr int RB = ScoreShape<VPL, DEEP>::RB;
  constexpr int RPW = ScoreShape<VPL, DEEP>::RPW;
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  // wave-uniform by construction; the compiler is told, so the buffer view below is scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const long s0 = (static_cast<long>(blockIdx.x) * kScoreWaves + wave) * RPW;
  // a wave past the pool has no rows but still takes part in the workgroup merge
  const int nrows = static_cast<int>(max(0L, min(static_cast<long>(RPW), n_slots - s0)));
  __shared__ UnitRun runs[kScoreWaves][2];
  if (lane == 0) {
    runs[wave][0].unit = -1;
    runs[wave][1].unit = -1;
  }

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
  const u32x4* rows = k + (static_cast<size_t>(seg) * n_slots + min(s0, static_cast<long>(n_slots))) *
                              row_vecs;
  const size_t uo = static_cast<size_t>(seg) * n_units;

  uint64_t acc = 0;       // this lane's share of the current unit's weighted sum
  int cur = -1, cnt = 0, f = 0, l = 0, n_runs = 0;
  uint32_t sysf = 0;
  // A finished run of rows of one unit: the wave's first and last runs go to LDS for the
  // workgroup merge (neighbouring waves mostly share them); a run between them belongs to this
  // wave alone and is published at once.
  auto flush = [&](bool last_run) {
    if (cur < 0) return;
    const uint64_t tot = wave_sum_u64(acc);
    if (n_runs == 0 || last_run) {
      if (lane == 0) runs[wave][n_runs == 0 ? 0 : 1] = UnitRun{tot, cur, cnt, f, l, sysf};
    } else if (lane == 0) {
      publish_run(UnitRun{tot, cur, cnt, f, l, sysf}, wsum + uo, len + uo, first + uo, last + uo,
                  flags + uo);
    }
    ++n_runs;
  };

  // A buffer view of the wave's rows: the load of an empty slot's row (or of a vector past the
  // row) gets an offset out of range and returns zeros without a memory access, so every load is
  // issued whatever the tags say.
  const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<u32x4*>(rows), 0, 16 * nrows * row_vecs, kBufFlags);
  for (int r0 = 0; r0 < nrows; r0 += RB) {
    u32x4 buf[RB][VPL];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int row = r0 + r;
      const int u = row < nrows ? readlane(uid, row) : -1;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int idx = lane + kWave * v;
        const int off = (u >= 0 && idx < row_vecs) ? 16 * (row * row_vecs + idx) : kOutOfBuf;
        buf[r][v] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, kNontemporal));
      }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      const int row = r0 + r;
      if (row >= nrows) break;
      const int u = readlane(uid, row);
      if (u < 0) continue;
      if (u != cur) {
        flush(false);
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
  flush(true);

  // Workgroup merge, in slot order: runs of one unit from consecutive waves add up to a single
  // publication.
  __syncthreads();
  if (threadIdx.x == 0) {
    UnitRun m = runs[0][0];
#pragma unroll
    for (int i = 1; i < 2 * kScoreWaves; ++i) {
      const UnitRun r = runs[i / 2][i % 2];
      if (r.unit < 0) continue;
      if (r.unit == m.unit) {
        m.wsum += r.wsum;
        m.cnt += r.cnt;
        m.first = min(m.first, r.first);
        m.last = max(m.last, r.last);
        m.sys |= r.sys;
      } else {
        if (m.unit >= 0) publish_run(m, wsum + uo, len + uo, first + uo, last + uo, flags + uo);
        m = r;
      }
    }
    if (m.unit >= 0) publish_run(m, wsum + uo, len + uo, first + uo, last + uo, flags + uo);
  }
}

template <bool BF16, int VPL>
hipError_t launch_score_t(const void* k, int n_seg, int n_slots, int row_vecs,
                          const int32_t* unit_id, const uint8_t* modality, const uint32_t wq[4],
                          int n_units, uint64_t* wsum, int32_t* len, int32_t* first,
                          int32_t* last, uint32_t* flags, int32_t* status, hipStream_t stream) {
  constexpr int RPW = ScoreShape<VPL, false>::RPW;
  static_assert(ScoreShape<VPL, true>::RPW == RPW, "one grid for both shapes");
  const long waves = (static_cast<long>(n_slots) + RPW - 1) / RPW;
  const dim3 grid(static_cast<unsigned>((waves + kScoreWaves - 1) / kScoreWaves),
                  static_cast<unsigned>(n_seg));
  if (waves * n_seg >= kShallowMinWaves)
    hipLaunchKernelGGL((score_kernel<BF16, VPL, false>), grid, dim3(kScoreWaves * kWave), 0,
                       stream, static_cast<const u32x4*>(k), n_slots, row_vecs, unit_id,
                       modality, wq[0], wq[1], wq[2], wq[3], n_units, wsum, len, first, last,
                       flags, status);
  else
    hipLaunchKernelGGL((score_kernel<BF16, VPL, true>), grid, dim3(kScoreWaves * kWave), 0,
                       stream, static_cast<const u32x4*>(k), n_slots, row_vecs, unit_id,
                       modality, wq[0], wq[1], wq[2], wq[3], n_units, wsum, len, first, last,
                       flags, status);
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
