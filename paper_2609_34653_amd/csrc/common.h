// Device-side helpers shared by the OmniTide gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "omnitide.h"

namespace omnitide {

constexpr int kWave = 64;

// Native 16-byte vector (usable with the nontemporal load/store builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// s_waitcnt operand for vmcnt(0) alone (gfx9 layout: vmcnt bits 3:0 and 15:14, expcnt 6:4 and
// lgkmcnt 11:8 at their maxima)
constexpr int kVmcntZero = 0x0f70;

// First error wins: only a zero status word is overwritten.
__device__ inline void set_status(int32_t* status, int32_t code) {
  if (status != nullptr) atomicCAS(status, 0, code);
}


// Lane moves by data-parallel primitives (DPP, register to register, no LDS round trip):
// row_shr:n shifts within each 16-lane row, row_bcast:15 / :31 hand lane 15 (31) to the next
// row(s).  Lanes without a source, and rows outside ROW_MASK, receive `fill`.  Every lane of the
// wave must be active.
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;
constexpr int kDppWaveShr1 = 0x138;     // lane i receives lane i - 1 (lane 0: fill)

template <int CTRL, int ROW_MASK>
__device__ inline int dpp_move(int fill, int v) {
  return __builtin_amdgcn_update_dpp(fill, v, CTRL, ROW_MASK, 0xf, false);
}

// Inclusive scans of a 32-bit value over the wave's lanes: within rows by four row shifts,
// then across rows by the two broadcasts.
__device__ inline int wave_scan_add_i32(int x) {
  x += dpp_move<kDppRowShr1, 0xf>(0, x);
  x += dpp_move<kDppRowShr2, 0xf>(0, x);
  x += dpp_move<kDppRowShr4, 0xf>(0, x);
  x += dpp_move<kDppRowShr8, 0xf>(0, x);
  x += dpp_move<kDppRowBcast15, 0xa>(0, x);
  x += dpp_move<kDppRowBcast31, 0xc>(0, x);
  return x;
}
__device__ inline int wave_scan_max_i32(int x, int lo) {
  x = max(x, dpp_move<kDppRowShr1, 0xf>(lo, x));
  x = max(x, dpp_move<kDppRowShr2, 0xf>(lo, x));
  x = max(x, dpp_move<kDppRowShr4, 0xf>(lo, x));
  x = max(x, dpp_move<kDppRowShr8, 0xf>(lo, x));
  x = max(x, dpp_move<kDppRowBcast15, 0xa>(lo, x));
  x = max(x, dpp_move<kDppRowBcast31, 0xc>(lo, x));
  return x;
}

// Maximum over the wave, the same in every lane.
__device__ inline int wave_max_i32(int v) {
  return __builtin_amdgcn_readlane(wave_scan_max_i32(v, INT32_MIN), kWave - 1);
}

// Exclusive running maximum over the wave's lanes (lane 0: lo).
__device__ inline int wave_exclusive_max_i32(int v, int lo) {
  return dpp_move<kDppWaveShr1, 0xf>(lo, wave_scan_max_i32(v, lo));
}

// Sum of a 64-bit value over the wave (modulo 2^64), the same in every lane: the inclusive
// scan of wave_scan_add_i32 with both halves moved by DPP and a 64-bit add per step.
template <int CTRL, int ROW_MASK>
__device__ inline uint64_t dpp_move_u64(uint64_t v) {
  const int lo = dpp_move<CTRL, ROW_MASK>(0, static_cast<int>(static_cast<uint32_t>(v)));
  const int hi = dpp_move<CTRL, ROW_MASK>(0, static_cast<int>(static_cast<uint32_t>(v >> 32)));
  return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}
__device__ inline uint64_t wave_sum_u64(uint64_t v) {
  v += dpp_move_u64<kDppRowShr1, 0xf>(v);
  v += dpp_move_u64<kDppRowShr2, 0xf>(v);
  v += dpp_move_u64<kDppRowShr4, 0xf>(v);
  v += dpp_move_u64<kDppRowShr8, 0xf>(v);
  v += dpp_move_u64<kDppRowBcast15, 0xa>(v);
  v += dpp_move_u64<kDppRowBcast31, 0xc>(v);
  const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v)), 63);
  const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(v >> 32)), 63);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// Sum over the wave, the same in every lane.
__device__ inline uint32_t wave_sum_u32(uint32_t v) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_readlane(wave_scan_add_i32(static_cast<int>(v)), kWave - 1));
}

// Position of set bit number n (0-based) of x; x has more than n set bits.
__device__ inline int nth_set_bit(uint32_t x, int n) {
  int pos = 0;
#pragma unroll
  for (int width = 16; width >= 1; width >>= 1) {
    const int c = __popc((x >> pos) & ((1u << width) - 1u));
    if (n >= c) {
      n -= c;
      pos += width;
    }
  }
  return pos;
}

// Byte arrays walked in 16-byte aligned blocks (absolute addresses): a block that holds a byte
// of the array is read whole, and its bytes outside the caller's range are ignored.  An aligned
// block never crosses a page, so the block of a valid byte is always mapped.
__device__ inline uintptr_t block16_floor(const uint8_t* p) {
  return reinterpret_cast<uintptr_t>(p) & ~static_cast<uintptr_t>(15);
}
__device__ inline void load_block16(uintptr_t addr, uint8_t (&b)[16]) {
  const u32x4 w = *reinterpret_cast<const u32x4*>(addr);
#pragma unroll
  for (int j = 0; j < 16; ++j) b[j] = static_cast<uint8_t>(w[j >> 2] >> (8 * (j & 3)));
}

template <typename T>
__device__ inline T readlane(T v, int lane) {
  return static_cast<T>(__builtin_amdgcn_readlane(static_cast<int>(v), lane));
}

// ---------------------------------------------------------------------------------------------
// Block-wide exclusive scans and reductions for one workgroup of up to 1024 threads.
// `scratch` must hold at least blockDim.x / 64 + 1 elements of T.

template <typename T>
__device__ inline T wave_inclusive_scan(T v) {
  if constexpr (sizeof(T) == 4) {
    // 32-bit integers wrap the same in either signedness
    return static_cast<T>(wave_scan_add_i32(static_cast<int>(v)));
  } else {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      T o = __shfl_up(v, off, kWave);
      if (lane >= off) v += o;
    }
    return v;
  }
}

// Returns the exclusive prefix of v over threads in thread order; *total gets the grand total.
// A one-wave workgroup scans in registers only (no LDS, no barrier).
template <typename T>
__device__ inline T block_exclusive_scan(T v, T* scratch, T* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int n_waves = (blockDim.x + kWave - 1) / kWave;
  T inc = wave_inclusive_scan(v);
  if (n_waves == 1) {
    *total = __shfl(inc, kWave - 1, kWave);
    return inc - v;
  }
  __syncthreads();
  if (lane == kWave - 1) scratch[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    T w = lane < n_waves ? scratch[lane] : T(0);
    T wi = wave_inclusive_scan(w);
    if (lane < n_waves) scratch[lane] = wi - w;
    if (lane == n_waves - 1) scratch[n_waves] = wi;
  }
  __syncthreads();
  T result = scratch[wave] + inc - v;
  *total = scratch[n_waves];
  __syncthreads();
  return result;
}

template <typename T>
__device__ inline T block_sum(T v, T* scratch) {
  T total;
  block_exclusive_scan(v, scratch, &total);
  return total;
}

// Exclusive running maximum over threads in thread order (identity `lo`); *total = overall max.
template <typename T>
__device__ inline T block_exclusive_max(T v, T lo, T* scratch, T* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int n_waves = (blockDim.x + kWave - 1) / kWave;
  T inc = v;
  if constexpr (sizeof(T) == 4) {
    inc = static_cast<T>(wave_scan_max_i32(static_cast<int>(v), static_cast<int>(lo)));
  } else {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      T o = __shfl_up(inc, off, kWave);
      if (lane >= off) inc = max(inc, o);
    }
  }
  T exc = __shfl_up(inc, 1, kWave);
  if (lane == 0) exc = lo;
  if (n_waves == 1) {
    *total = __shfl(inc, kWave - 1, kWave);
    return exc;
  }
  __syncthreads();
  if (lane == kWave - 1) scratch[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    T w = lane < n_waves ? scratch[lane] : lo;
    T wi = w;
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
      T o = __shfl_up(wi, off, kWave);
      if (lane >= off) wi = max(wi, o);
    }
    T we = __shfl_up(wi, 1, kWave);
    if (lane == 0) we = lo;
    if (lane < n_waves) scratch[lane] = we;
    if (lane == n_waves - 1) scratch[n_waves] = wi;
  }
  __syncthreads();
  T result = max(scratch[wave], exc);
  *total = scratch[n_waves];
  __syncthreads();
  return result;
}

}  // namespace omnitide
