// Device-side helpers shared by the OmniTide gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "omnitide.h"

namespace omnitide {

constexpr int kWave = 64;

// Native 16-byte vector (usable with the nontemporal load/store builtins).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// First error wins: only a zero status word is overwritten.
__device__ inline void set_status(int32_t* status, int32_t code) {
  if (status != nullptr) atomicCAS(status, 0, code);
}

__device__ inline uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ inline uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
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
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T o = __shfl_up(v, off, kWave);
    if (lane >= off) v += o;
  }
  return v;
}

// Returns the exclusive prefix of v over threads in thread order; *total gets the grand total.
template <typename T>
__device__ inline T block_exclusive_scan(T v, T* scratch, T* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int n_waves = (blockDim.x + kWave - 1) / kWave;
  T inc = wave_inclusive_scan(v);
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
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T o = __shfl_up(inc, off, kWave);
    if (lane >= off) inc = max(inc, o);
  }
  T exc = __shfl_up(inc, 1, kWave);
  if (lane == 0) exc = lo;
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
