// Measurement probe (not part of the method): the sustained rate of the bf16 matrix cores and the
// shader clock while they run, so that measured ceilings can be shown beside the published peak.
// Built into libomnitide_probe.so, used only by the benchmark.
//
// Every wave keeps four independent v_mfma_f32_32x32x16_bf16 accumulation chains in flight for
// `iters` iterations (operands stay in registers, no memory traffic).  Wave 0 of workgroup 0
// records the shader-clock counter and the 100 MHz wall-clock counter around its loop.
//
// The matrix cores' sustained rate depends on the operand bits (switching activity sets the
// power draw, and the clock drops to stay within the power limit): the first probe's operands
// are smooth per-lane constants, the second takes every lane's operands from a caller's table
// (for instance N(0,1) values rounded to bf16, the statistics of attention inputs).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void mfma_probe_kernel(int iters, float* __restrict__ sink,
                                                         uint64_t* __restrict__ clocks) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = static_cast<__bf16>(1.0f / (1 + lane + i));
    b[i] = static_cast<__bf16>(1.0f / (2 + lane + i));
  }
  floatx16 acc[4] = {floatx16{}, floatx16{}, floatx16{}, floatx16{}};
  const bool timer = blockIdx.x == 0 && threadIdx.x == 0;
  uint64_t c0 = 0, w0 = 0;
  if (timer) {
    c0 = clock64();
    w0 = wall_clock64();
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  }
  if (timer) {
    clocks[0] = clock64() - c0;
    clocks[1] = wall_clock64() - w0;
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[j][i];
  if (s == 12345.f) sink[blockIdx.x * blockDim.x + threadIdx.x] = s;   // keeps the loop alive
}

// Operands from a table: lane l of workgroup w loads entries ((w % 64) * 8 + i) * 64 + l,
// i = 0..7, of 16 bytes each, and every iteration issues eight MFMAs (two per chain) that pair
// those registers in rotation.
__global__ __launch_bounds__(256) void mfma_probe_ops_kernel(int iters,
                                                             const uint4* __restrict__ ops,
                                                             float* __restrict__ sink,
                                                             uint64_t* __restrict__ clocks) {
  const int lane = threadIdx.x & 63;
  bf16x8 a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    a[i] = __builtin_bit_cast(bf16x8, ops[((blockIdx.x % 64) * 8 + i) * 64 + lane]);
  floatx16 acc[4] = {floatx16{}, floatx16{}, floatx16{}, floatx16{}};
  const bool timer = blockIdx.x == 0 && threadIdx.x == 0;
  uint64_t c0 = 0, w0 = 0;
  if (timer) {
    c0 = clock64();
    w0 = wall_clock64();
  }
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[4 * r + j], a[(4 * r + j + 1) & 7],
                                                         acc[j], 0, 0, 0);
    }
  }
  if (timer) {
    clocks[0] = clock64() - c0;
    clocks[1] = wall_clock64() - w0;
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) s += acc[j][i];
  if (s == 12345.f) sink[blockIdx.x * blockDim.x + threadIdx.x] = s;   // keeps the loop alive
}

}  // namespace

extern "C" {

// Launches the probe on `stream`: n_wg workgroups of 4 waves, `iters` iterations of 4 MFMAs per
// wave (32,768 flops each).  clocks (device, 2 x uint64): shader-clock cycles and 100 MHz ticks
// of wave 0's loop.  sink (device): n_wg * 256 floats, never read.  Returns 0 or -8.
int omnitide_probe_mfma(int n_wg, int iters, float* sink, uint64_t* clocks, void* stream) {
  if (n_wg < 1 || iters < 1 || sink == nullptr || clocks == nullptr) return -2;
  hipLaunchKernelGGL(mfma_probe_kernel, dim3(n_wg), dim3(256), 0,
                     static_cast<hipStream_t>(stream), iters, sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : -8;
}

// The same with operands from `ops` (device, 64 x 8 x 64 entries of 16 bytes = 512 KiB): n_wg
// workgroups of 4 waves, `iters` iterations of 8 MFMAs per wave.  Returns 0, -2 or -8.
int omnitide_probe_mfma_ops(int n_wg, int iters, const void* ops, float* sink, uint64_t* clocks,
                            void* stream) {
  if (n_wg < 1 || iters < 1 || ops == nullptr || sink == nullptr || clocks == nullptr) return -2;
  hipLaunchKernelGGL(mfma_probe_ops_kernel, dim3(n_wg), dim3(256), 0,
                     static_cast<hipStream_t>(stream), iters, static_cast<const uint4*>(ops),
                     sink, clocks);
  return hipGetLastError() == hipSuccess ? 0 : -8;
}

}  // extern "C"
