// Split-KV combine shared by the chunk and decode attention kernels (one instantiation per
// translation unit).  Partials: part_o [n_split][n_rows][D] (unnormalised output against the
// split's reference m) and part_ml [n_split][n_rows] (m, l); rows are (segment, query token,
// query head) with L query tokens per segment.
#pragma once

#include "common.h"

namespace omnitide {
namespace {

// Stores four consecutive output values as float32, or rounded to bf16 (nearest even).
__device__ inline void store_out4(void* out, size_t idx, bool out_bf16, float a, float b, float c,
                                  float d) {
  if (out_bf16) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    const bf16x4 v = {static_cast<__bf16>(a), static_cast<__bf16>(b), static_cast<__bf16>(c),
                      static_cast<__bf16>(d)};
    *reinterpret_cast<bf16x4*>(static_cast<__bf16*>(out) + idx) = v;
  } else {
    *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = make_float4(a, b, c, d);
  }
}

// Merge split partials: out = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s, M = max_s m_s,
// splits in order.
// CH = splits loaded per step (4 for a few splits, 16 or 32 for many); BLOCK = threads per
// workgroup.
template <int D, int CH, int BLOCK = 256>
__global__ __launch_bounds__(BLOCK) void attn_combine_kernel(const float* __restrict__ part_o,
                                                           const float* __restrict__ part_ml,
                                                           int n_split, size_t n_rows,
                                                           const int32_t* __restrict__ n_ctx_g,
                                                           int L, int Hq, int cap,
                                                           void* __restrict__ out,
                                                           bool out_bf16) {
  constexpr int TPR = D / 4;                       // threads per row, 4 floats each
  const size_t row = static_cast<size_t>(blockIdx.x) * (BLOCK / TPR) + threadIdx.x / TPR;
  if (row >= n_rows) return;
  const int seg = static_cast<int>(row / (static_cast<size_t>(L) * Hq));
  // the segment's validity is checked only before the store, so that its load and the
  // partials' loads are in flight together (the partial buffers exist either way)
  const int nctx = n_ctx_g[seg];
  const int d4 = threadIdx.x % TPR;
  // One pass in fixed split order, kChunk splits at a time with all their loads in flight; the
  // running (M, num, den) is rescaled to each chunk's new maximum.
  constexpr int kChunk = CH;
  float M = -INFINITY, den = 0.f;
  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < n_split; s0 += kChunk) {
    float2 ml[kChunk];
    float4 ov[kChunk];
#pragma unroll
    for (int c = 0; c < kChunk; ++c) {
      const size_t pr = static_cast<size_t>(s0 + c) * n_rows + row;
      const bool in = s0 + c < n_split;
      ml[c] = in ? *reinterpret_cast<const float2*>(part_ml + 2 * pr) : make_float2(-INFINITY, 0.f);
      ov[c] = in ? *reinterpret_cast<const float4*>(part_o + pr * D + 4 * d4)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float cm = -INFINITY;
#pragma unroll
    for (int c = 0; c < kChunk; ++c) cm = fmaxf(cm, ml[c].x);
    const float Mn = fmaxf(M, cm);
    if (Mn == -INFINITY) continue;              // nothing visible in any split so far
    const float a = M == -INFINITY ? 0.f : exp2f(M - Mn);
    den *= a;
    num.x *= a;
    num.y *= a;
    num.z *= a;
    num.w *= a;
#pragma unroll
    for (int c = 0; c < kChunk; ++c) {
      const float w = ml[c].x == -INFINITY ? 0.f : exp2f(ml[c].x - Mn);
      den = fmaf(w, ml[c].y, den);
      num.x = fmaf(w, ov[c].x, num.x);
      num.y = fmaf(w, ov[c].y, num.y);
      num.z = fmaf(w, ov[c].z, num.z);
      num.w = fmaf(w, ov[c].w, num.w);
    }
    M = Mn;
  }
  if (nctx < L || nctx > cap) return;
  const float inv = den > 0.f ? 1.f / den : 0.f;
  store_out4(out, row * D + 4 * d4, out_bf16, num.x * inv, num.y * inv, num.z * inv,
             num.w * inv);
}

// Quad reductions (lanes 4i .. 4i+3) by DPP moves; every lane of the quad must be active.
constexpr int kDppQuadSwap1 = 0xb1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadSwap2 = 0x4e;   // quad_perm [2, 3, 0, 1]
template <int CTRL>
__device__ inline float quad_move(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
__device__ inline float quad_max(float v) {
  v = fmaxf(v, quad_move<kDppQuadSwap1>(v));
  return fmaxf(v, quad_move<kDppQuadSwap2>(v));
}
__device__ inline float quad_sum(float v) {
  v += quad_move<kDppQuadSwap1>(v);
  return v + quad_move<kDppQuadSwap2>(v);
}

// Many splits and few rows (decode): the four lanes of a quad share one row's four output values
// and take every fourth split each (all of a lane's loads in flight together); each lane keeps a
// running (M, num, den) as above, and the quad then merges its four by DPP moves: rescaled to
// the quad's maximum and summed (a fixed order, so the result is deterministic).  A row is
// D/4 quads, 2 rows per 256-thread workgroup at D = 128; a wave never straddles two rows.
template <int D>
__global__ __launch_bounds__(256) void attn_combine_quad_kernel(const float* __restrict__ part_o,
                                                              const float* __restrict__ part_ml,
                                                              int n_split, size_t n_rows,
                                                              const int32_t* __restrict__ n_ctx_g,
                                                              int L, int Hq, int cap,
                                                              void* __restrict__ out,
                                                              bool out_bf16) {
  constexpr int kTPS = 4;                          // lanes per (row, four values)
  constexpr int TPR = D / 4 * kTPS;                // threads per row
  static_assert(TPR % kWave == 0 && 256 % TPR == 0, "whole waves per row");
  constexpr int kPer = 8;                          // splits per lane per load batch
  const size_t row = static_cast<size_t>(blockIdx.x) * (256 / TPR) + threadIdx.x / TPR;
  if (row >= n_rows) return;                       // whole waves
  const int seg = static_cast<int>(row / (static_cast<size_t>(L) * Hq));
  const int nctx = n_ctx_g[seg];
  const int within = threadIdx.x % TPR;
  const int d4 = within / kTPS, ts = within % kTPS;
  float M = -INFINITY, den = 0.f;
  float4 num = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = ts; s0 < n_split; s0 += kTPS * kPer) {
    float2 ml[kPer];
    float4 ov[kPer];
#pragma unroll
    for (int c = 0; c < kPer; ++c) {
      const int sp = s0 + kTPS * c;
      const size_t pr = static_cast<size_t>(sp) * n_rows + row;
      const bool in = sp < n_split;
      ml[c] = in ? *reinterpret_cast<const float2*>(part_ml + 2 * pr) : make_float2(-INFINITY, 0.f);
      ov[c] = in ? *reinterpret_cast<const float4*>(part_o + pr * D + 4 * d4)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    float cm = -INFINITY;
#pragma unroll
    for (int c = 0; c < kPer; ++c) cm = fmaxf(cm, ml[c].x);
    const float Mn = fmaxf(M, cm);
    if (Mn == -INFINITY) continue;
    const float a = M == -INFINITY ? 0.f : exp2f(M - Mn);
    den *= a;
    num.x *= a;
    num.y *= a;
    num.z *= a;
    num.w *= a;
#pragma unroll
    for (int c = 0; c < kPer; ++c) {
      const float w = ml[c].x == -INFINITY ? 0.f : exp2f(ml[c].x - Mn);
      den = fmaf(w, ml[c].y, den);
      num.x = fmaf(w, ov[c].x, num.x);
      num.y = fmaf(w, ov[c].y, num.y);
      num.z = fmaf(w, ov[c].z, num.z);
      num.w = fmaf(w, ov[c].w, num.w);
    }
    M = Mn;
  }
  const float Mq = quad_max(M);
  // a lane without a visible key adds nothing (if no lane has one, every output is zero)
  const float a = (M == -INFINITY) ? 0.f : exp2f(M - Mq);
  den = quad_sum(den * a);
  num.x = quad_sum(num.x * a);
  num.y = quad_sum(num.y * a);
  num.z = quad_sum(num.z * a);
  num.w = quad_sum(num.w * a);
  if (ts != 0 || nctx < L || nctx > cap) return;
  const float inv = den > 0.f ? 1.f / den : 0.f;
  store_out4(out, row * D + 4 * d4, out_bf16, num.x * inv, num.y * inv, num.z * inv,
             num.w * inv);
}

// Launch the combine for n_rows rows.
template <int D>
hipError_t launch_combine(const float* part_o, const float* part_ml, int n_split, size_t n_rows,
                          const int32_t* n_ctx, int L, int Hq, int cap, void* out,
                          hipStream_t stream, bool out_bf16 = false) {
  constexpr int rows_per_block = 256 / (D / 4);
  const unsigned blocks = static_cast<unsigned>((n_rows + rows_per_block - 1) / rows_per_block);
  if (n_split <= 4)
    hipLaunchKernelGGL((attn_combine_kernel<D, 4>), dim3(blocks), dim3(256), 0, stream, part_o,
                       part_ml, n_split, n_rows, n_ctx, L, Hq, cap, out, out_bf16);
  else if (n_split <= 16)
    hipLaunchKernelGGL((attn_combine_kernel<D, 16>), dim3(blocks), dim3(256), 0, stream, part_o,
                       part_ml, n_split, n_rows, n_ctx, L, Hq, cap, out, out_bf16);
  else
    // many splits and few rows (decode): four lanes per output quad share the splits
    hipLaunchKernelGGL((attn_combine_quad_kernel<D>),
                       dim3(static_cast<unsigned>((n_rows + 256 / D - 1) / (256 / D))), dim3(256),
                       0, stream, part_o, part_ml, n_split, n_rows, n_ctx, L, Hq, cap, out,
                       out_bf16);
  return hipGetLastError();
}

}  // namespace
}  // namespace omnitide
