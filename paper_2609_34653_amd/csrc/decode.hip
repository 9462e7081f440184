// Decode attention over the compacted pool: the last n_q tokens of each segment (typically one
// generated token) attend to the whole context [0, n_ctx) (paper: Background -- decode generates
// one token at a time reusing the cached states; OmniPage ablation -- decode attention time
// over the native, OmniPage and eagerly compacted layouts).
//
// Bandwidth-bound: every (key, KV head) row is read once per call and serves all n_q * G query
// vectors of its group, so there is no matrix work worth the matrix cores.
//   grid      (key split, KV head, segment); the split count is chosen so that about 256
//             eight-wave workgroups run (one per CU), and a combine kernel merges the partials in
//             split order.
//   lanes     a group of D/8 lanes covers one key's D dimensions (16 bytes per lane, a fully
//             coalesced 2*D-byte read of the key's head slice); a wave covers 64/(D/8) keys per
//             load, kUnroll loads per iteration, and loads the next iteration's rows before
//             it processes the current ones.
//   scores    each lane holds 8 dimensions of every query vector in float; a dot product is a
//             reduction over the lane group.
//   softmax   float throughout (the probabilities are not rounded): running maximum per query
//             vector and lane group, rescaled once per kUnroll keys.
//   merge     the lane groups of a wave merge by lane exchanges, then the waves through LDS;
//             the result is the split's partial (or, with one split, the normalised output).
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "combine.h"

namespace omnitide {
namespace {

constexpr int kDecWaves = 8;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kUnroll = 4;                 // keys per lane group per iteration
constexpr int kDecTargetWGs = 256;       // one 8-wave workgroup per CU
constexpr int kMaxQG = 8;                  // query vectors per KV head (n_q * G)

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Sum over each aligned group of N lanes (N = 8 or 16), result in every lane of the group, with
// DPP lane permutations (no LDS): swap neighbours, swap pairs, mirror within 8 lanes (quad 0 <->
// quad 1), mirror within 16 lanes (8-lane halves).
template <int DPP>
__device__ inline float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), DPP, 0xf, 0xf, false));
}
template <int N>
__device__ inline float group_sum(float x) {
  static_assert(N == 8 || N == 16, "group of 8 or 16 lanes");
  x += dpp_f<0xB1>(x);    // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);    // quad_perm [2,3,0,1]
  x += dpp_f<0x141>(x);   // row_half_mirror
  if constexpr (N == 16) x += dpp_f<0x140>(x);   // row_mirror
  return x;
}

template <int D, int QG>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ n_ctx_g, int cap, int nq,
    int Hq, int Hkv, float scale_log2, float* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_ml, int n_split, int32_t* __restrict__ status) {
  constexpr int LPK = D / 8;               // lanes per key
  constexpr int KPW = kWave / LPK;         // keys per wave load
  constexpr int GROUPS = kDecWaves * KPW;  // lane groups per workgroup
  constexpr int STEP = GROUPS * kUnroll;   // keys per workgroup iteration
  const int split = blockIdx.x, g = blockIdx.y, seg = blockIdx.z;
  const int nctx = n_ctx_g[seg];
  if (nctx < nq || nctx > cap) {
    if (threadIdx.x == 0) set_status(status, OMNITIDE_E_CAPACITY);
    return;
  }
  const int G = Hq / Hkv;
  const int nqg = nq * G;
  const int j0 = static_cast<int>(static_cast<long>(nctx) * split / n_split);
  const int j1 = static_cast<int>(static_cast<long>(nctx) * (split + 1) / n_split);
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int cl = lane % LPK;               // dims 8cl .. 8cl+7
  const int grp = wave * KPW + lane / LPK; // lane group: one key per load

  // Query vector qi = (token i = qi / G, head g*G + qi % G); unused slots stay zero.
  float qv[QG][8];
  int lim[QG];
#pragma unroll
  for (int qi = 0; qi < QG; ++qi) {
    const bool ok = qi < nqg;
    const int i = ok ? qi / G : 0;
    const int h = g * G + (ok ? qi % G : 0);
    lim[qi] = ok ? nctx - nq + i : -1;     // keys <= lim are visible
    const u32x4 w = ok ? *reinterpret_cast<const u32x4*>(
                             q + ((static_cast<size_t>(seg) * nq + i) * Hq + h) * D + 8 * cl)
                       : u32x4{0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      qv[qi][2 * e] = bf16_lo(w[e]);
      qv[qi][2 * e + 1] = bf16_hi(w[e]);
    }
  }
  float m[QG], l[QG], o[QG][8];
#pragma unroll
  for (int qi = 0; qi < QG; ++qi) {
    m[qi] = -INFINITY;
    l[qi] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[qi][e] = 0.f;
  }
  const size_t row_stride = static_cast<size_t>(Hkv) * D;
  const uint16_t* kh = k + (static_cast<size_t>(seg) * cap * Hkv + g) * D + 8 * cl;
  const uint16_t* vh = v + (static_cast<size_t>(seg) * cap * Hkv + g) * D + 8 * cl;

  // Keys of iteration `base` for this lane group: base + u*GROUPS + grp; rows past j1 load row j0
  // (in range, ignored).  The next iteration's rows are loaded before this one is processed.
  constexpr bool kPrefetch = QG <= 4;     // keeps QG = 8 within 256 registers
  u32x4 kw[kUnroll], vw[kUnroll], kn[kUnroll], vn[kUnroll];
  auto load = [&](int base, u32x4 (&kd)[kUnroll], u32x4 (&vd)[kUnroll]) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int key = base + u * GROUPS + grp;
      const size_t r = static_cast<size_t>(key < j1 ? key : j0) * row_stride;
      kd[u] = *reinterpret_cast<const u32x4*>(kh + r);
      vd[u] = *reinterpret_cast<const u32x4*>(vh + r);
    }
  };
  if (j0 < j1) load(j0, kw, vw);
  for (int base = j0; base < j1; base += STEP) {
    if (kPrefetch && base + STEP < j1) load(base + STEP, kn, vn);
    int key[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) key[u] = base + u * GROUPS + grp;
#pragma unroll
    for (int qi = 0; qi < QG; ++qi) {
      float s[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc = fmaf(qv[qi][2 * e], bf16_lo(kw[u][e]), acc);
          acc = fmaf(qv[qi][2 * e + 1], bf16_hi(kw[u][e]), acc);
        }
        acc = group_sum<LPK>(acc);
        s[u] = (key[u] < j1 && key[u] <= lim[qi]) ? acc * scale_log2 : -INFINITY;
      }
      float mx = s[0];
#pragma unroll
      for (int u = 1; u < kUnroll; ++u) mx = fmaxf(mx, s[u]);
      const float m_new = fmaxf(m[qi], mx);
      if (m_new == -INFINITY) continue;    // nothing visible yet for this query vector
      const float alpha = __builtin_amdgcn_exp2f(m[qi] - m_new);
      m[qi] = m_new;
      float lsum = l[qi] * alpha;
      float acc8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc8[e] = o[qi][e] * alpha;
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const float p = __builtin_amdgcn_exp2f(s[u] - m_new);
        lsum += p;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc8[2 * e] = fmaf(p, bf16_lo(vw[u][e]), acc8[2 * e]);
          acc8[2 * e + 1] = fmaf(p, bf16_hi(vw[u][e]), acc8[2 * e + 1]);
        }
      }
      l[qi] = lsum;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[qi][e] = acc8[e];
    }
    if (kPrefetch) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        kw[u] = kn[u];
        vw[u] = vn[u];
      }
    } else if (base + STEP < j1) {
      load(base + STEP, kw, vw);
    }
  }

  // Merge the KPW lane groups of each wave (lanes LPK, 2 LPK, ... apart), then the waves.
#pragma unroll
  for (int qi = 0; qi < QG; ++qi) {
#pragma unroll
    for (int off = LPK; off < kWave; off <<= 1) {
      const float mo = __shfl_xor(m[qi], off, kWave);
      const float lo = __shfl_xor(l[qi], off, kWave);
      const float mn = fmaxf(m[qi], mo);
      const float a = m[qi] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[qi] - mn);
      const float b = mo == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mo - mn);
      l[qi] = a * l[qi] + b * lo;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[qi][e] = a * o[qi][e] + b * __shfl_xor(o[qi][e], off, kWave);
      m[qi] = mn;
    }
  }
  __shared__ float sm[kDecWaves][QG], sl[kDecWaves][QG];
  __shared__ float so[kDecWaves][QG][D];
  if (lane < LPK) {
#pragma unroll
    for (int qi = 0; qi < QG; ++qi) {
      if (lane == 0) {
        sm[wave][qi] = m[qi];
        sl[wave][qi] = l[qi];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) so[wave][qi][8 * cl + e] = o[qi][e];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < nqg * D; idx += kDecThreads) {
    const int qi = idx / D, d = idx % D;
    float M = -INFINITY;
    for (int gr = 0; gr < kDecWaves; ++gr) M = fmaxf(M, sm[gr][qi]);
    float num = 0.f, den = 0.f;
    if (M != -INFINITY) {
      for (int gr = 0; gr < kDecWaves; ++gr) {
        const float w = sm[gr][qi] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(sm[gr][qi] - M);
        num = fmaf(w, so[gr][qi][d], num);
        den = fmaf(w, sl[gr][qi], den);
      }
    }
    const int i = qi / G, h = g * G + qi % G;
    const size_t orow = (static_cast<size_t>(seg) * nq + i) * Hq + h;
    if (n_split == 1) {
      out[orow * D + d] = den > 0.f ? num / den : 0.f;
    } else {
      const size_t n_rows = static_cast<size_t>(gridDim.z) * nq * Hq;
      const size_t prow = static_cast<size_t>(split) * n_rows + orow;
      part_o[prow * D + d] = num;
      if (d == 0) *reinterpret_cast<float2*>(part_ml + 2 * prow) = make_float2(M, den);
    }
  }
}

template <int D, int QG>
hipError_t launch_decode_t(const DecodeArgs& a, int n_split, hipStream_t stream) {
  const dim3 grid(n_split, a.n_kv_heads, a.n_seg);
  const size_t n_rows = static_cast<size_t>(a.n_seg) * a.n_q * a.n_q_heads;
  float* part_o = static_cast<float*>(a.workspace);
  float* part_ml = part_o ? part_o + static_cast<size_t>(n_split) * n_rows * D : nullptr;
  const float scale_log2 = a.scale * 1.4426950408889634f;
  hipLaunchKernelGGL((decode_kernel<D, QG>), grid, dim3(kDecThreads), 0, stream,
                     static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                     static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.n_q, a.n_q_heads,
                     a.n_kv_heads, scale_log2, a.out, part_o, part_ml, n_split, a.d_status);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_split == 1) return e;
  return launch_combine<D>(part_o, part_ml, n_split, n_rows, a.n_ctx, a.n_q, a.n_q_heads, a.cap,
                           a.out, stream);
}

template <int D>
hipError_t launch_decode_d(const DecodeArgs& a, int n_split, hipStream_t stream) {
  const int qg = a.n_q * (a.n_q_heads / a.n_kv_heads);
  if (qg <= 1) return launch_decode_t<D, 1>(a, n_split, stream);
  if (qg <= 2) return launch_decode_t<D, 2>(a, n_split, stream);
  if (qg <= 4) return launch_decode_t<D, 4>(a, n_split, stream);
  return launch_decode_t<D, kMaxQG>(a, n_split, stream);
}

}  // namespace

int decode_num_splits(int n_seg, int cap, int n_kv_heads) {
  const long base = static_cast<long>(n_kv_heads) * n_seg;
  long s = kDecTargetWGs / base;
  s = std::min(s, static_cast<long>((cap + 63) / 64));
  return static_cast<int>(std::max(1L, std::min(s, 128L)));
}

size_t decode_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                              int head_dim) {
  const int s = decode_num_splits(n_seg, cap, n_kv_heads);
  if (s == 1) return 0;
  const size_t rows = static_cast<size_t>(n_seg) * n_q * n_q_heads;
  return static_cast<size_t>(s) * rows * (static_cast<size_t>(head_dim) + 2) * sizeof(float);
}

int decode_max_query_vectors() { return kMaxQG; }

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int s = decode_num_splits(a.n_seg, a.cap, a.n_kv_heads);
  if (a.head_dim == 128) return launch_decode_d<128>(a, s, stream);
  if (a.head_dim == 64) return launch_decode_d<64>(a, s, stream);
  return hipErrorInvalidValue;
}

}  // namespace omnitide
