// Decode attention over the compacted pool: the last n_q tokens of each segment (typically one
// generated token) attend to the whole context [0, n_ctx) (paper: Background -- decode generates
// one token at a time reusing the cached states; OmniPage ablation -- decode attention time
// over the native, OmniPage and eagerly compacted layouts).
//
// Bandwidth-bound: every (key, KV head) row is read once per call and serves all n_q * G <= 8
// query vectors of its group.  The products still go to the matrix cores: on the vector ALUs the
// per-key dot products, their cross-lane reductions and the P*V updates cost as much time as the
// loads themselves, while a 16x16 MFMA block with the query vectors as columns (half of them
// padding) costs almost nothing.
//   grid      (key split, KV head, segment); the split count is chosen so that about 256
//             eight-wave workgroups run (one per CU), and a combine kernel merges the partials in
//             split order.
//   waves     each wave owns 16 keys of every 128-key workgroup step and loads the next step's
//             keys before it works on the current ones: the K operands straight from global
//             memory into registers, the V rows by direct loads into a private double buffer in
//             LDS.  No workgroup barrier is needed until the waves merge.
//   products  S^T (16 keys x 16 columns) = K Q^T with v_mfma_f32_16x16x32_bf16 (lane l: key
//             l%16, dims 8(l/16).. of each 32-dim slice, a 16-byte load); its output gives lane
//             l column l%16 and keys 4(l/16)..+3, which is the P^T operand of
//             O^T (16 dims x 16 columns) += V^T P^T with v_mfma_f32_16x16x16_bf16.  V^T comes
//             from the LDS block through transposing reads.  Each probability enters twice, as
//             its bf16 rounding and as the bf16 rounding of the remainder, so it carries about
//             16 significant bits into the float accumulation.
//   softmax   float; per column an optimistic reference that moves only when a block's sum
//             would leave [0, 2^32) (as in the chunk attention), shared by the column's four
//             lane groups.
//   merge     the waves' (O, reference, sum) merge through LDS; the result is the split's
//             partial (or, with one split, the normalised output).
#include <algorithm>

#include "common.h"
#include "kernels.h"
#include "combine.h"

namespace omnitide {
namespace {

constexpr int kDecWaves = 8;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kKB = 16;                    // keys per wave per iteration (one 16x16 MFMA block)
constexpr int kKT = 64;                    // slots per tile of a span's tile list
constexpr int kStep = kDecWaves * kKB;     // keys per workgroup iteration
constexpr int kDecTargetWGs = 256;         // one eight-wave workgroup per CU
constexpr int kMaxQG = 8;                  // query vectors per KV head (n_q * G), <= 16

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<size_t>((const lds_void*)p));
}

// 16-byte direct global -> LDS load: lane i reads base + voff_i and writes 16 bytes at LDS byte
// address lds_base + 16 i (uniform base in SGPRs, per-lane 32-bit offset).  Inline assembly, so
// that the compiler's wait insertion does not treat it as a pending LDS write; the issuing wave,
// the only reader of the region it fills, waits for it with s_waitcnt vmcnt.  One wait state is
// required between the M0 write and the load; this file's kernels have no other M0 user.
__device__ inline void dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_base)
               : "memory");
}

// Transposing 64-bit LDS read: within a 16-lane group, lane i receives element i%4 of the
// 8-byte rows read by lanes i/4, 4+i/4, 8+i/4, 12+i/4.
__device__ inline shortx4 ld_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) shortx4*)(p));
}

// 32-byte unit swizzle of a key's row in a wave's V block: the four keys one 16-lane group
// reads (and the eight two groups read) land in distinct banks.
template <int D>
__device__ inline int vsw(int key) { return D == 128 ? (key & 7) : (key & 3); }

// One (query token, query head) vector per column of 16x16 MFMA blocks, keys as rows:
//   S^T (16 keys x 16 columns) = K (16 x d) Q^T with v_mfma_f32_16x16x32_bf16: the K operand
//       is the key's 16-byte piece straight from global memory (lane l: key l%16, dims
//       8(l/16).. of each 32-dim slice); lane l then holds column l%16, keys 4(l/16)..+3, which
//       is exactly the P^T operand layout of the 16x16x16 product.
//   O^T (16 dims x 16 columns) += V^T P^T with v_mfma_f32_16x16x16_bf16, once for the bf16
//       rounding of each probability and once for its remainder, so the probabilities enter
//       with about 16 significant bits; V^T comes from the wave's V block in LDS (direct
//       loads) through transposing reads.
// Each wave owns 16 keys of every 128-key workgroup step, prefetched one step ahead (K
// operands in registers, V in a private double buffer), so no workgroup barrier is needed
// until the waves merge.  Softmax reference per column: optimistic, as in the chunk attention.
// MODE kContig: keys are the contiguous rows [0, n_ctx) of the compacted pool.
// MODE kSpanTiles: keys are the slots [0, span) of a pool with holes (n_ctx_g holds the span);
// a step covers two 64-slot tiles of the span's tile list (four waves each), slot j is visible
// to query token i iff 0 <= key_pos[j] <= q_pos0 + i, and the V rows of empty slots are zeroed
// in the wave's LDS block before use (their bytes may be anything, NaN included).
// MODE kPosOrder: a pool with holes whose entries hold the positions 0 .. n-1 once each (n =
// q_pos0 + n_q; n_ctx_g holds the span): keys are taken in position order, position p from
// the slot list[p] names, so blocks, bounds and masks are those of kContig with n_ctx = n.  A
// wave loads the slot of its next block's key c16 one iteration ahead (a register), and its
// V keys' slots come from the lanes holding them.
template <int D, int MODE>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ n_ctx_g, int cap, int nq,
    int Hq, int Hkv, float scale_log2, float* __restrict__ out, float* __restrict__ part_o,
    float* __restrict__ part_ml, int n_split, int32_t* __restrict__ status,
    const int32_t* __restrict__ key_pos, const int32_t* __restrict__ qpos0_g,
    const int32_t* __restrict__ tile_list, const int32_t* __restrict__ n_active_g,
    int max_tiles) {
  // tile_list, n_active_g -- kSpanTiles: the visited tiles and their number; kPosOrder: the
  // slot of each position and the index's per-workgroup entry counts (max_tiles per segment).
  constexpr bool SPAN = MODE == kSpanTiles;
  constexpr bool POS = MODE == kPosOrder;
  constexpr int KC = D / 32;               // 32-dim slices (QK k-steps)
  constexpr int DB = D / 16;               // 16-dim blocks of the output
  constexpr int CHK = D / 8;               // 16-byte chunks per key row
  constexpr int CALLS = kKB * CHK / kWave; // direct loads per lane per V block
  constexpr int BLK = kKB * D;             // elements of one V block
  constexpr float kSumLimit = 4294967296.f;
  __shared__ __attribute__((aligned(1024))) uint16_t vbuf[kDecWaves][2][BLK];
  __shared__ float sm[kDecWaves][16], sl[kDecWaves][16];

  const int split = blockIdx.x, g = blockIdx.y, seg = blockIdx.z;
  int nctx = n_ctx_g[seg];                          // SPAN, POS: the span
  if (nctx < nq || nctx > cap) {
    if (threadIdx.x == 0) set_status(status, OMNITIDE_E_CAPACITY);
    return;
  }
  if constexpr (POS) {
    // the entries must be exactly the positions 0 .. q_pos0 + n_q - 1 (their number is checked
    // after the loop: every slot taken from the index is clamped, so the loop is safe either way)
    const int qp0 = qpos0_g[seg];
    if (qp0 < 0 || qp0 > nctx - nq) {
      if (threadIdx.x == 0) set_status(status, OMNITIDE_E_TAGS);
      return;
    }
    nctx = qp0 + nq;
  }
  const int G = Hq / Hkv;
  const int nqg = nq * G;
  // contiguous: keys [j0, j1); SPAN: steps [j0, j1) of the tile list (two tiles per step)
  const int n_units_all = SPAN ? (n_active_g[seg] + 1) / 2 : nctx;
  const int j0 = static_cast<int>(static_cast<long>(n_units_all) * split / n_split);
  const int j1 = static_cast<int>(static_cast<long>(n_units_all) * (split + 1) / n_split);
  const int n_act = SPAN ? n_active_g[seg] : 0;
  const size_t tl_base = static_cast<size_t>(seg) * max_tiles;
  const int32_t* kpos = SPAN ? key_pos + static_cast<size_t>(seg) * cap : nullptr;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int c16 = lane & 15, g4 = lane >> 4;

  // Q^T operand: column c16 = query vector (token c16 / G, head g*G + c16 % G); lane l holds
  // dims 32kc + 8 g4 .. +7.  Columns past n_q*G stay zero.
  const bool col_ok = c16 < nqg;
  const int tok = col_ok ? c16 / G : 0;
  // keys (contiguous: rows; SPAN: positions) <= lim are visible
  const int lim = SPAN ? qpos0_g[seg] + tok : (col_ok ? nctx - nq + tok : nctx - 1);
  bf16x8 qf[KC];
  {
    const uint16_t* qrow =
        q + ((static_cast<size_t>(seg) * nq + tok) * Hq + g * G + (col_ok ? c16 % G : 0)) * D;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc) {
      const u32x4 w = col_ok ? *reinterpret_cast<const u32x4*>(qrow + 32 * kc + 8 * g4)
                             : u32x4{0, 0, 0, 0};
      qf[kc] = __builtin_bit_cast(bf16x8, w);
    }
  }
  const size_t row_stride = static_cast<size_t>(Hkv) * D;
  const uint16_t* kh = k + (static_cast<size_t>(seg) * cap * Hkv + g) * D;
  const uint16_t* vh = v + (static_cast<size_t>(seg) * cap * Hkv + g) * D;
  // V block loads: LDS chunk cq*64 + lane of the block holds key (cq*64 + lane) / CHK, stored
  // at unit position ((that chunk) >> 1) ^ vsw(key); the lane fetches the global chunk that
  // belongs there.
  uint32_t voff[CALLS];
  int vkey[CALLS];
#pragma unroll
  for (int cq = 0; cq < CALLS; ++cq) {
    const int lc = cq * kWave + lane;
    const int key = lc / CHK, pc = lc % CHK;
    vkey[cq] = key;
    voff[cq] = 2u * static_cast<uint32_t>(8 * (2 * ((pc >> 1) ^ vsw<D>(key)) + (pc & 1)));
  }
  const uint32_t vlds = lds_addr(&vbuf[wave][0][0]);
  // keys of iteration it for this wave: base(it) + [0, 16).  Contiguous: base(it) = j0 +
  // it*kStep + 16*wave, rows past j1 - 1 clamped to it (read, then masked).  SPAN: base(it) =
  // 64*tile + 16*(wave % 4) with tile the list entry 2*(j0 + it) + wave / 4, rows past the span
  // clamped to its last slot; a wave past the list reads the span's first rows and masks them.
  // Every load is issued unconditionally, so the vmcnt waits below count exactly.
  auto block_base = [&](int it, bool& blk_ok) {
    if constexpr (SPAN) {
      const int a = 2 * (j0 + it) + (wave >> 2);
      blk_ok = a < n_act;
      return blk_ok ? kKT * tile_list[tl_base + a] + kKB * (wave & 3) : 0;
    } else {
      blk_ok = true;
      return j0 + it * kStep + kKB * wave;
    }
  };
  const int row_end = SPAN ? nctx : j1;      // rows >= row_end are clamped
  const int n_it = SPAN ? j1 - j0 : (j1 - j0 + kStep - 1) / kStep;
  // POS: slot of this lane's key c16 in the next block to issue (positions past row_end - 1
  // clamped), loaded one iteration ahead
  const int32_t* slot_of = POS ? tile_list + static_cast<size_t>(seg) * cap : nullptr;
  auto load_slot = [&](int it) {
    bool blk_ok;
    return slot_of[min(block_base(it, blk_ok) + c16, row_end - 1)];
  };
  int slot_next = 0;
  auto issue = [&](int it, int buf, bf16x8 (&ka)[KC], int (&kp)[5]) {
    bool blk_ok;
    const int kb0 = block_base(it, blk_ok);
    uint32_t kslot = 0;
    if constexpr (POS) kslot = min(static_cast<uint32_t>(slot_next), static_cast<uint32_t>(cap - 1));
    const int kr = POS ? static_cast<int>(kslot) : min(kb0 + c16, row_end - 1);
    const uint16_t* kp_ = kh + static_cast<size_t>(kr) * row_stride + 8 * g4;
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
      ka[kc] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(kp_ + 32 * kc));
    if constexpr (SPAN) {
      // positions of keys 4 g4 .. +3 (for the mask) and of key c16 (for the V zeroing)
#pragma unroll
      for (int i = 0; i < 4; ++i) kp[i] = kpos[min(kb0 + 4 * g4 + i, row_end - 1)];
      kp[4] = kpos[kr];
    }
    if constexpr (POS) {
      // V rows of keys vkey[cq] (< 16): their slots are held by lanes vkey[cq]; the host keeps
      // cap * Hkv * D * 2 below 2^32
#pragma unroll
      for (int cq = 0; cq < CALLS; ++cq) {
        const uint32_t vs = static_cast<uint32_t>(__shfl(static_cast<int>(kslot), vkey[cq], kWave));
        dma16(vh, voff[cq] + 2u * vs * static_cast<uint32_t>(row_stride),
              vlds + static_cast<uint32_t>((buf * BLK + cq * kWave * 8) * 2));
      }
      // the block after this one (the last iteration re-reads its own block's slot)
      slot_next = load_slot(min(it + 1, n_it - 1));
      return;
    }
    const int r0 = min(kb0, row_end - 1);
#pragma unroll
    for (int cq = 0; cq < CALLS; ++cq) {
      const int shift = min(kb0 + vkey[cq], row_end - 1) - r0;   // >= 0
      dma16(vh + static_cast<size_t>(r0) * row_stride,
            voff[cq] + 2u * static_cast<uint32_t>(shift * row_stride),
            vlds + static_cast<uint32_t>((buf * BLK + cq * kWave * 8) * 2));
    }
  };

  floatx4 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  bf16x8 kA[KC], kB[KC];
  int pA[5] = {-1, -1, -1, -1, -1}, pB[5] = {-1, -1, -1, -1, -1};
  // V^T operand read: lane (g4, i) takes dims 16db + i of keys 4g4 .. 4g4+3; the lanes of its
  // group read key 4g4 + (i >> 2), dims 16db + 4(i & 3) .. +3.
  const int vrow = 4 * g4 + (c16 >> 2);
  const int vsub = 4 * (c16 & 3);

  auto step = [&](auto bpar, int it) {
    constexpr int B = decltype(bpar)::value;
    bf16x8(&ka)[KC] = B == 0 ? kA : kB;
    bf16x8(&kn)[KC] = B == 0 ? kB : kA;
    const int(&pc)[5] = B == 0 ? pA : pB;
    int(&pn)[5] = B == 0 ? pB : pA;
    const bool more = it + 1 < n_it;
    floatx4 s = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < KC; ++kc)
      s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[kc], qf[kc], s, 0, 0, 0);
    const int(&kpc)[5] = pc;   // positions of this iteration's keys (SPAN)
    // the next iteration's loads go out once this one's K operands are consumed
    if (more) issue(it + 1, 1 - B, kn, pn);
    bool blk_ok;
    const int kb0 = block_base(it, blk_ok);
    const int key0 = kb0 + 4 * g4;
    if constexpr (SPAN) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (!blk_ok || key0 + i >= nctx || kpc[i] < 0 || kpc[i] > lim) s[i] = -INFINITY;
    } else if (kb0 + kKB > j1 || kb0 + kKB - 1 > nctx - nq) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (key0 + i >= j1 || key0 + i > lim) s[i] = -INFINITY;
    }
    float e[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(fmaf(s[i], scale_log2, -m_run));
    float ls = (e[0] + e[1]) + (e[2] + e[3]);
    if (__any(!(ls < kSumLimit))) {
      // exact block maximum per column (its four lane groups), move the reference, rescale
      float mx = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[2], s[3]));
      mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
      mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
      const float m_new = fmaxf(m_run, mx * scale_log2);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db] *= alpha;
      m_run = m_new;
#pragma unroll
      for (int i = 0; i < 4; ++i) e[i] = __builtin_amdgcn_exp2f(fmaf(s[i], scale_log2, -m_use));
    }
    // probabilities as bf16 plus bf16 remainder
    shortx4 ph, pl;
    float lsum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const __bf16 hi = static_cast<__bf16>(e[i]);
      const __bf16 lo = static_cast<__bf16>(e[i] - static_cast<float>(hi));
      ph[i] = __builtin_bit_cast(short, hi);
      pl[i] = __builtin_bit_cast(short, lo);
      lsum += static_cast<float>(hi) + static_cast<float>(lo);
    }
    l_run += lsum;
    // this iteration's V block has landed (the next one's loads may still be in flight: KC K
    // loads, in SPAN mode 5 position loads, CALLS direct loads)
    // (POS: the next block's slot load before them and the one after next's after them)
    constexpr int NEXT = CALLS + KC + (SPAN ? 5 : 0) + (POS ? 2 : 0);
    static_assert(NEXT == 8 || NEXT == 4 || NEXT == 13 || NEXT == 9 || NEXT == 10 || NEXT == 6,
                  "vmcnt immediates below");
    if (more) {
      if constexpr (NEXT == 13) asm volatile("s_waitcnt vmcnt(13)" ::: "memory");
      else if constexpr (NEXT == 10) asm volatile("s_waitcnt vmcnt(10)" ::: "memory");
      else if constexpr (NEXT == 9) asm volatile("s_waitcnt vmcnt(9)" ::: "memory");
      else if constexpr (NEXT == 6) asm volatile("s_waitcnt vmcnt(6)" ::: "memory");
      else if constexpr (NEXT == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
      else asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }
    if constexpr (SPAN) {
      // V rows of empty slots (and of a wave past the list) are zeroed by the four lanes of
      // their key, a quarter of the row each; the wave's own LDS reads below follow in order
      if (!blk_ok || kpc[4] < 0) {
        u32x4* row = reinterpret_cast<u32x4*>(&vbuf[wave][B][0] + c16 * D);
#pragma unroll
        for (int x = 0; x < CHK / 4; ++x) row[(CHK / 4) * g4 + x] = u32x4{0, 0, 0, 0};
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    const uint16_t* vb = &vbuf[wave][B][0] + vrow * D + vsub;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const shortx4 vt = ld_tr(vb + 16 * (db ^ vsw<D>(vrow)));
      o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, ph, o[db], 0, 0, 0);
      o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vt, pl, o[db], 0, 0, 0);
    }
  };
  if constexpr (POS) {
    if (n_it > 0) slot_next = load_slot(0);
  }
  if (n_it > 0) issue(0, 0, kA, pA);
  int it = 0;
  for (; it + 1 < n_it; it += 2) {
    step(std::integral_constant<int, 0>{}, it);
    step(std::integral_constant<int, 1>{}, it + 1);
  }
  if (it < n_it) step(std::integral_constant<int, 0>{}, it);

  if constexpr (POS) {
    // one wave per segment: the index's workgroup counts must add up to n_ctx entries
    if (split == 0 && g == 0 && wave == 0) {
      int c = 0;
      for (int b = lane; b < max_tiles; b += kWave)
        c += n_active_g[static_cast<size_t>(seg) * max_tiles + b];
      // the whole wave sums (a cross-lane scan), then one lane reports
      const int total = static_cast<int>(wave_sum_u32(static_cast<uint32_t>(c)));
      if (lane == 0 && total != nctx) set_status(status, OMNITIDE_E_TAGS);
    }
  }
  // merge the waves: per column the reference, the sum over the four lane groups, and O^T
  const float l_col = l_run + __shfl_xor(l_run, 16, kWave) + __shfl_xor(l_run, 32, kWave) +
                      __shfl_xor(l_run, 48, kWave);
  __syncthreads();                         // every wave is done with its V blocks
  // [wave][D][SCOL]: the LDS serves 32 lanes a cycle from 32 four-byte banks.  A store covers
  // 8 columns x lane groups (0, 1) in one half-wave and (2, 3) in the other, i.e. banks
  // c + 4 g SCOL; a load covers 32 consecutive dims of one column, banks d SCOL.  SCOL = 11
  // (odd, 4 SCOL = 12 mod 32) keeps both within distinct banks.
  constexpr int SCOL = kMaxQG + 3;
  float* so = reinterpret_cast<float*>(&vbuf[0][0][0]);
  static_assert(sizeof(vbuf) >= kDecWaves * D * SCOL * sizeof(float), "merge buffer");
  if (g4 == 0) {
    sm[wave][c16] = m_run;
    sl[wave][c16] = l_col;
  }
  if (c16 < kMaxQG) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) so[(wave * D + 16 * db + 4 * g4 + i) * SCOL + c16] = o[db][i];
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
        num = fmaf(w, so[(gr * D + d) * SCOL + qi], num);
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

template <int D>
hipError_t launch_decode_t(const DecodeArgs& a, int n_split, hipStream_t stream) {
  const dim3 grid(n_split, a.n_kv_heads, a.n_seg);
  const size_t n_rows = static_cast<size_t>(a.n_seg) * a.n_q * a.n_q_heads;
  float* part_o = n_split > 1 ? static_cast<float*>(a.workspace) : nullptr;
  float* part_ml = part_o ? part_o + static_cast<size_t>(n_split) * n_rows * D : nullptr;
  const float scale_log2 = a.scale * 1.4426950408889634f;
  if (a.key_pos != nullptr && a.pos_order) {
    // position order: the position index after the partials
    int32_t* slot_of = reinterpret_cast<int32_t*>(
        static_cast<uint8_t*>(a.workspace) +
        align256(n_split > 1 ? static_cast<size_t>(n_split) * n_rows * (D + 2) * 4 : 0));
    hipError_t e = launch_pos_index(a.key_pos, a.n_ctx, a.q_pos0, a.n_seg, a.cap, a.n_q,
                                    slot_of, stream, a.d_status);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((decode_kernel<D, kPosOrder>), grid, dim3(kDecThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.n_q, a.n_q_heads,
                       a.n_kv_heads, scale_log2, a.out, part_o, part_ml, n_split, a.d_status,
                       a.key_pos, a.q_pos0, slot_of,
                       slot_of + static_cast<size_t>(a.n_seg) * a.cap, pos_index_blocks(a.cap));
  } else if (a.key_pos != nullptr) {
    // span mode: the tile tables after the partials
    uint8_t* tbl = static_cast<uint8_t*>(a.workspace) +
                   align256(n_split > 1 ? static_cast<size_t>(n_split) * n_rows * (D + 2) * 4 : 0);
    hipError_t e = launch_span_tiles(a.key_pos, a.n_ctx, a.n_seg, a.cap, a.n_q, a.skip_empty,
                                     tbl, stream);
    if (e != hipSuccess) return e;
    const SpanTiles T = span_tiles_at(tbl, a.n_seg, a.cap);
    hipLaunchKernelGGL((decode_kernel<D, kSpanTiles>), grid, dim3(kDecThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.n_q, a.n_q_heads,
                       a.n_kv_heads, scale_log2, a.out, part_o, part_ml, n_split, a.d_status,
                       a.key_pos, a.q_pos0, T.list, T.n_active, (a.cap + kKT - 1) / kKT);
  } else {
    hipLaunchKernelGGL((decode_kernel<D, kContig>), grid, dim3(kDecThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.n_q, a.n_q_heads,
                       a.n_kv_heads, scale_log2, a.out, part_o, part_ml, n_split, a.d_status,
                       nullptr, nullptr, nullptr, nullptr, 0);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_split == 1) return e;
  return launch_combine<D>(part_o, part_ml, n_split, n_rows, a.n_ctx, a.n_q, a.n_q_heads, a.cap,
                           a.out, stream);
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

size_t decode_span_workspace_bytes(int n_seg, int cap, int n_q, int n_q_heads, int n_kv_heads,
                                   int head_dim) {
  // the tile tables (tile traversals) or the position index (position order)
  return align256(decode_workspace_bytes(n_seg, cap, n_q, n_q_heads, n_kv_heads, head_dim)) +
         std::max(span_tiles_bytes(n_seg, cap), pos_index_bytes(n_seg, cap));
}

int decode_max_query_vectors() { return kMaxQG; }

hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream) {
  const int s = decode_num_splits(a.n_seg, a.cap, a.n_kv_heads);
  if (a.head_dim == 128) return launch_decode_t<128>(a, s, stream);
  if (a.head_dim == 64) return launch_decode_t<64>(a, s, stream);
  return hipErrorInvalidValue;
}

}  // namespace omnitide
