// Chunk prefill attention over [compacted history || chunk]: flash-style, bf16 MFMA on gfx950.
//
// Decomposition
//   rows     for KV head g the L*G query rows (position p, head g*G + r) are flattened as
//            m = p*G + r and tiled 128 per workgroup (4 waves x 32): GQA packing, so one K/V
//            tile staged in LDS serves G query heads.
//   keys     64-key tiles; a workgroup's key range ends at its last row's causal limit; with
//            n_split > 1 the tile range is cut into equal parts and a combine kernel merges the
//            partial (O, max, sum) in fixed split order.
//   products S^T = K Q^T and O^T = V^T P^T with v_mfma_f32_32x32x16_bf16.  Computing the
//            transposed scores puts one query column in each lane, so the softmax row statistics
//            are lane-local (plus one exchange between the two 32-lane halves).
//   layout   the keys of an S^T tile are permuted when K rows are read from LDS so that lane half
//            h holds keys 16h..16h+15 of the tile in register order; its probabilities then form
//            the B operand of the P*V product directly (8 consecutive keys per operand).  V
//            stays row-major in LDS; its V^T operand is gathered by transposing LDS reads.
//   softmax  fp32, base-2 exponent with scale*log2(e) folded into the scores; the causal mask is
//            applied only to tiles that reach past the workgroup's first row's limit.  The
//            exponentials are taken against a reference that moves only when a row's tile sum
//            would leave a bounded range (no per-tile row maximum, rare rescaling); row sums are
//            taken over the rounded bf16 probabilities with dot2 instructions.
//   loop     unrolled by two, so every LDS buffer is addressed statically; the score MFMAs of the
//            next tile are interleaved with this tile's exponentials.
//   order    workgroups that share a (KV head, split) are mapped onto one XCD (workgroups are
//            dealt round-robin over 8 XCDs), so their K/V re-reads hit that XCD's L2.
#include <algorithm>

#include <mutex>

#include "common.h"
#include "kernels.h"
#include "combine.h"

namespace omnitide {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kKT = 64;                  // keys per tile
constexpr int kRowsWG = kAttnWaves * 32; // query rows per workgroup
constexpr int kNumXcd = 8;
constexpr int kTargetWGs = 512;          // two resident workgroups on each of 256 CUs

// LDS layout: two K and two V tile buffers, each row-major [64 keys][D]:
//   K  16-byte chunks XOR-swizzled by kswz(key), so the 8 (and 16) lanes one LDS cycle serves
//      read distinct bank groups when they fetch rows perm_key(0..31) of the S^T tile.
//   V  32-byte units XOR-swizzled by vswz(key); the V^T operand of O^T = V^T P^T is gathered
//      with the transposing 64-bit LDS read (ds_read_b64_tr_b16): within a 16-lane group, lane i
//      receives element i%4 of the 8-byte rows read by lanes i/4, 4+i/4, 8+i/4, 12+i/4, i.e.
//      one dimension of four consecutive keys.  Each group reads four rows x 32 bytes; the
//      swizzle puts them (and the neighbouring group's) in distinct banks.
// Tiles are copied global -> LDS by the 16-byte direct loads (no register staging); a lane's LDS
// destination is fixed (lane-contiguous), so the swizzles are realised by choosing which global
// chunk each lane fetches.
template <int D>
struct Smem {
  static constexpr int TILE_ELEMS = kKT * D;
  static constexpr int CHUNKS = D / 8;                         // 16-byte chunks per row
  static constexpr int CALLS = TILE_ELEMS / 8 / kWave / kAttnWaves;  // 1 KB loads per wave
  // a lane's pieces cover keys k0 + (64 / CALLS) * cq with k0 < 64 / CALLS
  static_assert(kAttnWaves * kWave / CHUNKS == kKT / CALLS, "key step of a lane's pieces");
};

__device__ inline int kswz(int key) {
  return (key & 3) | ((key >> 2) & 4) | ((key << 1) & 8);
}
template <int D>
__device__ inline int vswz(int key) {
  return D == 128 ? ((key & 3) ^ ((key & 1) << 2)) : (key & 3);
}

__device__ inline floatx16 mfma(bf16x8 a, bf16x8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// S^T row r of a 32x32 MFMA tile holds key perm_key(r): lane half h, accumulator i <-> key 16h+i.
__device__ inline int perm_key(int r) { return 16 * ((r & 7) >> 2) + 4 * (r >> 3) + (r & 3); }

__device__ inline u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }

typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

__device__ inline shortx4 ld_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) shortx4*)(p));
}

__device__ inline uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<size_t>((const lds_void*)p));
}

// 16-byte direct global -> LDS load: lane i reads base + voff_i and writes 16 bytes at LDS byte
// address lds_base + 16 i.  Written as inline assembly (uniform base in SGPRs, per-lane 32-bit
// offset) so that issuing it costs no vector instructions and so that the compiler's wait
// insertion does not treat it as a pending LDS write (it would otherwise make later LDS reads of
// other buffers wait for it).  Callers wait for it explicitly (s_waitcnt vmcnt(0) + barrier)
// before any lane reads the buffer it fills.  One wait state is required between the M0 write
// and the load.  M0 is not listed as clobbered (the compiler reserves it and ignores such
// clobbers): this file's kernels have no other M0 user, so no compiler value lives in M0.
__device__ inline void dma16(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_base)
               : "memory");
}
// The same for 4 bytes per lane (lane i writes LDS byte address lds_base + 4 i).
__device__ inline void dma4(const void* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_base)
               : "memory");
}

// max(x over both 32-lane halves): v_permlane32_swap exchanges the halves without LDS.
// This lane's index in its wave, recomputed (two instructions) at the point of use.  The span
// paths index by lane only now and then; a fresh value there spares the register allocator a
// long-lived copy, which it would otherwise spill and reload behind the tile prefetches.
__device__ inline int lane_now() {
  int r;   // volatile: not hoisted out of the loop (where it would be spilled again)
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(r));
  return r;
}

__device__ inline float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int B, class T>
__device__ inline T& pick(T& a, T& b) {
  if constexpr (B == 0) return a; else return b;
}

// Key traversals of attn_kernel:
//   kContig    keys are the contiguous rows [0, n_ctx) of the compacted pool, the chunk last.
//   kSpanTiles keys are the slots [0, span) of a pool with holes (n_ctx_g holds the span); slot j
//              is visible to query i iff 0 <= key_pos[j] <= q_pos0 + i; only the active tiles
//              listed by span_list_kernel are visited, and a tile is masked only if it holds an
//              empty slot or a position past the workgroup's first row.
//   kPosOrder  a pool with holes whose entries hold the positions 0 .. n-1 once each (n = q_pos0
//              + L; n_ctx_g holds the span): keys are taken in position order, position p from
//              the slot list[p] names (pos_index_kernel), so the tiles, bounds and causal masks
//              are those of kContig with n_ctx = n; only the tile loads are gathers.
template <int D, int MODE>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ v, const int32_t* __restrict__ n_ctx_g, int cap, int L, int Hq,
    int Hkv, float scale_log2, void* __restrict__ out, bool out_bf16,
    float* __restrict__ part_o, float* __restrict__ part_ml, int n_mt, int n_split,
    int32_t* __restrict__ status,
    const int32_t* __restrict__ key_pos, const int32_t* __restrict__ qpos0_g,
    const int4* __restrict__ tile_info, const int32_t* __restrict__ list,
    const int32_t* __restrict__ list_n, int max_tiles) {
  // list, list_n -- kSpanTiles: the visited tiles and their number; kPosOrder: the slot of each
  // position and the index's per-workgroup entry counts (max_tiles of them per segment).
  constexpr bool SPAN = MODE == kSpanTiles;
  constexpr bool POS = MODE == kPosOrder;
  using S = Smem<D>;
  // Tile buffers K0, K1, V0, V1 at fixed offsets (every access below names its buffer at
  // compile time, so LDS addresses are immediates).
  __shared__ __attribute__((aligned(1024))) uint16_t lds[4 * S::TILE_ELEMS];
  __shared__ int32_t kpos_lds[SPAN ? kKT : 1];     // positions of the current tile's keys
  __shared__ __attribute__((aligned(16))) int32_t slot_ring[POS ? 4 * kKT : 1];  // tiles t..t+3

  const int seg = blockIdx.y;
  int nctx = n_ctx_g[seg];                         // SPAN, POS: the span
  if (nctx < L || nctx > cap) {
    if (threadIdx.x == 0) set_status(status, OMNITIDE_E_CAPACITY);
    return;
  }
  if constexpr (POS) {
    // the entries must be exactly the positions 0 .. q_pos0 + L - 1 (their number is checked
    // after the loop: the index clamps every slot it hands out, so the loop is safe either way)
    const int qp0 = qpos0_g[seg];
    if (qp0 < 0 || qp0 > nctx - L) {
      if (threadIdx.x == 0) set_status(status, OMNITIDE_E_TAGS);
      return;
    }
    nctx = qp0 + L;
  }
  // XCD-aware order: blocks b with equal b % 8 run on one XCD; give them consecutive work ids.
  const int nb = gridDim.x, b = blockIdx.x;
  const int xcd = b % kNumXcd, q8 = nb / kNumXcd, r8 = nb % kNumXcd;
  const int lin = (xcd < r8 ? xcd * (q8 + 1) : r8 * (q8 + 1) + (xcd - r8) * q8) + b / kNumXcd;
  const int mt = lin % n_mt;
  const int split = (lin / n_mt) % n_split;
  const int g = lin / (n_mt * n_split);

  const int G = Hq / Hkv;
  const int rows = L * G;
  const int kept = SPAN ? qpos0_g[seg] : nctx - L;  // logical position of chunk query 0
  const int m0 = mt * kRowsWG;
  const int p_lo = m0 / G;
  const int p_hi = min(L - 1, (m0 + kRowsWG - 1) / G);
  const int kmax = kept + p_hi + 1;               // keys [0, kmax) are needed by this workgroup
  const int n_tiles = SPAN ? list_n[seg] : (kmax + kKT - 1) / kKT;
  const int t_begin = static_cast<int>(static_cast<long>(n_tiles) * split / n_split);
  const int t_end = static_cast<int>(static_cast<long>(n_tiles) * (split + 1) / n_split);
  const int full_lim = kept + p_lo;               // keys <= full_lim are visible to every row

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int col = lane & 31;
  const int h = lane >> 5;
  const int m = m0 + wave * 32 + col;
  const bool row_ok = m < rows;
  const int p = row_ok ? m / G : L - 1;
  const int head = g * G + (row_ok ? m % G : 0);
  const int lim = kept + p;

  // Q^T operand: lane holds q[p][head][16c + 8h .. +8] for every 16-wide chunk c of d.
  bf16x8 qf[D / 16];
  {
    const uint16_t* qrow = q + ((static_cast<size_t>(seg) * L + p) * Hq + head) * D;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      u32x4 t = row_ok ? ld16(qrow + 16 * c + 8 * h) : u32x4{0, 0, 0, 0};
      qf[c] = __builtin_bit_cast(bf16x8, t);
    }
  }

  const size_t kv_seg = static_cast<size_t>(seg) * cap;
  const int row_stride = Hkv * D;
  // Per-lane byte offsets of this lane's 16-byte pieces inside a tile (the same for every
  // tile): piece cq covers linear chunk (wave + kAttnWaves*cq)*64 + lane of the swizzled tile.
  uint32_t koff[S::CALLS], voff[S::CALLS];
  int krowl[S::CALLS];
#pragma unroll
  for (int cq = 0; cq < S::CALLS; ++cq) {
    const int lc = (wave + kAttnWaves * cq) * kWave + lane;
    const int key = lc / S::CHUNKS, pc = lc % S::CHUNKS;
    const int row = POS ? 0 : key * row_stride;   // POS: the row comes from the slot index
    krowl[cq] = key;
    koff[cq] = 2u * (row + 8 * (pc ^ (kswz(key) & (S::CHUNKS - 1))));
    voff[cq] = 2u * (row + 8 * (2 * ((pc >> 1) ^ vswz<D>(key)) + (pc & 1)));
  }
  const uint16_t* k_head = k + (kv_seg * Hkv + g) * D;
  const uint16_t* v_head = v + (kv_seg * Hkv + g) * D;
  const uint32_t lds_wave = lds_addr(lds) + static_cast<uint32_t>(wave * kWave * 16);
  // Direct global -> LDS copy of one tensor's tile t into buffer `buf` (0,1 = K; 2,3 = V).  In a
  // boundary tile, rows past n_ctx are clamped to a valid row here and zeroed after arrival.
  auto issue = [&](const uint16_t* head_base, const uint32_t* offs, int t, int buf) {
    const int j0 = t * kKT;
    const uint16_t* tile = head_base + static_cast<size_t>(j0) * row_stride;
    const uint32_t dst = lds_wave + static_cast<uint32_t>(buf * S::TILE_ELEMS * 2);
    if constexpr (POS) {
      // key r of tile t is the entry at position 64t + r (positions past n_ctx were clamped to
      // n_ctx - 1 when the ring was filled); this lane's keys krowl[0] + KS * cq have adjacent
      // ring words, read at once.  The host keeps cap * Hkv * D * 2 below 2^32.
      typedef int32_t SlotVec __attribute__((ext_vector_type(S::CALLS)));
      const SlotVec sl = *reinterpret_cast<const SlotVec*>(slot_ring + (t & 3) * kKT +
                                                           krowl[0] * S::CALLS);
#pragma unroll
      for (int cq = 0; cq < S::CALLS; ++cq) {
        const uint32_t slot = min(static_cast<uint32_t>(sl[cq]), static_cast<uint32_t>(cap - 1));
        dma16(head_base, offs[cq] + 2u * slot * static_cast<uint32_t>(row_stride),
              dst + static_cast<uint32_t>(cq * kAttnWaves * kWave * 16));
      }
      return;
    }
    if (j0 + kKT <= nctx) {
#pragma unroll
      for (int cq = 0; cq < S::CALLS; ++cq)
        dma16(tile, offs[cq], dst + static_cast<uint32_t>(cq * kAttnWaves * kWave * 16));
    } else {
#pragma unroll
      for (int cq = 0; cq < S::CALLS; ++cq) {
        // Base at row min(j0, n_ctx-1) so every lane offset stays non-negative (the hardware
        // zero-extends it): lane row min(j0+key, n_ctx-1) lies 0..kKT-1 rows past the base.
        const int r0 = min(j0, nctx - 1);
        const int shift = min(j0 + krowl[cq], nctx - 1) - r0 - krowl[cq];
        dma16(head_base + static_cast<size_t>(r0) * row_stride,
              offs[cq] + 2u * static_cast<uint32_t>(shift * row_stride),
              dst + static_cast<uint32_t>(cq * kAttnWaves * kWave * 16));
      }
    }
  };
  auto zero_rows = [&](int t, int buf) {
    const int j0 = t * kKT;
    uint16_t* base = lds + buf * S::TILE_ELEMS;
    for (int idx = tid; idx < kKT * S::CHUNKS; idx += kAttnThreads)
      if (j0 + idx / S::CHUNKS >= nctx)
        *reinterpret_cast<u32x4*>(base + 8 * idx) = u32x4{0, 0, 0, 0};
  };

  // SPAN: the a-th visited tile is list[a]; tile_info holds its (largest position, has an
  // empty slot, occupancy bits 0-31, occupancy bits 32-63).
  const size_t tl_base = static_cast<size_t>(seg) * max_tiles;
  auto tile_of = [&](int a) -> int {
    if constexpr (SPAN) return list[tl_base + a]; else return a;
  };
  // POS: wave 0 copies the slots of positions 64t .. 64t+63 (clamped to n_ctx - 1) into ring
  // entry t & 3 (a direct load, waited for with the tile loads before the loop barrier).  Word i
  // of an entry holds key (i % CALLS) * KS + i / CALLS, KS = 64 / CALLS: the CALLS keys a lane
  // loads rows for (krowl[0] + KS * cq) are adjacent.
  auto load_ring = [&](int t) {
    constexpr int KS = kKT / S::CALLS;
    const int p = min(t * kKT + (lane % S::CALLS) * KS + lane / S::CALLS, nctx - 1);
    dma4(list + static_cast<size_t>(seg) * cap, 4u * static_cast<uint32_t>(p),
         lds_addr(slot_ring) + static_cast<uint32_t>((t & 3) * kKT * 4));
  };
  // SPAN: wave 0 holds the positions of the next V tile's keys (one per lane, -1 past the span)
  int kp_next = -1;
  auto load_kpos = [&](int t) {
    const int j = t * kKT + lane_now();
    kp_next = j < nctx ? key_pos[static_cast<size_t>(seg) * cap + j] : -1;
  };

  floatx16 o[D / 32];
#pragma unroll
  for (int dt = 0; dt < D / 32; ++dt) o[dt] = floatx16{};
  // m_run: the reference the exponentials are taken against (-inf until this row has seen a
  // visible key).  It is not kept equal to the running maximum: the exponentials of a tile are
  // computed optimistically against it and only if some row's tile sum reaches 2^32 (or is not
  // finite: no reference yet) does the wave fall back to the exact tile maximum, move the
  // reference, rescale and recompute.  Every probability and every partial sum therefore stays
  // below 2^32 x tile count, far from fp32 overflow, and the final division by the sum taken
  // against the same reference makes the result independent of where the reference sits.
  float m_run = -INFINITY, l_run = 0.f;
  const int krow = perm_key(col);
  const int fk = kswz(krow) & (S::CHUNKS - 1);
  // transposing V reads: this lane's role inside its 16-lane group
  const int gi = lane & 15, gq = (lane >> 4) & 1;
  const int vsl = vswz<D>(gi >> 2);
  const int v_lane_off = (gi >> 2) * D + 8 * ((gi & 3) >> 1) + 4 * (gi & 1);
  constexpr int NQK = 2 * (D / 16);                // score MFMAs per tile (two 32-key halves)
  constexpr int EPS = 32 / NQK;                    // exponentials per interleave segment
  constexpr float kSumLimit = 4294967296.f;        // 2^32

  auto kop = [&](const uint16_t* kb, int i) {      // K operand of score MFMA i
    const int st = i & 1, c = i >> 1;
    return __builtin_bit_cast(bf16x8, ld16(kb + (32 * st + krow) * D + 8 * ((2 * c + h) ^ fk)));
  };

  if (t_begin < t_end) {
    if constexpr (POS) {
      if (wave == 0) {
        for (int a = 0; a < 3 && t_begin + a < t_end; ++a) load_ring(t_begin + a);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
    issue(k_head, koff, tile_of(t_begin), 0);
    issue(v_head, voff, tile_of(t_begin), 2);
    if constexpr (SPAN) {
      if (wave == 0) load_kpos(tile_of(t_begin));
    }
    if (t_begin + 1 < t_end) issue(k_head, koff, tile_of(t_begin + 1), 1);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (!SPAN && t_begin * kKT + kKT > nctx) {
      zero_rows(t_begin, 0);
      __syncthreads();
    }
    floatx16 sA[2] = {floatx16{}, floatx16{}}, sB[2];
#pragma unroll
    for (int i = 0; i < NQK; ++i) sA[i & 1] = mfma(kop(lds, i), qf[i >> 1], sA[i & 1]);

    // One iteration for tile t with B = (t - t_begin) & 1: scores of t are in s_cur (computed
    // by the previous iteration); K(t+1) is in K buffer 1-B, V(t) in V buffer B.  The iteration
    // issues K(t+2) into K buffer B and V(t+1) into V buffer 1-B.
    auto step = [&](auto par, int t) {
      constexpr int B = decltype(par)::value;
      floatx16(&s_cur)[2] = pick<B>(sA, sB);
      floatx16(&s_nxt)[2] = pick<B>(sB, sA);
      const uint16_t* Kn = lds + (1 - B) * S::TILE_ELEMS;
      const uint16_t* Vs = lds + (2 + B) * S::TILE_ELEMS;
      const int j0 = t * kKT;
      const bool has_next = t + 1 < t_end;
      __builtin_amdgcn_s_waitcnt(0);      // this wave's pieces of K(t+1) and V(t) have landed
      // SPAN: t indexes the tile list.  The V rows of the tile's empty slots (their contents are
      // arbitrary) are zeroed by the lanes that loaded them, before the barrier publishes the
      // tile; a key is then masked by the tile's occupancy bits, or, in a tile holding a
      // position past the workgroup's first row, by its published position.
      int4 info = int4{0, 0, 0, 0};
      if constexpr (SPAN) {
        info = tile_info[tl_base + tile_of(t)];
        if (info.y != 0) {
          const uint64_t valid = static_cast<uint64_t>(static_cast<uint32_t>(info.z)) |
                                 (static_cast<uint64_t>(static_cast<uint32_t>(info.w)) << 32);
          uint16_t* vb = lds + (2 + B) * S::TILE_ELEMS;
#pragma unroll
          for (int cq = 0; cq < S::CALLS; ++cq) {
            if (((valid >> (((wave + kAttnWaves * cq) * kWave + lane_now()) / S::CHUNKS)) & 1) == 0)
              *reinterpret_cast<u32x4*>(vb + 8 * ((wave + kAttnWaves * cq) * kWave + lane_now())) =
                  u32x4{0, 0, 0, 0};
          }
        }
      }
      __syncthreads();                    // ... everyone's; iteration t-1 is finished
      bool masked;
      bool causal = false;
      if constexpr (SPAN) {
        causal = info.x > full_lim;
        masked = info.y != 0 || causal;
        if (causal) {
          if (wave == 0) kpos_lds[lane_now()] = kp_next;
          __syncthreads();
        }
        if (t + 2 < t_end) issue(k_head, koff, tile_of(t + 2), B);
        if (has_next) {
          issue(v_head, voff, tile_of(t + 1), 3 - B);
          if (wave == 0) load_kpos(tile_of(t + 1));
        }
      } else {
        if ((has_next && j0 + 2 * kKT > nctx) || j0 + kKT > nctx) {
          if (has_next) zero_rows(t + 1, 1 - B);
          zero_rows(t, 2 + B);
          __syncthreads();
        }
        if (t + 2 < t_end) issue(k_head, koff, t + 2, B);
        if (has_next) issue(v_head, voff, t + 1, 3 - B);
        if constexpr (POS) {
          // ring entry (t + 3) & 3 held tile t - 1's slots, last read two iterations ago
          if (wave == 0 && t + 3 < t_end) load_ring(t + 3);
        }
        masked = j0 + kKT - 1 > full_lim;  // causal mask: only tiles past the first row's limit
      }

      if (masked) {
        if (SPAN && !causal) {
          // occupancy bits of this lane's keys 32st + 16h + i
          const uint32_t half_bits[2] = {static_cast<uint32_t>(info.z) >> (16 * h),
                                         static_cast<uint32_t>(info.w) >> (16 * h)};
#pragma unroll
          for (int st = 0; st < 2; ++st) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
              if (((half_bits[st] >> i) & 1) == 0) s_cur[st][i] = -INFINITY;
          }
        } else {
#pragma unroll
          for (int st = 0; st < 2; ++st) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
              if constexpr (SPAN) {
                const int kp = kpos_lds[32 * st + 16 * h + i];
                if (kp < 0 || kp > lim) s_cur[st][i] = -INFINITY;
              } else {
                if (j0 + 32 * st + 16 * h + i > lim) s_cur[st][i] = -INFINITY;
              }
            }
          }
        }
      }

      // Interleave: segment i issues score MFMA i of the next tile and then EPS exponentials
      // of this tile, so the vector ALU works while the matrix core runs (a wave issues in
      // order).  In the last iteration the next-K buffer holds a stale tile; the scores
      // computed from it are discarded, which keeps the loop body branch-free.
      // Each segment also rounds its completed pairs of probabilities into the P operand and
      // adds them to the row sum (in the same pair order and chains as the rowsum below), so
      // no vector work is left between the two MFMA phases.
      static_assert(EPS % 2 == 0, "whole pairs per segment");
      float e[32];
      bf16x8 pf[2][2];
      const bf16x2 one2 = {static_cast<__bf16>(1.f), static_cast<__bf16>(1.f)};
      float ls_run[2] = {0.f, 0.f};
      {
        s_nxt[0] = floatx16{};
        s_nxt[1] = floatx16{};
        const float m_use = m_run;
        bf16x8 ka0 = kop(Kn, 0), ka1 = kop(Kn, 1);
#pragma unroll
        for (int i = 0; i < NQK; ++i) {
          const bf16x8 ka = (i & 1) ? ka1 : ka0;
          s_nxt[i & 1] = mfma(ka, qf[i >> 1], s_nxt[i & 1]);
          if (i + 2 < NQK) {
            if (i & 1) ka1 = kop(Kn, i + 2); else ka0 = kop(Kn, i + 2);
          }
#pragma unroll
          for (int j = 0; j < EPS; ++j) {
            const int x = i * EPS + j;
            e[x] = __builtin_amdgcn_exp2f(fmaf(s_cur[x >> 4][x & 15], scale_log2, -m_use));
          }
#pragma unroll
          for (int j = 0; j < EPS; j += 2) {
            const int x = i * EPS + j;
            const __bf16 b0 = static_cast<__bf16>(e[x]), b1 = static_cast<__bf16>(e[x + 1]);
            pf[x >> 4][(x >> 3) & 1][x & 7] = b0;
            pf[x >> 4][(x >> 3) & 1][(x & 7) + 1] = b1;
            const bf16x2 pr = {b0, b1};
            ls_run[(x >> 1) & 1] =
                __builtin_amdgcn_fdot2_f32_bf16(pr, one2, ls_run[(x >> 1) & 1], false);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      auto pack = [&]() {
#pragma unroll
        for (int x = 0; x < 32; ++x) pf[x >> 4][(x >> 3) & 1][x & 7] = static_cast<__bf16>(e[x]);
      };
      // Row sum of the rounded probabilities (exactly the weights the P*V product uses), two
      // bf16 pairs per instruction against (1, 1), in two chains.
      auto rowsum = [&]() {
        float ls[2] = {0.f, 0.f};
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const bf16x8 v8 = pf[x >> 3][(x >> 2) & 1];
          const int j = x & 3;
          const bf16x2 pr = {v8[2 * j], v8[2 * j + 1]};
          ls[x & 1] = __builtin_amdgcn_fdot2_f32_bf16(pr, one2, ls[x & 1], false);
        }
        return ls[0] + ls[1];
      };
      float lsum = ls_run[0] + ls_run[1];
      if (__any(!(lsum < kSumLimit))) {
        // Slow path: exact tile maximum, move the reference, rescale, recompute the tile.
        float mx = -INFINITY;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
#pragma unroll
          for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s_cur[st][i]);
        }
        mx = max_halves(mx) * scale_log2;
        const float m_new = fmaxf(m_run, mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) o[dt] *= alpha;
        m_run = m_new;
#pragma unroll
        for (int x = 0; x < 32; ++x)
          e[x] = __builtin_amdgcn_exp2f(fmaf(s_cur[x >> 4][x & 15], scale_log2, -m_use));
        pack();
        lsum = rowsum();
      }
      l_run += lsum;

      // O^T += V^T P^T: the V^T operand (dims 32dt.., keys 32st+16h+8cc..+8) from two
      // transposing reads of four keys each, read three products ahead (the order pinned by
      // the segment fences; the scheduler would otherwise move the reads next to their use).
      constexpr int NPV = 4 * (D / 32);
      auto vop = [&](int i) {
        const int dt = i % (D / 32), cc = (i / (D / 32)) & 1, st = i / (2 * (D / 32));
        const int unit = (2 * dt + gq) ^ vsl;
        const uint16_t* vp = Vs + (32 * st + 16 * h + 8 * cc) * D + 16 * unit + v_lane_off;
        const shortx4 lo = ld_tr(vp);
        const shortx4 hi = ld_tr(vp + 4 * D);
        return __builtin_bit_cast(bf16x8,
                                  __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      };
      bf16x8 va[4] = {vop(0), vop(1), vop(2), bf16x8{}};
#pragma unroll
      for (int i = 0; i < NPV; ++i) {
        if (i + 3 < NPV) va[(i + 3) % 4] = vop(i + 3);
        const int dt = i % (D / 32), cc = (i / (D / 32)) & 1, st = i / (2 * (D / 32));
        o[dt] = mfma(va[i % 4], pf[st][cc], o[dt]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    int t = t_begin;
    for (; t + 1 < t_end; t += 2) {
      step(std::integral_constant<int, 0>{}, t);
      step(std::integral_constant<int, 1>{}, t + 1);
    }
    if (t < t_end) step(std::integral_constant<int, 0>{}, t);
  }

  if constexpr (POS) {
    // one wave per segment: the index's workgroup counts must add up to n_ctx entries
    if (blockIdx.x == 0 && wave == 0) {
      int c = 0;
      for (int b = lane; b < max_tiles; b += kWave)
        c += list_n[static_cast<size_t>(seg) * max_tiles + b];
      // the whole wave sums (a cross-lane scan), then one lane reports
      const int total = static_cast<int>(wave_sum_u32(static_cast<uint32_t>(c)));
      if (lane == 0 && total != nctx) set_status(status, OMNITIDE_E_TAGS);
    }
  }
  const float l_tot = sum_halves(l_run);
  if (!row_ok) return;
  const size_t orow = (static_cast<size_t>(seg) * L + p) * Hq + head;
  if (n_split == 1) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int qd = 0; qd < 4; ++qd)
        store_out4(out, orow * D + 32 * dt + 8 * qd + 4 * h, out_bf16, o[dt][4 * qd] * inv,
                   o[dt][4 * qd + 1] * inv, o[dt][4 * qd + 2] * inv, o[dt][4 * qd + 3] * inv);
    }
  } else {
    const size_t n_rows_all = static_cast<size_t>(gridDim.y) * L * Hq;
    const size_t prow = static_cast<size_t>(split) * n_rows_all + orow;
    float* dst = part_o + prow * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) {
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        float4 val = make_float4(o[dt][4 * qd], o[dt][4 * qd + 1], o[dt][4 * qd + 2],
                                 o[dt][4 * qd + 3]);
        *reinterpret_cast<float4*>(dst + 32 * dt + 8 * qd + 4 * h) = val;
      }
    }
    if (h == 0) *reinterpret_cast<float2*>(part_ml + 2 * prow) = make_float2(m_run, l_tot);
  }
}

// Active tiles of a span.  span_info_kernel: one wave per 64-slot tile of [0, span) (a grid of
// workgroups) records the tile's largest key position, whether it holds an empty slot (or
// slots past the span), its 64 occupancy bits and whether it is visited (it holds an entry, or
// every tile of the span is visited).  span_list_kernel: one workgroup per segment lists the
// visited tiles, in order.
constexpr int kSpanThreads = 1024;
constexpr int kInfoThreads = 256;

__global__ __launch_bounds__(kInfoThreads) void span_info_kernel(
    const int32_t* __restrict__ key_pos, const int32_t* __restrict__ span_g, int cap, int L,
    int max_tiles, int skip_empty, int4* __restrict__ tile_info, uint8_t* __restrict__ act_g) {
  const int seg = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int t = blockIdx.x * (kInfoThreads / kWave) + threadIdx.x / kWave;
  const int span = span_g[seg];
  if (span < L || span > cap) return;            // reported by the attention kernel
  if (t * kKT >= span) return;
  const int j = t * kKT + lane;
  const int p = j < span ? key_pos[static_cast<size_t>(seg) * cap + j] : -1;
  const uint64_t valid = __ballot(p >= 0);
  const int mx = wave_max_i32(p);
  if (lane == 0) {
    const size_t tb = static_cast<size_t>(seg) * max_tiles;
    tile_info[tb + t] = make_int4(mx, valid != ~0ull ? 1 : 0,
                                  static_cast<int>(valid & 0xffffffffu),
                                  static_cast<int>(valid >> 32));
    act_g[tb + t] = (valid != 0 || !skip_empty) ? 1 : 0;
  }
}

__global__ __launch_bounds__(kSpanThreads) void span_list_kernel(
    const uint8_t* __restrict__ act_g, const int32_t* __restrict__ span_g, int cap, int L,
    int max_tiles, int32_t* __restrict__ tile_list, int32_t* __restrict__ n_active_g) {
  __shared__ int32_t scr[kSpanThreads / kWave + 1];
  const int seg = blockIdx.x;
  const int tid = threadIdx.x;
  const int span = span_g[seg];
  const size_t tb = static_cast<size_t>(seg) * max_tiles;
  if (span < L || span > cap) {
    if (tid == 0) n_active_g[seg] = 0;
    return;
  }
  const int n_tiles = (span + kKT - 1) / kKT;
  int running = 0;
  for (int base = 0; base < n_tiles; base += kSpanThreads) {
    const int t = base + tid;
    const int f = t < n_tiles ? act_g[tb + t] : 0;
    int total;
    const int off = block_exclusive_scan(f, scr, &total);
    if (f) tile_list[tb + running + off] = t;
    running += total;
  }
  if (tid == 0) n_active_g[seg] = running;
}

// Position index of a span whose entries should hold the positions 0 .. n-1 once each (n =
// q_pos0 + chunk_len): slot_of[p] = the slot holding position p, built in one launch without
// clearing.  One thread per slot j of the span exchanges j into slot_of[key_pos[j]] and gets
// the previous content back: a slot written by an earlier call (anything, even garbage), or one
// written by this call if the position is held twice.  It is the latter exactly when that slot
// lies inside the span and holds the same position now, which is reported as OMNITIDE_E_TAGS,
// as is a position >= n.  Each workgroup stores its count of entries (so no accumulator needs
// clearing); the attention kernels compare their sum with n, which reports a missing position.
// With no position repeated, none >= n and n entries, every slot_of[0, n) was written by this
// call.  Segments with an invalid span or q_pos0 are left to the attention kernels.
__global__ __launch_bounds__(kInfoThreads) void pos_index_kernel(
    const int32_t* __restrict__ key_pos, const int32_t* __restrict__ span_g,
    const int32_t* __restrict__ qpos0_g, int cap, int L, int32_t* __restrict__ slot_of,
    int32_t* __restrict__ counts, int32_t* __restrict__ status) {
  __shared__ int32_t wave_counts[kInfoThreads / kWave];
  const int seg = blockIdx.y;
  const int span = span_g[seg];
  const int qp0 = qpos0_g[seg];
  const bool seg_ok = span >= L && span <= cap && qp0 >= 0 && qp0 <= span - L;
  const int n = seg_ok ? qp0 + L : 0;
  const int j = blockIdx.x * kInfoThreads + static_cast<int>(threadIdx.x);
  const size_t sb = static_cast<size_t>(seg) * cap;
  const int p = seg_ok && j < span ? key_pos[sb + j] : -1;
  if (p >= n) {
    set_status(status, OMNITIDE_E_TAGS);
  } else if (p >= 0) {
    const int old = atomicExch(&slot_of[sb + p], j);
    if (old != j && old >= 0 && old < span && key_pos[sb + old] == p)
      set_status(status, OMNITIDE_E_TAGS);
  }
  const uint64_t c = __ballot(p >= 0);
  if ((threadIdx.x & (kWave - 1)) == 0) wave_counts[threadIdx.x / kWave] = __popcll(c);
  __syncthreads();
  if (threadIdx.x == 0) {
    int total = 0;
    for (int w = 0; w < kInfoThreads / kWave; ++w) total += wave_counts[w];
    counts[static_cast<size_t>(seg) * gridDim.x + blockIdx.x] = total;
  }
}

}  // namespace

// Tables of n_seg segments: int4 info, int32 list, int32 counts, then the byte flags (the
// caller places buf on a 256-byte boundary).
SpanTiles span_tiles_at(void* buf, int n_seg, int cap) {
  const size_t nt = static_cast<size_t>(n_seg) * ((cap + kKT - 1) / kKT);
  uint8_t* b = static_cast<uint8_t*>(buf);
  SpanTiles T;
  T.info = reinterpret_cast<int4*>(b);
  T.list = reinterpret_cast<int32_t*>(b + nt * sizeof(int4));
  T.n_active = T.list + nt;
  T.act = reinterpret_cast<uint8_t*>(T.n_active + n_seg);
  return T;
}

size_t span_tiles_bytes(int n_seg, int cap) {
  const size_t nt = static_cast<size_t>(n_seg) * ((cap + kKT - 1) / kKT);
  return nt * (sizeof(int4) + sizeof(int32_t) + 1) + static_cast<size_t>(n_seg) * sizeof(int32_t);
}

// Position index of n_seg segments (kPosOrder): int32 slot_of[n_seg][cap], then the
// per-workgroup entry counts [n_seg][pos_index_blocks(cap)].
int pos_index_blocks(int cap) { return (cap + kInfoThreads - 1) / kInfoThreads; }

size_t pos_index_bytes(int n_seg, int cap) {
  return static_cast<size_t>(n_seg) * (static_cast<size_t>(cap) + pos_index_blocks(cap)) *
         sizeof(int32_t);
}

hipError_t launch_pos_index(const int32_t* key_pos, const int32_t* span, const int32_t* q_pos0,
                            int n_seg, int cap, int L, int32_t* slot_of, hipStream_t stream,
                            int32_t* d_status) {
  int32_t* counts = slot_of + static_cast<size_t>(n_seg) * cap;
  hipLaunchKernelGGL(pos_index_kernel, dim3(pos_index_blocks(cap), n_seg), dim3(kInfoThreads), 0,
                     stream, key_pos, span, q_pos0, cap, L, slot_of, counts, d_status);
  return hipGetLastError();
}

hipError_t launch_span_tiles(const int32_t* key_pos, const int32_t* span, int n_seg, int cap,
                             int min_span, bool skip_empty, void* buf, hipStream_t stream) {
  const int max_tiles = (cap + kKT - 1) / kKT;
  const SpanTiles T = span_tiles_at(buf, n_seg, cap);
  const int per_block = kInfoThreads / kWave;
  hipLaunchKernelGGL(span_info_kernel, dim3((max_tiles + per_block - 1) / per_block, n_seg),
                     dim3(kInfoThreads), 0, stream, key_pos, span, cap, min_span, max_tiles,
                     skip_empty ? 1 : 0, T.info, T.act);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(span_list_kernel, dim3(n_seg), dim3(kSpanThreads), 0, stream, T.act, span,
                     cap, min_span, max_tiles, T.list, T.n_active);
  return hipGetLastError();
}

namespace {

template <int D>
hipError_t launch_attn_t(const AttnArgs& a, int n_split, hipStream_t stream) {
  const int G = a.n_q_heads / a.n_kv_heads;
  const int n_mt = (a.chunk_len * G + kRowsWG - 1) / kRowsWG;
  const dim3 grid(n_mt * a.n_kv_heads * n_split, a.n_seg);
  const size_t n_rows = static_cast<size_t>(a.n_seg) * a.chunk_len * a.n_q_heads;
  float* part_o = n_split > 1 ? static_cast<float*>(a.workspace) : nullptr;
  float* part_ml = part_o ? part_o + static_cast<size_t>(n_split) * n_rows * D : nullptr;
  const float scale_log2 = a.scale * 1.4426950408889634f;
  if (a.key_pos != nullptr && a.pos_order) {
    // position order: the position index after the partials
    int32_t* slot_of = reinterpret_cast<int32_t*>(
        static_cast<uint8_t*>(a.workspace) +
        align256(n_split > 1 ? static_cast<size_t>(n_split) * n_rows * (D + 2) * 4 : 0));
    hipError_t e = launch_pos_index(a.key_pos, a.n_ctx, a.q_pos0, a.n_seg, a.cap, a.chunk_len,
                                    slot_of, stream, a.d_status);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_kernel<D, kPosOrder>), grid, dim3(kAttnThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.chunk_len,
                       a.n_q_heads, a.n_kv_heads, scale_log2, a.out, a.out_bf16, part_o, part_ml,
                       n_mt, n_split, a.d_status, a.key_pos, a.q_pos0, nullptr, slot_of,
                       slot_of + static_cast<size_t>(a.n_seg) * a.cap, pos_index_blocks(a.cap));
  } else if (a.key_pos != nullptr) {
    // span mode: tile table after the partials
    const int max_tiles = (a.cap + kKT - 1) / kKT;
    uint8_t* tbl = static_cast<uint8_t*>(a.workspace) +
                   align256(n_split > 1 ? static_cast<size_t>(n_split) * n_rows * (D + 2) * 4 : 0);
    const SpanTiles T = span_tiles_at(tbl, a.n_seg, a.cap);
    int4* tile_info = T.info;
    int32_t* tile_list = T.list;
    int32_t* n_active = T.n_active;
    hipError_t e = launch_span_tiles(a.key_pos, a.n_ctx, a.n_seg, a.cap, a.chunk_len,
                                     a.skip_empty, tbl, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_kernel<D, kSpanTiles>), grid, dim3(kAttnThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.chunk_len,
                       a.n_q_heads, a.n_kv_heads, scale_log2, a.out, a.out_bf16, part_o, part_ml,
                       n_mt, n_split, a.d_status, a.key_pos, a.q_pos0, tile_info, tile_list,
                       n_active, max_tiles);
  } else {
    hipLaunchKernelGGL((attn_kernel<D, kContig>), grid, dim3(kAttnThreads), 0, stream,
                       static_cast<const uint16_t*>(a.q), static_cast<const uint16_t*>(a.k),
                       static_cast<const uint16_t*>(a.v), a.n_ctx, a.cap, a.chunk_len,
                       a.n_q_heads, a.n_kv_heads, scale_log2, a.out, a.out_bf16, part_o, part_ml,
                       n_mt, n_split, a.d_status, nullptr, nullptr, nullptr, nullptr, nullptr, 0);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_split == 1) return e;
  return launch_combine<D>(part_o, part_ml, n_split, n_rows, a.n_ctx, a.chunk_len, a.n_q_heads,
                           a.cap, a.out, stream, a.out_bf16);
}

}  // namespace

int attn_num_splits(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                    int head_dim) {
  (void)head_dim;
  const int G = n_q_heads / n_kv_heads;
  const long n_mt = (static_cast<long>(chunk_len) * G + kRowsWG - 1) / kRowsWG;
  const long base = n_mt * n_kv_heads * n_seg;
  const long tiles = (cap + kKT - 1) / kKT;
  long s = kTargetWGs / base;
  s = std::min(s, tiles / 4);
  return static_cast<int>(std::max(1L, std::min(s, 16L)));
}

size_t attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                            int head_dim) {
  const int s = attn_num_splits(n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim);
  if (s == 1) return 0;
  const size_t rows = static_cast<size_t>(n_seg) * chunk_len * n_q_heads;
  return static_cast<size_t>(s) * rows * (static_cast<size_t>(head_dim) + 2) * sizeof(float);
}

size_t span_attn_workspace_bytes(int n_seg, int cap, int chunk_len, int n_q_heads,
                                 int n_kv_heads, int head_dim) {
  // the tile table (tile traversals) or the position index (position order) after the partials
  return align256(attn_workspace_bytes(n_seg, cap, chunk_len, n_q_heads, n_kv_heads, head_dim)) +
         std::max(span_tiles_bytes(n_seg, cap), pos_index_bytes(n_seg, cap));
}

int span_attn_max_cap() { return 32768 * kKT; }

namespace {

// float32 -> bf16 (round to nearest even), four values per thread; n is a multiple of 4.
__global__ __launch_bounds__(256) void cast_bf16_kernel(const float4* __restrict__ src,
                                                        uint2* __restrict__ dst, size_t n4) {
  for (size_t i = static_cast<size_t>(blockIdx.x) * 256 + threadIdx.x; i < n4;
       i += static_cast<size_t>(gridDim.x) * 256) {
    const float4 x = src[i];
    const __bf16 b[4] = {static_cast<__bf16>(x.x), static_cast<__bf16>(x.y),
                         static_cast<__bf16>(x.z), static_cast<__bf16>(x.w)};
    dst[i] = make_uint2(static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b[0])) |
                            (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b[1])) << 16),
                        static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b[2])) |
                            (static_cast<uint32_t>(__builtin_bit_cast(uint16_t, b[3])) << 16));
  }
}

hipError_t cast_bf16(const void* src, void* dst, size_t n, hipStream_t stream) {
  const size_t n4 = n / 4;
  const unsigned blocks = static_cast<unsigned>(std::min<size_t>((n4 + 255) / 256, 4096));
  if (blocks == 0) return hipSuccess;
  hipLaunchKernelGGL(cast_bf16_kernel, dim3(blocks), dim3(256), 0, stream,
                     static_cast<const float4*>(src), static_cast<uint2*>(dst), n4);
  return hipGetLastError();
}

}  // namespace

size_t attn_cast_bytes(int n_seg, int cap, int chunk_len, int n_q_heads, int n_kv_heads,
                       int head_dim) {
  const size_t q = static_cast<size_t>(n_seg) * chunk_len * n_q_heads * head_dim;
  const size_t kv = static_cast<size_t>(n_seg) * cap * n_kv_heads * head_dim;
  return align256(q * 2) + 2 * align256(kv * 2);
}

hipError_t launch_attn(const AttnArgs& a, hipStream_t stream) {
  const int s = attn_num_splits(a.n_seg, a.cap, a.chunk_len, a.n_q_heads, a.n_kv_heads,
                                a.head_dim);
  AttnArgs b = a;
  if (a.in_f32) {
    // bf16 copies of q, k and v after the partials
    uint8_t* w = static_cast<uint8_t*>(a.workspace) +
                 align256(attn_workspace_bytes(a.n_seg, a.cap, a.chunk_len, a.n_q_heads,
                                               a.n_kv_heads, a.head_dim));
    const size_t nq = static_cast<size_t>(a.n_seg) * a.chunk_len * a.n_q_heads * a.head_dim;
    const size_t nkv = static_cast<size_t>(a.n_seg) * a.cap * a.n_kv_heads * a.head_dim;
    void* q16 = w;
    void* k16 = w + align256(nq * 2);
    void* v16 = w + align256(nq * 2) + align256(nkv * 2);
    hipError_t e = cast_bf16(a.q, q16, nq, stream);
    if (e == hipSuccess) e = cast_bf16(a.k, k16, nkv, stream);
    if (e == hipSuccess) e = cast_bf16(a.v, v16, nkv, stream);
    if (e != hipSuccess) return e;
    b.q = q16;
    b.k = k16;
    b.v = v16;
  }
  if (a.head_dim == 128) return launch_attn_t<128>(b, s, stream);
  if (a.head_dim == 64) return launch_attn_t<64>(b, s, stream);
  return hipErrorInvalidValue;
}

// Fixed scratch of omnitide_chunk_attn_noalloc: the split-KV partials live in this array, one
// copy per device, held until the process ends.  Host code never passes the array's name to a
// kernel (on the host it is only a stand-in for the symbol): the device address comes from
// hipGetSymbolAddress, taken once per device with that device current, and is cached here.
static __device__ __align__(256) uint8_t scratch[OMNITIDE_NOALLOC_SCRATCH_BYTES];
// Splits times row-tile workgroups never exceed kTargetWGs and a row tile holds kRowsWG rows, so
// the partials need at most kTargetWGs * kRowsWG * (128 + 2) floats: every valid shape fits.
static_assert(static_cast<size_t>(kTargetWGs) * kRowsWG * (128 + 2) * sizeof(float) <=
                  OMNITIDE_NOALLOC_SCRATCH_BYTES,
              "the split heuristic can exceed the fixed scratch");

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(hipStream_t stream, void** ptr) {
  int dev = -1;
  hipError_t e = stream != nullptr ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    int cur = -1;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t r = hipSetDevice(cur);
      if (e == hipSuccess) e = r;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_attn_noalloc(const AttnArgs& a, hipStream_t stream) {
  AttnArgs b = a;
  b.workspace = nullptr;
  if (attn_workspace_bytes(a.n_seg, a.cap, a.chunk_len, a.n_q_heads, a.n_kv_heads,
                           a.head_dim) > 0) {
    const hipError_t e = noalloc_scratch(stream, &b.workspace);
    if (e != hipSuccess) return e;
  }
  return launch_attn(b, stream);
}

}  // namespace omnitide
