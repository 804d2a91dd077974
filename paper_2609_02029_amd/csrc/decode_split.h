// decode_split.h -- split phase of the decode attention over per-head grouped
// caches (gfx950, wave64, VALU) for the 16-bit cache formats, bf16 and
// binary16; instantiated once per format by decode_split_<format>.hip.  fp8
// caches take the matrix-core kernel of decode_mfma.h (included below, it
// shares this file's work decomposition, helpers and launcher).
//
// What is computed (paper: Eqs. conditional-attention-weight and
// conditional-attention, exact scaled dot-product logit): for every sequence b
// and query head qh of a layer, over the slots [0, n_valid) of KV head
// h = qh / G,
//     out = sum_s exp(z_s - m) v_s / sum_s exp(z_s - m),   z_s = scale q.k_s.
// Softmax is invariant to the order of the slots, so ring slots are read in
// slot order and never unwrapped (keys are post-RoPE, positions are not used).
//
// Work decomposition.  One launch covers the (b, h) "items" of a layer.
// Each item gets workgroups in proportion to its 64-slot tiles (the host
// picks T tiles per workgroup for the whole launch, about four workgroups
// per CU, and gives an item of n tiles ceil(n / T) workgroups), so the grid
// is balanced by bytes, not by unit (full and windowed heads of one layer
// differ by up to ~56x in length).  Workgroup j of an item takes its tiles
// j, j + nwg, ... and walks them one after another with all four waves on
// the same tile (split_body below).  The G query heads of an item share every
// K/V byte read.
//
// Inside a wave, per tile (one stream of 16-byte buffer loads per lane with
// PF loads always in flight, running on into the next tile):
//   q.k   one lane per slot: the K tile is stored slot-minor in 8-element
//         channel chunks, so chunk g of the tile is contiguous and lane t
//         reads its own slot's chunk; q is uniform and comes through scalar
//         loads.  bf16 keys: v_dot2_f32_bf16 multiplies bf16 pairs (q as an
//         SGPR operand) with fp32 accumulate; binary16 keys meet q staged in
//         LDS as binary16 (each head under a power of
//         two that keeps every component within 2^31 of its largest exact)
//         in v_dot2_f32_f16.  Each wave covers a quarter of the channels;
//         the quarters are summed through LDS.
//   softmax  online, base 2 (log2(e) folded into the scale); the tile max is
//         one DPP row reduction plus four lane reads per head.
//   p.v   lanes own 8 channels of one row (V row-major, a wave reads whole
//         rows contiguously); p is broadcast through a per-wave LDS slice.
//         The values are widened to fp32 (exactly) and take one fp32 FMA per
//         (row, channel, head) with the fp32 weights.
//         The V buffer descriptor of a tile ends at row n_valid, so rows
//         past it read as zero (and their p is zero).
// The fused append writes the new token, in the cache format, into its slot
// at the start of the one workgroup whose tiles hold that slot, before any
// of its waves read.
// A workgroup either writes the final output (an item with one workgroup) or
// a partial (m, l, acc) that the combine kernel merges: m* = max m_j,
// l* = sum l_j 2^(m_j - m*), out = sum acc_j 2^(m_j - m*) / l*.
#pragma once

#include <hip/hip_ext.h>

#include <utility>

#include "hwkv_internal.h"
#include "kv_format.h"

namespace hwkv {
namespace {

// Calls f(std::integral_constant<int, J>{}) for J = 0 .. N-1 (fully
// unrolled: every index is a compile-time constant).
template <typename F, int... Js>
__device__ __forceinline__ void static_for_impl(F &f,
                                                std::integer_sequence<int, Js...>) {
  (f(std::integral_constant<int, Js>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Load batching (compile-time).
#ifndef HWKV_DECODE_PREFETCH
#define HWKV_DECODE_PREFETCH 4     // 16-byte chunk loads in flight
#endif
#ifndef HWKV_DECODE_AUX
#define HWKV_DECODE_AUX 2  // cache-policy bits of the streaming loads (nt)
#endif
#ifndef HWKV_DECODE_MINWAVES
#define HWKV_DECODE_MINWAVES 4
#endif
constexpr int kWaves = kDecodeWaves;             // waves per workgroup
constexpr int kPrefetch = HWKV_DECODE_PREFETCH;  // 16-byte loads in flight
// VGPR budget: four waves per SIMD (four workgroups per CU); eight q heads
// per KV head (64 value accumulators per lane), and six with binary16 keys
// at head_dim 256, need the budget of three
constexpr int split_waves_per_eu(int D, int G, int F) {
  if (HWKV_DECODE_MINWAVES <= 2) return HWKV_DECODE_MINWAVES;
  return (G == 8 || (F == HWKV_KV_F16 && G == 6 && D >= 256)) ? HWKV_DECODE_MINWAVES - 1
                                                              : HWKV_DECODE_MINWAVES;
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef const __attribute__((address_space(4))) u32x4_t cu32x4_t;

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c,
                                         false);
}

__device__ __forceinline__ float bf_lo(uint32_t x) {
  return __uint_as_float(x << 16);
}
__device__ __forceinline__ float bf_hi(uint32_t x) {
  return __uint_as_float(x & 0xffff0000u);
}

// Raw buffer loads: SGPR descriptor + 32-bit byte offset; reads past
// the descriptor's num_records return zero.

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base,
                                                            uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0,
                                           (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 bload(__amdgpu_buffer_rsrc_t r, int offset) {
  const u32x4_t v =
      __builtin_amdgcn_raw_buffer_load_b128(r, offset, 0, HWKV_DECODE_AUX);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// One chunk (8 elements) of format F: a 16- or 8-byte buffer load at a
// per-lane offset plus a wave-uniform one (soffset, an SGPR: no vector add);
// the range check applies to their sum.
template <int F>
__device__ __forceinline__ typename KvFormat<F>::Chunk bload_chunk(
    __amdgpu_buffer_rsrc_t r, int offset, int soffset = 0) {
  if constexpr (KvFormat<F>::kBytes == 2) {
    const u32x4_t v =
        __builtin_amdgcn_raw_buffer_load_b128(r, offset, soffset, HWKV_DECODE_AUX);
    return make_uint4(v.x, v.y, v.z, v.w);
  } else {
    const u32x2_t v =
        __builtin_amdgcn_raw_buffer_load_b64(r, offset, soffset, HWKV_DECODE_AUX);
    return make_uint2(v.x, v.y);
  }
}

__device__ __forceinline__ float h_lo(uint32_t x) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(x & 0xffffu));
}
__device__ __forceinline__ float h_hi(uint32_t x) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)(x >> 16));
}

// fp8 codes 2i, 2i + 1 of a word as one bf16 pair (exact), low code first.
template <bool HI>
__device__ __forceinline__ uint32_t fp8x2_bf16x2(uint32_t w) {
  return __builtin_bit_cast(uint32_t,
                            __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HI));
}


// The 8 elements of a V chunk widened to fp32 (exact).
template <int F>
__device__ __forceinline__ void widen8(typename KvFormat<F>::Chunk x, float (&vf)[8]) {
  if constexpr (F == HWKV_KV_BF16) {
    vf[0] = bf_lo(x.x); vf[1] = bf_hi(x.x); vf[2] = bf_lo(x.y); vf[3] = bf_hi(x.y);
    vf[4] = bf_lo(x.z); vf[5] = bf_hi(x.z); vf[6] = bf_lo(x.w); vf[7] = bf_hi(x.w);
  } else {
    vf[0] = h_lo(x.x); vf[1] = h_hi(x.x); vf[2] = h_lo(x.y); vf[3] = h_hi(x.y);
    vf[4] = h_lo(x.z); vf[5] = h_hi(x.z); vf[6] = h_lo(x.w); vf[7] = h_hi(x.w);
  }
}

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                         0xF, 0xF, false));
}

__device__ __forceinline__ float lane_read(float v, int lane) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// Maximum over the 64 lanes (result uniform).  Within rows of 16 lanes:
// quad_perm(1,0,3,2), quad_perm(2,3,0,1), row_half_mirror, row_mirror; then
// the four row results are read out.
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp<0xB1>(v));
  v = fmaxf(v, dpp<0x4E>(v));
  v = fmaxf(v, dpp<0x141>(v));
  v = fmaxf(v, dpp<0x140>(v));
  return fmaxf(fmaxf(lane_read(v, 0), lane_read(v, 16)),
               fmaxf(lane_read(v, 32), lane_read(v, 48)));
}

__device__ __forceinline__ float wave_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  return (lane_read(v, 0) + lane_read(v, 16)) +
         (lane_read(v, 32) + lane_read(v, 48));
}

template <int D, int G, int F>
struct SplitSmem {
  static constexpr int PST = (G + 3) & ~3;  // weights per slot (fp32), 16-byte rows
  struct Tile {
    float lg[2][G][kWaves][64];     // partial logits (head, wave, slot), by tile parity
    float p[64 * PST];              // the tile's weights (slot, head)
  };
  // separate areas (not a union): the epilogue's writes need no barrier
  // behind the last tile's reads
  struct {
    Tile t;                                               // the tile walk
    __attribute__((aligned(16))) float acc[kWaves][G][D];  // epilogue: wave sums
  } u;
  float alpha[G];                   // the tile's rescale of each head's sums
  float m[G], l[G];                 // the workgroup's shift and normaliser
  // binary16 keys: the item's q as binary16 pairs (head-major), and each
  // head's logit scale
  __attribute__((aligned(16))) uint32_t q16[F == HWKV_KV_F16 ? G * D / 2 : 4];
  float qsc[G];
};

// x of lane l and x of lane l ^ 32 for two values at once (VALU lane swap):
// returns x0 + x0' in lanes 0..31 and x1 + x1' in lanes 32..63.
__device__ __forceinline__ float half_sum_pair(float x0, float x1) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, x0),
                                                  __builtin_bit_cast(int, x1), false, false);
  return __builtin_bit_cast(float, (int)r[0]) + __builtin_bit_cast(float, (int)r[1]);
}

// A wave-uniform 64-bit value in scalar registers.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint64_t u = (uint64_t)x;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// One element of the page table read through the vector memory path: its
// wait is ordered with the streaming loads (in issue order), so it does not
// hold up the scalar loads of q the way a scalar load of the table would.
// The value stays in a vector register until it is used (a read of it right
// away would wait for every load in flight).
__device__ __forceinline__ int page_entry(const int32_t *table, int idx) {
  const __amdgpu_buffer_rsrc_t r = make_rsrc(table, (uint32_t)(idx + 1) * 4u);
  return __builtin_amdgcn_raw_buffer_load_b32(r, 0, idx * 4, 0);
}

// The split phase with PFW chunk loads in flight per lane.
//
// A workgroup owns tiles j, j + nwg, j + 2 nwg, ... of its item (j is its
// index among the item's nwg workgroups) and walks them one after another
// with all four waves on the same tile: wave w takes the tile's K chunks
// 4i + w and its V steps 4i + w (i = 0 .. NC/4 - 1), so at every step the
// four waves read four adjacent chunk-rows of the tile, and at any moment the
// launch's workgroups read a compact band of each unit (tile k of every
// workgroup) rather than every tile of the layer at once.  Each wave forms
// partial logits over its channels; the four partials of a slot meet in LDS,
// where the owner of each head (wave h mod 4) adds them up and runs the
// head's online softmax, and passes the weights and the rescale factor of
// the running sums back through LDS; every wave accumulates p.v over its own
// rows.  Two workgroup barriers per tile.
template <int D, int G, int F, int PFW>
__device__ __forceinline__ void split_body(const DecodeArgs &a) {
  using Chunk = typename KvFormat<F>::Chunk;
  constexpr int EB = KvFormat<F>::kBytes;  // bytes per element
  constexpr int LB = 8 * EB;        // bytes per chunk
  constexpr int NC = D / 8;         // chunks per row
  constexpr int RPS = 64 / NC;      // rows per V step
  constexpr int NCW = NC / kWaves;  // a wave's K chunks, and V steps, per tile
  constexpr int PIECES = 2 * NCW;   // a wave's loads per tile
  // loads in flight per lane; the ring slot of a load is its piece number
  // mod PF, the same in every tile
  constexpr int PF = PFW < PIECES ? PFW : PIECES;
  constexpr int PST = SplitSmem<D, G, F>::PST;
  static_assert(NC % kWaves == 0, "the four waves share a tile's chunks");
  static_assert(PIECES % PF == 0, "ring slots repeat from tile to tile");
  static_assert(F == HWKV_KV_BF16 || F == HWKV_KV_F16, "16-bit formats (fp8: decode_mfma)");
  __shared__ SplitSmem<D, G, F> sm;

  const DecodeItems &it = a.it;
  const int blk = blockIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  // The item and its fields in one round of independent loads, lane i
  // reading item i's (entries of split_begin past the launch's items hold
  // INT32_MAX): the item is the number of items that begin at or before
  // this workgroup, less one, and its fields are read from its lane.  (A
  // search over split_begin would be a chain of dependent loads before the
  // first tile load of every workgroup.)
  static_assert(kMaxItems == 64, "one lane per item");
  const int sb_l = it.split_begin[lane];
  const int sb1_l = it.split_begin[lane + 1];
  const int nv_l = it.n_valid[lane];
  const int ns_l = it.new_slot[lane];
  const int pto_l = it.pto[lane];
  const int qrow_l = it.q_row[lane];
  const int64_t koff_l = it.k_off[lane];
  const int64_t voff_l = it.v_off[lane];
  const int item = __builtin_amdgcn_readfirstlane(__popcll(__ballot(sb_l <= blk)) - 1);
  auto pick = [&](int v) { return __builtin_amdgcn_readlane(v, item); };
  auto pick64 = [&](int64_t v) {
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)v, item);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)v >> 32), item);
    return (int64_t)(((uint64_t)hi << 32) | lo);
  };
  const int j = blk - pick(sb_l);                          // workgroup of the item
  const int nwg = pick(sb1_l) - pick(sb_l);
  const int nv = pick(nv_l);
  const int new_slot = pick(ns_l);
  const int q_row = pick(qrow_l);
  const int c8 = lane % NC;
  const int rsub = lane / NC;
  const int n_tiles = (nv + 63) / 64;
  const int pto = pick(pto_l);
  // read out of their lanes here, not under the paged test below (where the
  // compiler would otherwise move their loads, a second round trip)
  int64_t koff_i = pick64(koff_l), voff_i = pick64(voff_l);
  asm volatile("" : "+s"(koff_i), "+s"(voff_i));
  // the item's K tiles and V rows, or the page pool of a paged unit (the
  // offsets are uniform; said so, or the compiler may keep them in vector
  // registers and then fail to feed them to the scalar operands below)
  const int64_t koff = uniform64(pto >= 0 ? a.pool_off : koff_i);
  const int64_t voff = uniform64(pto >= 0 ? a.pool_off + kPageTokens * D : voff_i);
  uint8_t *const kbase = static_cast<uint8_t *>(a.cache) + koff * EB;
  uint8_t *const vbase = static_cast<uint8_t *>(a.cache) + voff * EB;

  // K tile t and the V rows of tile t (pg: its page, for a paged unit)
  auto k_tile = [&](int t, int pg) -> uint8_t * {
    if (pto >= 0)
      return kbase + (size_t)pg * 2 * kPageTokens * D * EB +
             (size_t)(t % (kPageTokens / 64)) * NC * 64 * LB;
    return kbase + (size_t)t * NC * 64 * LB;
  };
  auto v_tile = [&](int t, int pg) -> uint8_t * {
    if (pto >= 0)
      return vbase + (size_t)pg * 2 * kPageTokens * D * EB +
             (size_t)(t % (kPageTokens / 64)) * 64 * D * EB;
    return vbase + (size_t)t * 64 * D * EB;
  };
  auto page_of = [&](int t) -> int {
    return pto >= 0 ? page_entry(a.page_table, pto + t / (kPageTokens / 64)) : 0;
  };
  // K: the whole tile (slots past n_valid are masked); V: rows [0, n_valid)
  // only, so that rows past it read as zero.  A tile that does not exist
  // (has == false) gets empty descriptors: its loads return zero and touch
  // no memory, so the loads of a tile's ring are issued the same way
  // whether or not a next tile follows (a load behind a branch makes the
  // compiler copy the ring's registers where the paths meet, and a copy of
  // a register with a load in flight waits for every load in flight).
  auto k_rsrc = [&](int t, int pg, bool has = true) {
    return make_rsrc(k_tile(t, __builtin_amdgcn_readfirstlane(pg)),
                     has ? (uint32_t)(NC * 64 * LB) : 0u);
  };
  auto v_rsrc = [&](int t, int pg, bool has = true) {
    return make_rsrc(v_tile(t, __builtin_amdgcn_readfirstlane(pg)),
                     has ? (uint32_t)(min(64, nv - 64 * t) * D * EB) : 0u);
  };

  // The walk visits logical tiles; logical tile 0 is the tile that holds
  // new_slot (and that tile's logical number is 0), so that the new token's
  // tile is always the first tile of workgroup 0, which stores the token
  // before any of its waves read.  The order of the tiles does not change
  // the softmax.
  const int tile_new = new_slot >= 0 ? new_slot / 64 : 0;
  auto phys = [&](int lt) {
    return __builtin_amdgcn_readfirstlane(lt == 0 ? tile_new : (lt == tile_new ? 0 : lt));
  };
  // fused append: workgroup 0 stores the new token first; its waves then
  // read it from the cache like any other slot
  // (the same condition as new_slot >= 0 && j == 0, made explicitly uniform:
  // written plainly, the compiler fails with an illegal VGPR to SGPR copy)
  const bool writes_new =
      __builtin_amdgcn_readfirstlane((int)(new_slot >= 0 && j == 0)) != 0;
  if (writes_new && threadIdx.x < 2 * NC) {
    const int tn = new_slot / 64;
    const int pg = pto >= 0 ? a.page_table[pto + tn / (kPageTokens / 64)] : 0;
    const size_t src = (size_t)it.kv_row[item] * D;
    if (threadIdx.x < NC) {
      const int g = threadIdx.x;
      store_chunk<F>(k_tile(tn, pg) + ((size_t)g * 64 + new_slot % 64) * LB,
                     encode8<F>(*reinterpret_cast<const uint4 *>(a.k_new + src + g * 8),
                                it.k_scale[item]));
    } else {
      const int g = threadIdx.x - NC;
      store_chunk<F>(v_tile(tn, pg) + (size_t)(new_slot % 64) * D * EB + g * LB,
                     encode8<F>(*reinterpret_cast<const uint4 *>(a.v_new + src + g * 8),
                                it.v_scale[item]));
    }
  }

  // The softmax of head h is run by wave h % 4 (its owner), which keeps the
  // head's running shift m and lane sums l; every wave keeps acc over its
  // own rows for every head and rescales it with the owner's factor.
  constexpr int OWN = (G + kWaves - 1) / kWaves;   // heads a wave owns, at most
  float m[OWN], l[OWN], acc[G][8];
#pragma unroll
  for (int o = 0; o < OWN; ++o) {
    m[o] = -INFINITY;
    l[o] = 0.f;
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  // the first tile (its page entry is read before q, so that waiting for it
  // does not wait for q)
  int t = j;                     // logical tile
  int tp = phys(t);              // its place in the unit
  int pg = page_of(tp);
  // binary16 keys: every head's q in one round of loads, issued before the
  // first tile's loads (a step's q is cold; its conversion below then waits
  // for q alone, not for the tile).  Buffer loads: with plain loads here the
  // compiler fails with an illegal VGPR to SGPR copy.  Lanes past D read the
  // head's last four values again (D = 64, 128), which leaves its max as is.
  constexpr int QR = (D + 255) / 256;
  uint2 w[F == HWKV_KV_F16 ? G : 1][QR];
  if constexpr (F == HWKV_KV_F16) {
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(a.q + (size_t)q_row * D, (uint32_t)(G * D * 2));
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int r = 0; r < QR; ++r) {
        const int c = min(256 * r + 4 * lane, D - 4);
        const u32x2_t x = __builtin_amdgcn_raw_buffer_load_b64(qr, (h * D + c) * 2, 0, 0);
        w[h][r] = make_uint2(x.x, x.y);
      }
  }
  // Only this workgroup reads the new slot in this launch: a workgroup-scope
  // release/acquire around the barrier orders the store before its loads
  // (agent scope would write back and invalidate the whole L2).
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");

  // per-lane parts of the piece addresses (the step is in soffset)
  const int kl = lane * LB;                    // K: lane = slot
  const int vl = rsub * D * EB + c8 * LB;      // V: row rsub of the step, 8 channels
  // piece q of a tile: K chunk 4q + w, or V step 4(q - NCW) + w.  Both are
  // 64 LB bytes long (a K chunk of 64 slots; RPS rows of D elements), so the
  // offset of piece q is (4 (q mod NCW) + w) 64 LB: the wave's part is in
  // wso (an SGPR), the step's part an immediate added to it.
  static_assert(RPS * D * EB == 64 * LB, "K chunks and V steps are equally long");
  const int wso = wave * 64 * LB;
  auto ld = [&](__amdgpu_buffer_rsrc_t kr, __amdgpu_buffer_rsrc_t vr, auto qc) -> Chunk {
    constexpr int q = decltype(qc)::value;
    constexpr int step = kWaves * (q % NCW) * 64 * LB;
    int so = wso;
    asm volatile("" : "+s"(so));   // one SGPR add per load, not one SGPR per piece
    if constexpr (q < NCW)
      return bload_chunk<F>(kr, kl, so + step);
    else
      return bload_chunk<F>(vr, vl, so + step);
  };
  // q chunk c of head h is qw[h NC + c - wave] (the wave's chunks are
  // c = 4i + wave)
  const cu32x4_t *const qw = (const cu32x4_t *)(a.q + (size_t)q_row * D) + wave;
  float *const pl = sm.u.t.p;

  __amdgpu_buffer_rsrc_t krs = k_rsrc(tp, pg), vrs = v_rsrc(tp, pg);
  // q is read through scalar loads during the walk, and a step's q is cold
  // (in HBM).  One vector load per lane touching its own 64-byte piece of
  // the item's q, issued with the first tile's loads, brings q's lines into
  // L2 in the shadow of those loads; the value is only consumed at the end
  // of the kernel, so nothing waits for it early.  (Binary16 keys stage q
  // through LDS instead.)
  uint32_t qtouch = 0;
  if constexpr (F != HWKV_KV_F16)
    qtouch = reinterpret_cast<const uint32_t *>(a.q + (size_t)q_row * D)[min(lane * 16, G * D / 2 - 1)];
  Chunk buf[PF];
  static_for<PF>([&](auto jc) { buf[jc.value] = ld(krs, vrs, jc); });
  // binary16 keys: q goes to LDS as binary16, head h scaled by the power of
  // two 2^sh that puts its largest |q| in [2^14, 2^15), so that every
  // component within a factor 2^31 of it converts exactly; the head's logit
  // scale takes 2^-sh back (sh is capped so that the scale stays normal).
  // The keys' binary16 pairs then meet q in v_dot2_f32_f16 (exact products,
  // fp32 sums), as bf16 keys meet q in v_dot2_f32_bf16.
  if constexpr (F == HWKV_KV_F16) {
    int ez;
    (void)frexpf(a.scale_log2, &ez);
#pragma unroll
    for (int h = 0; h < G; ++h) {
      if (h % kWaves != wave) continue;   // wave h % 4 stages head h
      float mx = 0.0f;
#pragma unroll
      for (int r = 0; r < QR; ++r)
        mx = fmaxf(mx, fmaxf(fmaxf(fabsf(bf_lo(w[h][r].x)), fabsf(bf_hi(w[h][r].x))),
                             fmaxf(fabsf(bf_lo(w[h][r].y)), fabsf(bf_hi(w[h][r].y)))));
      mx = wave_max(mx);
      int ex;
      (void)frexpf(mx, &ex);               // mx in [2^(ex-1), 2^ex)
      const int sh = __builtin_amdgcn_readfirstlane(min(mx > 0.0f ? 15 - ex : 0, ez + 120));
#pragma unroll
      for (int r = 0; r < QR; ++r) {
        const int c = 256 * r + 4 * lane;
        if (c < D) {
          const uint2 x = w[h][r];
          const f16x2_t lo = {(_Float16)ldexpf(bf_lo(x.x), sh), (_Float16)ldexpf(bf_hi(x.x), sh)};
          const f16x2_t hi = {(_Float16)ldexpf(bf_lo(x.y), sh), (_Float16)ldexpf(bf_hi(x.y), sh)};
          *reinterpret_cast<uint2 *>(&sm.q16[(h * D + c) / 2]) =
              make_uint2(__builtin_bit_cast(uint32_t, lo), __builtin_bit_cast(uint32_t, hi));
        }
      }
      if (lane == 0) sm.qsc[h] = ldexpf(a.scale_log2, -sh);
    }
    // LDS only: the tile's loads stay in flight across this barrier
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
  }
  // logit scale (base 2); binary16 keys: the scale of each head the wave
  // owns, with its q shift taken back
  const float zscale = a.scale_log2;
  float zsc[OWN];
#pragma unroll
  for (int o = 0; o < OWN; ++o) {
    const int h = min(wave + kWaves * o, G - 1);
    zsc[o] = F == HWKV_KV_F16 ? __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                                               __builtin_bit_cast(int, sm.qsc[h])))
                              : zscale;
  }
  for (int k = 0;; ++k) {
    const bool has_next = t + nwg < n_tiles;
    // the next tile and its page: its first PF loads are issued during the
    // last PF pieces of this tile, with descriptors built at those loads
    // (so that they are not live, beside q, through the whole tile)
    const int tn = has_next ? t + nwg : -1;
    const int tnp = has_next ? phys(tn) : 0;
    const int pgn = has_next ? page_of(tnp) : 0;
    // after consuming piece q, issue the load PF pieces later in the stream
    auto issue = [&](auto qc) {
      constexpr int q = decltype(qc)::value;
      constexpr int qn = q + PF;
      if constexpr (qn < PIECES) {
        buf[q % PF] = ld(krs, vrs, std::integral_constant<int, qn>{});
      } else {
        int tt = tnp;
        asm volatile("" : "+s"(tt));   // descriptors built here, not kept live
        buf[q % PF] = ld(k_rsrc(tt, pgn, has_next), v_rsrc(tt, pgn, has_next),
                         std::integral_constant<int, qn - PIECES>{});
      }
    };
    uint64_t qaddr = (uint64_t)qw;
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = 0.f;

    // ---- partial q.k over the wave's chunks.  The empty asm statements make
    // the accumulators and the q address opaque at each step boundary, so
    // that every step issues its own loads and does its own arithmetic,
    // instead of the compiler hoisting a tile's loads and spilling.  q chunks
    // are read one step ahead of their use (scalar loads; q is uniform).
    // (8 q heads, or binary16 keys, whose q is widened to fp32 SGPRs: no
    // double buffer, its SGPRs do not fit beside the rest)
#ifndef HWKV_DECODE_QAHEAD
#define HWKV_DECODE_QAHEAD 0
#endif
    constexpr bool QAHEAD = HWKV_DECODE_QAHEAD && G < 8 && F != HWKV_KV_F16;
    u32x4_t qc[G];
    if constexpr (QAHEAD) {
#pragma unroll
      for (int h = 0; h < G; ++h) qc[h] = qw[h * NC];
    }
    static_for<NCW>([&](auto jc) {
      constexpr int q = decltype(jc)::value;
#pragma unroll
      for (int h = 0; h < G; ++h) asm volatile("" : "+v"(s[h]));
      asm volatile("" : "+s"(qaddr));
      const Chunk x = buf[q % PF];
      issue(jc);
      const cu32x4_t *qj = (const cu32x4_t *)qaddr;
      if constexpr (!QAHEAD && F != HWKV_KV_F16) {
#pragma unroll
        for (int h = 0; h < G; ++h) qc[h] = qj[h * NC + kWaves * q];
      }
      u32x4_t qn[G];
      if constexpr (QAHEAD && q + 1 < NCW) {
#pragma unroll
        for (int h = 0; h < G; ++h) qn[h] = qj[h * NC + kWaves * (q + 1)];
      }
      if constexpr (F == HWKV_KV_BF16) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          s[h] = dot2(qc[h].x, x.x, s[h]);
          s[h] = dot2(qc[h].y, x.y, s[h]);
          s[h] = dot2(qc[h].z, x.z, s[h]);
          s[h] = dot2(qc[h].w, x.w, s[h]);
        }
      } else {
        // binary16 keys: q chunk (kWaves q + wave) of head h from LDS (one
        // address for every lane: a broadcast read).  The 16-byte vectors are
        // reinterpreted whole and split into pairs by shuffles: bit-casting
        // single elements of the u32x4 vector instead made this toolchain
        // feed the first element to all four products.
        const u32x4_t *q16 = reinterpret_cast<const u32x4_t *>(sm.q16) + kWaves * q + wave;
        const f16x8_t kv = __builtin_bit_cast(f16x8_t, u32x4_t{x.x, x.y, x.z, x.w});
#pragma unroll
        for (int h = 0; h < G; ++h) {
          const f16x8_t qv = __builtin_bit_cast(f16x8_t, q16[h * NC]);
          s[h] = __builtin_amdgcn_fdot2(__builtin_shufflevector(qv, qv, 0, 1),
                                        __builtin_shufflevector(kv, kv, 0, 1), s[h], false);
          s[h] = __builtin_amdgcn_fdot2(__builtin_shufflevector(qv, qv, 2, 3),
                                        __builtin_shufflevector(kv, kv, 2, 3), s[h], false);
          s[h] = __builtin_amdgcn_fdot2(__builtin_shufflevector(qv, qv, 4, 5),
                                        __builtin_shufflevector(kv, kv, 4, 5), s[h], false);
          s[h] = __builtin_amdgcn_fdot2(__builtin_shufflevector(qv, qv, 6, 7),
                                        __builtin_shufflevector(kv, kv, 6, 7), s[h], false);
        }
      }
      if constexpr (QAHEAD && q + 1 < NCW) {
#pragma unroll
        for (int h = 0; h < G; ++h) qc[h] = qn[h];
      }
    });

    // ---- the four partial logits of each slot meet in LDS (buffers
    // alternate with the tile, so one barrier per tile suffices for them: a
    // wave can only reach this tile's buffer again after every wave has
    // passed the next tile's barrier, i.e. after every owner has read it)
#pragma unroll
    for (int h = 0; h < G; ++h) sm.u.t.lg[k & 1][h][wave][lane] = s[h];
    __syncthreads();

    // ---- online softmax, base 2, of the heads this wave owns
    const bool valid = 64 * tp + lane < nv;
#pragma unroll
    for (int o = 0; o < OWN; ++o) {
      const int h = wave + kWaves * o;
      if (h < G) {  // uniform
        float z = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) z += sm.u.t.lg[k & 1][h][w][lane];  // fixed order
        z = valid ? z * zsc[o] : -INFINITY;
        const float mnew = fmaxf(m[o], wave_max(z));
        float alpha = 1.0f;
        if (mnew > m[o]) {  // uniform
          alpha = exp2f(m[o] - mnew);
          l[o] *= alpha;
          m[o] = mnew;
        }
        const float p = exp2f(z - mnew);
        l[o] += p;
        pl[lane * PST + h] = p;
        if (lane == 0) sm.alpha[h] = alpha;
      }
    }
    __syncthreads();
    // every wave rescales its sums of the heads whose shift moved
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float alpha = __builtin_bit_cast(
          float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, sm.alpha[h])));
      if (alpha != 1.0f) {  // uniform
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= alpha;
      }
    }

    // ---- p.v over the wave's V steps (rows (4i + w) RPS + rsub)
    // p of a step's row is read from LDS one step ahead (pc: this step,
    // pn: the next), so the LDS latency overlaps a step of work
    float pc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) pc[h] = pl[(wave * RPS + rsub) * PST + h];
    static_for<NCW>([&](auto jc) {
      constexpr int i = decltype(jc)::value;
      constexpr int q = NCW + i;
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          asm volatile("" : "+v"(acc[h][e]), "+v"(acc[h][e + 1]));
      const Chunk x = buf[q % PF];
      issue(std::integral_constant<int, q>{});
      float pn[G];
      if constexpr (i + 1 < NCW) {
#pragma unroll
        for (int h = 0; h < G; ++h)
          pn[h] = pl[((kWaves * (i + 1) + wave) * RPS + rsub) * PST + h];
      }
      float vf[8];
      widen8<F>(x, vf);
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pc[h], vf[e], acc[h][e]);
      if constexpr (i + 1 < NCW) {
#pragma unroll
        for (int h = 0; h < G; ++h) pc[h] = pn[h];
      }
    });
    if (!has_next) break;
    t = tn;
    tp = tnp;
    pg = pgn;
    krs = k_rsrc(tp, pg);
    vrs = v_rsrc(tp, pg);
  }

  // ---- the workgroup's partial.  Each head's owner gives its shift m and
  // normaliser l (the lane sums added up); every wave applied the owners'
  // rescale factors to its sums, so acc, which holds each wave's own rows,
  // is summed as it is: over the lanes that share a channel chunk (lane,
  // lane ^ NC, ..., lane ^ 32 -- the last step pairs channel e with e + 4 in
  // one lane swap, so lanes 0..31 end with channels 0..3 and lanes 32..63
  // with channels 4..7 of their chunk), then over the waves in LDS.
#pragma unroll
  for (int o = 0; o < OWN; ++o) {
    const int h = wave + kWaves * o;
    if (h < G) {  // uniform
      const float lh = wave_sum(l[o]);
      if (lane == 0) {
        sm.m[h] = m[o];
        sm.l[h] = lh;
      }
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int off = 16; off >= NC; off >>= 1)
        acc[h][e] += __shfl_xor(acc[h][e], off);
    }
  }
  const int half = lane >> 5;
  float red[G][4];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[h][e] = half_sum_pair(acc[h][e], acc[h][e + 4]);
  if ((lane & 31) < NC) {
#pragma unroll
    for (int h = 0; h < G; ++h)
      *reinterpret_cast<float4 *>(&sm.u.acc[wave][h][c8 * 8 + 4 * half]) =
          make_float4(red[h][0], red[h][1], red[h][2], red[h][3]);
  }
  __syncthreads();

  const int pidx = it.ws_split0 + blk;   // this workgroup's partial
  for (int idx = threadIdx.x; idx < G * D / 4; idx += kWaves * 64) {
    const int h = idx / (D / 4), c = (idx % (D / 4)) * 4;
    float4 A = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float4 x = *reinterpret_cast<const float4 *>(&sm.u.acc[w][h][c]);
      A.x += x.x;
      A.y += x.y;
      A.z += x.z;
      A.w += x.w;
    }
    const float L = sm.l[h];
    // streaming (non-temporal) stores: nothing here is read again by this
    // kernel
    if (nwg == 1) {
      const float inv = 1.0f / L;
      __builtin_nontemporal_store(f32x4_t{A.x * inv, A.y * inv, A.z * inv, A.w * inv},
                                  reinterpret_cast<f32x4_t *>(&a.out[((size_t)q_row + h) * D + c]));
    } else {
      __builtin_nontemporal_store(
          f32x4_t{A.x, A.y, A.z, A.w},
          reinterpret_cast<f32x4_t *>(&a.part_acc[((size_t)pidx * G + h) * D + c]));
      if (c == 0)
        __builtin_nontemporal_store(
            f32x2_t{sm.m[h], L}, reinterpret_cast<f32x2_t *>(&a.part_ml[((size_t)pidx * G + h) * 2]));
    }
  }
  asm volatile("" ::"v"(qtouch));   // the q touch above, consumed
}


template <int F>
constexpr int kSplitDepth = kPrefetch;

template <int D, int G, int F>
__global__ __launch_bounds__(kWaves * 64)
__attribute__((amdgpu_waves_per_eu(split_waves_per_eu(D, G, F)))) void decode_split(DecodeArgs a) {
  split_body<D, G, F, kSplitDepth<F>>(a);
}

// Compute units of the current device (cached per device).
inline int device_cus() {
  static int cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] <= 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n < 1)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// Calls F<D, G>::run(args...) for the runtime (D, G) of a cache.
template <template <int, int> class F, typename... Args>
hipError_t dispatch_dg(int D, int G, Args &&...args) {
#define HWKV_G(DD)                                                   \
  switch (G) {                                                       \
    case 1: return F<DD, 1>::run(args...);                           \
    case 2: return F<DD, 2>::run(args...);                           \
    case 4: return F<DD, 4>::run(args...);                           \
    case 6: return F<DD, 6>::run(args...);                           \
    case 8: return F<DD, 8>::run(args...);                           \
    default: return hipErrorInvalidValue;                            \
  }
  switch (D) {
    case 64: HWKV_G(64)
    case 128: HWKV_G(128)
    case 256: HWKV_G(256)
    default: return hipErrorInvalidValue;
  }
#undef HWKV_G
}

}  // namespace
}  // namespace hwkv

#include "decode_mfma.h"

namespace hwkv {
namespace {

template <int F>
struct SplitLaunch {
  template <int D, int G>
  struct At {
    static hipError_t run(const DecodeArgs &a, int n, hipStream_t s, hipEvent_t e0,
                          hipEvent_t e1) {
      // fp8 caches on the matrix cores (decode_mfma.h), 16-bit ones on VALU
      if constexpr (F == HWKV_KV_FP8_E4M3)
        hipExtLaunchKernelGGL((decode_mfma<D, G>), dim3(n), dim3(kWaves * 64), 0, s, e0,
                              e1, 0, a);
      else
        hipExtLaunchKernelGGL((decode_split<D, G, F>), dim3(n), dim3(kWaves * 64), 0,
                              s, e0, e1, 0, a);
      return hipGetLastError();
    }
  };
};

}  // namespace

template <int F>
hipError_t launch_decode_split_fmt(int D, int G, const DecodeArgs &a,
                                   int n_splits, hipStream_t s, hipEvent_t e0,
                                   hipEvent_t e1) {
  return dispatch_dg<SplitLaunch<F>::template At>(D, G, a, n_splits, s, e0, e1);
}

}  // namespace hwkv
