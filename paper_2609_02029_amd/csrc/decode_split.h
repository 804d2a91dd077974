// decode_split.h -- split phase of the decode attention over per-head grouped
// caches (gfx950, wave64, VALU), templated on the cache format; instantiated
// once per format by decode_split_<format>.hip.
//
// What is computed (paper: Eqs. conditional-attention-weight and
// conditional-attention, exact scaled dot-product logit): for every sequence b
// and query head qh of a layer, over the slots [0, n_valid) of KV head
// h = qh / G,
//     out = sum_s exp(z_s - m) v_s / sum_s exp(z_s - m),   z_s = scale q.k_s.
// Softmax is invariant to the order of the slots, so ring slots are read in
// slot order and never unwrapped (keys are post-RoPE, positions are not used).
//
// Work decomposition.  One launch covers the (b, h) "items" of a layer; each
// item's slots are cut into splits of kWaves * kTilesPerWave * 64 tokens and
// every split is one workgroup, so the grid is balanced by bytes, not by unit
// (full and windowed heads of one layer differ by up to ~56x in length).  The
// G query heads of an item share every K/V byte read.  A split is one page
// of a paged full unit, whose workgroup reads that page only.
//
// Inside a wave, per 64-slot tile (one stream of chunk-sized buffer loads per
// lane -- 16 bytes, or 8 for fp8 -- with kPrefetch, or kPrefetch8, loads
// always in flight):
//   q.k   one lane per slot: the K tile is stored slot-minor in 8-element
//         channel chunks, so chunk g of the tile is contiguous and lane t
//         reads its own slot's chunk; q is uniform and comes through scalar
//         loads.  bf16 keys: v_dot2_f32_bf16 multiplies bf16 pairs (q as an
//         SGPR operand) with fp32 accumulate; fp8 keys are first widened to
//         bf16 pairs (exact: every E4M3 value is a bf16 value) and take the
//         same path, with the K scale folded into the logit scale; binary16
//         keys meet the fp32-widened q in fp32 FMAs.  No cross-lane
//         reduction is needed for the logits.
//   softmax  online, base 2 (log2(e) folded into the scale); the tile max is
//         one DPP row reduction plus four lane reads per head.
//   p.v   lanes own 8 channels of one row (V row-major, a wave reads whole
//         rows contiguously); p is broadcast through a per-wave LDS slice.
//         bf16 and binary16 values are widened to fp32 (exactly) and take
//         one fp32 FMA per (row, channel, head) with the fp32 weights; fp8
//         values go over token pairs in binary16 (v_dot2_f32_f16, the
//         weights rounded to binary16, the normaliser in fp32), and the fp8
//         V scale multiplies the workgroup's result.
//         The V buffer descriptor ends at row n_valid, so rows past it read
//         as zero (and their p is zero).
// The fused append writes the new token, in the cache format, into its slot
// at the start of the one workgroup whose split holds that slot, before any
// of its waves read.
// The waves of a workgroup are merged in LDS; a split either writes the final
// output (single-split items) or a partial (m, l, acc) that the combine
// kernel merges: m* = max m_j, l* = sum l_j 2^(m_j - m*),
// out = sum acc_j 2^(m_j - m*) / l*.
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

// Split geometry and load batching (compile-time; see decode_split_tokens).
#ifndef HWKV_DECODE_WAVES
#define HWKV_DECODE_WAVES 4
#endif
#ifndef HWKV_DECODE_TPW
#define HWKV_DECODE_TPW 1
#endif
#ifndef HWKV_DECODE_PREFETCH
#define HWKV_DECODE_PREFETCH 4     // 16-byte chunk loads in flight
#endif
#ifndef HWKV_DECODE_PREFETCH8
#define HWKV_DECODE_PREFETCH8 8    // 8-byte (fp8) chunk loads in flight
#endif
#ifndef HWKV_DECODE_AUX
#define HWKV_DECODE_AUX 2  // cache-policy bits of the streaming loads (nt)
#endif
#ifndef HWKV_DECODE_MINWAVES
#define HWKV_DECODE_MINWAVES 4
#endif
#ifndef HWKV_DECODE_ROT
#define HWKV_DECODE_ROT 7  // a tile's starting step: (ROT * tile) mod steps
#endif
constexpr int kWaves = HWKV_DECODE_WAVES;        // waves per workgroup
constexpr int kTilesPerWave = HWKV_DECODE_TPW;   // 64-slot tiles per wave
constexpr int kPrefetch = HWKV_DECODE_PREFETCH;  // 16-byte loads in flight
constexpr int kPrefetch8 = HWKV_DECODE_PREFETCH8;  // 8-byte loads in flight
constexpr int kMinWavesPerEU = HWKV_DECODE_MINWAVES;  // VGPR budget
// A split is one page of a paged full unit: its workgroup reads one page.
static_assert(kWaves * kTilesPerWave * kTile == kPageTokens && kTilesPerWave == 1,
              "a decode split must be one page of 4 tiles, one per wave");

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
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

// fp8 codes 2i, 2i + 1 of a word as one binary16 pair (exact: every E4M3
// value is a binary16 value), low code first.
template <bool HI>
__device__ __forceinline__ f16x2_t fp8x2_f16x2(uint32_t w) {
  return __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(w, 1.0f, HI);
}

// The 8 elements of a V chunk widened to fp32 (exact for every format).
template <int F>
__device__ __forceinline__ void widen8(typename KvFormat<F>::Chunk x, float (&vf)[8]) {
  if constexpr (F == HWKV_KV_BF16) {
    vf[0] = bf_lo(x.x); vf[1] = bf_hi(x.x); vf[2] = bf_lo(x.y); vf[3] = bf_hi(x.y);
    vf[4] = bf_lo(x.z); vf[5] = bf_hi(x.z); vf[6] = bf_lo(x.w); vf[7] = bf_hi(x.w);
  } else if constexpr (F == HWKV_KV_F16) {
    vf[0] = h_lo(x.x); vf[1] = h_hi(x.x); vf[2] = h_lo(x.y); vf[3] = h_hi(x.y);
    vf[4] = h_lo(x.z); vf[5] = h_hi(x.z); vf[6] = h_lo(x.w); vf[7] = h_hi(x.w);
  } else {
    const f32x2_t a0 = __builtin_amdgcn_cvt_pk_f32_fp8(x.x, false);
    const f32x2_t a1 = __builtin_amdgcn_cvt_pk_f32_fp8(x.x, true);
    const f32x2_t a2 = __builtin_amdgcn_cvt_pk_f32_fp8(x.y, false);
    const f32x2_t a3 = __builtin_amdgcn_cvt_pk_f32_fp8(x.y, true);
    vf[0] = a0.x; vf[1] = a0.y; vf[2] = a1.x; vf[3] = a1.y;
    vf[4] = a2.x; vf[5] = a2.y; vf[6] = a3.x; vf[7] = a3.y;
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

template <int D, int G>
struct SplitSmem {
  static constexpr int NC = D / 8;
  static constexpr int PST = (G + 3) & ~3;  // p stride per slot
  float m[kWaves][G];
  float l[kWaves][G];
  float p[kWaves][64 * PST];                // per-wave p broadcast, tile loop
  __attribute__((aligned(16))) float acc[kWaves][G][D];   // per-wave partials
};

// x of lane l and x of lane l ^ 32 for two values at once (VALU lane swap):
// returns x0 + x0' in lanes 0..31 and x1 + x1' in lanes 32..63.
__device__ __forceinline__ float half_sum_pair(float x0, float x1) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, x0),
                                                  __builtin_bit_cast(int, x1), false, false);
  return __builtin_bit_cast(float, (int)r[0]) + __builtin_bit_cast(float, (int)r[1]);
}

// The split phase with PFW chunk loads in flight per lane; instantiated by
// decode_split (the default depth) and decode_split_deep (twice as deep).
template <int D, int G, int F, int PFW>
__device__ __forceinline__ void split_body(const DecodeArgs &a) {
  using Chunk = typename KvFormat<F>::Chunk;
  constexpr int EB = KvFormat<F>::kBytes;  // bytes per element
  constexpr int LB = 8 * EB;        // bytes per chunk
  constexpr int NC = D / 8;         // chunks per row
  constexpr int RPS = 64 / NC;      // rows per wave step in p.v
  constexpr int PST = SplitSmem<D, G>::PST;
  // loads in flight per lane (at most one tile's K chunks); the ring slot of
  // a load is its step number mod PF across tiles, so PF must divide 2 NC.
  // 8-byte loads keep twice as many in flight, for the same bytes.
  constexpr int PF = PFW < NC ? PFW : NC;
  // fp8 values: p.v over token pairs with v_dot2_f32_f16 -- a lane's two
  // consecutive p.v steps read rows r and r + RPS of the same channels, whose
  // codes widen exactly to binary16 pairs; the weights enter the product
  // rounded to binary16 (the normaliser keeps the fp32 weights)
  constexpr bool PAIR = F == HWKV_KV_FP8_E4M3;
  static_assert(NC % 2 == 0, "p.v steps come in pairs");
  static_assert((2 * NC) % PF == 0, "prefetch depth must divide 2 NC");
  __shared__ SplitSmem<D, G> sm;

  const DecodeItems &it = a.it;
  const int blk = blockIdx.x;
  int lo = 0, hi = it.n_items - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (it.split_begin[mid] <= blk)
      lo = mid;
    else
      hi = mid - 1;
  }
  const int item = lo;
  const int split = blk - it.split_begin[item];
  const int nsplit = it.split_begin[item + 1] - it.split_begin[item];
  const int nv = it.n_valid[item];
  const int new_slot = it.new_slot[item];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int c8 = lane % NC;
  const int rsub = lane / NC;

  // Region this workgroup reads: the item's rows, or for a paged unit the
  // page of this split (rows r0 .. r0 + 255 of the unit); every address
  // below is relative to the region's first row r0.
  uint8_t *kbase, *vbase;
  int r0 = 0, rows = nv;
  if (it.pto[item] >= 0) {
    const int64_t pg = a.page_table[it.pto[item] + split];
    kbase = static_cast<uint8_t *>(a.cache) +
            (a.pool_off + pg * 2 * kPageTokens * D) * EB;
    vbase = kbase + kPageTokens * D * EB;
    r0 = split * kPageTokens;
    rows = min(nv - r0, kPageTokens);
  } else {
    kbase = static_cast<uint8_t *>(a.cache) + it.k_off[item] * EB;
    vbase = static_cast<uint8_t *>(a.cache) + it.v_off[item] * EB;
  }
  // q is uniform across the workgroup: read it through the scalar path
  // (constant address space), so v_dot2 takes it as an SGPR operand
  const cu32x4_t *qc = (const cu32x4_t *)(a.q + (size_t)it.q_row[item] * D);
  // Tiles of the item are dealt to its waves with a stride: wave wl of the
  // item's nw waves takes tiles wl, wl + nw, ...  At any moment the item's
  // waves then read a compact window of the cache instead of one far-apart
  // region each, which keeps the DRAM traffic local.
  const int n_tiles = (nv + 63) / 64;
  const int nw = nsplit * kWaves;
  const int wl = split * kWaves + wave;
  // fused append: the workgroup that reads new_slot stores the new token
  // first; its waves then read it from the cache like any other slot
  const bool writes_new =
      new_slot >= 0 && ((new_slot / 64) % nw) / kWaves == split;
  if (writes_new && threadIdx.x < 2 * NC) {
    const size_t src = (size_t)it.kv_row[item] * D;
    if (threadIdx.x < NC) {
      const int g = threadIdx.x;
      store_chunk<F>(
          kbase + (((size_t)((new_slot - r0) / 64) * NC + g) * 64 + new_slot % 64) * LB,
          encode8<F>(*reinterpret_cast<const uint4 *>(a.k_new + src + g * 8),
                     it.k_scale[item]));
    } else {
      const int g = threadIdx.x - NC;
      store_chunk<F>(vbase + (size_t)(new_slot - r0) * D * EB + g * LB,
                     encode8<F>(*reinterpret_cast<const uint4 *>(a.v_new + src + g * 8),
                                it.v_scale[item]));
    }
  }

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  }
  float *pl = sm.p[wave];
  // Only this workgroup reads the new slot in this launch: a workgroup-scope
  // release/acquire around the barrier orders the store before its loads
  // (agent scope would write back and invalidate the whole L2).
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");

  // K: every tile up to the last occupied one; V: rows [0, nv) only
  const __amdgpu_buffer_rsrc_t krs =
      make_rsrc(kbase, (uint32_t)(((rows + 63) / 64) * 64 * D * EB));
  const __amdgpu_buffer_rsrc_t vrs = make_rsrc(vbase, (uint32_t)(rows * D * EB));
  // logit scale (base 2), with the fp8 K scale folded in
  const float zscale =
      F == HWKV_KV_FP8_E4M3 ? a.scale_log2 * it.k_scale[item] : a.scale_log2;

  // Each tile is a stream of 2 NC chunk loads per lane: NC K chunks (one
  // lane per slot), then NC steps of V rows (lanes own channel slices).  It
  // is consumed with PF loads always in flight: the V loads of a tile are on
  // their way while its last K chunks and the softmax are computed, and the
  // first K loads of the wave's next tile while its last V rows are.
  //
  // The wave walks its tile's K chunks, and its V rows, from a tile-dependent
  // starting step and wraps round (the q chunks and the weights follow).
  // Every wave starts at the same moment; without the rotation all of them
  // would read the same offset of tiles a whole tile apart at each step,
  // which crowds their requests onto a few HBM channels.  The V steps keep
  // the fp8 token pairs (steps 2s, 2s + 1) together.
  auto rot_k = [](int tile) { return (HWKV_DECODE_ROT * tile) & (NC - 1); };
  auto rot_v = [](int tile) { return (HWKV_DECODE_ROT * tile) & (NC - 1) & (PAIR ? ~1 : ~0); };
  Chunk buf[PF];
  int t = wl;
  int rk = rot_k(t), rv = rot_v(t);
  int kofs = (t * 64 - r0) * D * EB + lane * LB;
  if (t < n_tiles) static_for<PF>([&](auto jc) {
    buf[jc.value] = bload_chunk<F>(krs, kofs, ((jc.value + rk) & (NC - 1)) * 64 * LB);
  });
  for (int k = 0; k < kTilesPerWave && t < n_tiles; ++k) {
    const int slot0 = t * 64;
    const int slot = slot0 + lane;
    const int tn = t + nw;
    const bool has_next = k + 1 < kTilesPerWave && tn < n_tiles;
    int rk_n = rot_k(tn);
    int vofs = (slot0 - r0 + rsub) * D * EB + c8 * LB;
    int kofs_n = (tn * 64 - r0) * D * EB + lane * LB;
    uint64_t qaddr = (uint64_t)qc;
    // load j of this tile's stream: K chunk (j + rk) mod NC, or V step
    // (j - NC + rv) mod NC; V's descriptor ends at row n_valid, so the
    // rows past it read as zero
    auto ld = [&](auto jc) -> Chunk {
      constexpr int j = decltype(jc)::value;
      if constexpr (j < NC)   // K: the chunk step is uniform
        return bload_chunk<F>(krs, kofs, ((j + rk) & (NC - 1)) * 64 * LB);
      else
        return bload_chunk<F>(vrs, vofs + ((j - NC + rv) & (NC - 1)) * RPS * D * EB);
    };
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = 0.f;

    // ---- q.k, one K chunk per step.  The empty asm statements make the
    // accumulators, the offsets and the q address opaque at each step
    // boundary, so that every step issues its own loads (one load PF steps
    // ahead, the step's q chunk) and does its own arithmetic, instead of the
    // compiler hoisting the loads of the whole tile and spilling.
    // q chunks are read one step ahead of their use (qc: this step's chunk,
    // qn: the next one), so the scalar-load latency overlaps a step of work.
    u32x4_t qc[G];
    {
      const cu32x4_t *q0 = (const cu32x4_t *)qaddr;
#pragma unroll
      for (int h = 0; h < G; ++h) qc[h] = q0[h * NC + rk];
    }
    static_for<NC>([&](auto jc) {
      constexpr int j = decltype(jc)::value;
#pragma unroll
      for (int h = 0; h < G; ++h) asm volatile("" : "+v"(s[h]));
      asm volatile("" : "+v"(kofs), "+v"(vofs), "+s"(qaddr), "+s"(rk), "+s"(rv));
      const Chunk x = buf[j % PF];
      buf[j % PF] = ld(std::integral_constant<int, j + PF>{});
      u32x4_t qn[G];
      if constexpr (j + 1 < NC) {
        const cu32x4_t *qj = (const cu32x4_t *)qaddr;
        const int qi = (j + 1 + rk) & (NC - 1);
#pragma unroll
        for (int h = 0; h < G; ++h) qn[h] = qj[h * NC + qi];
      }
      if constexpr (F == HWKV_KV_BF16) {
#pragma unroll
        for (int h = 0; h < G; ++h) {
          s[h] = dot2(qc[h].x, x.x, s[h]);
          s[h] = dot2(qc[h].y, x.y, s[h]);
          s[h] = dot2(qc[h].z, x.z, s[h]);
          s[h] = dot2(qc[h].w, x.w, s[h]);
        }
      } else if constexpr (F == HWKV_KV_FP8_E4M3) {
        const uint32_t k0 = fp8x2_bf16x2<false>(x.x), k1 = fp8x2_bf16x2<true>(x.x);
        const uint32_t k2 = fp8x2_bf16x2<false>(x.y), k3 = fp8x2_bf16x2<true>(x.y);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          s[h] = dot2(qc[h].x, k0, s[h]);
          s[h] = dot2(qc[h].y, k1, s[h]);
          s[h] = dot2(qc[h].z, k2, s[h]);
          s[h] = dot2(qc[h].w, k3, s[h]);
        }
      } else {
        float kf[8];
        widen8<F>(x, kf);
#pragma unroll
        for (int h = 0; h < G; ++h) {
          s[h] = fmaf(bf_lo(qc[h].x), kf[0], s[h]);
          s[h] = fmaf(bf_hi(qc[h].x), kf[1], s[h]);
          s[h] = fmaf(bf_lo(qc[h].y), kf[2], s[h]);
          s[h] = fmaf(bf_hi(qc[h].y), kf[3], s[h]);
          s[h] = fmaf(bf_lo(qc[h].z), kf[4], s[h]);
          s[h] = fmaf(bf_hi(qc[h].z), kf[5], s[h]);
          s[h] = fmaf(bf_lo(qc[h].w), kf[6], s[h]);
          s[h] = fmaf(bf_hi(qc[h].w), kf[7], s[h]);
        }
      }
      if constexpr (j + 1 < NC) {
#pragma unroll
        for (int h = 0; h < G; ++h) qc[h] = qn[h];
      }
    });

    // ---- online softmax, base 2 (the first V loads are already in flight)
    const bool valid = slot < nv;
    // token-pair order of the binary16 weights: token t is half (t / RPS) % 2
    // of pair (t / 2 RPS) RPS + t % RPS, whose G weights are G dwords
    const int ppid = (lane / (2 * RPS)) * RPS + lane % RPS;
    const int phalf = (lane / RPS) & 1;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float z = valid ? s[h] * zscale : -INFINITY;
      const float mnew = fmaxf(m[h], wave_max(z));
      if (mnew > m[h]) {  // uniform
        const float alpha = exp2f(m[h] - mnew);
        l[h] *= alpha;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] *= alpha;
        m[h] = mnew;
      }
      const float p = exp2f(z - mnew);
      l[h] += p;
      if constexpr (PAIR)
        reinterpret_cast<_Float16 *>(pl)[2 * (ppid * G + h) + phalf] = (_Float16)p;
      else
        pl[lane * PST + h] = p;
    }

    // ---- p.v, one step of RPS rows per step; lanes own channels 8 c8 ..
    auto issue = [&](auto jc) {  // the load PF steps after step j
      constexpr int j = decltype(jc)::value;
      constexpr int jn = j + PF;
      if constexpr (jn < 2 * NC) {
        buf[j % PF] = ld(std::integral_constant<int, jn>{});
      } else {
        if (has_next)
          buf[j % PF] = bload_chunk<F>(krs, kofs_n, ((jn - 2 * NC + rk_n) & (NC - 1)) * 64 * LB);
      }
    };
    if constexpr (PAIR) {
      // steps 2s and 2s + 1 read rows r = rsub + 2s RPS and r + RPS: the
      // first step keeps its chunk and reads the pair's weights (so the LDS
      // latency overlaps a step), the second builds the binary16 pairs
      // (v_r[c], v_r+RPS[c]) and takes one v_dot2 per (head, channel)
      const uint32_t *pp = reinterpret_cast<const uint32_t *>(pl);
      int pofs = rsub * G;
      uint32_t pw[G];
      Chunk xp;
      static_for<NC>([&](auto jc) {
        constexpr int js = decltype(jc)::value;
        constexpr int j = NC + js;
#pragma unroll
        for (int h = 0; h < G; ++h)
#pragma unroll
          for (int e = 0; e < 8; e += 2)
            asm volatile("" : "+v"(acc[h][e]), "+v"(acc[h][e + 1]));
        asm volatile("" : "+v"(vofs), "+v"(kofs_n), "+v"(pofs), "+s"(rv), "+s"(rk_n));
        const Chunk x = buf[j % PF];
        issue(std::integral_constant<int, j>{});
        if constexpr (js % 2 == 0) {
          xp = x;
          const int pi = ((js + rv) & (NC - 1)) / 2;   // the step pair's weights
#pragma unroll
          for (int h = 0; h < G; ++h) pw[h] = pp[pofs + pi * RPS * G + h];
        } else {
          const uint32_t w0 = __builtin_amdgcn_perm(x.x, xp.x, 0x05010400u);
          const uint32_t w1 = __builtin_amdgcn_perm(x.x, xp.x, 0x07030602u);
          const uint32_t w2 = __builtin_amdgcn_perm(x.y, xp.y, 0x05010400u);
          const uint32_t w3 = __builtin_amdgcn_perm(x.y, xp.y, 0x07030602u);
          const f16x2_t v[8] = {fp8x2_f16x2<false>(w0), fp8x2_f16x2<true>(w0),
                                fp8x2_f16x2<false>(w1), fp8x2_f16x2<true>(w1),
                                fp8x2_f16x2<false>(w2), fp8x2_f16x2<true>(w2),
                                fp8x2_f16x2<false>(w3), fp8x2_f16x2<true>(w3)};
#pragma unroll
          for (int h = 0; h < G; ++h) {
            const f16x2_t ph = __builtin_bit_cast(f16x2_t, pw[h]);
#pragma unroll
            for (int e = 0; e < 8; ++e)
              acc[h][e] = __builtin_amdgcn_fdot2(ph, v[e], acc[h][e], false);
          }
        }
      });
    } else {
    // p of a step's rows is read from LDS one step ahead (pc: this step,
    // pn: the next), so the LDS latency overlaps a step of work.
    int pofs = rsub * PST;
    float pc[G];
#pragma unroll
    for (int h = 0; h < G; ++h) pc[h] = pl[pofs + (rv & (NC - 1)) * RPS * PST + h];
    static_for<NC>([&](auto jc) {
      constexpr int js = decltype(jc)::value;
      constexpr int j = NC + js;
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; e += 2)
          asm volatile("" : "+v"(acc[h][e]), "+v"(acc[h][e + 1]));
      asm volatile("" : "+v"(vofs), "+v"(kofs_n), "+v"(pofs), "+s"(rv), "+s"(rk_n));
      const Chunk x = buf[j % PF];
      issue(std::integral_constant<int, j>{});
      float pn[G];
      if constexpr (js + 1 < NC) {
        const int pi = (js + 1 + rv) & (NC - 1);
#pragma unroll
        for (int h = 0; h < G; ++h) pn[h] = pl[pofs + pi * RPS * PST + h];
      }
      float vf[8];
      widen8<F>(x, vf);
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pc[h], vf[e], acc[h][e]);
      if constexpr (js + 1 < NC) {
#pragma unroll
        for (int h = 0; h < G; ++h) pc[h] = pn[h];
      }
    });
    }
    t = tn;
    kofs = kofs_n;
    rk = rk_n;
    rv = rot_v(tn);
  }

  // ---- wave partials: l over all lanes; acc over the lanes that share a
  // channel chunk (lane, lane ^ NC, ..., lane ^ 32).  The last step pairs
  // channel e with e + 4 in one lane swap, so lanes 0..31 end with channels
  // 0..3 and lanes 32..63 with channels 4..7 of their chunk.
#pragma unroll
  for (int h = 0; h < G; ++h) {
    l[h] = wave_sum(l[h]);
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
      *reinterpret_cast<float4 *>(&sm.acc[wave][h][c8 * 8 + 4 * half]) =
          make_float4(red[h][0], red[h][1], red[h][2], red[h][3]);
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      sm.m[wave][h] = m[h];
      sm.l[wave][h] = l[h];
    }
  }
  __syncthreads();

  // ---- merge the waves (wave 0 of every split has at least one tile), 4
  // channels per thread and step
  float *part = a.ws + (size_t)(it.ws_split0 + blk) * (G * (D + 2));
  const float vsc = F == HWKV_KV_FP8_E4M3 ? it.v_scale[item] : 1.0f;
  for (int idx = threadIdx.x; idx < G * D / 4; idx += kWaves * 64) {
    const int h = idx / (D / 4), c = (idx % (D / 4)) * 4;
    float M = sm.m[0][h];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sm.m[w][h]);
    float L = 0.f;
    float4 A = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = exp2f(sm.m[w][h] - M);
      L += sm.l[w][h] * f;
      const float4 x = *reinterpret_cast<const float4 *>(&sm.acc[w][h][c]);
      A.x += x.x * f;
      A.y += x.y * f;
      A.z += x.z * f;
      A.w += x.w * f;
    }
    if constexpr (F == HWKV_KV_FP8_E4M3) {  // the V scale of the codes
      A.x *= vsc;
      A.y *= vsc;
      A.z *= vsc;
      A.w *= vsc;
    }
    if (nsplit == 1) {
      const float inv = 1.0f / L;
      *reinterpret_cast<float4 *>(&a.out[((size_t)it.q_row[item] + h) * D + c]) =
          make_float4(A.x * inv, A.y * inv, A.z * inv, A.w * inv);
    } else {
      float *dst = &part[2 * G + h * D + c];
      if constexpr ((2 * G) % 4 == 0) {     // partial records 16-byte aligned
        *reinterpret_cast<float4 *>(dst) = A;
      } else {
        dst[0] = A.x;
        dst[1] = A.y;
        dst[2] = A.z;
        dst[3] = A.w;
      }
      if (c == 0) {
        part[h] = M;
        part[G + h] = L;
      }
    }
  }
}


template <int F>
constexpr int kSplitDepth = KvFormat<F>::kBytes == 2 ? kPrefetch : kPrefetch8;

template <int D, int G, int F>
__global__ __launch_bounds__(kWaves * 64)
__attribute__((amdgpu_waves_per_eu(kMinWavesPerEU))) void decode_split(DecodeArgs a) {
  split_body<D, G, F, kSplitDepth<F>>(a);
}

// For launches with fewer split workgroups than CUs: the chip is not full,
// so each wave keeps twice as many loads in flight.  (With the chip full the
// default depth is faster: the arithmetic between loads is what the other
// resident waves hide.)
template <int D, int G, int F>
__global__ __launch_bounds__(kWaves * 64)
__attribute__((amdgpu_waves_per_eu(kMinWavesPerEU))) void decode_split_deep(DecodeArgs a) {
  split_body<D, G, F, 2 * kSplitDepth<F>>(a);
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

template <int F>
struct SplitLaunch {
  template <int D, int G>
  struct At {
    static hipError_t run(const DecodeArgs &a, int n, hipStream_t s, hipEvent_t e0,
                          hipEvent_t e1) {
      // (8 q heads per kv head: the deeper ring does not fit the registers)
      if constexpr (G < 8) {
        if (n < device_cus()) {
          hipExtLaunchKernelGGL((decode_split_deep<D, G, F>), dim3(n), dim3(kWaves * 64), 0,
                                s, e0, e1, 0, a);
          return hipGetLastError();
        }
      }
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
