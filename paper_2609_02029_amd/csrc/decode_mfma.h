// decode_mfma.h -- split phase of the decode attention on the matrix cores
// (gfx950), for fp8-E4M3 caches.  Same work decomposition, fused append and
// partial format as decode_split (decode_split.h), which serves the 16-bit
// formats; over fp8 codes that kernel spends three times their VALU work per
// byte and is bound by it, so here the products go to the matrix cores.
//
// Wave w of the workgroup takes slots [16w, 16w + 16) of every tile and all
// of their channels, so it forms complete logits on its own and keeps its own
// online softmax: no partial logits meet in LDS and no workgroup barrier
// falls inside the walk.  Per tile:
//   S = K Q^T   v_mfma_f32_16x16x32_bf16: A = K (16 slots x 32 channels:
//               lane (g, r) holds slot r's channels 8g .. 8g + 7, one 8-byte
//               chunk load straight from the slot-minor K tile, its codes
//               widened to bf16 -- exact, every E4M3 value is a bf16 value),
//               B = Q^T (32 channels x 16 columns; column c is q head c, the
//               columns past G are zero).  Lane (g, c) ends with the logits of
//               slots 4g .. 4g + 3 for head c.
//   O += P V    v_mfma_f32_16x16x16_bf16: A = P (16 heads x 16 slots, exactly
//               the weights lane (g, c) formed), B = V (16 slots x 16
//               channels): lane (g, c) reads the codes of channel 16 vb + c in
//               rows 4g .. 4g + 3 of the wave's rows from LDS and widens them.
//               The weights go in as two bf16 terms, hi = round(p) and lo =
//               round(p - hi), which carry p to within 2^-18 of itself, with
//               fp32 accumulation.
// A wave's 16 V rows go from global memory straight into its own LDS area
// (buffer_load ... lds); K goes into registers.  The next tile's loads are
// issued as soon as this tile's K and V have been read, and run during its
// softmax and products.  At the end the four waves' (m, l, acc) are merged in
// LDS exactly (each rescaled to the largest shift) into the workgroup's
// partial; the fp8 V scale multiplies it there, and the K scale is folded
// into the logit scale.
#pragma once

// Included by decode_split.h after its helpers.

namespace hwkv {
namespace {

typedef __bf16 mbf16x8_t __attribute__((ext_vector_type(8)));
typedef short mi16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_mvoid_t;

// S += K Q^T over 32 channels (16 slots x 16 heads), bf16 operands
__device__ __forceinline__ f32x4_t mfma_kq(u32x4_t k, u32x4_t q, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(mbf16x8_t, k),
                                                 __builtin_bit_cast(mbf16x8_t, q), c, 0, 0, 0);
}

// O += P V over 16 slots (16 heads x 16 channels), bf16 operands
__device__ __forceinline__ f32x4_t mfma_pv(u32x2_t p, u32x2_t v, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(mi16x4_t, p),
                                                   __builtin_bit_cast(mi16x4_t, v), c, 0, 0, 0);
}

// Two fp32 values as a bf16 pair (round to nearest even), low first
__device__ __forceinline__ uint32_t pack_bf16x2(float x, float y) {
  const f32x2_t f = {x, y};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// 16 bytes per lane from a buffer into the LDS block of the instruction (lane
// i fills bytes [16 i, 16 i + 16) of it); reads past the descriptor's range
// return zero.  (A device function of its own: written in the kernel body,
// the builtin keeps the host pass from emitting the kernel's stub.)
__device__ __forceinline__ void buf_to_lds(__amdgpu_buffer_rsrc_t r, uint8_t *lds_block,
                                           int voffset) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_mvoid_t *)lds_block, 16, voffset, 0, 0,
                                           HWKV_DECODE_AUX);
}

template <int D, int G>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(2)))
void decode_mfma(DecodeArgs a) {
  static_assert(G <= 8, "the epilogue keeps G <= 8 heads of acc per wave");
  constexpr int F = HWKV_KV_FP8_E4M3;
  constexpr int EB = 1;                // bytes per element
  constexpr int LB = 8;                // bytes per (chunk, slot) of a K tile
  constexpr int NC = D / 8;            // chunks per slot
  constexpr int KB = D / 32;           // K products per tile and wave
  constexpr int VB = D / 16;           // 16-channel blocks of the output
  constexpr int VROW = D * EB;         // bytes per V row
  constexpr int VW = 16 * VROW;        // a wave's 16 V rows of a tile
  constexpr int VLD = VW / 1024;       // direct loads per wave and tile (1 KiB each)
  static_assert(VW % 1024 == 0, "whole 1-KiB loads");
  // a wave's area: its V rows during the walk, its acc in the epilogue
  constexpr int AW = VW > G * D * 4 ? VW : G * D * 4;
  __shared__ __attribute__((aligned(1024))) uint8_t vsm[kWaves * AW];
  __shared__ float sml[kWaves][2][8];

  const DecodeItems &it = a.it;
  const int blk = blockIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int g4 = lane >> 4, l16 = lane & 15;
  // the item: one round of lane loads, as in decode_split
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
  const int j = blk - pick(sb_l);
  const int nwg = pick(sb1_l) - pick(sb_l);
  const int nv = pick(nv_l);
  const int new_slot = pick(ns_l);
  const int q_row = pick(qrow_l);
  const int n_tiles = (nv + 63) / 64;
  const int pto = pick(pto_l);
  int64_t koff_i = pick64(koff_l), voff_i = pick64(voff_l);
  asm volatile("" : "+s"(koff_i), "+s"(voff_i));
  const int64_t koff = uniform64(pto >= 0 ? a.pool_off : koff_i);
  const int64_t voff = uniform64(pto >= 0 ? a.pool_off + kPageTokens * D : voff_i);
  uint8_t *const kbase = static_cast<uint8_t *>(a.cache) + koff * EB;
  uint8_t *const vbase = static_cast<uint8_t *>(a.cache) + voff * EB;
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
  // only, so that rows past it read as zero; a tile that does not exist gets
  // empty descriptors (its loads return zero and touch no memory)
  auto k_rsrc = [&](int t, int pg, bool has) {
    return make_rsrc(k_tile(t, __builtin_amdgcn_readfirstlane(pg)),
                     has ? (uint32_t)(NC * 64 * LB) : 0u);
  };
  auto v_rsrc = [&](int t, int pg, bool has) {
    return make_rsrc(v_tile(t, __builtin_amdgcn_readfirstlane(pg)),
                     has ? (uint32_t)(min(64, nv - 64 * t) * D * EB) : 0u);
  };
  // logical tile 0 is the tile that holds new_slot (see decode_split)
  const int tile_new = new_slot >= 0 ? new_slot / 64 : 0;
  auto phys = [&](int lt) {
    return __builtin_amdgcn_readfirstlane(lt == 0 ? tile_new : (lt == tile_new ? 0 : lt));
  };
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

  // the first tile, and q: lane (g, c) holds head c's channels 32 cb + 8 g ..
  // + 7 for every 32-channel block cb (zero for c >= G); buffer loads, issued
  // before the barrier and consumed after the first tile's loads
  int t = j;
  int tp = phys(t);
  int pg = page_of(tp);
  u32x4_t qb[KB];
  {
    const __amdgpu_buffer_rsrc_t qr =
        make_rsrc(a.q + (size_t)q_row * D, (uint32_t)(G * D * 2));
    const int qo = (l16 < G ? l16 * D * 2 : G * D * 2) + 16 * g4;   // past the range: zero
#pragma unroll
    for (int cb = 0; cb < KB; ++cb)
      qb[cb] = __builtin_amdgcn_raw_buffer_load_b128(qr, qo + 64 * cb, 0, 0);
  }
  // a wave's V area starts zeroed, so that no row of it ever holds bits that
  // were not loaded from the cache (rows past n_valid read as zero anyway)
  {
    uint4 *z = reinterpret_cast<uint4 *>(vsm + wave * AW);
#pragma unroll
    for (int i = 0; i < VW / 1024; ++i) z[i * 64 + lane] = make_uint4(0u, 0u, 0u, 0u);
  }
  // only this workgroup reads the new slot in this launch (see decode_split)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");

  // per-lane load offsets: K chunk 4 cb + g of slot 16 w + c; the wave's V
  // rows, contiguous in the tile and in its LDS area (direct load n, lane i:
  // bytes n KiB + 16 i of both)
  const int kl = ((g4 * 64) + 16 * wave + l16) * LB;
  const int vsrc = 16 * wave * VROW + 16 * lane;
  // codes of row 4 g + i, channel 16 vb + c: byte i VROW + 16 vb of vrd
  const uint8_t *const vrd = vsm + wave * AW + 4 * g4 * VROW + l16;

  uint2 kreg[KB];
  auto issue = [&](int tq, int pq, bool has) {
    const __amdgpu_buffer_rsrc_t kr = k_rsrc(tq, pq, has);
    const __amdgpu_buffer_rsrc_t vr = v_rsrc(tq, pq, has);
#pragma unroll
    for (int cb = 0; cb < KB; ++cb)
      kreg[cb] = bload_chunk<F>(kr, kl + cb * 4 * 64 * LB, 0);
#pragma unroll
    for (int n = 0; n < VLD; ++n) buf_to_lds(vr, vsm + wave * AW + n * 1024, vsrc + n * 1024);
  };
  issue(tp, pg, true);

  // logit scale (base 2) with the K scale of the codes
  const float zs = a.scale_log2 * it.k_scale[item];

  // the lane's head c: running shift m (base 2, lazily raised: the weights
  // stay below 2^8) and the sum of its slots' weights
  float m = -1e30f, lsum = 0.0f;
  f32x4_t o[VB];
#pragma unroll
  for (int vb = 0; vb < VB; ++vb) o[vb] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (;;) {
    const bool has_next = t + nwg < n_tiles;
    const int tn = has_next ? t + nwg : t;
    const int tnp = phys(tn);
    const int pgn = has_next ? page_of(tnp) : 0;
    // S = K Q^T
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < KB; ++cb) {   // the codes of 8 channels as bf16 (exact)
      const u32x4_t kx = {fp8x2_bf16x2<false>(kreg[cb].x), fp8x2_bf16x2<true>(kreg[cb].x),
                          fp8x2_bf16x2<false>(kreg[cb].y), fp8x2_bf16x2<true>(kreg[cb].y)};
      s = mfma_kq(kx, qb[cb], s);
    }
    // this tile's V: the four codes of channel 16 vb + c in rows 4 g ..
    // 4 g + 3, as bf16
    u32x2_t vr[VB];
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) {
      const uint32_t w = (uint32_t)vrd[16 * vb] | ((uint32_t)vrd[VROW + 16 * vb] << 8) |
                         ((uint32_t)vrd[2 * VROW + 16 * vb] << 16) |
                         ((uint32_t)vrd[3 * VROW + 16 * vb] << 24);
      vr[vb] = u32x2_t{fp8x2_bf16x2<false>(w), fp8x2_bf16x2<true>(w)};
    }
    // both consumed (the LDS reads complete) before the next tile's loads
    // overwrite the registers and the LDS area
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) asm volatile("" ::"v"(vr[vb]) : "memory");
    issue(tnp, pgn, has_next);

    // online softmax of the lane's head over its four slots
    const int slot0 = 64 * tp + 16 * wave + 4 * g4;
    float z[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) z[i] = slot0 + i < nv ? s[i] * zs : -INFINITY;
    float mx = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (__any(mx > m + 8.0f)) {
      const float mn = fmaxf(m, mx);
      const float alpha = exp2f(m - mn);
      m = mn;
      lsum *= alpha;
      // acc rows are heads 4 g + r: their factors come from lanes 4 g + r
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float al = __shfl(alpha, 4 * g4 + r);
#pragma unroll
        for (int vb = 0; vb < VB; ++vb) o[vb][r] *= al;
      }
    }
    float p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[i] = exp2f(z[i] - m);
      lsum += p[i];
    }
    // the weights as hi + lo bf16 terms
    u32x2_t ph, pl;
    ph.x = pack_bf16x2(p[0], p[1]);
    ph.y = pack_bf16x2(p[2], p[3]);
    pl.x = pack_bf16x2(p[0] - bf_lo(ph.x), p[1] - bf_hi(ph.x));
    pl.y = pack_bf16x2(p[2] - bf_lo(ph.y), p[3] - bf_hi(ph.y));
#pragma unroll
    for (int vb = 0; vb < VB; ++vb) {
      o[vb] = mfma_pv(ph, vr[vb], o[vb]);
      o[vb] = mfma_pv(pl, vr[vb], o[vb]);
    }
    if (!has_next) break;
    t = tn;
    tp = tnp;
    pg = pgn;
  }

  // ---- the workgroup's partial: every wave's (m, l, acc) in its own area
  // (after the last, empty, loads have landed), then an exact merge
  __builtin_amdgcn_s_waitcnt(0);
  float lt = lsum + __shfl_xor(lsum, 16);
  lt += __shfl_xor(lt, 32);
  if (lane < G) {
    sml[wave][0][lane] = m;
    sml[wave][1][lane] = lt;
  }
  float *const accw = reinterpret_cast<float *>(vsm + wave * AW);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int h = 4 * g4 + r;
    if (h < G) {
#pragma unroll
      for (int vb = 0; vb < VB; ++vb) accw[h * D + 16 * vb + l16] = o[vb][r];
    }
  }
  __syncthreads();

  const int pidx = it.ws_split0 + blk;
  const float vsc = it.v_scale[item];
  for (int idx = threadIdx.x; idx < G * D / 4; idx += kWaves * 64) {
    const int h = idx / (D / 4), c = (idx % (D / 4)) * 4;
    float M = sml[0][0][h];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sml[w][0][h]);
    float L = 0.f;
    float4 A = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = exp2f(sml[w][0][h] - M);
      const float4 x =
          *reinterpret_cast<const float4 *>(vsm + w * AW + ((size_t)h * D + c) * 4);
      L += sml[w][1][h] * f;
      A.x += x.x * f;
      A.y += x.y * f;
      A.z += x.z * f;
      A.w += x.w * f;
    }
    A.x *= vsc;   // the V scale of the codes
    A.y *= vsc;
    A.z *= vsc;
    A.w *= vsc;
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
            f32x2_t{M, L}, reinterpret_cast<f32x2_t *>(&a.part_ml[((size_t)pidx * G + h) * 2]));
    }
  }
}

}  // namespace
}  // namespace hwkv
