// write_kernels.hip -- prefill materialisation and ring-buffer append into
// the per-head grouped cache (gfx950).  Chunk copies of 8 elements, stored in
// the cache format (kv_format.h); the only other arithmetic is the
// slot <-> position map.
//
// Retained set of a finite unit at length n: {p < S} U {p >= n - w} (the
// paper's J_t(w) window plus an additive sink prefix); slot(p) = p for full
// units and sinks, S + ((p - S) mod w) otherwise.  After materialising the
// chunk [p0, p1) a ring slot j >= S holds the one position
// p in [p1 - w, p1) with p = j (mod w), namely p = b + ((j - b) mod w) with
// b = p1 - w, provided p >= S; the chunk writes slot j iff that p lies in
// [p0, p1).  Iterating over destination slots makes every K tile write a
// full, coalesced chunk-per-lane store and never touches slots the chunk
// does not own, so prefill never forms a full-length cache.
#include <algorithm>

#include "hwkv_internal.h"
#include "kv_format.h"

namespace hwkv {
namespace {

// One workgroup per (destination tile, kv head): 64 slots x D channels.
template <int D, int F>
__global__ __launch_bounds__(256) void prefill_write(WriteArgs a) {
  constexpr int NC = D / 8;
  constexpr int EB = KvFormat<F>::kBytes;
  constexpr int LB = 8 * EB;
  __shared__ int64_t src_row[kTile];  // source row of each slot, or -1
  const int h = blockIdx.y;
  const WriteHead &wh = a.head[h];
  int x = blockIdx.x, tile = -1;
#pragma unroll
  for (int r = 0; r < 3; ++r) {
    if (tile < 0) {
      if (x < wh.n_tiles[r])
        tile = wh.tile0[r] + x;
      else
        x -= wh.n_tiles[r];
    }
  }
  if (tile < 0) return;  // uniform: past this head's tiles

  const int64_t w = wh.window;
  const int64_t S = a.n_sinks;
  if (threadIdx.x < kTile) {
    const int64_t j = (int64_t)tile * kTile + threadIdx.x;
    int64_t p = -1;
    if (w == 0 || j < S) {
      p = j;
    } else if (j < S + w) {
      const int64_t b = a.p1 - w;
      int64_t r = (j - b) % w;
      if (r < 0) r += w;
      p = b + r;
      if (p < S) p = -1;
    }
    src_row[threadIdx.x] = (p >= a.p0 && p < a.p1) ? p - a.p0 : -1;
  }
  __syncthreads();

  uint8_t *const cache = static_cast<uint8_t *>(a.cache);
  uint8_t *kt, *vt;     // this tile's K tile and its first V row
  if (wh.pto >= 0) {    // paged: tile `tile % 4` of page tile / 4
    constexpr int TPP = kPageTokens / kTile;
    const int64_t pg = a.page_table[wh.pto + tile / TPP];
    const int64_t base = a.pool_off + pg * 2 * kPageTokens * D;
    kt = cache + (base + (int64_t)(tile % TPP) * kTile * D) * EB;
    vt = cache + (base + (int64_t)kPageTokens * D + (int64_t)(tile % TPP) * kTile * D) * EB;
  } else {
    kt = cache + (wh.k_off + (size_t)tile * kTile * D) * EB;
    vt = cache + (wh.v_off + (size_t)tile * kTile * D) * EB;
  }
  const size_t row_stride = (size_t)a.n_kv_heads * D;
  // K: thread -> (chunk g, slot), slot fastest: coalesced tile stores
  for (int e = threadIdx.x; e < kTile * NC; e += 256) {
    const int sl = e & (kTile - 1), g = e >> 6;
    const int64_t r = src_row[sl];
    if (r < 0) continue;
    const uint4 val =
        *reinterpret_cast<const uint4 *>(a.k + r * row_stride + h * D + g * 8);
    store_chunk<F>(kt + ((size_t)g * kTile + sl) * LB, encode8<F>(val, wh.k_scale));
  }
  // V: thread -> (slot, chunk g), chunk fastest: row-contiguous both sides
  for (int e = threadIdx.x; e < kTile * NC; e += 256) {
    const int sl = e / NC, g = e % NC;
    const int64_t r = src_row[sl];
    if (r < 0) continue;
    const uint4 val =
        *reinterpret_cast<const uint4 *>(a.v + r * row_stride + h * D + g * 8);
    store_chunk<F>(vt + (size_t)sl * D * EB + g * LB, encode8<F>(val, wh.v_scale));
  }
}

// One workgroup of 64 lanes per (sequence, kv head): lanes [0, NC) copy K
// chunks into the tile layout, lanes [NC, 2 NC) copy the V row.
template <int D, int F>
__global__ __launch_bounds__(64) void append_token(AppendArgs a) {
  constexpr int NC = D / 8;
  constexpr int EB = KvFormat<F>::kBytes;
  constexpr int LB = 8 * EB;
  const int i = blockIdx.x;
  const int t = threadIdx.x;
  const int slot = a.slot[i];
  const size_t src = (size_t)a.kv_row[i] * D;
  uint8_t *const cache = static_cast<uint8_t *>(a.cache);
  // the K region and V region holding `slot`, and its row r in them
  int64_t koff, voff;
  int r = slot;
  if (a.pto[i] >= 0) {  // paged: row slot % 256 of page slot / 256
    const int64_t pg = a.page_table[a.pto[i] + slot / kPageTokens];
    koff = a.pool_off + pg * 2 * kPageTokens * D;
    voff = koff + (int64_t)kPageTokens * D;
    r = slot % kPageTokens;
  } else {
    koff = a.k_off[i];
    voff = a.v_off[i];
  }
  if (t < NC) {
    uint8_t *kt = cache + (koff + (size_t)(r / kTile) * kTile * D) * EB;
    const uint4 val = *reinterpret_cast<const uint4 *>(a.k_new + src + t * 8);
    store_chunk<F>(kt + ((size_t)t * kTile + r % kTile) * LB,
                   encode8<F>(val, a.k_scale[i]));
  } else if (t < 2 * NC) {
    const int g = t - NC;
    const uint4 val = *reinterpret_cast<const uint4 *>(a.v_new + src + g * 8);
    store_chunk<F>(cache + (voff + (size_t)r * D) * EB + g * LB,
                   encode8<F>(val, a.v_scale[i]));
  }
}

// Installs page-table entries before the kernels that read them (kernels
// on one stream run in order, so the next launch sees the entries).
__global__ __launch_bounds__(512) void page_update(PageUpdateArgs a) {
  for (int i = threadIdx.x; i < a.n; i += 512) a.table[a.idx[i]] = a.page[i];
}

// 8 fp8 codes as 8 bf16 values (exact: every E4M3 value is a bf16 value).
__device__ __forceinline__ uint4 widen_fp8x8(uint2 c) {
  auto w = [](uint32_t x, bool hi) -> uint32_t {
    return __builtin_bit_cast(uint32_t, hi ? __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, true)
                                           : __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, false));
  };
  return make_uint4(w(c.x, false), w(c.x, true), w(c.y, false), w(c.y, true));
}

// Staging of an fp8 cache for prefill attention: the occupied rows of each
// (unit, sequence) of a layer widened to bf16 code values, in the layout of
// a bf16 cache (K tiles chunk for chunk, V rows), into an image the bf16
// kernel reads.  blockIdx.y: the unit; blockIdx.z: 0 = K, 1 = V.  Whole K
// tiles are staged (rows past the occupied ones are never read).
template <int D>
__global__ __launch_bounds__(256) void stage_units(StageArgs a) {
  constexpr int NC = D / 8;
  constexpr int TPP = kPageTokens / kTile;
  const StageUnit &su = a.unit[blockIdx.y];
  const bool isv = blockIdx.z != 0;
  const int64_t n = isv ? (int64_t)su.n_rows * NC
                        : (int64_t)((su.n_rows + kTile - 1) / kTile) * kTile * NC;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < n;
       c += (int64_t)gridDim.x * 256) {
    int64_t src;
    if (su.pto < 0) {
      src = (isv ? su.src_v_off : su.src_k_off) + c * 8;
    } else if (!isv) {          // K chunk c: tile t, position r in the tile
      const int64_t t = c / (kTile * NC), r = c % (kTile * NC);
      const int64_t pg = a.page_table[su.pto + t / TPP];
      src = a.pool_off + pg * 2 * kPageTokens * D + (t % TPP) * kTile * D + r * 8;
    } else {                    // V chunk c: row j, chunk g
      const int64_t j = c / NC, g = c % NC;
      const int64_t pg = a.page_table[su.pto + j / kPageTokens];
      src = a.pool_off + pg * 2 * kPageTokens * D + (int64_t)kPageTokens * D +
            (j % kPageTokens) * D + g * 8;
    }
    const uint2 codes = *reinterpret_cast<const uint2 *>(a.cache + src);
    *reinterpret_cast<uint4 *>(a.image + (isv ? su.dst_v_off : su.dst_k_off) + c * 8) =
        widen_fp8x8(codes);
  }
}

// The chunk's own K and V as the cache will store them: fp8 codes (code(x /
// s) of the unit's scale) widened to bf16 code values, or binary16 values.
template <int D, int F>
__global__ __launch_bounds__(256) void stage_chunk(StageChunkArgs a) {
  constexpr int NC = D / 8;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < a.n_chunks;
       c += (int64_t)gridDim.x * 256) {
    const int h = (int)((c / NC) % a.n_kv_heads);
    const uint4 k = *reinterpret_cast<const uint4 *>(a.k + c * 8);
    const uint4 v = *reinterpret_cast<const uint4 *>(a.v + c * 8);
    if constexpr (F == HWKV_KV_F16) {
      *reinterpret_cast<uint4 *>(a.k_out + c * 8) = encode8<HWKV_KV_F16>(k, 1.0f);
      *reinterpret_cast<uint4 *>(a.v_out + c * 8) = encode8<HWKV_KV_F16>(v, 1.0f);
    } else {
      *reinterpret_cast<uint4 *>(a.k_out + c * 8) =
          widen_fp8x8(encode8<HWKV_KV_FP8_E4M3>(k, a.k_scale[h]));
      *reinterpret_cast<uint4 *>(a.v_out + c * 8) =
          widen_fp8x8(encode8<HWKV_KV_FP8_E4M3>(v, a.v_scale[h]));
    }
  }
}

// Calls L<D, F>::run(args...) for the runtime (D, format).
template <template <int, int> class L, typename... Args>
hipError_t dispatch_df(int fmt, int D, Args &&...args) {
#define HWKV_F(DD)                                                        \
  switch (fmt) {                                                          \
    case HWKV_KV_BF16: return L<DD, HWKV_KV_BF16>::run(args...);          \
    case HWKV_KV_F16: return L<DD, HWKV_KV_F16>::run(args...);            \
    case HWKV_KV_FP8_E4M3: return L<DD, HWKV_KV_FP8_E4M3>::run(args...);  \
    default: return hipErrorInvalidValue;                                 \
  }
  switch (D) {
    case 64: HWKV_F(64)
    case 128: HWKV_F(128)
    case 256: HWKV_F(256)
    default: return hipErrorInvalidValue;
  }
#undef HWKV_F
}

template <int D, int F>
struct WriteLaunch {
  static hipError_t run(const WriteArgs &a, int max_tiles, hipStream_t s) {
    hipLaunchKernelGGL((prefill_write<D, F>), dim3(max_tiles, a.n_kv_heads),
                       dim3(256), 0, s, a);
    return hipGetLastError();
  }
};

template <int D, int F>
struct AppendLaunch {
  static hipError_t run(const AppendArgs &a, hipStream_t s) {
    hipLaunchKernelGGL((append_token<D, F>), dim3(a.n_items), dim3(64), 0, s, a);
    return hipGetLastError();
  }
};

}  // namespace

hipError_t launch_prefill_write(int fmt, int D, const WriteArgs &a,
                                int max_tiles, hipStream_t s) {
  return dispatch_df<WriteLaunch>(fmt, D, a, max_tiles, s);
}

hipError_t launch_append(int fmt, int D, const AppendArgs &a, hipStream_t s) {
  return dispatch_df<AppendLaunch>(fmt, D, a, s);
}

hipError_t launch_stage_units(int D, const StageArgs &a, hipStream_t s) {
  const int64_t per = 256;
  const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>((a.max_chunks + per - 1) / per, 2048)),
                  (unsigned)a.n_units, 2);
  switch (D) {
    case 64: hipLaunchKernelGGL(stage_units<64>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(stage_units<128>, grid, dim3(256), 0, s, a); break;
    case 256: hipLaunchKernelGGL(stage_units<256>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_stage_chunk(int D, const StageChunkArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>((a.n_chunks + 255) / 256, 4096)));
  if (a.fmt != HWKV_KV_F16 && a.fmt != HWKV_KV_FP8_E4M3) return hipErrorInvalidValue;
#define HWKV_SC(DD)                                                                   \
  if (a.fmt == HWKV_KV_F16)                                                           \
    hipLaunchKernelGGL((stage_chunk<DD, HWKV_KV_F16>), grid, dim3(256), 0, s, a);     \
  else                                                                                \
    hipLaunchKernelGGL((stage_chunk<DD, HWKV_KV_FP8_E4M3>), grid, dim3(256), 0, s, a)
  switch (D) {
    case 64: HWKV_SC(64); break;
    case 128: HWKV_SC(128); break;
    case 256: HWKV_SC(256); break;
    default: return hipErrorInvalidValue;
  }
#undef HWKV_SC
  return hipGetLastError();
}

hipError_t launch_page_update(const PageUpdateArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(page_update, dim3(1), dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace hwkv
