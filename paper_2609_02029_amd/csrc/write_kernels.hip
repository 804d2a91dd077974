// write_kernels.hip -- prefill materialisation and ring-buffer append into
// the per-head grouped cache (gfx950).  Pure 16-byte copies; the only
// arithmetic is the slot <-> position map.
//
// Retained set of a finite unit at length n: {p < S} U {p >= n - w} (the
// paper's J_t(w) window plus an additive sink prefix); slot(p) = p for full
// units and sinks, S + ((p - S) mod w) otherwise.  After materialising the
// chunk [p0, p1) a ring slot j >= S holds the one position
// p in [p1 - w, p1) with p = j (mod w), namely p = b + ((j - b) mod w) with
// b = p1 - w, provided p >= S; the chunk writes slot j iff that p lies in
// [p0, p1).  Iterating over destination slots makes every K tile write a
// full, coalesced 16-byte-per-lane store and never touches slots the chunk
// does not own, so prefill never forms a full-length cache.
#include "hwkv_internal.h"

namespace hwkv {
namespace {

// One workgroup per (destination tile, kv head): 64 slots x D channels.
template <int D>
__global__ __launch_bounds__(256) void prefill_write(WriteArgs a) {
  constexpr int NC = D / 8;
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

  uint16_t *kt = a.cache + wh.k_off + (size_t)tile * kTile * D;
  uint16_t *vt = a.cache + wh.v_off + (size_t)tile * kTile * D;
  const size_t row_stride = (size_t)a.n_kv_heads * D;
  // K: thread -> (chunk g, slot), slot fastest: coalesced tile stores
  for (int e = threadIdx.x; e < kTile * NC; e += 256) {
    const int sl = e & (kTile - 1), g = e >> 6;
    const int64_t r = src_row[sl];
    if (r < 0) continue;
    const uint4 val =
        *reinterpret_cast<const uint4 *>(a.k + r * row_stride + h * D + g * 8);
    *reinterpret_cast<uint4 *>(kt + ((size_t)g * kTile + sl) * 8) = val;
  }
  // V: thread -> (slot, chunk g), chunk fastest: row-contiguous both sides
  for (int e = threadIdx.x; e < kTile * NC; e += 256) {
    const int sl = e / NC, g = e % NC;
    const int64_t r = src_row[sl];
    if (r < 0) continue;
    const uint4 val =
        *reinterpret_cast<const uint4 *>(a.v + r * row_stride + h * D + g * 8);
    *reinterpret_cast<uint4 *>(vt + (size_t)sl * D + g * 8) = val;
  }
}

// One workgroup of 64 lanes per (sequence, kv head): lanes [0, NC) copy K
// chunks into the tile layout, lanes [NC, 2 NC) copy the V row.
template <int D>
__global__ __launch_bounds__(64) void append_token(AppendArgs a) {
  constexpr int NC = D / 8;
  const int i = blockIdx.x;
  const int t = threadIdx.x;
  const int slot = a.slot[i];
  const size_t src = (size_t)a.kv_row[i] * D;
  if (t < NC) {
    uint16_t *kt = a.cache + a.k_off[i] + (size_t)(slot / kTile) * kTile * D;
    const uint4 val = *reinterpret_cast<const uint4 *>(a.k_new + src + t * 8);
    *reinterpret_cast<uint4 *>(kt + ((size_t)t * kTile + slot % kTile) * 8) =
        val;
  } else if (t < 2 * NC) {
    const int g = t - NC;
    const uint4 val = *reinterpret_cast<const uint4 *>(a.v_new + src + g * 8);
    *reinterpret_cast<uint4 *>(a.cache + a.v_off[i] + (size_t)slot * D +
                               g * 8) = val;
  }
}

}  // namespace

hipError_t launch_prefill_write(int D, const WriteArgs &a, int max_tiles,
                                hipStream_t s) {
  const dim3 grid(max_tiles, a.n_kv_heads);
  switch (D) {
    case 64: hipLaunchKernelGGL(prefill_write<64>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(prefill_write<128>, grid, dim3(256), 0, s, a); break;
    case 256: hipLaunchKernelGGL(prefill_write<256>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_append(int D, const AppendArgs &a, hipStream_t s) {
  switch (D) {
    case 64: hipLaunchKernelGGL(append_token<64>, dim3(a.n_items), dim3(64), 0, s, a); break;
    case 128: hipLaunchKernelGGL(append_token<128>, dim3(a.n_items), dim3(64), 0, s, a); break;
    case 256: hipLaunchKernelGGL(append_token<256>, dim3(a.n_items), dim3(64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hwkv
