// probe_kernels.hip -- read-bandwidth probes for the decode roofline (gfx950).
//
// Loads only, non-temporal (the split kernel's cache policy): the loaded
// words are folded into one value, which is written to *sink only if it
// equals an impossible pattern, so the loads stay.
//  * flat: consecutive wavefronts read consecutive 1 KiB pieces (16 bytes a
//    lane) and stride by the whole grid, PF loads in flight per lane.  At
//    any moment the grid reads one compact window of the buffer: the
//    practical ceiling of a streaming read.
//  * tiles: the decode split kernel's walk without its arithmetic.  One
//    64 KiB tile per wavefront (32 KiB of K then 32 KiB of V: 64 slots at
//    head_dim 256 in bf16), four wavefronts per workgroup on consecutive
//    tiles, the 32 chunk loads of each half from step 7t mod 32 on, PF
//    loads in flight (4 in the split kernel).
#include "hwkv_internal.h"

namespace hwkv {
namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// a load in flight stays a whole 16-byte value until it is consumed (a fold
// at issue would wait for it there); non-temporal, as the split kernel's
// streaming loads are
__device__ __forceinline__ u32x4_t load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 2);
}
__device__ __forceinline__ uint32_t fold(u32x4_t v) { return v.x ^ v.y ^ v.z ^ v.w; }

constexpr uint32_t kImpossible = 0x9e3779b9u;

template <int PF>
__global__ __launch_bounds__(256) void probe_flat(const ProbeArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int nw = gridDim.x * 4;
  const int pieces = (int)(a.bytes >> 10);
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t *>(a.buf), (short)0, (int)a.bytes, 0x00020000);
  const int n = w < pieces ? (pieces - w + nw - 1) / nw : 0;   // this wave's pieces
  uint32_t acc = 0;
  u32x4_t buf[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i)
    buf[i] = i < n ? load16(r, (w + i * nw) * 1024 + lane * 16) : u32x4_t{0, 0, 0, 0};
  for (int i0 = 0; i0 < n; i0 += PF) {
#pragma unroll
    for (int i = 0; i < PF; ++i) {
      acc ^= fold(buf[i]);
      const int j = i0 + i + PF;
      buf[i] = j < n ? load16(r, (w + j * nw) * 1024 + lane * 16) : u32x4_t{0, 0, 0, 0};
    }
  }
  if (acc == kImpossible) a.sink[0] = 1.0f;
}

template <int PF>
__global__ __launch_bounds__(256) void probe_tiles(const ProbeArgs a) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ntiles = (int)(a.bytes >> 16);
  if (t >= ntiles) return;                           // uniform per wave
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t *>(a.buf), (short)0, (int)a.bytes, 0x00020000);
  const int rot = (7 * t) & 31;
  int base = t * 65536 + lane * 16;
  auto off = [&](int j) {                            // load j of the tile's 64
    const int half = j >> 5, step = ((j & 31) + rot) & 31;
    return base + half * 32768 + step * 1024;
  };
  uint32_t acc = 0;
  u32x4_t buf[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i) buf[i] = load16(r, off(i));
#pragma unroll
  for (int j = 0; j < 64; ++j) {
    // opaque at each step, as in the split kernel: one load issued per step,
    // PF in flight, rather than the tile's loads hoisted together
    asm volatile("" : "+v"(base), "+v"(acc));
    acc ^= fold(buf[j % PF]);
    if (j + PF < 64) buf[j % PF] = load16(r, off(j + PF));
  }
  if (acc == kImpossible) a.sink[0] = 1.0f;
}

}  // namespace

hipError_t launch_probe(const ProbeArgs &a, int n_cus, hipStream_t s) {
  if (a.pattern == 1) {                            // waves_per_simd: loads in flight
    const dim3 grid((unsigned)(((a.bytes >> 16) + 3) / 4)), block(256);
    switch (a.waves_per_simd) {
      case 2: hipLaunchKernelGGL(probe_tiles<2>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(probe_tiles<4>, grid, block, 0, s, a); break;
      case 8: hipLaunchKernelGGL(probe_tiles<8>, grid, block, 0, s, a); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  // 4 SIMDs per CU, 4 wavefronts per workgroup: waves_per_simd workgroups per CU
  const dim3 grid((unsigned)(n_cus * a.waves_per_simd)), block(256);
  switch (a.waves_per_simd) {
    case 2: hipLaunchKernelGGL(probe_flat<4>, grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL(probe_flat<2>, grid, block, 0, s, a); break;
    case 8: hipLaunchKernelGGL(probe_flat<1>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hwkv
