// read_probe.hip -- read-bandwidth probes beside the decode roofline
// (gfx950); measurement tooling, built into its own library
// (_lib/libhwkv_probe.so), which the benchmark's probe workload loads.  Not
// part of the runtime's ABI.
//
//   int hwkv_read_probe(const void *buf, int64_t bytes, int32_t pattern,
//                       int32_t depth, float *sink, void *stream);
//
// One pass of 16-byte non-temporal loads (the decode split kernel's cache
// policy) over bytes [0, bytes) of the device buffer `buf`, enqueued on
// `stream`.  Loads only: the loaded words are folded into one value, written
// to *sink only if it equals an impossible pattern, so the loads stay.
//   pattern 0  flat grid-stride sweep: consecutive wavefronts read
//              consecutive 1 KiB pieces and stride by the grid; `depth`
//              (2, 4 or 8) wavefronts per SIMD of the device, 8 / depth
//              loads in flight per lane.  At any moment the grid reads one
//              compact window of the buffer: the practical ceiling of a
//              streaming read.
//   pattern 1  the decode split kernel's walk without its arithmetic: the
//              buffer's first half stands for the K tiles (32 KiB each), its
//              second half for the V rows of the same tiles; two workgroups
//              of four wavefronts per CU, workgroup j walking tiles j,
//              j + G, ... with the four wavefronts on the same tile
//              (wavefront w: K chunks 4i + w, then V steps 4i + w, 1 KiB
//              each); `depth` (2, 4 or 8) loads in flight per lane (the
//              split kernel keeps 4).
// buf and sink are device pointers; bytes a positive multiple of 65,536
// below 2^31.  Returns 0, 1 (invalid argument) or 5 (launch error).
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

struct ProbeArgs {
  const uint8_t *buf;
  int64_t bytes;                 // a multiple of 64 KiB below 2^31
  float *sink;                   // written only for an impossible fold
};

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

// The cooperative strided walk: 16 pieces of 1 KiB per wavefront per tile
// (8 K chunks, 8 V steps); the ring of PF loads runs on into the next tile.
template <int PF>
__global__ __launch_bounds__(256) void probe_walk(const ProbeArgs a) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ntiles = (int)(a.bytes >> 16);
  const int half = ntiles * 32768;               // K tiles, then V rows
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t *>(a.buf), (short)0, (int)a.bytes, 0x00020000);
  int t = blockIdx.x;
  if (t >= ntiles) return;                       // uniform per workgroup
  auto off = [&](int tile, int q) {              // piece q of a tile (0..15)
    return (q < 8 ? 0 : half) + tile * 32768 + (4 * (q & 7) + w) * 1024 + lane * 16;
  };
  uint32_t acc = 0;
  u32x4_t buf[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i) buf[i] = load16(r, off(t, i));
  for (;;) {
    const int tn = t + (int)gridDim.x;
    const bool more = tn < ntiles;
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      asm volatile("" : "+v"(acc));
      acc ^= fold(buf[q % PF]);
      if (q + PF < 16) {
        buf[q % PF] = load16(r, off(t, q + PF));
      } else {
        // a tile that does not exist reads past the range: zero, no traffic
        buf[q % PF] = load16(r, more ? off(tn, q + PF - 16) : (int)a.bytes);
      }
    }
    __syncthreads();                             // the split kernel's tile barrier
    if (!more) break;
    t = tn;
  }
  if (acc == kImpossible) a.sink[0] = 1.0f;
}

}  // namespace

extern "C" int hwkv_read_probe(const void *buf, int64_t bytes, int32_t pattern,
                               int32_t depth, float *sink, void *stream) {
  if (!buf || !sink) return 1;
  if (bytes <= 0 || bytes % 65536 != 0 || bytes > (int64_t)INT32_MAX) return 1;
  if (pattern != 0 && pattern != 1) return 1;
  if (depth != 2 && depth != 4 && depth != 8) return 1;
  int dev = 0, n_cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n_cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      n_cus < 1)
    return 5;
  const ProbeArgs a{static_cast<const uint8_t *>(buf), bytes, sink};
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 block(256);
  if (pattern == 1) {
    const dim3 grid((unsigned)(2 * n_cus));
    switch (depth) {
      case 2: hipLaunchKernelGGL(probe_walk<2>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(probe_walk<4>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(probe_walk<8>, grid, block, 0, s, a); break;
    }
  } else {
    // 4 SIMDs per CU, 4 wavefronts per workgroup: depth workgroups per CU
    const dim3 grid((unsigned)(n_cus * depth));
    switch (depth) {
      case 2: hipLaunchKernelGGL(probe_flat<4>, grid, block, 0, s, a); break;
      case 4: hipLaunchKernelGGL(probe_flat<2>, grid, block, 0, s, a); break;
      default: hipLaunchKernelGGL(probe_flat<1>, grid, block, 0, s, a); break;
    }
  }
  return hipGetLastError() == hipSuccess ? 0 : 5;
}
