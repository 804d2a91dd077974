// decode_kernels.hip -- merge phase of the split-K decode attention, and the
// launchers of both phases.  The split kernel (decode_split.h) is compiled
// once per cache format, in decode_split_<format>.hip.
#include "decode_split.h"

#include <algorithm>

namespace hwkv {

// Instantiated in the per-format sources.
extern template hipError_t launch_decode_split_fmt<HWKV_KV_BF16>(
    int, int, const DecodeArgs &, int, hipStream_t, hipEvent_t, hipEvent_t);
extern template hipError_t launch_decode_split_fmt<HWKV_KV_F16>(
    int, int, const DecodeArgs &, int, hipStream_t, hipEvent_t, hipEvent_t);
extern template hipError_t launch_decode_split_fmt<HWKV_KV_FP8_E4M3>(
    int, int, const DecodeArgs &, int, hipStream_t, hipEvent_t, hipEvent_t);

namespace {

// Merge geometry (compile-time).
#ifndef HWKV_COMBINE_THREADS
#define HWKV_COMBINE_THREADS 256
#endif
#ifndef HWKV_COMBINE_CHAN
#define HWKV_COMBINE_CHAN 32
#endif
#ifndef HWKV_COMBINE_UNROLL
#define HWKV_COMBINE_UNROLL 4
#endif
constexpr int kCombineThreads = HWKV_COMBINE_THREADS;  // per merge workgroup
constexpr int kCombineChan = HWKV_COMBINE_CHAN;        // channels per workgroup
constexpr int kCombineUnroll = HWKV_COMBINE_UNROLL;  // splits per thread per round

// One workgroup per (item, query head of the group, kCombineChan-channel
// chunk).  Its threads are R rows of kCombineChan / 4 lanes, a lane owning 4
// channels (one 16-byte load per split, so a row reads whole 128-byte
// lines).  Thread (r, q) merges its channels over splits r, r + R, r + 2R,
// ...; each round issues the loads of kCombineUnroll splits before using any
// of them, so a round costs one memory round trip (R * kCombineUnroll = 128
// splits per round).  The rows are then merged: the common
// shift through LDS, the weighted sums across the rows of a wavefront by
// lane shuffles, and across the wavefronts in LDS.  The merge is a
// kernel of its own: ordering the partials of other workgroups inside the
// split kernel would need device-scope fences, which write back and
// invalidate the L2 under every workgroup's stream.
template <int D, int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine(
    DecodeArgs a) {
  constexpr int CW = kCombineChan < D ? kCombineChan : D;
  constexpr int CH = D / CW;
  constexpr int LPR = CW / 4;                     // lanes per row
  constexpr int R = kCombineThreads / LPR;        // rows
  constexpr int U = kCombineUnroll;
  constexpr int NWV = kCombineThreads / 64;      // wavefronts
  static_assert(R <= 64, "the row shifts are reduced by one wavefront");
  static_assert(64 % LPR == 0, "a row lies within one wavefront");
  __shared__ float sM[R], sL[NWV], sMx;
  __shared__ float4 sA[NWV][LPR];
  const DecodeItems &it = a.it;
  const int bid = blockIdx.x;
  const int item = bid / (G * CH);
  const int h = (bid / CH) % G;
  const int ch = bid % CH;
  if (item >= it.n_items) return;
  const int sb = it.split_begin[item];
  const int ns = it.split_begin[item + 1] - sb;
  if (ns <= 1) return;
  const int tid = threadIdx.x;
  const int r = tid / LPR, q = tid % LPR;
  const int c = ch * CW + 4 * q;
  // partial j of the item: acc row (j, h) is D floats (whole 128-byte lines
  // per row of lanes), (m, l) of (j, h) two floats
  const float *acc_base = a.part_acc + ((size_t)(it.ws_split0 + sb) * G + h) * D + c;
  const float *ml_base = a.part_ml + ((size_t)(it.ws_split0 + sb) * G + h) * 2;

  float M = -INFINITY, L = 0.f;
  float4 A = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int j0 = r; j0 < ns; j0 += R * U) {
    float mj[U], lj[U];
    float4 aj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {  // every load of the round is in flight
      const int j = min(j0 + u * R, ns - 1);
      const float2 ml = *reinterpret_cast<const float2 *>(ml_base + (size_t)j * G * 2);
      mj[u] = ml.x;
      lj[u] = ml.y;
      aj[u] = *reinterpret_cast<const float4 *>(acc_base + (size_t)j * G * D);
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (j0 + u * R >= ns) mj[u] = -INFINITY;
    float Mn = M;
#pragma unroll
    for (int u = 0; u < U; ++u) Mn = fmaxf(Mn, mj[u]);
    const float f = exp2f(M - Mn);
    L *= f;
    A.x *= f;
    A.y *= f;
    A.z *= f;
    A.w *= f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float e = exp2f(mj[u] - Mn);
      L += lj[u] * e;
      A.x += aj[u].x * e;
      A.y += aj[u].y * e;
      A.z += aj[u].z * e;
      A.w += aj[u].w * e;
    }
    M = Mn;
  }
  // rows: the common shift max_r M_r (row 0 always has a split, ns >= 2);
  // rows without a split have M_r = -inf, weight 0 and zero sums
  if (q == 0) sM[r] = M;
  __syncthreads();
  if (tid < 64) {
    float mx = tid < R ? sM[tid] : -INFINITY;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if (tid == 0) sMx = mx;
  }
  __syncthreads();
  const float f = (M == -INFINITY) ? 0.f : exp2f(M - sMx);
  L *= f;
  A.x *= f;
  A.y *= f;
  A.z *= f;
  A.w *= f;
  // sum over the rows of a wavefront (lanes q, q + LPR, ...), then over the
  // wavefronts in LDS
#pragma unroll
  for (int off = LPR; off < 64; off <<= 1) {
    L += __shfl_xor(L, off);
    A.x += __shfl_xor(A.x, off);
    A.y += __shfl_xor(A.y, off);
    A.z += __shfl_xor(A.z, off);
    A.w += __shfl_xor(A.w, off);
  }
  const int wv = tid >> 6, lane = tid & 63;
  if (lane < LPR) {
    sA[wv][lane] = A;
    if (lane == 0) sL[wv] = L;
  }
  __syncthreads();
  if (tid < LPR) {
    float Lx = 0.f;
    float4 Ax = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int w = 0; w < NWV; ++w) {
      const float4 x = sA[w][tid];
      Lx += sL[w];
      Ax.x += x.x;
      Ax.y += x.y;
      Ax.z += x.z;
      Ax.w += x.w;
    }
    const float inv = 1.0f / Lx;
    *reinterpret_cast<float4 *>(&a.out[((size_t)it.q_row[item] + h) * D + ch * CW + 4 * tid]) =
        make_float4(Ax.x * inv, Ax.y * inv, Ax.z * inv, Ax.w * inv);
  }
}

template <int D, int G>
hipError_t launch_combine_dg(const DecodeArgs &a, int n_combine,
                             hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  hipExtLaunchKernelGGL((decode_combine<D, G>), dim3(n_combine),
                        dim3(kCombineThreads), 0, s, e0, e1, 0, a);
  return hipGetLastError();
}

template <int D, int G>
struct CombineLaunch {
  static hipError_t run(const DecodeArgs &a, int n, hipStream_t s, hipEvent_t e0,
                        hipEvent_t e1) {
    return launch_combine_dg<D, G>(a, n, s, e0, e1);
  }
};

}  // namespace

int decode_workgroup_target(int fmt, int D, int G) {
  // at most one workgroup per SIMD slot the register budget holds (the fp8
  // kernel, on the matrix cores, holds two waves per SIMD)
  const int per_cu4 = fmt == HWKV_KV_FP8_E4M3
                          ? std::min(kDecodeWgPerCuX4, 8)
                          : std::min(kDecodeWgPerCuX4, 4 * split_waves_per_eu(D, G, fmt));
  return std::max(1, per_cu4 * device_cus() / 4);
}
int decode_combine_blocks_per_item(int D, int G) {
  return G * (D / (kCombineChan < D ? kCombineChan : D));
}

hipError_t launch_decode_split(int fmt, int D, int G, const DecodeArgs &a,
                               int n_splits, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
  switch (fmt) {
    case HWKV_KV_BF16:
      return launch_decode_split_fmt<HWKV_KV_BF16>(D, G, a, n_splits, s, e0, e1);
    case HWKV_KV_F16:
      return launch_decode_split_fmt<HWKV_KV_F16>(D, G, a, n_splits, s, e0, e1);
    case HWKV_KV_FP8_E4M3:
      return launch_decode_split_fmt<HWKV_KV_FP8_E4M3>(D, G, a, n_splits, s, e0, e1);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_decode_combine(int D, int G, const DecodeArgs &a,
                                 int n_combine_blocks, hipStream_t s, hipEvent_t e0,
                                 hipEvent_t e1) {
  return dispatch_dg<CombineLaunch>(D, G, a, n_combine_blocks, s, e0, e1);
}

}  // namespace hwkv
