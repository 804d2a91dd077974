// decode_kernels.hip -- merge phase of the split-K decode attention, and the
// launchers of both phases.  The split kernel (decode_split.h) is compiled
// once per cache format, in decode_split_<format>.hip.
#include "decode_split.h"

namespace hwkv {

// Instantiated in the per-format sources.
extern template hipError_t launch_decode_split_fmt<HWKV_KV_BF16>(
    int, int, const DecodeArgs &, int, hipStream_t);
extern template hipError_t launch_decode_split_fmt<HWKV_KV_F16>(
    int, int, const DecodeArgs &, int, hipStream_t);
extern template hipError_t launch_decode_split_fmt<HWKV_KV_FP8_E4M3>(
    int, int, const DecodeArgs &, int, hipStream_t);

namespace {

// One workgroup per (item, query head of the group, kCombineChan-channel
// chunk).  Thread (r, c) merges channel c of splits r, r + R, r + 2R, ...
// (R = rows of the workgroup); each round issues the loads of kCombineUnroll
// splits before using any of them, so a round costs one memory round trip.
// The rows are then merged in LDS.  The merge is a kernel of its own:
// ordering the partials of other workgroups inside the split kernel would
// need device-scope fences, which write back and invalidate the L2 under
// every workgroup's stream.
template <int D, int G>
__global__ __launch_bounds__(kCombineThreads) void decode_combine(
    DecodeArgs a) {
  constexpr int CW = kCombineChan < D ? kCombineChan : D;
  constexpr int CH = D / CW;
  constexpr int R = kCombineThreads / CW;
  constexpr int PS = G * (D + 2);
  constexpr int U = kCombineUnroll;
  __shared__ float sM[R], sL[R];
  __shared__ float sA[R][CW];
  const DecodeItems &it = a.it;
  const int bid = blockIdx.x;
  const int item = bid / (G * CH);
  const int h = (bid / CH) % G;
  const int ch = bid % CH;
  if (item >= it.n_items) return;
  const int sb = it.split_begin[item];
  const int ns = it.split_begin[item + 1] - sb;
  if (ns <= 1) return;
  const int r = threadIdx.x / CW, cl = threadIdx.x % CW;
  const int c = ch * CW + cl;
  const float *base = a.ws + (size_t)(it.ws_split0 + sb) * PS;

  float M = -INFINITY, L = 0.f, A = 0.f;
  for (int j0 = r; j0 < ns; j0 += R * U) {
    float mj[U], lj[U], aj[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {  // every load of the round is in flight
      const int j = min(j0 + u * R, ns - 1);
      const float *pj = base + (size_t)j * PS;
      mj[u] = pj[h];
      lj[u] = pj[G + h];
      aj[u] = pj[2 * G + h * D + c];
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (j0 + u * R >= ns) mj[u] = -INFINITY;
    float Mn = M;
#pragma unroll
    for (int u = 0; u < U; ++u) Mn = fmaxf(Mn, mj[u]);
    const float f = exp2f(M - Mn);
    L *= f;
    A *= f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float e = exp2f(mj[u] - Mn);
      L += lj[u] * e;
      A += aj[u] * e;
    }
    M = Mn;
  }
  if (cl == 0) {
    sM[r] = M;
    sL[r] = L;
  }
  sA[r][cl] = A;
  __syncthreads();
  if (threadIdx.x < CW) {
    float Mx = sM[0];
    for (int w = 1; w < R; ++w) Mx = fmaxf(Mx, sM[w]);
    float Lx = 0.f, Ax = 0.f;
    for (int w = 0; w < R; ++w) {
      const float f = exp2f(sM[w] - Mx);
      Lx += sL[w] * f;
      Ax += sA[w][threadIdx.x] * f;
    }
    a.out[((size_t)it.q_row[item] + h) * D + c] = Ax / Lx;
  }
}

template <int D, int G>
hipError_t launch_combine_dg(const DecodeArgs &a, int n_combine,
                             hipStream_t s) {
  hipLaunchKernelGGL((decode_combine<D, G>), dim3(n_combine),
                     dim3(kCombineThreads), 0, s, a);
  return hipGetLastError();
}

template <int D, int G>
struct CombineLaunch {
  static hipError_t run(const DecodeArgs &a, int n, hipStream_t s) {
    return launch_combine_dg<D, G>(a, n, s);
  }
};

}  // namespace

int decode_split_tokens() { return kWaves * kTilesPerWave * kTile; }
int decode_combine_blocks_per_item(int D, int G) {
  return G * (D / (kCombineChan < D ? kCombineChan : D));
}

hipError_t launch_decode_split(int fmt, int D, int G, const DecodeArgs &a,
                               int n_splits, hipStream_t s) {
  switch (fmt) {
    case HWKV_KV_BF16:
      return launch_decode_split_fmt<HWKV_KV_BF16>(D, G, a, n_splits, s);
    case HWKV_KV_F16:
      return launch_decode_split_fmt<HWKV_KV_F16>(D, G, a, n_splits, s);
    case HWKV_KV_FP8_E4M3:
      return launch_decode_split_fmt<HWKV_KV_FP8_E4M3>(D, G, a, n_splits, s);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_decode_combine(int D, int G, const DecodeArgs &a,
                                 int n_combine_blocks, hipStream_t s) {
  return dispatch_dg<CombineLaunch>(D, G, a, n_combine_blocks, s);
}

}  // namespace hwkv
