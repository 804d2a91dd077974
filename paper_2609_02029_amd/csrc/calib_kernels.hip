// calib_kernels.hip -- scores of the calibration replay (gfx950).
//
// For every sampled query row and query head, the stabilised cosine of each
// candidate window's output against the full-history output (Appendix,
// calibration score, Eq. stabilized-cosine: a vector whose norm is at most
// 1e-12 counts as zero; two zero vectors score 1, exactly one scores 0), and
// per (candidate, kv head) the mean of those scores over the rows and the
// head's G query heads (Eq. conditional-similarity).  fp32 throughout: one
// wavefront per (row, q head) with lanes over channels and DPP/lane-read
// reductions; one workgroup per (candidate, kv head) for the means.  The
// partials of the one-pass replay are merged into candidates here too.
#include "hwkv_internal.h"

namespace hwkv {
namespace {

__device__ __forceinline__ float wave_sum64(float v) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ float cos_stab(float uv, float uu, float vv) {
  const float eps = 1e-12f;
  const float nu = sqrtf(uu), nv = sqrtf(vv);
  const bool zu = nu <= eps, zv = nv <= eps;
  if (zu && zv) return 1.0f;
  if (zu || zv) return 0.0f;
  return uv / (nu * nv);
}

template <int D>
__global__ __launch_bounds__(256) void calib_scores(const CalibArgs a) {
  constexpr int PER = D / 64;                      // channels per lane
  const int wave = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int rq = a.n_rows * a.n_q_heads;
  if (wave >= rq) return;                          // uniform per wave
  const size_t vec = (size_t)rq * D;               // one candidate's outputs
  const float *full = a.outs + (size_t)a.n_cand * vec + (size_t)wave * D;
  float f[PER];
  float ff = 0.f;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    f[i] = full[lane + 64 * i];
    ff += f[i] * f[i];
  }
  ff = wave_sum64(ff);
  for (int k = 0; k < a.n_cand; ++k) {
    const float *o = a.outs + (size_t)k * vec + (size_t)wave * D;
    float uv = 0.f, uu = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const float x = o[lane + 64 * i];
      uv += x * f[i];
      uu += x * x;
    }
    uv = wave_sum64(uv);
    uu = wave_sum64(uu);
    if (lane == 0) a.scores[(size_t)k * rq + wave] = cos_stab(uv, uu, ff);
  }
  if (a.ref) {
    const float *r = a.ref + (size_t)wave * D;
    float uv = 0.f, rr = 0.f;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const float x = r[lane + 64 * i];
      uv += x * f[i];
      rr += x * x;
    }
    uv = wave_sum64(uv);
    rr = wave_sum64(rr);
    if (lane == 0) a.check[wave] = cos_stab(uv, ff, rr);
  }
}

// one workgroup per (candidate k, kv head h): mean of scores[k][r][h G + g]
__global__ __launch_bounds__(256) void calib_means(const CalibArgs a) {
  __shared__ float part[4];
  const int hkv = a.n_q_heads / a.group;
  const int k = blockIdx.x / hkv, h = blockIdx.x % hkv;
  const int n = a.n_rows * a.group;
  const float *sc = a.scores + (size_t)k * a.n_rows * a.n_q_heads;
  float s = 0.f;
  for (int i = threadIdx.x; i < n; i += 256) {
    const int r = i / a.group, g = i - r * a.group;
    s += sc[(size_t)r * a.n_q_heads + h * a.group + g];
  }
  s = wave_sum64(s);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0)
    a.means[(size_t)k * hkv + h] = ((part[0] + part[1]) + (part[2] + part[3])) / (float)n;
}

// Merge of the one-pass replay: one wavefront per column c, lanes over
// channels, every candidate in one walk over the column's split partials.
// Candidate k < K of column c (row position t) holds the sinks and the keys
// s >= e = t + 1 - w_k; e <= S means every key, as the full candidate (k = K)
// does.  Its parts: the sinks' partial; the partial of split j (keys
// [j T, (j + 1) T), T = 32 tiles_per_split) when all of the split's keys are
// >= e, i.e. j >= j_k with j_k = e / T + (e > (e / T) T) (0 for e <= S); the
// window's edge partial when e lies inside split e / T.  The windows ascend,
// so j_k does not increase with k: walking the splits from the top down with
// a running (M, L, acc) over splits [j, n_splits), candidate k is complete
// when the walk has added split j_k, and takes the running state, its edge
// partial and the sinks.  out = sum acc 2^((m - M) c) / sum l 2^((m - M) c),
// M = max m over the parts with l > 0 (m in logit units, c = scale log2 e);
// the running state carries its own shift and is rescaled as it rises.
template <int D>
__global__ __launch_bounds__(256) void replay_merge(const ReplayMergeArgs a) {
  constexpr int PER = D / 64;
  const int col = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int K = a.n_windows;
  if (col >= a.n_cols) return;                     // uniform per wave
  const int h = (col % a.n_q_heads) / a.group;     // the column's kv head
  const int t = a.rows[col / a.n_q_heads];
  const int S = a.n_sinks;
  const int T = 32 * a.tiles_per_split;
  const float c2 = a.scale_log2 * a.k_scale[h];
  const float vs = a.v_scale[h];
  const size_t stride = (size_t)a.n_cols * (D + 4);
  const float *pc = a.part + (size_t)col * (D + 4);
  // the sinks' partial
  const float *ps = pc + (size_t)a.n_splits * stride;
  const bool sinks = S > 0 && ps[1] > 0.0f;
  float sm = -1e30f, sl = 0.0f, sacc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) sacc[i] = 0.0f;
  if (sinks) {
    sm = ps[0];
    sl = ps[1];
#pragma unroll
    for (int i = 0; i < PER; ++i) sacc[i] = ps[4 + lane + 64 * i];
  }
  // the first split of candidate k's own keys
  auto first_split = [&](int k) -> int {
    const int e = t + 1 - a.windows[k];
    if (e <= S) return 0;
    const int je = e / T;
    return e > je * T ? je + 1 : je;
  };
  // running state over the splits added so far
  float M = -1e30f, L = 0.0f, acc[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) acc[i] = 0.0f;
  // candidate k (K: the full one) from the running state, its edge partial
  // (k < K and the edge inside a split) and the sinks
  auto finish = [&](int k) {
    float *orow = a.outs + ((size_t)k * a.n_cols + col) * D;
    float em = -1e30f, el = 0.0f, eacc[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) eacc[i] = 0.0f;
    if (k < K) {
      const int e = t + 1 - a.windows[k];
      if (e > S && e > (e / T) * T) {
        const float2 ml =
            *reinterpret_cast<const float2 *>(a.win_ml + ((size_t)k * a.n_cols + col) * 2);
        em = ml.x;
        el = ml.y;
        if (el > 0.0f) {
#pragma unroll
          for (int i = 0; i < PER; ++i) eacc[i] = orow[lane + 64 * i];
        }
      }
    }
    float Mx = -1e30f;
    if (L > 0.0f) Mx = M;
    if (el > 0.0f) Mx = fmaxf(Mx, em);
    if (sinks) Mx = fmaxf(Mx, sm);
    const float fr = L > 0.0f ? __builtin_amdgcn_exp2f((M - Mx) * c2) : 0.0f;
    const float fe = el > 0.0f ? __builtin_amdgcn_exp2f((em - Mx) * c2) : 0.0f;
    const float fs = sinks ? __builtin_amdgcn_exp2f((sm - Mx) * c2) : 0.0f;
    const float inv = vs / (L * fr + el * fe + sl * fs);
#pragma unroll
    for (int i = 0; i < PER; ++i)
      orow[lane + 64 * i] = (acc[i] * fr + eacc[i] * fe + sacc[i] * fs) * inv;
  };
  int k = 0;                                       // the next candidate to finish
  // split j's partial, loaded one split ahead of its use
  float nm = 0.0f, nl = 0.0f, nacc[PER];
  auto load = [&](int j) {
    const float *pj = pc + (size_t)j * stride;
    nm = pj[0];
    nl = pj[1];
#pragma unroll
    for (int i = 0; i < PER; ++i) nacc[i] = pj[4 + lane + 64 * i];
  };
  if (a.n_splits > 0) load(a.n_splits - 1);
  for (int j = a.n_splits - 1; j >= 0; --j) {
    while (k < K && first_split(k) > j) finish(k++);   // complete before split j
    const float m = nm, l = nl;
    float x[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) x[i] = nacc[i];
    if (j > 0) load(j - 1);
    if (l > 0.0f) {                                // uniform: empty splits add nothing
      const float Mn = fmaxf(M, m);
      const float f0 = L > 0.0f ? __builtin_amdgcn_exp2f((M - Mn) * c2) : 0.0f;
      const float f1 = __builtin_amdgcn_exp2f((m - Mn) * c2);
      L = L * f0 + l * f1;
#pragma unroll
      for (int i = 0; i < PER; ++i) acc[i] = acc[i] * f0 + x[i] * f1;
      M = Mn;
    }
  }
  while (k < K) finish(k++);                       // the candidates holding every split
  finish(K);
}

}  // namespace

hipError_t launch_replay_merge(int D, const ReplayMergeArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)(((size_t)a.n_cols + 3) / 4)), block(256);
  switch (D) {
    case 64: hipLaunchKernelGGL(replay_merge<64>, grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL(replay_merge<128>, grid, block, 0, s, a); break;
    case 256: hipLaunchKernelGGL(replay_merge<256>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_calib_scores(int D, const CalibArgs &a, hipStream_t s) {
  const int waves = a.n_rows * a.n_q_heads;
  const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
  switch (D) {
    case 64: hipLaunchKernelGGL(calib_scores<64>, grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL(calib_scores<128>, grid, block, 0, s, a); break;
    case 256: hipLaunchKernelGGL(calib_scores<256>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_calib_means(const CalibArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)(a.n_cand * (a.n_q_heads / a.group))), block(256);
  hipLaunchKernelGGL(calib_means, grid, block, 0, s, a);
  return hipGetLastError();
}

}  // namespace hwkv
