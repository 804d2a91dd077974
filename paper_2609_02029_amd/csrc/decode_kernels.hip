// decode_kernels.hip -- split-K decode attention over per-head grouped caches
// (gfx950, wave64, VALU).
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
// G query heads of an item share every K/V byte read.
//
// Inside a wave, per 64-slot tile:
//   q.k   one lane per slot: the K tile is stored slot-minor in 16-byte
//         channel chunks, so chunk g of the tile is 1 KiB contiguous and lane
//         t reads its own slot's chunk; q is staged once per workgroup in LDS
//         and read as a broadcast, and v_dot2_f32_bf16 multiplies bf16 pairs
//         with fp32 accumulate.
//         No cross-lane reduction is needed for the logits.
//   softmax  online, base 2 (log2(e) folded into the scale); the tile max is
//         one DPP row reduction plus four lane reads per head.
//   p.v   lanes own 8 channels of one row (V row-major, a wave reads whole
//         rows contiguously); p is broadcast through a per-wave LDS slice.
// The waves of a workgroup are merged in LDS; a split either writes the final
// output (single-split items) or a partial (m, l, acc) that the combine
// kernel merges: m* = max m_j, l* = sum l_j 2^(m_j - m*),
// out = sum acc_j 2^(m_j - m*) / l*.
#include "hwkv_internal.h"

namespace hwkv {
namespace {

constexpr int kWaves = 4;         // waves per workgroup
constexpr int kTilesPerWave = 2;  // 64-slot tiles per wave per split
constexpr int kMinWavesPerEU = 3; // register budget: <= 168 VGPRs per lane

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

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
__global__ __launch_bounds__(kWaves * 64)
__attribute__((amdgpu_waves_per_eu(kMinWavesPerEU))) void decode_split(
    DecodeArgs a) {
  constexpr int NC = D / 8;         // 16-byte chunks per row
  constexpr int RPS = 64 / NC;      // rows per wave step in p.v
  constexpr int PST = (G + 3) & ~3; // p stride per slot in LDS
  __shared__ uint4 q_lds[G * NC];
  __shared__ float p_lds[kWaves][64 * PST];
  __shared__ float mrg_acc[kWaves][G][D];
  __shared__ float mrg_m[kWaves][G];
  __shared__ float mrg_l[kWaves][G];

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
  const int nv = it.n_valid[item];
  const int new_slot = it.new_slot[item];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int c8 = lane % NC;
  const int rsub = lane / NC;

  uint16_t *kbase = a.cache + it.k_off[item];
  uint16_t *vbase = a.cache + it.v_off[item];
  {
    const uint4 *qg =
        reinterpret_cast<const uint4 *>(a.q + (size_t)it.q_row[item] * D);
    for (int e = threadIdx.x; e < G * NC; e += kWaves * 64) q_lds[e] = qg[e];
  }
  // the fused append reads the new token from k_new / v_new (new_slot >= 0
  // only when they are given)
  const uint4 *knew = reinterpret_cast<const uint4 *>(
      a.k_new + (size_t)(new_slot >= 0 ? it.kv_row[item] : 0) * D);
  const uint4 *vnew = reinterpret_cast<const uint4 *>(
      a.v_new + (size_t)(new_slot >= 0 ? it.kv_row[item] : 0) * D);

  float m[G], l[G], acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = -INFINITY;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  }
  float *pl = p_lds[wave];
  __syncthreads();

  for (int k = 0; k < kTilesPerWave; ++k) {
    const int tile = (split * kTilesPerWave + k) * kWaves + wave;
    const int slot0 = tile * 64;
    if (slot0 >= nv) break;

    // ---- q.k: one lane per slot
    const int slot = slot0 + lane;
    const bool is_new = slot == new_slot;
    uint4 *kt = reinterpret_cast<uint4 *>(kbase + (size_t)tile * 64 * D) + lane;
    const uint4 *ksrc = is_new ? knew : kt;
    const int kstr = is_new ? 1 : 64;
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = 0.f;
#pragma unroll 2
    for (int g = 0; g < NC; ++g) {
      const uint4 kk = ksrc[g * kstr];
      if (is_new) kt[g * 64] = kk;
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const uint4 qq = q_lds[h * NC + g];
        s[h] = dot2(qq.x, kk.x, s[h]);
        s[h] = dot2(qq.y, kk.y, s[h]);
        s[h] = dot2(qq.z, kk.z, s[h]);
        s[h] = dot2(qq.w, kk.w, s[h]);
      }
    }

    // ---- online softmax, base 2
    const bool valid = slot < nv;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float z = valid ? s[h] * a.scale_log2 : -INFINITY;
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
      pl[lane * PST + h] = p;
    }

    // ---- p.v: lanes own channels [8 c8, 8 c8 + 8) of row rsub of a step
    const int rows = min(64, nv - slot0);
    uint4 *vt = reinterpret_cast<uint4 *>(vbase + (size_t)slot0 * D);
#pragma unroll 4
    for (int st = 0; st < 64 / RPS; ++st) {
      if (st * RPS >= rows) break;
      const int r = st * RPS + rsub;
      const bool rv = r < rows;
      const int rc = rv ? r : rows - 1;
      const bool rn = (slot0 + rc) == new_slot;
      const uint4 *vsrc = rn ? vnew + c8 : vt + rc * NC + c8;
      const uint4 vv = *vsrc;
      if (rn) vt[rc * NC + c8] = vv;
      float pv[G];
#pragma unroll
      for (int h = 0; h < G; ++h) pv[h] = rv ? pl[r * PST + h] : 0.f;
      const float vf[8] = {bf_lo(vv.x), bf_hi(vv.x), bf_lo(vv.y), bf_hi(vv.y),
                           bf_lo(vv.z), bf_hi(vv.z), bf_lo(vv.w), bf_hi(vv.w)};
#pragma unroll
      for (int h = 0; h < G; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(pv[h], vf[e], acc[h][e]);
    }
  }

  // ---- wave partials: l over all lanes, acc over lanes sharing a chunk
#pragma unroll
  for (int h = 0; h < G; ++h) {
    l[h] = wave_sum(l[h]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int off = 32; off >= NC; off >>= 1)
        acc[h][e] += __shfl_xor(acc[h][e], off);
    }
  }
  if (rsub == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) mrg_acc[wave][h][c8 * 8 + e] = acc[h][e];
  }
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      mrg_m[wave][h] = m[h];
      mrg_l[wave][h] = l[h];
    }
  }
  __syncthreads();

  // ---- merge the waves (every split has a valid tile in wave 0)
  const int nsplit = it.split_begin[item + 1] - it.split_begin[item];
  float *part = a.ws + (size_t)(it.ws_split0 + blk) * (G * (D + 2));
  for (int idx = threadIdx.x; idx < G * D; idx += kWaves * 64) {
    const int h = idx / D, c = idx % D;
    float M = mrg_m[0][h];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) M = fmaxf(M, mrg_m[w][h]);
    float L = 0.f, A = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float f = exp2f(mrg_m[w][h] - M);
      L += mrg_l[w][h] * f;
      A += mrg_acc[w][h][c] * f;
    }
    if (nsplit == 1) {
      a.out[((size_t)it.q_row[item] + h) * D + c] = A / L;
    } else {
      part[2 * G + h * D + c] = A;
      if (c == 0) {
        part[h] = M;
        part[G + h] = L;
      }
    }
  }
}

// One workgroup per (item, query head of the group, 64-channel chunk).
template <int D, int G>
__global__ __launch_bounds__(256) void decode_combine(DecodeArgs a) {
  constexpr int CH = D / 64;
  constexpr int PS = G * (D + 2);
  __shared__ float sl[4][64];
  __shared__ float sa[4][64];
  const DecodeItems &it = a.it;
  const int bid = blockIdx.x;
  const int item = bid / (G * CH);
  const int h = (bid / CH) % G;
  const int ch = bid % CH;
  if (item >= it.n_items) return;
  const int sb = it.split_begin[item];
  const int ns = it.split_begin[item + 1] - sb;
  if (ns <= 1) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = ch * 64 + lane;
  const float *base = a.ws + (size_t)(it.ws_split0 + sb) * PS;

  float M = -INFINITY;
  for (int j = lane; j < ns; j += 64) M = fmaxf(M, base[(size_t)j * PS + h]);
  M = wave_max(M);
  float L = 0.f, A = 0.f;
  for (int j = wave; j < ns; j += 4) {
    const float *pj = base + (size_t)j * PS;
    const float f = exp2f(pj[h] - M);
    L += pj[G + h] * f;
    A += pj[2 * G + h * D + c] * f;
  }
  sl[wave][lane] = L;
  sa[wave][lane] = A;
  __syncthreads();
  if (wave == 0) {
    L = (sl[0][lane] + sl[1][lane]) + (sl[2][lane] + sl[3][lane]);
    A = (sa[0][lane] + sa[1][lane]) + (sa[2][lane] + sa[3][lane]);
    a.out[((size_t)it.q_row[item] + h) * D + c] = A / L;
  }
}

template <int D, int G>
hipError_t launch_dg(const DecodeArgs &a, int n_splits, int n_combine,
                     hipStream_t s) {
  hipLaunchKernelGGL((decode_split<D, G>), dim3(n_splits), dim3(kWaves * 64),
                     0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || n_combine == 0) return e;
  hipLaunchKernelGGL((decode_combine<D, G>), dim3(n_combine), dim3(256), 0, s,
                     a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_d(int G, const DecodeArgs &a, int n_splits, int n_combine,
                    hipStream_t s) {
  switch (G) {
    case 1: return launch_dg<D, 1>(a, n_splits, n_combine, s);
    case 2: return launch_dg<D, 2>(a, n_splits, n_combine, s);
    case 4: return launch_dg<D, 4>(a, n_splits, n_combine, s);
    case 6: return launch_dg<D, 6>(a, n_splits, n_combine, s);
    case 8: return launch_dg<D, 8>(a, n_splits, n_combine, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

int decode_split_tokens() { return kWaves * kTilesPerWave * kTile; }

hipError_t launch_decode(int D, int G, const DecodeArgs &a, int n_splits,
                         int n_combine_blocks, hipStream_t s) {
  switch (D) {
    case 64: return launch_d<64>(G, a, n_splits, n_combine_blocks, s);
    case 128: return launch_d<128>(G, a, n_splits, n_combine_blocks, s);
    case 256: return launch_d<256>(G, a, n_splits, n_combine_blocks, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace hwkv
