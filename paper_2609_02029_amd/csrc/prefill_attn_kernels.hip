// prefill_attn_kernels.hip -- sink + window causal attention of one prefill
// chunk on bf16 MFMA (gfx950).
//
// Query token t of the chunk [p0, p1), query head q of KV head h = q / G,
// attends over R(t + 1) restricted to [0, t]: positions s <= t with s < S or
// s >= t + 1 - w (every s <= t for a full unit) -- the windowed attention of
// the paper's conditional attention equations with the sink prefix of its
// StreamingLLM control.  Keys below p0 come from the cache as it stands
// before the chunk is materialised (sinks, plus the ring for a finite unit,
// whose residency at length p0 covers every s >= p0 + 1 - w); keys in
// [p0, t] come from the chunk's own K/V.
//
// Formulation.  A workgroup owns one KV head and 32 * NW consecutive
// (token, q-head) columns of that head (column c = token * G + g), one
// 32-column block per wavefront.  Per key tile of 32 positions it computes
//     S^T = K Q^T           (v_mfma_f32_32x32x16_bf16, K from LDS, Q^T held
//                            in registers for the whole kernel)
//     O^T += V^T P^T        (V^T from LDS, P^T straight from the S^T
//                            accumulator registers)
// In the 32x32 accumulator layout a lane owns one column and 16 key rows, so
// the softmax max and sum are in-lane plus one swap between the two lane
// halves.  The P^T operand needs 8 keys per lane in MFMA k order; instead of
// moving P, the keys of each 16-key step are permuted (k index 8*half + j is
// key 16*step + 8*(j/4) + 4*half + j%4, exactly the rows a lane already holds)
// and V^T is stored in LDS in that permuted key order.
//
// Online softmax in base 2 with a lazy rescale: the running shift m only
// moves when a tile's maximum exceeds it by more than 8 (log2 units), so the
// O^T accumulators are rescaled rarely; any shift gives the same quotient
// and terms stay below 2^8.  Tiles no column of a wavefront can see are
// skipped by that wavefront; tiles every column sees skip the mask.
#include "hwkv_internal.h"

namespace hwkv {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kKeys = 32;                  // keys per tile
constexpr int kVRow = kKeys * 2 + 16;      // bytes per V^T row in LDS (odd x 16)

__device__ __forceinline__ u32x4_t ld16(const uint16_t *p) {
  return *reinterpret_cast<const u32x4_t *>(p);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

// Byte offset, within a V^T row, of the 4-key quad kq (keys 4kq .. 4kq+3):
// key 16s + 8jh + 4h + jl is stored at 16s + 8h + 4jh + jl.
__device__ __forceinline__ int quad_pos(int kq) {
  return (4 * (kq >> 2) + 2 * (kq & 1) + ((kq >> 1) & 1)) * 8;
}

template <int D, int NW>
struct Prefill {
  static constexpr int NT = NW * 64;
  static constexpr int DC = D / 8;                 // 16-byte channel chunks
  static constexpr int KS = D / 16;                // k-steps of S^T
  static constexpr int DB = D / 32;                // 32-channel blocks of O^T
  static constexpr int KBYTES = DC * kKeys * 16;   // K tile [DC][32][8]
  static constexpr int VBYTES = D * kVRow;         // V^T tile [D][permuted 32]
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int KLD = (DC * kKeys + NT - 1) / NT;   // K chunks / thread
  static constexpr int VLD = (D + NT - 1) / NT;            // V groups / thread
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void prefill_attn(const PrefillAttnArgs a) {
  using P = Prefill<D, NW>;
  constexpr int NT = P::NT, DC = P::DC, KS = P::KS, DB = P::DB;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * P::STAGE];

  const int nb = a.n_col_blocks;
  const int h = a.head_order[blockIdx.x / nb];
  const int cb = nb - 1 - (int)(blockIdx.x % nb);   // later tokens first
  const PrefillAttnHead &hd = a.head[h];
  const int G = a.group;
  const int Hq = a.n_kv_heads * G;
  const int ncols = a.n_tokens * G;
  const int c_first = cb * 32 * NW;
  const int c_last = min(c_first + 32 * NW, ncols) - 1;
  // positions and slots fit in 32 bits (max_ctx < 2^24)
  const int p0 = a.p0;
  const int S = a.n_sinks;
  const int W = hd.window;                          // 0 = full
  const int ta = p0 + c_first / G, tb = p0 + c_last / G;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, cl = lane & 31;

  // this wavefront's columns and this lane's column
  const int wc0 = c_first + 32 * wave;
  const bool wave_live = wc0 <= c_last;
  const int wc_last = min(wc0 + 31, c_last);
  const int t_lo = p0 + min(wc0, c_last) / G, t_hi = p0 + wc_last / G;
  const int c = wc0 + cl;
  const bool col_ok = c <= c_last;
  const int cc = min(c, c_last);
  const int tl = cc / G, g = cc - tl * G;
  const int t = p0 + tl;
  const size_t q_row = ((size_t)tl * Hq + (size_t)h * G + g) * D;

  u32x4_t qv[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qv[ks] = col_ok ? ld16(a.q + q_row + 16 * ks + 8 * half) : u32x4_t{0, 0, 0, 0};

  // key ranges: [ra0, ra1) then [rb0, rb1)
  const int lo = (W == 0) ? 0 : max(0, ta + 1 - W);
  int ra1, rb0 = 0, rb1 = 0;
  if (lo <= S) {
    ra1 = tb + 1;
  } else {
    ra1 = S;
    rb0 = lo;
    rb1 = tb + 1;
  }
  const int na = (ra1 + kKeys - 1) / kKeys;
  const int ntiles = na + (rb1 - rb0 + kKeys - 1) / kKeys;

  const uint16_t *kc = a.cache + hd.k_off;
  const uint16_t *vc = a.cache + hd.v_off;
  const size_t in_stride = (size_t)a.n_kv_heads * D;
  const uint16_t *kin = a.k + (size_t)h * D;
  const uint16_t *vin = a.v + (size_t)h * D;

  auto tile_range = [&](int i, int *s0, int *se) {
    if (i < na) {
      *s0 = i * kKeys;
      *se = ra1;
    } else {
      *s0 = rb0 + (i - na) * kKeys;
      *se = rb1;
    }
  };
  // Cache slot of position s < p0 of a tile starting at s0: sinks and full
  // units map to themselves; ring positions s >= b0 = max(s0, S) sit at
  // S + ((b0 - S) mod W + (s - b0)) mod W, with s - b0 < 32.
  struct Ring {
    int b0, rb;
  };
  auto ring_of = [&](int s0) -> Ring {
    Ring r;
    r.b0 = max(s0, S);
    r.rb = (W == 0) ? 0 : (r.b0 - S) % W;
    return r;
  };
  auto slot_of = [&](const Ring &r, int s) -> int {
    if (W == 0 || s < S) return s;
    int off = r.rb + (s - r.b0);
    while (off >= W) off -= W;
    return S + off;
  };

  // staging registers of the next tile
  u32x4_t kreg[P::KLD];
  u32x4_t vreg[P::VLD][4];

  auto stage_load = [&](int i) {
    int s0, se;
    tile_range(i, &s0, &se);
    const Ring rg = ring_of(s0);
#pragma unroll
    for (int j = 0; j < P::KLD; ++j) {
      const int e = tid + j * NT;
      const int key = e & (kKeys - 1), dc = e / kKeys;
      const int s = s0 + key;
      u32x4_t x = {0, 0, 0, 0};
      if (e < DC * kKeys && s < se) {
        if (s >= p0) {
          x = ld16(kin + (size_t)(s - p0) * in_stride + dc * 8);
        } else {
          const int sl = slot_of(rg, s);
          x = ld16(kc + ((sl >> 6) * DC + dc) * (kTile * 8) + (sl & 63) * 8);
        }
      }
      kreg[j] = x;
    }
#pragma unroll
    for (int j = 0; j < P::VLD; ++j) {
      const int gi = tid + j * NT;
      const int kq = gi & 7, dc = gi >> 3;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int s = s0 + 4 * kq + e;
        u32x4_t x = {0, 0, 0, 0};
        if (gi < D && s < se) {
          if (s >= p0)
            x = ld16(vin + (size_t)(s - p0) * in_stride + dc * 8);
          else
            x = ld16(vc + slot_of(rg, s) * D + dc * 8);
        }
        vreg[j][e] = x;
      }
    }
  };

  auto stage_store = [&](int buf) {
    uint8_t *kl = smem + buf * P::STAGE;
    uint8_t *vl = kl + P::KBYTES;
#pragma unroll
    for (int j = 0; j < P::KLD; ++j) {
      const int e = tid + j * NT;
      if (e < DC * kKeys)
        *reinterpret_cast<u32x4_t *>(kl + e * 16) = kreg[j];
    }
#pragma unroll
    for (int j = 0; j < P::VLD; ++j) {
      const int gi = tid + j * NT;
      if (gi < D) {
        const int kq = gi & 7, dc = gi >> 3;
        uint8_t *dst = vl + (dc * 8) * kVRow + quad_pos(kq);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          // channels 2m (low halves) and 2m + 1 (high halves) of 4 keys
          uint32_t x0 = vreg[j][0][m], x1 = vreg[j][1][m];
          uint32_t x2 = vreg[j][2][m], x3 = vreg[j][3][m];
          uint2 lo2, hi2;
          lo2.x = (x0 & 0xFFFFu) | (x1 << 16);
          lo2.y = (x2 & 0xFFFFu) | (x3 << 16);
          hi2.x = (x0 >> 16) | (x1 & 0xFFFF0000u);
          hi2.y = (x2 >> 16) | (x3 & 0xFFFF0000u);
          *reinterpret_cast<uint2 *>(dst + (2 * m) * kVRow) = lo2;
          *reinterpret_cast<uint2 *>(dst + (2 * m + 1) * kVRow) = hi2;
        }
      }
    }
  };

  const float c2 = a.scale_log2;
  const float tau = 8.0f / c2;                  // lazy-rescale slack (raw units)
  float m = -1e30f;                              // running shift (raw units)
  float l = 0.0f;                                // this lane's partial sum
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;

  if (ntiles > 0) {
    stage_load(0);
    stage_store(0);
  }
  __syncthreads();

  for (int i = 0; i < ntiles; ++i) {
    if (i + 1 < ntiles) stage_load(i + 1);
    int s0, se;
    tile_range(i, &s0, &se);
    const int slast = min(s0 + kKeys, se) - 1;
    const bool skip = !wave_live || s0 > t_hi ||
                      (W != 0 && s0 >= S && slast < t_lo + 1 - W);
    if (!skip) {
      const uint8_t *kl = smem + (i & 1) * P::STAGE;
      const uint8_t *vl = kl + P::KBYTES;
      f32x16_t st;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4_t kx =
            *reinterpret_cast<const u32x4_t *>(kl + ((2 * ks + half) * kKeys + cl) * 16);
        st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, kx), __builtin_bit_cast(bf16x8_t, qv[ks]), st, 0,
            0, 0);
      }
      const bool full_vis = s0 + kKeys <= se && slast <= t_lo &&
                            (W == 0 || slast < S || s0 >= t_hi + 1 - W);
      if (!full_vis) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int s = s0 + (r >> 2) * 8 + half * 4 + (r & 3);
          const bool vis = s < se && s <= t && (W == 0 || s < S || s >= t + 1 - W);
          if (!vis) st[r] = -__builtin_inff();
        }
      }
      float mx = st[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, st[r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      if (__any(mx > m + tau)) {
        const float mn = fmaxf(m, mx);
        const float alpha = __builtin_amdgcn_exp2f((m - mn) * c2);
        m = mn;
        l *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      }
      const float mc = m * c2;
      float pr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[r], c2, -mc));
        l += pr[r];
      }
      u32x4_t pb[2];
#pragma unroll
      for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int j = 0; j < 4; ++j) pb[s][j] = pack_bf16(pr[8 * s + 2 * j], pr[8 * s + 2 * j + 1]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const u32x4_t vx = *reinterpret_cast<const u32x4_t *>(
              vl + (32 * db + cl) * kVRow + 32 * s + 16 * half);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, vx), __builtin_bit_cast(bf16x8_t, pb[s]), o[db],
              0, 0, 0);
        }
      }
    }
    if (i + 1 < ntiles) stage_store((i + 1) & 1);
    __syncthreads();
  }

  if (!col_ok) return;
  const float lt = l + __shfl_xor(l, 32);
  const float inv = 1.0f / lt;
  float *orow = a.out + q_row;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int rq = 0; rq < 4; ++rq) {
      float4 v;
      v.x = o[db][4 * rq + 0] * inv;
      v.y = o[db][4 * rq + 1] * inv;
      v.z = o[db][4 * rq + 2] * inv;
      v.w = o[db][4 * rq + 3] * inv;
      *reinterpret_cast<float4 *>(orow + 32 * db + 8 * rq + 4 * half) = v;
    }
}

}  // namespace

int prefill_attn_columns_per_block() { return 32 * kPrefillWaves; }

hipError_t launch_prefill_attn(int D, const PrefillAttnArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)(a.n_col_blocks * a.n_kv_heads));
  const dim3 block(kPrefillWaves * 64);
  switch (D) {
    case 64: hipLaunchKernelGGL((prefill_attn<64, kPrefillWaves>), grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL((prefill_attn<128, kPrefillWaves>), grid, block, 0, s, a); break;
    case 256: hipLaunchKernelGGL((prefill_attn<256, kPrefillWaves>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hwkv
