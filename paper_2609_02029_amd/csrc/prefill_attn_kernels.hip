// prefill_attn_kernels.hip -- sink + window causal attention of one prefill
// chunk on bf16 or binary16 MFMA (gfx950).
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
// The calibration replay (replay_attn, below) uses the same tiles, operand
// layouts and softmax on a traced history, for every candidate in one pass.
//
// Formulation.  A workgroup owns one KV head and 32 * NW consecutive
// (token, q-head) columns of that head (column c = token * G + g), one
// 32-column block per wavefront.  Per key tile of 32 positions it computes
//     S^T = K Q^T           (v_mfma_f32_32x32x16_bf16, K from LDS, Q^T held
//                            in registers for the whole kernel)
//     O^T += V^T P^T        (V^T from LDS by transposing reads, P^T straight
//                            from the S^T accumulator registers)
// In the 32x32 accumulator layout a lane owns one column and 16 key rows, so
// the softmax max and sum are in-lane plus one swap between the two lane
// halves.  The P^T operand needs 8 keys per lane in MFMA k order; instead of
// moving P, the keys of each 16-key step are permuted (k index 8*half + j is
// key 16*step + 8*(j/4) + 4*half + j%4, exactly the rows a lane already
// holds), and the V^T operand is read in that key order.
//
// Data movement.  K and V tiles go from global memory straight into LDS
// (global_load_lds_dwordx4: lane i of an instruction fills bytes
// [16i, 16i + 16) of the instruction's LDS block; each lane picks its own
// source), double-buffered, one barrier per tile, no staging registers.
// Both tiles are stored as rows of one 16-byte channel chunk for the 32
// keys (512 B), two rows per load instruction; in odd rows key k sits at
// position k ^ 4.  Lane L of every load then fetches key (L % 32) ^
// (4 (L / 32)) -- one key per lane and tile, so its cache slot and row
// addresses are worked out once per tile -- at chunk 2n + L / 32.
//   K tile: rows contiguous.  The S^T operand (a lane's key, 8 channels of
//           one chunk) is one 16-byte read; a half-wave reads a whole row.
//   V tile: row pairs spaced 1 KiB + 128 B apart.  ds_read_b64_tr_b16 over
//           a 16-lane group turns 4 keys x 16 channels of V into 4 keys of
//           one channel per lane -- the V^T operand.  A half-wave (two
//           16-lane groups: the same 4 keys, adjacent 16-channel pieces)
//           touches four 64-byte pieces that the odd-row swizzle and the pair
//           pad place on disjoint banks of the 256-byte-wide LDS.
// Every operand address is a per-lane base plus a compile-time offset.
// Keys past the tile's range read a zero row, so they are exact zeros (and
// masked).
//
// Binary16 caches (prefill_attn<.., true>): the same tiles, loads and
// layouts (both formats are 2-byte elements), on v_mfma_f32_32x32x16_f16.
// The keys and values enter as stored; q (bf16) is converted to binary16
// after scaling by a power of two 2^sh common to the wavefront that puts the
// wavefront's largest |q| in [2^14, 2^15), which is exact for every
// component within a factor 2^31 of it, and the logit scale takes 2^-sh back.
// The softmax weights enter the value product as binary16 with a 2^7 bias
// (they are at most 2^8 before it, so at most 2^15 after), which keeps the
// small ones clear of binary16's subnormal range; the running sum carries the
// same bias, so the quotient is unchanged.
//
// Online softmax in base 2 with a lazy rescale: the running shift m only
// moves when a tile's maximum exceeds it by more than 8 (log2 units), so the
// O^T accumulators are rescaled rarely; any shift gives the same quotient
// and terms stay below 2^8.  Tiles no column of a wavefront can see are
// skipped by that wavefront; tiles every column sees skip the mask.
#include "hwkv_internal.h"

namespace hwkv {

// A zero row (head_dim <= 256): the source of every key past a tile's range
__device__ __attribute__((aligned(16))) uint32_t g_zero_row[128] = {};

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kKeys = 32;                  // keys per tile
// Operand reads from LDS issued ahead of the products (sched_group_barrier
// masks: matrix-core instructions, LDS reads)
constexpr int kPipeK = 4;                  // K operands (one 16-byte read each)
constexpr int kPipeV = 3;                  // V operands (two 8-byte reads each)
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

__device__ __forceinline__ u32x4_t ld16(const uint16_t *p) {
  return *reinterpret_cast<const u32x4_t *>(p);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ uint32_t pack_f16(float lo, float hi) {
  const f32x2_t f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2_t));
}

// 32x32x16 MFMA on 2-byte operands: binary16 (F16) or bf16
template <bool F16>
__device__ __forceinline__ f32x16_t mfma16(u32x4_t a, u32x4_t b, f32x16_t c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// 16 bytes from global memory into the LDS block of the issuing instruction
__device__ __forceinline__ void g2lds(const void *src, uint8_t *lds_block) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_t *)lds_block, 16, 0, 0);
}

__device__ __forceinline__ void wait_loads() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// x of lane l and x of lane l ^ 32 in both lanes (VALU lane swap)
__device__ __forceinline__ void halves(float x, float *a, float *b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(int, x),
                                                  __builtin_bit_cast(int, x), false, false);
  *a = __builtin_bit_cast(float, (int)r[0]);      // x of the lower-half lane
  *b = __builtin_bit_cast(float, (int)r[1]);      // x of the upper-half lane
}


template <int D, int NW>
struct Prefill {
  static constexpr int DC = D / 8;                 // 16-byte channel chunks
  static constexpr int KS = D / 16;                // k-steps of S^T
  static constexpr int DB = D / 32;                // 32-channel blocks of O^T
  static constexpr int NINST = DC / 2;             // loads per tile (K or V), 2 rows each
  static constexpr int KBYTES = NINST * 1024;      // K tile
  static constexpr int VPAIR = 1024 + 128;         // bytes per V row pair (padded)
  static constexpr int VBYTES = NINST * VPAIR;     // V tile
  static constexpr int STAGE = KBYTES + VBYTES;
  static constexpr int IPW = (NINST + NW - 1) / NW;   // per wave and tile, each of K, V
};

template <int D, int NW, bool F16>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void prefill_attn(const PrefillAttnArgs a) {
  using P = Prefill<D, NW>;
  constexpr int KS = P::KS, DB = P::DB, DC = P::DC;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * P::STAGE];

  const int nb = a.n_col_blocks;
  const int h = a.head_order[blockIdx.x / nb];
  const int cb = nb - 1 - (int)(blockIdx.x % nb);   // later tokens first
  const PrefillAttnHead &hd = a.head[h];
  const int G = a.group;
  const int Hq = a.n_kv_heads * G;
  const int ncols = a.n_tokens * G;
  const int c_first = cb * 32 * NW;
  const int c_last = min(c_first + 32 * NW, ncols) - 1;
  // positions and slots fit in 32 bits (max_ctx < 2^24).  Query row r sits
  // at position p0 + r.
  const int p0 = a.p0;
  auto pos = [&](int r) -> int { return p0 + r; };
  const int S = a.n_sinks;
  const int W = hd.window;                          // 0 = full
  const int ta = pos(c_first / G), tb = pos(c_last / G);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // uniform across the wavefront: keeps the per-wave tile tests and the LDS
  // block of every load in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, cl = lane & 31;

  // this wavefront's columns and this lane's column
  const int wc0 = c_first + 32 * wave;
  const bool wave_live = wc0 <= c_last;
  const int wc_last = min(wc0 + 31, c_last);
  const int t_lo = pos(min(wc0, c_last) / G), t_hi = pos(wc_last / G);
  const int c = wc0 + cl;
  const bool col_ok = c <= c_last;
  const int cc = min(c, c_last);
  const int tl = cc / G, g = cc - tl * G;
  const int t = pos(tl);
  const size_t q_row = ((size_t)tl * Hq + (size_t)h * G + g) * D;

  u32x4_t qv[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qv[ks] = col_ok ? ld16(a.q + q_row + 16 * ks + 8 * half) : u32x4_t{0, 0, 0, 0};

  // key ranges: [0, ra1) then [rb0, rb1)
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
  const uint16_t *zero = reinterpret_cast<const uint16_t *>(g_zero_row);

  auto tile_range = [&](int i, int *s0, int *se) {
    if (i < na) {
      *s0 = i * kKeys;
      *se = ra1;
    } else {
      *s0 = rb0 + (i - na) * kKeys;
      *se = rb1;
    }
  };

  // The key this lane loads in every tile.
  const int lkey = cl ^ (4 * half);
  // Ring slot of the load tile's positions: positions s >= b0 = max(s0, S)
  // sit at S + (rb + s - b0) mod W with rb = (b0 - S) mod W; rb follows b0
  // from tile to tile (b0 never decreases).
  int ld_b0 = S, ld_rb = 0;
  auto issue_loads = [&](int i, int buf) {
    int s0, se;
    tile_range(i, &s0, &se);
    const int b0 = max(s0, S);
    if (W != 0) {
      const int step = b0 - ld_b0;
      int rb = ld_rb + step;
      if (step > kKeys || W < kKeys)
        rb %= W;                                   // range switch, tiny windows
      else
        rb = rb >= W ? rb - W : rb;
      ld_rb = rb;
    }
    ld_b0 = b0;
    const int s = s0 + lkey;
    const uint16_t *kp, *vp;
    int kstep;                                     // elements per K chunk
    if (s >= se) {
      kp = zero;
      vp = zero;
      kstep = 8;
    } else if (s >= p0) {
      kp = kin + (size_t)(s - p0) * in_stride;
      vp = vin + (size_t)(s - p0) * in_stride;
      kstep = 8;
    } else {
      int sl = s;
      if (W != 0 && s >= S) {
        int off = ld_rb + (s - b0);                // < W + 32
        if (W >= kKeys)
          off = off >= W ? off - W : off;
        else
          off = off % W;                           // tiny windows only
        sl = S + off;
      }
      if (hd.pto >= 0) {
        // paged full unit: the tile's 32 keys (s0 is a multiple of 32) lie
        // in page s0 / 256, at rows sl % 256 of it
        const int64_t pg = a.page_table[hd.pto + (s0 >> 8)];
        const uint16_t *pk = a.cache + a.pool_off + pg * 2 * kPageTokens * D;
        const int sp = sl & (kPageTokens - 1);
        kp = pk + (size_t)((sp >> 6) * DC) * (kTile * 8) + (sp & 63) * 8;
        vp = pk + (size_t)kPageTokens * D + (size_t)sp * D;
      } else {
        kp = kc + (size_t)((sl >> 6) * DC) * (kTile * 8) + (sl & 63) * 8;
        vp = vc + (size_t)sl * D;
      }
      kstep = kTile * 8;
    }
    uint8_t *kl = smem + buf * P::STAGE;
    uint8_t *vl = kl + P::KBYTES;
#pragma unroll
    for (int j = 0; j < P::IPW; ++j) {
      const int n = wave + j * NW;
      if (P::NINST % NW != 0 && n >= P::NINST) break;   // uniform per wave
      const int ch = 2 * n + half;
      g2lds(kp + ch * kstep, kl + n * 1024);
      g2lds(vp + ch * 8, vl + n * P::VPAIR);
    }
  };

  // logit scale, base 2, with the stored keys' scale (1 but for fp8 caches);
  // uniform, so kept in a scalar register (the 256-channel kernel has no
  // vector register to spare for it)
  float c2 = __builtin_bit_cast(
      float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, a.scale_log2 * hd.k_scale)));
  if constexpr (F16) {
    // q to binary16 under the wavefront's power of two 2^sh; c2 takes 2^-sh
    // (sh is capped so that c2 stays a normal number)
    float mx = 0.0f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x0 = __builtin_bit_cast(float, qv[ks][j] << 16);
        const float x1 = __builtin_bit_cast(float, qv[ks][j] & 0xffff0000u);
        mx = fmaxf(mx, fmaxf(fabsf(x0), fabsf(x1)));
      }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    mx = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, mx)));
    int ex, ec;
    (void)frexpf(mx, &ex);                      // mx in [2^(ex-1), 2^ex)
    (void)frexpf(c2, &ec);
    int sh = mx > 0.0f ? 15 - ex : 0;
    sh = min(sh, ec + 120);
    sh = __builtin_amdgcn_readfirstlane(sh);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x0 = __builtin_bit_cast(float, qv[ks][j] << 16);
        const float x1 = __builtin_bit_cast(float, qv[ks][j] & 0xffff0000u);
        qv[ks][j] = pack_f16(ldexpf(x0, sh), ldexpf(x1, sh));
      }
    c2 = ldexpf(c2, -sh);
  }
  const float tau = 8.0f / c2;                  // lazy-rescale slack (raw units)
  constexpr float pbias = F16 ? 7.0f : 0.0f;    // log2 of the weights' bias
  float m = -1e30f;                              // running shift (raw units)
  float l = 0.0f;                                // this lane's partial sum
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;

  // S^T operand: key cl of chunk row 2ks + half (odd rows swizzled).
  const int klane = half * 512 + lkey * 16;
  // V^T operand: 16-lane group gq = lane / 16, local lane mq.  For k-step s
  // and half hh of its 8 keys, lane (gq, mq) reads 8 bytes of key
  // 16s + 8hh + 4(gq / 2) + mq / 4 at channel 32db + 16(gq % 2) + 4(mq % 4),
  // i.e. in chunk row 4db + 2(gq % 2) + (mq % 4) / 2 of parity (mq / 2) % 2.
  const int gq = lane >> 4, mq = lane & 15;
  const int vpar = (mq >> 1) & 1;
  const int vkey0 = 4 * (gq >> 1) + (mq >> 2);
  const int vlane = (gq & 1) * P::VPAIR + vpar * 512 + (vkey0 ^ (4 * vpar)) * 16 + (mq & 1) * 8;

  issue_loads(0, 0);

  for (int i = 0; i < ntiles; ++i) {
    wait_loads();
    __syncthreads();
    if (i + 1 < ntiles) issue_loads(i + 1, (i + 1) & 1);
    int s0, se;
    tile_range(i, &s0, &se);
    const int slast = min(s0 + kKeys, se) - 1;
    const bool skip = !wave_live || s0 > t_hi ||
                      (W != 0 && s0 >= S && slast < t_lo + 1 - W);
    if (skip) continue;
    const uint8_t *kl = smem + (i & 1) * P::STAGE + klane;
    const uint8_t *vl = smem + (i & 1) * P::STAGE + P::KBYTES + vlane;
    f32x16_t st;
#pragma unroll
    for (int r = 0; r < 16; ++r) st[r] = 0.0f;
    {
      u32x4_t kx[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kx[ks] = *reinterpret_cast<const u32x4_t *>(kl + ks * 1024);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) st = mfma16<F16>(kx[ks], qv[ks], st);
      // K operand reads run kPipeK products ahead of their use (left to
      // itself the scheduler reads each operand just before its product and
      // waits out the LDS latency every time)
      constexpr int PK = kPipeK < KS ? kPipeK : KS;
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, PK, 0);
#pragma unroll
      for (int i = 0; i < KS - PK; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, PK, 0);
    }
    const bool full_vis = s0 + kKeys <= se && slast <= t_lo &&
                          (W == 0 || slast < S || s0 >= t_hi + 1 - W);
    if (!full_vis) {
      // key of row r: e + cr, cr = 8 (r / 4) + r % 4; e and e - t are made
      // opaque so the per-row offsets stay compile-time constants on the
      // uniform side of each comparison
      int e = s0 + 4 * half, d = e - t;
      asm volatile("" : "+v"(e), "+v"(d));
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int cr = (r >> 2) * 8 + (r & 3);
        const bool vis = (e < se - cr) & (d <= -cr) &
                         ((W == 0) | (e < S - cr) | (d >= 1 - W - cr));
        if (!vis) st[r] = -__builtin_inff();
      }
    }
    float mx = st[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, st[r]);
    {
      float lo_half, hi_half;
      halves(mx, &lo_half, &hi_half);
      mx = fmaxf(lo_half, hi_half);
    }
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
    const float mc = m * c2 - pbias;
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
      for (int j = 0; j < 4; ++j)
        pb[s][j] = F16 ? pack_f16(pr[8 * s + 2 * j], pr[8 * s + 2 * j + 1])
                       : pack_bf16(pr[8 * s + 2 * j], pr[8 * s + 2 * j + 1]);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        i16x4_t v2[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          v2[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t *)(vl + 2 * db * P::VPAIR + (16 * s + 8 * hh) * 16));
        const u32x4_t va = __builtin_bit_cast(
            u32x4_t, __builtin_shufflevector(v2[0], v2[1], 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = mfma16<F16>(va, pb[s], o[db]);
      }
    }
    // V operand reads (two per product) run kPipeV products ahead
    {
      constexpr int PV = kPipeV < 2 * DB ? kPipeV : 2 * DB;
      __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * PV, 1);
#pragma unroll
      for (int i = 0; i < 2 * DB - PV; ++i) {
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 1);
        __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 1);
      }
      __builtin_amdgcn_sched_group_barrier(kSchedMfma, PV, 1);
    }
  }

  float l_lo, l_hi;
  halves(l, &l_lo, &l_hi);
  if (!col_ok) return;
  const float lt = l_lo + l_hi;
  const float inv = hd.v_scale / lt;     // the stored values' scale (fp8)
  // the output row, recomputed here rather than kept live through the loop
  int c_out = c;
  asm volatile("" : "+v"(c_out));
  const int tl_o = c_out / G, g_o = c_out - tl_o * G;
  float *orow = a.out + ((size_t)tl_o * Hq + (size_t)h * G + g_o) * D;
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


// Calibration replay in one pass.  Workgroups and columns as in prefill_attn
// (column c = row * G + g of one KV head, row r at position rows[r]); the
// keys are the traced history, each candidate window w holds the sinks
// [0, S) and the suffix [max(S, t + 1 - w), t] of row position t, and the
// full candidate holds every s <= t.  The suffixes are nested, so a column
// walks its keys once, from the top tile down: when the walk has added every
// key at or above a window's edge t + 1 - w, the running (m, l, acc) is that
// window's share of the split, written out there.  A tile holding an edge is
// added in up to two passes of the V^T P^T product per edge: the keys at or
// above the edge, then the rest.  Split y < n_splits covers key tiles
// [y tps, (y + 1) tps) of [0, t_last] without the sinks; split n_splits adds
// the sinks alone.  replay_merge assembles each candidate.
template <int D, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2)))
void replay_attn(const ReplayAttnArgs a) {
  using P = Prefill<D, NW>;
  constexpr int KS = P::KS, DB = P::DB;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * P::STAGE];
  __shared__ int swin[kMaxWindows];

  const int nb = a.n_col_blocks;
  const int h = blockIdx.x / nb;
  const int cb = nb - 1 - (int)(blockIdx.x % nb);   // later rows first
  const int G = a.group;
  const int Hq = a.n_kv_heads * G;
  const int ncols = a.n_rows * G;
  const int c_first = cb * 32 * NW;
  const int c_last = min(c_first + 32 * NW, ncols) - 1;
  const int32_t *rows = a.rows;
  const int S = a.n_sinks;
  const int K = a.n_windows;
  const int tb = rows[c_last / G];                  // the block's last position

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5, cl = lane & 31;
  const int wc0 = c_first + 32 * wave;
  const bool wave_live = wc0 <= c_last;
  const int wc_last = min(wc0 + 31, c_last);
  const int t_lo = rows[min(wc0, c_last) / G], t_hi = rows[wc_last / G];
  const int c = wc0 + cl;
  const bool col_ok = c <= c_last;
  const int cc = min(c, c_last);
  const int tl = cc / G, g = cc - tl * G;
  const int t = rows[tl];
  const size_t q_row = ((size_t)tl * Hq + (size_t)h * G + g) * D;
  const size_t n_cols = (size_t)a.n_rows * Hq;
  // the lane's column id (row * Hq + h * G + g), recomputed where it is
  // needed rather than kept live through the tile loop
  auto column_id = [&]() -> size_t {
    int cx = wc0 + (int)(threadIdx.x & 31);
    asm volatile("" : "+v"(cx));
    const int ccx = min(cx, c_last), tx = ccx / G;
    return (size_t)tx * Hq + (size_t)h * G + (size_t)(ccx - tx * G);
  };

  // this workgroup's key tiles
  const int ntiles = tb / kKeys + 1;
  const bool sink_pass = (int)blockIdx.y == a.n_splits;
  int i_lo, i_hi;
  if (sink_pass) {
    i_lo = 0;
    i_hi = min(ntiles, (S + kKeys - 1) / kKeys);
  } else {
    i_lo = blockIdx.y * a.tiles_per_split;
    i_hi = min(ntiles, i_lo + a.tiles_per_split);
  }
  if (i_lo >= i_hi) {                               // uniform: an empty split
    if (col_ok && half == 0) {
      float *pp = a.part + ((size_t)blockIdx.y * n_cols + q_row / D) * (D + 4);
      pp[0] = -1e30f;
      pp[1] = 0.0f;
    }
    return;
  }
  for (int i = tid; i < K; i += NW * 64) swin[i] = a.windows[i];

  u32x4_t qv[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qv[ks] = col_ok ? ld16(a.q + q_row + 16 * ks + 8 * half) : u32x4_t{0, 0, 0, 0};

  const size_t in_stride = (size_t)a.n_kv_heads * D;
  const uint16_t *kin = a.k + (size_t)h * D;
  const uint16_t *vin = a.v + (size_t)h * D;
  const uint16_t *zero = reinterpret_cast<const uint16_t *>(g_zero_row);
  // the key this lane loads in every tile (see prefill_attn)
  const int lkey = cl ^ (4 * half);
  auto issue_loads = [&](int i, int buf) {
    const int s = i * kKeys + lkey;
    const uint16_t *kp = s <= tb ? kin + (size_t)s * in_stride : zero;
    const uint16_t *vp = s <= tb ? vin + (size_t)s * in_stride : zero;
    uint8_t *kl = smem + buf * P::STAGE;
    uint8_t *vl = kl + P::KBYTES;
#pragma unroll
    for (int j = 0; j < P::IPW; ++j) {
      const int n = wave + j * NW;
      if (P::NINST % NW != 0 && n >= P::NINST) break;   // uniform per wave
      const int ch = 2 * n + half;
      g2lds(kp + ch * 8, kl + n * 1024);
      g2lds(vp + ch * 8, vl + n * P::VPAIR);
    }
  };

  // logit scale, base 2, with the keys' scale; uniform (scalar register)
  const float c2 = __builtin_bit_cast(
      float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, a.scale_log2 * a.k_scale[h])));
  float m = -1e30f;                              // running shift (raw units)
  float l = 0.0f;                                // this lane's partial sum
  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;

  const int klane = half * 512 + lkey * 16;
  const int gq = lane >> 4, mq = lane & 15;
  const int vpar = (mq >> 1) & 1;
  const int vkey0 = 4 * (gq >> 1) + (mq >> 2);
  const int vlane = (gq & 1) * P::VPAIR + vpar * 512 + (vkey0 ^ (4 * vpar)) * 16 + (mq & 1) * 8;

  issue_loads(i_hi - 1, 0);
  __syncthreads();                               // swin
  // The lane's next window: the first whose edge lies below this split's top
  // (windows with an edge at or above it have no key here).  An edge at or
  // below S means the window holds every key: it is the full candidate.
  const int top = i_hi * kKeys;
  int kn = 0;
  int edge = INT_MIN;
  if (!sink_pass) {
    while (kn < K && t + 1 - swin[kn] >= top) ++kn;
    edge = (kn < K && t + 1 - swin[kn] > S) ? t + 1 - swin[kn] : INT_MIN;
  }

  // V^T P^T over the keys of rows [lo, hi) of this lane's tile rows (key of
  // row r: s0 + 4 half + 8 (r / 4) + r % 4), adding their weights to l
  auto add_keys = [&](const float (&pr)[16], int s0, int lo, int hi, const uint8_t *vl) {
    u32x4_t pb[2];
    const int e = s0 + 4 * half;
    float ls = 0.0f;
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r0 = 8 * s + 2 * j, r1 = r0 + 1;
        const int k0 = e + (r0 >> 2) * 8 + (r0 & 3), k1 = e + (r1 >> 2) * 8 + (r1 & 3);
        const float p0 = (k0 >= lo && k0 < hi) ? pr[r0] : 0.0f;
        const float p1 = (k1 >= lo && k1 < hi) ? pr[r1] : 0.0f;
        ls += p0 + p1;
        pb[s][j] = pack_bf16(p0, p1);
      }
    l += ls;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        i16x4_t v2[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh)
          v2[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4_t *)(vl + 2 * db * P::VPAIR + (16 * s + 8 * hh) * 16));
        const bf16x8_t va = __builtin_bit_cast(
            bf16x8_t, __builtin_shufflevector(v2[0], v2[1], 0, 1, 2, 3, 4, 5, 6, 7));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            va, __builtin_bit_cast(bf16x8_t, pb[s]), o[db], 0, 0, 0);
      }
    }
  };

  const int n_it = i_hi - i_lo;
  for (int it = 0; it < n_it; ++it) {
    const int i = i_hi - 1 - it;                 // tiles from the top down
    wait_loads();
    __syncthreads();
    if (it + 1 < n_it) issue_loads(i - 1, (it + 1) & 1);
    const int s0 = i * kKeys;
    const bool skip = !wave_live || s0 > t_hi ||
                      (sink_pass ? s0 >= S : s0 + kKeys <= S);
    if (skip) continue;
    const uint8_t *kl = smem + (it & 1) * P::STAGE + klane;
    const uint8_t *vl = smem + (it & 1) * P::STAGE + P::KBYTES + vlane;
    // S^T of the tile, masked: visible keys are s <= t, and s < S in the
    // sink pass, s >= S otherwise
    const bool full_vis = s0 + kKeys - 1 <= t_lo && (sink_pass ? s0 + kKeys <= S : s0 >= S);
    auto logits = [&]() -> f32x16_t {
      f32x16_t st;
#pragma unroll
      for (int r = 0; r < 16; ++r) st[r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4_t kx = *reinterpret_cast<const u32x4_t *>(kl + ks * 1024);
        st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, kx), __builtin_bit_cast(bf16x8_t, qv[ks]), st, 0, 0, 0);
      }
      if (!full_vis) {
        int e = s0 + 4 * half, d = e - t;
        asm volatile("" : "+v"(e), "+v"(d));
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int cr = (r >> 2) * 8 + (r & 3);
          const bool vis = (d <= -cr) & (sink_pass ? (e < S - cr) : (e >= S - cr));
          if (!vis) st[r] = -__builtin_inff();
        }
      }
      return st;
    };
    // a window's partial at its edge, for the lanes whose edge lies in this
    // tile; those lanes move to their next window
    auto edge_partials = [&](bool act) {
      float l_lo, l_hi;
      halves(l, &l_lo, &l_hi);
      if (act && wc0 + cl <= c_last) {
        const size_t col_id = column_id();
        float *wa = a.win_acc + ((size_t)kn * n_cols + col_id) * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int rq = 0; rq < 4; ++rq)
            *reinterpret_cast<float4 *>(wa + 32 * db + 8 * rq + 4 * half) =
                make_float4(o[db][4 * rq + 0], o[db][4 * rq + 1], o[db][4 * rq + 2],
                            o[db][4 * rq + 3]);
        if (half == 0)
          *reinterpret_cast<float2 *>(a.win_ml + ((size_t)kn * n_cols + col_id) * 2) =
              make_float2(m, l_lo + l_hi);
      }
      if (act) {
        ++kn;
        edge = (kn < K && t + 1 - swin[kn] > S) ? t + 1 - swin[kn] : INT_MIN;
      }
    };

    float mc;
    {
      const f32x16_t st = logits();
      float mx = st[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, st[r]);
      {
        float lo_half, hi_half;
        halves(mx, &lo_half, &hi_half);
        mx = fmaxf(lo_half, hi_half);
      }
      if (__any((mx - m) * c2 > 8.0f)) {        // lazy rescale: shift moves by > 8
        const float mn = fmaxf(m, mx);
        const float alpha = __builtin_amdgcn_exp2f((m - mn) * c2);
        m = mn;
        l *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      }
      mc = m * c2;
      float pr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[r], c2, -mc));
      // First pass: a lane whose next window edge lies in this tile adds the
      // keys at or above the edge; every other lane adds the whole tile.
      const bool act = edge >= s0;
      add_keys(pr, s0, act ? edge : s0, s0 + kKeys, vl);
    }
    if (__any(edge >= s0)) {                     // uniform; rare
      // Further passes, each over the keys below the last edge taken: the
      // logits and weights are recomputed from the tile (same shift, same
      // values) rather than kept live through the passes.
      bool act = edge >= s0;                     // the lanes of the first pass
      int cut = act ? edge : s0;                 // keys [s0, cut) not added yet
      while (true) {
        edge_partials(act);
        if (!__any(cut > s0)) break;
        act = edge >= s0;                        // the lane's next edge, below cut
        const int lo = act ? edge : s0;
        const f32x16_t st = logits();
        float pr[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(st[r], c2, -mc));
        add_keys(pr, s0, lo, cut, vl);
        cut = lo;
      }
    }
  }

  float l_lo, l_hi;
  halves(l, &l_lo, &l_hi);
  if (wc0 + cl > c_last) return;
  float *pp = a.part + ((size_t)blockIdx.y * n_cols + column_id()) * (D + 4);
  if (half == 0) {
    pp[0] = m;
    pp[1] = l_lo + l_hi;
  }
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int rq = 0; rq < 4; ++rq)
      *reinterpret_cast<float4 *>(pp + 4 + 32 * db + 8 * rq + 4 * half) =
          make_float4(o[db][4 * rq + 0], o[db][4 * rq + 1], o[db][4 * rq + 2],
                      o[db][4 * rq + 3]);
}

}  // namespace

int prefill_attn_columns_per_block() { return 32 * kPrefillWaves; }

hipError_t launch_prefill_attn(int D, bool f16, const PrefillAttnArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)(a.n_col_blocks * a.n_kv_heads));
  const dim3 block(kPrefillWaves * 64);
#define HWKV_PA(DD, FF) \
  hipLaunchKernelGGL((prefill_attn<DD, kPrefillWaves, FF>), grid, block, 0, s, a)
  switch (D) {
    case 64: if (f16) HWKV_PA(64, true); else HWKV_PA(64, false); break;
    case 128: if (f16) HWKV_PA(128, true); else HWKV_PA(128, false); break;
    case 256: if (f16) HWKV_PA(256, true); else HWKV_PA(256, false); break;
    default: return hipErrorInvalidValue;
  }
#undef HWKV_PA
  return hipGetLastError();
}

hipError_t launch_replay_attn(int D, const ReplayAttnArgs &a, hipStream_t s) {
  const dim3 grid((unsigned)(a.n_col_blocks * a.n_kv_heads),
                  (unsigned)(a.n_splits + (a.n_sinks > 0 ? 1 : 0)));
  const dim3 block(kPrefillWaves * 64);
  switch (D) {
    case 64: hipLaunchKernelGGL((replay_attn<64, kPrefillWaves>), grid, block, 0, s, a); break;
    case 128: hipLaunchKernelGGL((replay_attn<128, kPrefillWaves>), grid, block, 0, s, a); break;
    case 256: hipLaunchKernelGGL((replay_attn<256, kPrefillWaves>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace hwkv
