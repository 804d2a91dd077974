// kv_format.h -- cache formats p_KV of the stored keys and values (gfx950).
//
// The paper's storage accounting carries the cache format p_KV through the
// effective bytes per element b^K, b^V (Method, Eq. nominal-storage), and a
// format that changes numerical execution is used by every consumer of the
// cache.  Three formats are stored:
//   bf16      the input format, stored as is (b = 2);
//   f16       IEEE binary16, round to nearest even, overflow to infinity
//             (b = 2);
//   fp8-e4m3  OCP FP8 E4M3 ("E4M3FN": 1 sign, 4 exponent bits of bias 7,
//             3 mantissa bits; subnormals m * 2^-9; no infinities; S.1111.111
//             is NaN; largest finite 448), stored as code(x / s) with a
//             per-(layer, KV head) fp32 scale s, separately for K and V: the
//             quotient is the correctly rounded fp32 division, then rounded to
//             nearest even and saturated to +-448; NaN stays NaN (b = 1).
// The value of a stored element is its decoded value (times s for fp8).
//
// Every format stores 8 elements per chunk (16 bytes for the 16-bit formats,
// 8 bytes for fp8), so the tile layout of hwkv_internal.h holds for all three
// with the chunk as its unit.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "hwkv.h"

namespace hwkv {

template <int F>
struct KvFormat;

template <>
struct KvFormat<HWKV_KV_BF16> {
  static constexpr int kBytes = 2;
  using Chunk = uint4;
};
template <>
struct KvFormat<HWKV_KV_F16> {
  static constexpr int kBytes = 2;
  using Chunk = uint4;
};
template <>
struct KvFormat<HWKV_KV_FP8_E4M3> {
  static constexpr int kBytes = 1;
  using Chunk = uint2;
};

// OCP E4M3 code of the fp32 value y: round to nearest even, saturate finite
// and infinite magnitudes >= 448 to 448, NaN to S.1111.111.  The sign bit of
// the code is the sign bit of y (so -0 and negative values that round to zero
// give 0x80).
__device__ __forceinline__ uint32_t e4m3_encode(float y) {
  const uint32_t u = __builtin_bit_cast(uint32_t, y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7fffffffu;
  if (a > 0x7f800000u) return sign | 0x7fu;       // NaN
  if (a >= 0x43e00000u) return sign | 0x7eu;      // |y| >= 448: saturate
  if (a < 0x3c800000u) {                          // |y| < 2^-6: subnormal step
    // |y| * 2^9 is exact; rounding it to an integer in 0..8 gives the code
    // (8 is the smallest normal, 2^-6, whose code is 0x08)
    const float t = __builtin_bit_cast(float, a) * 512.0f;
    return sign | (uint32_t)__builtin_rintf(t);
  }
  // normal: move the exponent from bias 127 to bias 7 and keep 3 mantissa
  // bits, rounding the 20 dropped bits to nearest even (a carry out of the
  // mantissa raises the exponent, which is the correct result)
  const uint32_t v = a - (120u << 23);
  uint32_t r = v >> 20;
  const uint32_t rem = v & 0xfffffu;
  r += (rem > 0x80000u || (rem == 0x80000u && (r & 1u))) ? 1u : 0u;
  return sign | r;
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
  return __builtin_bit_cast(float, h << 16);
}

// Stores 8 bf16 input elements (a 16-byte chunk) in format F.  `s` is the
// fp8 scale (unused otherwise).
template <int F>
__device__ __forceinline__ typename KvFormat<F>::Chunk encode8(uint4 x, float s) {
  if constexpr (F == HWKV_KV_BF16) {
    return x;
  } else if constexpr (F == HWKV_KV_F16) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    uint32_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const _Float16 lo = (_Float16)bf16_bits_to_f32(w[i] & 0xffffu);
      const _Float16 hi = (_Float16)bf16_bits_to_f32(w[i] >> 16);
      o[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) |
             ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  } else {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    uint32_t o[2] = {0u, 0u};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t c0 = e4m3_encode(__fdiv_rn(bf16_bits_to_f32(w[i] & 0xffffu), s));
      const uint32_t c1 = e4m3_encode(__fdiv_rn(bf16_bits_to_f32(w[i] >> 16), s));
      o[i / 2] |= (c0 | (c1 << 8)) << (16 * (i % 2));
    }
    return make_uint2(o[0], o[1]);
  }
}

template <int F>
__device__ __forceinline__ void store_chunk(uint8_t *dst, typename KvFormat<F>::Chunk c) {
  *reinterpret_cast<typename KvFormat<F>::Chunk *>(dst) = c;
}

}  // namespace hwkv
