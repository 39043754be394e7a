// a4: per-32 MX quantisation of one block of 32 bf16 activations (shared by
// the standalone quantiser and the grouped GEMM's preparation kernel).
//
// A 64-byte load, the block maximum, the scale exponent (smallest power of
// two that fits the maximum), 32 round-to-nearest-even element codes, and one
// packed store:
//   e4m3  32 bytes, element j in byte j;
//   e2m3  24 bytes, element j in bits [6j, 6j+6) of the little-endian block;
//   e2m1  16 bytes, element 2i in the low nibble of byte i.
// These are the register layouts the matrix cores read, so the GEMM loads a
// lane's 32-element operand as one contiguous run of bytes. Inside the
// grouped GEMM's workspace an e2m3 block sits in a 32-byte slot (its 24 bytes,
// then 8 unused), so its activation rows have the FP8 rows' byte geometry
// (SLOT = true).
#pragma once

#include "moe_dev.h"

namespace moe {

// 16 e2m3 codes, one per byte of w[0..3] (code j in byte j % 4 of w[j / 4]),
// packed at 6 bits each into 12 bytes (code j at bits 6j).
__device__ __forceinline__ void pack6x16(const uint32_t* w, uint32_t* p) {
  uint64_t lo = 0, hi = 0;  // codes 0..9 in lo (60 bits), 10..15 in hi
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const uint64_t c = (w[j / 4] >> (8 * (j % 4))) & 0x3fu;
    if (j < 10) lo |= c << (6 * j);
    else hi |= c << (6 * (j - 10));
  }
  // 96 bits: lo holds bits 0..59, hi bits 60..95
  const uint64_t b0 = lo | (hi << 60), b1 = hi >> 4;
  p[0] = (uint32_t)b0;
  p[1] = (uint32_t)(b0 >> 32);
  p[2] = (uint32_t)b1;
}

// Quantise block b (32 consecutive elements of x) into codes and scales[b].
template <int FMT, bool SLOT = false>
__device__ __forceinline__ void quant_block(const uint16_t* __restrict__ x, long b,
                                            uint8_t* __restrict__ codes,
                                            uint8_t* __restrict__ scales) {
  const uint4* src = reinterpret_cast<const uint4*>(x + b * 32);
  uint32_t w[16];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint4 r = src[i];
    w[4 * i] = r.x;
    w[4 * i + 1] = r.y;
    w[4 * i + 2] = r.z;
    w[4 * i + 3] = r.w;
  }
  float v[32];
  float amax = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    v[2 * i] = bf16_to_f32(w[i] & 0xffffu);
    v[2 * i + 1] = bf16_to_f32(w[i] >> 16);
    amax = fmaxf(amax, fmaxf(fabsf(v[2 * i]), fabsf(v[2 * i + 1])));
  }
  const int X = mx_scale_exp<FMT>(amax);
  scales[b] = (uint8_t)(X + 127);
  if constexpr (FMT == 0) {
    uint4* dst = reinterpret_cast<uint4*>(codes + b * 32);
    uint32_t p[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      p[i] = e4m3_pack4(ldexpf(v[4 * i], -X), ldexpf(v[4 * i + 1], -X), ldexpf(v[4 * i + 2], -X),
                        ldexpf(v[4 * i + 3], -X));
    dst[0] = make_uint4(p[0], p[1], p[2], p[3]);
    dst[1] = make_uint4(p[4], p[5], p[6], p[7]);
    return;
  }
  uint32_t c[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) c[i] = mx_encode<FMT>(ldexpf(v[i], -X));
  if constexpr (FMT == 4) {
    uint32_t p[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t q = 0;
#pragma unroll
      for (int j = 0; j < 8; ++j) q |= c[8 * i + j] << (4 * j);
      p[i] = q;
    }
    *reinterpret_cast<uint4*>(codes + b * 16) = make_uint4(p[0], p[1], p[2], p[3]);
  } else {
    uint32_t p[6] = {0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const int bit = 6 * j, word = bit >> 5, sh = bit & 31;
      p[word] |= c[j] << sh;
      if (sh > 26) p[word + 1] |= c[j] >> (32 - sh);
    }
    uint2* dst = reinterpret_cast<uint2*>(codes + b * (SLOT ? 32 : 24));
    dst[0] = make_uint2(p[0], p[1]);
    dst[1] = make_uint2(p[2], p[3]);
    dst[2] = make_uint2(p[4], p[5]);
  }
}

}  // namespace moe
