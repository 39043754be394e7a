// Device-side helpers shared by the gfx950 kernels of the routed-MoE layer.
//
// Number formats (bit definitions; see include/moe.h):
//   - bf16 <-> fp32 with round-to-nearest-even;
//   - MX element encoders for e4m3 / e2m3 / e2m1 and the per-32 block scale
//     exponent rule (smallest power of two that fits the block maximum);
//   - wrappers around the CDNA4 block-scaled matrix-core instruction
//     V_MFMA_SCALE_F32_16X16X128_F8F6F4.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

namespace moe {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// Compile-time loop: f(std::integral_constant<int, i>) for i = 0 .. N-1.
template <int... Is, typename F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, Is...>, F&& f) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;  // quiet NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// ---------------------------------------------------------------------------
// MX element formats. FMT is the matrix-core operand format code:
//   0 = e4m3 (FP8), 2 = e2m3 (FP6), 4 = e2m1 (FP4).
// ---------------------------------------------------------------------------
template <int FMT> struct Elem;
template <> struct Elem<0> {   // e4m3: bias 7, max 448 = 1.75 * 2^8, 0x7f is NaN
  static constexpr int kEBits = 4, kMBits = 3, kBias = 7, kMaxCode = 0x7e, kEMax = 8, kBits = 8;
  static constexpr float kMaxMant = 1.75f;
};
template <> struct Elem<2> {   // e2m3: bias 1, max 7.5 = 1.875 * 2^2
  static constexpr int kEBits = 2, kMBits = 3, kBias = 1, kMaxCode = 0x1f, kEMax = 2, kBits = 6;
  static constexpr float kMaxMant = 1.875f;
};
template <> struct Elem<4> {   // e2m1: bias 1, max 6 = 1.5 * 2^2
  static constexpr int kEBits = 2, kMBits = 1, kBias = 1, kMaxCode = 0x7, kEMax = 2, kBits = 4;
  static constexpr float kMaxMant = 1.5f;
};

// Block scale exponent: the smallest X in [-127, 127] with
// amax <= maxval * 2^X; amax == 0 gives 0. Writing amax = m * 2^f with m in
// [1, 2): X = f - emax if m <= max_mant, else f - emax + 1.
template <int FMT>
__device__ __forceinline__ int mx_scale_exp(float amax) {
  using E = Elem<FMT>;
  if (!(amax > 0.0f)) return 0;
  int ex;
  float m = frexpf(amax, &ex);  // amax = m * 2^ex, m in [0.5, 1)
  int x = (2.0f * m <= E::kMaxMant) ? (ex - 1 - E::kEMax) : (ex - E::kEMax);
  return x < -127 ? -127 : (x > 127 ? 127 : x);
}

// Round q (already divided by the block scale, |q| <= maxval) to the nearest
// element code, ties to even; the sign bit is q's sign bit.
template <int FMT>
__device__ __forceinline__ uint32_t mx_encode(float q) {
  using E = Elem<FMT>;
  constexpr int kEMin = 1 - E::kBias;
  const uint32_t sign = __float_as_uint(q) >> 31;
  const float a = fabsf(q);
  int ex = (int)((__float_as_uint(a) >> 23) & 0xffu) - 127;  // floor(log2 a) for normal a
  int e = ex < kEMin ? kEMin : ex;
  int n = (int)rintf(ldexpf(a, E::kMBits - e));  // exact scaling, then RNE
  if (n >= (1 << (E::kMBits + 1))) {             // rounded up into the next binade
    e += 1;
    n >>= 1;
  }
  uint32_t ef, mf;
  if (e == kEMin && n < (1 << E::kMBits)) {
    ef = 0;
    mf = (uint32_t)n;
  } else {
    ef = (uint32_t)(e - kEMin + 1);
    mf = (uint32_t)(n - (1 << E::kMBits));
  }
  uint32_t mag = (ef << E::kMBits) | mf;
  if (mag > (uint32_t)E::kMaxCode) mag = E::kMaxCode;
  return (sign << (E::kEBits + E::kMBits)) | mag;
}

// Four values already divided by their block scale (|q| <= 448) to e4m3
// codes, packed little-endian (value 0 in byte 0), by the hardware
// conversion: OCP e4m3, round to nearest even, subnormals kept, the sign of
// zero kept -- the same codes as mx_encode<0>.
__device__ __forceinline__ uint32_t e4m3_pack4(float a, float b, float c, float d) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return (uint32_t)w;
}

// ---------------------------------------------------------------------------
// Matrix core: D(16x16) += A(16x128) . B(128x16) with one E8M0 scale per lane
// per operand. Lane l supplies row (l % 16) of A and column (l % 16) of B for
// the 32-element K block (l / 16); its scale register holds that block's
// scale in the byte selected by OPSA / OPSB. D: lane l holds
// D[4 * (l / 16) + i][l % 16] in element i.
// FA is the A operand's element format code; B is always FP4 e2m1.
// ---------------------------------------------------------------------------
template <int FA, int OPSA, int OPSB>
__device__ __forceinline__ v4f mfma_scaled_16x16x128(const v8i& a, const v8i& b, const v4f& c,
                                                     int sa, int sb) {
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c, FA, 4, OPSA, sa, OPSB, sb);
}

// Wave-wide shuffles (ds_bpermute based).
__device__ __forceinline__ float shfl_xor_f(float v, int m) { return __shfl_xor(v, m, kWave); }
__device__ __forceinline__ int shfl_xor_i(int v, int m) { return __shfl_xor(v, m, kWave); }

// Value of the exchange partner at butterfly level L of a wave-wide
// reduction, by VALU lane moves (no LDS round trip): L = 0, 1 swap lanes
// inside each quad (xor 1, xor 2), L = 2, 3 rotate each row of 16 by 4 and 8
// (for a commutative reduction this covers the row like xor 4, xor 8), L = 4
// swaps rows 0 <-> 1 and 2 <-> 3, L = 5 the two halves of the wave.
template <int L>
__device__ __forceinline__ int wave_partner(int v) {
  if constexpr (L == 0) return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);
  if constexpr (L == 1) return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);
  if constexpr (L == 2) return __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);
  if constexpr (L == 3) return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false);
  const int lane = (int)(threadIdx.x % kWave);
  if constexpr (L == 4) {
    const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
    return (int)(((lane >> 4) & 1) ? r[0] : r[1]);
  }
  const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
  return (int)((lane >> 5) ? r[0] : r[1]);
}

// Wave-wide arg-max of (value, index) pairs: the largest value, ties to the
// lower index; every lane ends with the result (a unique answer, so the
// reduction order does not matter).
__device__ __forceinline__ void wave_argmax(float& bv, int& bi) {
  auto step = [&](float ov, int oi) {
    if (ov > bv || (ov == bv && oi < bi)) {
      bv = ov;
      bi = oi;
    }
  };
  step(__int_as_float(wave_partner<0>(__float_as_int(bv))), wave_partner<0>(bi));
  step(__int_as_float(wave_partner<1>(__float_as_int(bv))), wave_partner<1>(bi));
  step(__int_as_float(wave_partner<2>(__float_as_int(bv))), wave_partner<2>(bi));
  step(__int_as_float(wave_partner<3>(__float_as_int(bv))), wave_partner<3>(bi));
  step(__int_as_float(wave_partner<4>(__float_as_int(bv))), wave_partner<4>(bi));
  step(__int_as_float(wave_partner<5>(__float_as_int(bv))), wave_partner<5>(bi));
}

// Lane j's value (j wave-uniform), read through a scalar register.
__device__ __forceinline__ float lane_value(float v, int j) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), j));
}

// Map a linear workgroup id to a logical tile id so that consecutive logical
// ids run on the same XCD: the dispatcher sends workgroup b to XCD b % 8.
// n must be a multiple of 8.
__device__ __forceinline__ int xcd_remap(int b, int n) { return (b & 7) * (n >> 3) + (b >> 3); }

// Exclusive scan of v over the block (blockDim.x == 1024); returns the prefix
// and writes the block total to *total.
__device__ __forceinline__ int block_exclusive_scan_1024(int v, int* total) {
  __shared__ int wsum[16];
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  int inc = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int o = __shfl_up(inc, d, kWave);
    if (lane >= d) inc += o;
  }
  if (lane == kWave - 1) wsum[w] = inc;
  __syncthreads();
  if (w == 0) {
    int s = lane < 16 ? wsum[lane] : 0;
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) {
      const int o = __shfl_up(s, d, kWave);
      if (lane >= d) s += o;
    }
    if (lane < 16) wsum[lane] = s;  // inclusive
  }
  __syncthreads();
  const int before = w ? wsum[w - 1] : 0;
  *total = wsum[15];
  __syncthreads();
  return before + inc - v;
}

}  // namespace moe
