// a7: fixed-order combine of the per-(token, slot) fp32 partials.
//
// out[t, h] = bf16_rne(acc), acc = 0, acc = fmaf(w[t, j], P[t*k_total + j, h], acc)
// for j = 0 .. k_total-1 in this order. No atomics, so the result is the
// same bits on every run. Two layouts of the same arithmetic:
//  - few tokens: one thread per 8 consecutive h, two 16-byte loads per slot
//    (all slots in flight at once), one 16-byte store;
//  - many tokens (the partials far exceed the caches and are read once): one
//    thread per 4 consecutive h, one 16-byte non-temporal load per slot, so
//    each load instruction of a wave reads 1 KiB of one partial row
//    contiguously (measured 5.3 -> 6.2 TB/s on a 537 MB partial buffer).
#include "moe_dev.h"
#include "moe_launch.h"

namespace moe {

// KT > 0: the slot count is known at compile time, so every slot's loads
// are issued before the first multiply-add (the adds still run in slot
// order); KT == 0: any slot count, one slot at a time.
template <int KT>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ P,
                                                      const float* __restrict__ w, int T, int H,
                                                      int kt, uint16_t* __restrict__ out) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int h8 = H / 8;
  if (idx >= (long)T * h8) return;
  const int t = (int)(idx / h8), c = (int)(idx % h8);
  if constexpr (KT > 0) kt = KT;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto add = [&](float wj, const float4& p0, const float4& p1) {
    acc[0] = fmaf(wj, p0.x, acc[0]);
    acc[1] = fmaf(wj, p0.y, acc[1]);
    acc[2] = fmaf(wj, p0.z, acc[2]);
    acc[3] = fmaf(wj, p0.w, acc[3]);
    acc[4] = fmaf(wj, p1.x, acc[4]);
    acc[5] = fmaf(wj, p1.y, acc[5]);
    acc[6] = fmaf(wj, p1.z, acc[6]);
    acc[7] = fmaf(wj, p1.w, acc[7]);
  };
  const float4* src = reinterpret_cast<const float4*>(P + (size_t)t * kt * H) + 2 * c;
  const size_t row4 = (size_t)H / 4;  // float4 per partial row
  if constexpr (KT > 0) {
    float4 p[KT][2];
    float wv[KT];
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      p[j][0] = src[j * row4];
      p[j][1] = src[j * row4 + 1];
      wv[j] = w[(size_t)t * KT + j];
    }
#pragma unroll
    for (int j = 0; j < KT; ++j) add(wv[j], p[j][0], p[j][1]);
  } else {
    for (int j = 0; j < kt; ++j) add(w[(size_t)t * kt + j], src[j * row4], src[j * row4 + 1]);
  }
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(acc[2 * i]) | (f32_to_bf16_rne(acc[2 * i + 1]) << 16);
  reinterpret_cast<uint4*>(out + (size_t)t * H)[c] = make_uint4(o[0], o[1], o[2], o[3]);
}

typedef float f4v __attribute__((ext_vector_type(4)));

template <int KT>
__global__ __launch_bounds__(256) void combine_wide_kernel(const float* __restrict__ P,
                                                           const float* __restrict__ w, int T,
                                                           int H, uint16_t* __restrict__ out) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int h4 = H / 4;
  if (idx >= (long)T * h4) return;
  const int t = (int)(idx / h4), c = (int)(idx % h4);
  const f4v* src = reinterpret_cast<const f4v*>(P + (size_t)t * KT * H) + c;
  const size_t row4 = (size_t)H / 4;
  f4v p[KT];
  float wv[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    p[j] = __builtin_nontemporal_load(src + j * row4);
    wv[j] = w[(size_t)t * KT + j];
  }
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    acc[0] = fmaf(wv[j], p[j].x, acc[0]);
    acc[1] = fmaf(wv[j], p[j].y, acc[1]);
    acc[2] = fmaf(wv[j], p[j].z, acc[2]);
    acc[3] = fmaf(wv[j], p[j].w, acc[3]);
  }
  reinterpret_cast<uint2*>(out + (size_t)t * H)[c] =
      make_uint2(f32_to_bf16_rne(acc[0]) | (f32_to_bf16_rne(acc[1]) << 16),
                 f32_to_bf16_rne(acc[2]) | (f32_to_bf16_rne(acc[3]) << 16));
}

// Tokens from which the wide layout is used.
constexpr int kWideTokens = 256;

hipError_t launch_combine(const float* partials, const float* w, int T, int H, int k_total,
                          uint16_t* out, hipStream_t s) {
  if (T >= kWideTokens && k_total >= 1 && k_total <= 16) {
    const long n4 = (long)T * (H / 4);
    const dim3 g4((int)((n4 + 255) / 256)), b4(256);
    switch (k_total) {
#define MOE_COMBINE_WIDE(K)                                                                   \
  case K:                                                                                     \
    hipLaunchKernelGGL(combine_wide_kernel<K>, g4, b4, 0, s, partials, w, T, H, out);        \
    break;
      MOE_COMBINE_WIDE(1) MOE_COMBINE_WIDE(2) MOE_COMBINE_WIDE(3) MOE_COMBINE_WIDE(4)
      MOE_COMBINE_WIDE(5) MOE_COMBINE_WIDE(6) MOE_COMBINE_WIDE(7) MOE_COMBINE_WIDE(8)
      MOE_COMBINE_WIDE(9) MOE_COMBINE_WIDE(10) MOE_COMBINE_WIDE(11) MOE_COMBINE_WIDE(12)
      MOE_COMBINE_WIDE(13) MOE_COMBINE_WIDE(14) MOE_COMBINE_WIDE(15) MOE_COMBINE_WIDE(16)
#undef MOE_COMBINE_WIDE
    }
    return hipGetLastError();
  }
  const long n = (long)T * (H / 8);
  if (n == 0) return hipSuccess;
  const dim3 grid((int)((n + 255) / 256)), block(256);
  switch (k_total) {
#define MOE_COMBINE_KT(K)                                                                  \
  case K:                                                                                  \
    hipLaunchKernelGGL(combine_kernel<K>, grid, block, 0, s, partials, w, T, H, k_total, out); \
    break;
    MOE_COMBINE_KT(1) MOE_COMBINE_KT(2) MOE_COMBINE_KT(3) MOE_COMBINE_KT(4) MOE_COMBINE_KT(5)
    MOE_COMBINE_KT(6) MOE_COMBINE_KT(7) MOE_COMBINE_KT(8) MOE_COMBINE_KT(9) MOE_COMBINE_KT(10)
    MOE_COMBINE_KT(11) MOE_COMBINE_KT(12) MOE_COMBINE_KT(13) MOE_COMBINE_KT(14) MOE_COMBINE_KT(15)
    MOE_COMBINE_KT(16)
#undef MOE_COMBINE_KT
    default:
      hipLaunchKernelGGL(combine_kernel<0>, grid, block, 0, s, partials, w, T, H, k_total, out);
  }
  return hipGetLastError();
}

}  // namespace moe
