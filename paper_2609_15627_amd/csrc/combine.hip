// a7: fixed-order combine of the per-(token, slot) fp32 partials.
//
// out[t, h] = bf16_rne(acc), acc = 0, acc = fmaf(w[t, j], P[t*k_total + j, h], acc)
// for j = 0 .. k_total-1 in this order. One thread per 8 consecutive h:
// two 16-byte loads per slot, one 16-byte store. No atomics, so the result is
// the same bits on every run.
#include "moe_dev.h"
#include "moe_launch.h"

namespace moe {

__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ P,
                                                      const float* __restrict__ w, int T, int H,
                                                      int kt, uint16_t* __restrict__ out) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int h8 = H / 8;
  if (idx >= (long)T * h8) return;
  const int t = (int)(idx / h8), c = (int)(idx % h8);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < kt; ++j) {
    const float wj = w[(size_t)t * kt + j];
    const float4* src = reinterpret_cast<const float4*>(P + ((size_t)t * kt + j) * H) + 2 * c;
    const float4 p0 = src[0], p1 = src[1];
    acc[0] = fmaf(wj, p0.x, acc[0]);
    acc[1] = fmaf(wj, p0.y, acc[1]);
    acc[2] = fmaf(wj, p0.z, acc[2]);
    acc[3] = fmaf(wj, p0.w, acc[3]);
    acc[4] = fmaf(wj, p1.x, acc[4]);
    acc[5] = fmaf(wj, p1.y, acc[5]);
    acc[6] = fmaf(wj, p1.z, acc[6]);
    acc[7] = fmaf(wj, p1.w, acc[7]);
  }
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = f32_to_bf16_rne(acc[2 * i]) | (f32_to_bf16_rne(acc[2 * i + 1]) << 16);
  reinterpret_cast<uint4*>(out + (size_t)t * H)[c] = make_uint4(o[0], o[1], o[2], o[3]);
}

hipError_t launch_combine(const float* partials, const float* w, int T, int H, int k_total,
                          uint16_t* out, hipStream_t s) {
  const long n = (long)T * (H / 8);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(combine_kernel, dim3((int)((n + 255) / 256)), dim3(256), 0, s, partials, w, T,
                     H, k_total, out);
  return hipGetLastError();
}

}  // namespace moe
