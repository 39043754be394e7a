// a4: per-32 MX quantisation of bf16 activations, one thread per block of 32
// consecutive elements (the block arithmetic is quant_block in quant_dev.h).
#include "moe_launch.h"
#include "quant_dev.h"

namespace moe {

int act_bits(int fmt) { return fmt == kFmtBf16 ? 16 : (fmt == 0 ? 8 : (fmt == 2 ? 6 : 4)); }
int ws_act_bits(int fmt) { return fmt == 2 ? 8 : act_bits(fmt); }

template <int FMT>
__global__ __launch_bounds__(256) void quant_act_kernel(const uint16_t* __restrict__ x, long nblk,
                                                        uint8_t* __restrict__ codes,
                                                        uint8_t* __restrict__ scales) {
  const long b = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (b < nblk) quant_block<FMT>(x, b, codes, scales);
}

hipError_t launch_quantize_act(const uint16_t* x, long rows, int K, int fmt, uint8_t* codes,
                               uint8_t* scales, hipStream_t s) {
  const long nblk = rows * (K / 32);
  if (nblk == 0) return hipSuccess;
  const int blocks = (int)((nblk + 255) / 256);
  if (fmt == 0)
    hipLaunchKernelGGL(quant_act_kernel<0>, dim3(blocks), dim3(256), 0, s, x, nblk, codes, scales);
  else if (fmt == 2)
    hipLaunchKernelGGL(quant_act_kernel<2>, dim3(blocks), dim3(256), 0, s, x, nblk, codes, scales);
  else
    hipLaunchKernelGGL(quant_act_kernel<4>, dim3(blocks), dim3(256), 0, s, x, nblk, codes, scales);
  return hipGetLastError();
}

}  // namespace moe
