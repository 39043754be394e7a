// The expert-weight layout of the grouped GEMM: FP4 code rows (K/2 bytes
// each) in groups of 16, each group's bytes ordered by 64-byte K piece, then
// by row. One K piece of a group (16 rows x 128 K elements) is then 1 KiB of
// contiguous memory, which is what every kernel that reads weights fetches
// per load instruction (a 16-row operand block of the 16x16x128 product, or
// one 16-row DMA instruction of the LDS-tiled geometries): the weight stream
// reads whole contiguous KiB instead of 64-byte pieces of 16 rows spread
// over 16 * K/2 bytes. Byte c of K piece q of row 16 g + r sits at
// 16 g * K/2 + 1024 q + 64 r + c. A group occupies the same byte range in
// both layouts, so row and expert offsets are unchanged.
#include "moe_launch.h"

namespace moe {

// One thread per 16 output bytes; indices in 64 bits (a whole model's
// weights pass in one call).
__global__ __launch_bounds__(256) void pack_fp4_kernel(const uint8_t* __restrict__ w,
                                                       uint8_t* __restrict__ out, long nchunk,
                                                       int kbytes) {
  const long o = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= nchunk) return;
  const long gbytes = 16L * kbytes;  // bytes of one 16-row group
  const long byte = 16 * o;
  const long grp = byte / gbytes;
  const int within = (int)(byte - grp * gbytes);
  const int q = within >> 10, r = (within >> 6) & 15, c = within & 63;
  const long src = grp * gbytes + (long)r * kbytes + 64L * q + c;
  *reinterpret_cast<uint4*>(out + byte) = *reinterpret_cast<const uint4*>(w + src);
}

hipError_t launch_pack_fp4(const uint8_t* w, uint8_t* out, long rows, int K, hipStream_t s) {
  const int kbytes = K / 2;
  const long nchunk = rows * kbytes / 16;
  if (nchunk == 0) return hipSuccess;
  const long blocks = (nchunk + 255) / 256;
  hipLaunchKernelGGL(pack_fp4_kernel, dim3((unsigned)blocks), dim3(256), 0, s, w, out, nchunk,
                     kbytes);
  return hipGetLastError();
}

}  // namespace moe
