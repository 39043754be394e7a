// a5 / a6: grouped FP4 expert GEMMs, weight-streaming geometry with register
// double buffering (one wave per workgroup).
//
// Work item: (row tile of up to 16 sorted rows of one expert, N tile). Every
// workgroup streams its N tile of the expert's packed FP4 weights from HBM
// exactly once, over the whole K extent, and multiplies it with the tile's
// activation rows on the block-scaled matrix cores (16x16x128, FP4 weights
// consumed directly: no unpacking, no offline expansion -- the paper found
// that expanding FP4 to INT8 doubled weight traffic and slowed the gate
// kernel; Rejected or reverted directions).
//
// Operands go straight from global memory into registers, double-buffered
// one step of 128*J K elements ahead (frag_load / stream_k). The weight
// rows' E8M0 scales are the exception: each workgroup copies its rows' whole
// scale rows into LDS once, up front (whole contiguous lines), and the K
// loop reads them there. Gathering a few scale bytes per row per step from global
// memory re-touched each 128-byte scale line over the whole K loop, long
// enough for it to leave L2 between uses: measured on the decode layer, the
// weight scales were fetched about six times over (0.65 GB of 2.58 GB).
//
// Stage 1 (gate/up): each wave owns 16*NBW h columns; it streams those gate
// rows and the matching up rows, so SwiGLU and the per-32 re-quantisation of
// h (the quantisation block spans two 16-column tiles of the same wave) run in
// registers. Stage 2 (down): each wave owns 16*NBW output columns of H and
// writes fp32 partials to the unique row a = sorted[r] of every assignment.
#include "gemm_common.h"
#include "gemm_launch.h"

namespace moe {

// Copy nbytes (a multiple of 16, 16-byte aligned at both ends) of
// contiguous global memory to LDS: whole 1 KiB runs per wave instruction.
// Plain loads and LDS stores rather than LDS DMA: with a DMA pending, the
// compiler's wait insertion cannot tell the later global loads apart and
// waits for all of them in the streaming loop.
__device__ __forceinline__ void copy_rows_to_lds(uint8_t* dst, const uint8_t* src, int nbytes,
                                                 int lane) {
  for (int o = 16 * lane; o < nbytes; o += 1024)
    *reinterpret_cast<v4u*>(dst + o) = *reinterpret_cast<const v4u*>(src + o);
}

// Copy 16 gathered rows of kb bytes each (kb a multiple of 4) to LDS as a
// dense [16][kb] block; rows(r) gives row r's address.
template <typename RowFn>
__device__ __forceinline__ void copy_gather16_to_lds(uint8_t* dst, RowFn rows, int kb, int lane) {
  const int words = kb / 4;  // 4-byte pieces per row
  for (int q = lane; q < 16 * words; q += 64)
    *reinterpret_cast<uint32_t*>(dst + 4 * q) =
        *reinterpret_cast<const uint32_t*>(rows(q / words) + 4 * (q % words));
}

// Registers of one K step: activation pieces + scales, NB weight rows + scales.
template <int FA, int J, int NB>
struct Frag {
  static constexpr int kAV = J * ActBytes<FA>::kBlock / 16;
  v4u a[kAV];
  uint32_t as;
  v4u b[NB][J];
  uint32_t bs[NB];
};

// gather_scales on a weight scale row held in LDS (byte offset `o`).
template <int J>
__device__ __forceinline__ uint32_t gather_scales_lds(uint32_t o, int g) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const uint32_t* w = reinterpret_cast<const uint32_t*>(lds + o);
  uint32_t r = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) r |= ((w[j] >> (8 * g)) & 0xffu) << (8 * j);
  return r;
}

// Loads of one K step starting at 32-element block `step` (a multiple of 4).
// Product j of the step covers the 128 elements [step*32 + 128j, +128):
//  - a weight lane (column c16, lane group g) supplies block step + 4j + g,
//    16 contiguous bytes; one load instruction reads 64 contiguous bytes of
//    each of the wave's 16 rows;
//  - an FP4 activation lane does the same on its row;
//  - an FP8 activation lane supplies 16-element halves: the matrix core reads
//    an FP8 lane's bytes 0-15 as K = 16g.. and bytes 16-31 as K = 64 + 16g..
//    of the product's 128 (an FP4 lane's 32 elements are K = 32g..), so it
//    takes elements [16g, 16g+16) and [64+16g, 64+16g+16) of the product;
//  - scales: the scale lane g is block g of the product (block 4j + g).
//  - every lane loads unconditionally (rows past the tile's end read a valid
//    row of the tile; their accumulator rows are never stored), so the loop
//    holds no branches around loads and the waits count exact.
template <int FA, int J, int NB, bool NT>
__device__ __forceinline__ void frag_load(Frag<FA, J, NB>& f, const uint8_t* a_row,
                                          uint32_t as_lds, const uint8_t* const* b_rows,
                                          const uint32_t* bs_lds, int step, int g) {
  {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if constexpr (FA == 0) {
        const uint8_t* base = a_row + (size_t)step * 32 + 128 * j + 16 * g;
        f.a[2 * j] = ld16<false>(base);
        f.a[2 * j + 1] = ld16<false>(base + 64);
      } else {
        f.a[j] = ld16<false>(a_row + (size_t)(step + 4 * j + g) * 16);
      }
    }
    f.as = gather_scales_lds<J>(as_lds + step, g);
  }
#pragma unroll
  for (int n = 0; n < NB; ++n) {
#pragma unroll
    for (int j = 0; j < J; ++j) f.b[n][j] = ld16<NT>(b_rows[n] + (size_t)(step + 4 * j + g) * 16);
    f.bs[n] = gather_scales_lds<J>(bs_lds[n] + step, g);
  }
}

template <int FA, int J, int NB>
__device__ __forceinline__ void frag_mma(const Frag<FA, J, NB>& f, v4f* acc) {
  static_for<J>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    v8i a;
    if constexpr (FA == 0) {
      const v4u lo = f.a[2 * j], hi = f.a[2 * j + 1];
      a = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    } else {
      const v4u lo = f.a[j];
      a = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
    }
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const v4u bq = f.b[n][j];
      const v8i b = v8i{(int)bq.x, (int)bq.y, (int)bq.z, (int)bq.w, 0, 0, 0, 0};
      acc[n] = mfma_scaled_16x16x128<FA, j, j>(a, b, acc[n], (int)f.as, (int)f.bs[n]);
    }
  });
}

// Full K loop for one wave: NB weight rows (16 each, one per lane column),
// one 16-row activation tile. K = nblk32 * 32 with nblk32 % 4 == 0. Steps of
// 4J blocks are double-buffered: the steady-state loop always has the next
// step's loads in flight while the current step's products run, with no
// branch around a load, so each wait covers exactly the step it needs. A
// tail of single 128-element steps follows.
template <int FA, int J, int NB, bool NT>
__device__ __forceinline__ void stream_k(const uint8_t* a_row, uint32_t as_lds,
                                         const uint8_t* const* b_rows, const uint32_t* bs_lds,
                                         int nblk32, int g, v4f* acc) {
  const int kc_blocks = 4 * J;
  const int nsteps = nblk32 / kc_blocks;
  if (nsteps > 0) {
    Frag<FA, J, NB> f0, f1;
    frag_load<FA, J, NB, NT>(f0, a_row, as_lds, b_rows, bs_lds, 0, g);
    int c = 0;
    for (; c + 2 < nsteps; c += 2) {  // f0 holds step c; steps c + 1 and c + 2 exist
      frag_load<FA, J, NB, NT>(f1, a_row, as_lds, b_rows, bs_lds, (c + 1) * kc_blocks, g);
      frag_mma<FA, J, NB>(f0, acc);
      frag_load<FA, J, NB, NT>(f0, a_row, as_lds, b_rows, bs_lds, (c + 2) * kc_blocks, g);
      frag_mma<FA, J, NB>(f1, acc);
    }
    if (c + 1 < nsteps) {
      frag_load<FA, J, NB, NT>(f1, a_row, as_lds, b_rows, bs_lds, (c + 1) * kc_blocks, g);
      frag_mma<FA, J, NB>(f0, acc);
      frag_mma<FA, J, NB>(f1, acc);
    } else {
      frag_mma<FA, J, NB>(f0, acc);
    }
  }
  for (int blk = nsteps * kc_blocks; blk < nblk32; blk += 4) {
    Frag<FA, 1, NB> f;
    frag_load<FA, 1, NB, NT>(f, a_row, as_lds, b_rows, bs_lds, blk, g);
    frag_mma<FA, 1, NB>(f, acc);
  }
}

template <int FA, int J, int NBW, bool NT, int WPB>
__global__ __launch_bounds__(64 * WPB) void s1_stream_kernel(S1Args p) {
  static_assert(NBW % 2 == 0, "a quantisation block spans two 16-column tiles");
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int hc0 = nt * (WPB * NBW * 16) + w * (NBW * 16);  // first h column of this wave

  const int tok = p.sorted[row0 + (c16 < nrows ? c16 : 0)] / p.k_total;
  const uint8_t* a_row = p.xq + (size_t)tok * (p.H / 32) * kAB;

  // Scale rows to LDS first: the tile's 16 activation rows, then the wave's
  // 16 NBW gate rows and the matching up rows; the K loop streams the codes.
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int kb = p.H / 32;
  const size_t ebase = (size_t)e * 2 * p.I;
  uint8_t* my = lds + w * ((2 * NBW + 1) * 16 * kb);
  copy_gather16_to_lds(
      my,
      [&](int r) {
        const int t = p.sorted[row0 + (r < nrows ? r : 0)] / p.k_total;
        return p.xs + (size_t)t * kb;
      },
      kb, lane);
  uint8_t* myb = my + 16 * kb;
  copy_rows_to_lds(myb, p.w13s + (ebase + hc0) * kb, NBW * 16 * kb, lane);
  copy_rows_to_lds(myb + NBW * 16 * kb, p.w13s + (ebase + p.I + hc0) * kb, NBW * 16 * kb, lane);
  const uint32_t as_lds = (uint32_t)(my - lds) + c16 * kb;
  const uint8_t* b_rows[2 * NBW];
  uint32_t bs_lds[2 * NBW];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t gr = ebase + hc0 + 16 * b + c16;  // gate row
    const size_t ur = gr + p.I;                    // up row
    b_rows[b] = p.w13 + gr * (p.H / 2);
    b_rows[NBW + b] = p.w13 + ur * (p.H / 2);
    bs_lds[b] = (uint32_t)(myb - lds) + (16 * b + c16) * kb;
    bs_lds[NBW + b] = (uint32_t)(myb - lds) + (NBW * 16 + 16 * b + c16) * kb;
  }
  v4f acc[2 * NBW];
#pragma unroll
  for (int n = 0; n < 2 * NBW; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k<FA, J, 2 * NBW, NT>(a_row, as_lds, b_rows, bs_lds, p.H / 32, g, acc);

  s1_epilogue<FA, NBW>(acc, p, row0, nrows, hc0, g, c16);
}

template <int FA, int J, int NBW, bool NT, int WPB>
__global__ __launch_bounds__(64 * WPB) void s2_stream_kernel(S2Args p) {
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int nc0 = nt * (WPB * NBW * 16) + w * (NBW * 16);  // first output column of this wave

  const size_t ar = (size_t)row0 + (c16 < nrows ? c16 : 0);
  const uint8_t* a_row = p.hq + ar * (p.I / 32) * kAB;

  // Scale rows to LDS first: the tile's 16 activation rows, then the wave's
  // 16 NBW consecutive weight rows.
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int kb = p.I / 32;
  uint8_t* my = lds + w * ((NBW + 1) * 16 * kb);
  copy_gather16_to_lds(
      my, [&](int r) { return p.hs + ((size_t)row0 + (r < nrows ? r : 0)) * kb; }, kb, lane);
  uint8_t* myb = my + 16 * kb;
  copy_rows_to_lds(myb, p.w2s + ((size_t)e * p.H + nc0) * kb, NBW * 16 * kb, lane);
  const uint32_t as_lds = (uint32_t)(my - lds) + c16 * kb;
  const uint8_t* b_rows[NBW];
  uint32_t bs_lds[NBW];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t rr = (size_t)e * p.H + nc0 + 16 * b + c16;
    b_rows[b] = p.w2 + rr * (p.I / 2);
    bs_lds[b] = (uint32_t)(myb - lds) + (16 * b + c16) * kb;
  }
  v4f acc[NBW];
#pragma unroll
  for (int n = 0; n < NBW; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k<FA, J, NBW, NT>(a_row, as_lds, b_rows, bs_lds, p.I / 32, g, acc);

  s2_epilogue<NBW>(acc, p, row0, nrows, nc0, g, c16);
}

template <int FA, int NBW1>
static void launch_s1(const S1Args& p, long mt, hipStream_t s) {
  S1Args q = p;
  q.t.n_ntiles = p.I / (NBW1 * 16);
  q.t.ngroup = n_group_of(q.t.n_ntiles);
  const long n = mt * q.t.n_ntiles;
  hipLaunchKernelGGL((s1_stream_kernel<FA, 2, NBW1, false, 1>), dim3((int)((n + 7) / 8 * 8)),
                     dim3(64), (2 * NBW1 + 1) * 16 * (p.H / 32), s, q);
}

template <int FA, int NBW2>
static void launch_s2(const S2Args& p, long mt, hipStream_t s) {
  S2Args q = p;
  q.t.n_ntiles = p.H / (NBW2 * 16);
  q.t.ngroup = n_group_of(q.t.n_ntiles);
  const long n = mt * q.t.n_ntiles;
  hipLaunchKernelGGL((s2_stream_kernel<FA, 2, NBW2, false, 1>), dim3((int)((n + 7) / 8 * 8)),
                     dim3(64), (NBW2 + 1) * 16 * (p.I / 32), s, q);
}

// One wave per workgroup, steps of 256 K elements, 32 h columns per wave in
// stage 1 and 64 output columns per wave in stage 2. Measured alternatives
// (non-temporal weight loads, 2 or 4 waves per workgroup, 128- or 512-element
// steps, deeper register rings, direct-to-LDS rings, persistent waves) were
// slower on the decode layer.
void launch_s1_stream(const S1Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_s1<0, 2>(p, mt, s);
  else launch_s1<4, 2>(p, mt, s);
}

void launch_s2_stream(const S2Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_s2<0, 4>(p, mt, s);
  else launch_s2<4, 4>(p, mt, s);
}

// ---------------------------------------------------------------------------
// Probe: one 16x16x128 product with the GEMM's operand and scale placement.
// ---------------------------------------------------------------------------
template <int FA>
__global__ void probe_kernel(const uint8_t* a, const uint8_t* sa, const uint8_t* b,
                             const uint8_t* sb, float* d) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int lane = threadIdx.x, g = lane >> 4, c16 = lane & 15;
  // scales live in LDS as in the GEMM: row c16's four bytes of A at 4 c16,
  // of B at 64 + 4 c16
  if (g == 0) {
    *reinterpret_cast<uint32_t*>(lds + 4 * c16) = *reinterpret_cast<const uint32_t*>(sa + 4 * c16);
    *reinterpret_cast<uint32_t*>(lds + 64 + 4 * c16) =
        *reinterpret_cast<const uint32_t*>(sb + 4 * c16);
  }
  __syncthreads();
  constexpr int kAB = ActBytes<FA>::kBlock;
  const uint8_t* ar = a + (size_t)c16 * 4 * kAB;
  const uint8_t* br = b + (size_t)c16 * 64;
  const uint32_t bso = 64 + 4 * c16;
  v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
  Frag<FA, 1, 1> f;
  frag_load<FA, 1, 1, false>(f, ar, 4 * c16, &br, &bso, 0, g);
  frag_mma<FA, 1, 1>(f, &acc);
#pragma unroll
  for (int i = 0; i < 4; ++i) d[(4 * g + i) * 16 + c16] = acc[i];
}

hipError_t launch_probe(const uint8_t* a, const uint8_t* sa, int fmt, const uint8_t* b,
                        const uint8_t* sb, float* d, hipStream_t s) {
  if (fmt == 0)
    hipLaunchKernelGGL(probe_kernel<0>, dim3(1), dim3(64), 128, s, a, sa, b, sb, d);
  else if (fmt == 4)
    hipLaunchKernelGGL(probe_kernel<4>, dim3(1), dim3(64), 128, s, a, sa, b, sb, d);
  else
    return hipErrorNotSupported;
  return hipGetLastError();
}

}  // namespace moe
