// a5 / a6: grouped FP4 expert GEMMs, weight-streaming geometry with register
// double or triple buffering (one wave per workgroup, or for stage 1 two
// waves that split the K extent).
//
// Work item: (row tile of up to 16 sorted rows of one expert, N tile). Every
// workgroup streams its N tile of the expert's packed FP4 weights from HBM
// exactly once, over the whole K extent, and multiplies it with the tile's
// activation rows on the block-scaled matrix cores (16x16x128, FP4 weights
// consumed directly: no unpacking, no offline expansion -- the paper found
// that expanding FP4 to INT8 doubled weight traffic and slowed the gate
// kernel; Rejected or reverted directions).
//
// Measured on the decode layer, and what it shaped:
//  - under full HBM load a load takes tens of microseconds, so a
//    workgroup's start (tile, sorted row, token, then scale rows: a chain of
//    dependent loads) is as long as its streaming. The first step's code
//    loads go out before the scale rows are staged, so those two latencies
//    overlap. (Streaming two N tiles per workgroup to pay the chain once was
//    slower: fewer, longer workgroups leave a ragged last wave.)
//  - weight scales gathered a few bytes per row per step from global memory
//    were fetched about six times over (each 128-byte line re-touched across
//    the whole K loop, long enough to leave L2) and made each step wait for
//    all outstanding loads. The workgroup copies its whole scale rows into
//    LDS by DMA instead;
//  - the compiler's wait insertion only counts exactly while every
//    outstanding vector memory operation is an ordinary load it can see: an
//    LDS DMA, an inline-asm LDS read, or stores in flight make it wait for
//    everything. So one explicit full wait follows the prologue, and the
//    step loop has no DMA, no stores and no wave-wide branch around a load;
//    each step's loads go out as one group ahead of the products that do not
//    need them;
//  - a decode tile holds two or three of its 16 rows: lanes of the rows past
//    the end skip their activation loads (lane-masked; they multiply zeros),
//    which made stage 1 about 3% faster.
//
// Stage 1 (gate/up): each wave owns 16*NBW h columns; it streams those gate
// rows and the matching up rows, so SwiGLU and the per-32 re-quantisation of
// h (the quantisation block spans two 16-column tiles of the same wave) run
// in registers. Stage 2 (down): each wave owns 16*NBW output columns and
// writes fp32 partials to the unique row a = sorted[r] of every assignment.
#include "gemm_common.h"
#include "gemm_launch.h"

namespace moe {



// 16 gathered rows of kb bytes each (kb a multiple of 4) to LDS as a dense
// [16][kb] block by 4-byte DMA; rows(r) gives row r's address.
template <typename RowFn>
__device__ __forceinline__ void dma_gather16(uint8_t* dst, RowFn rows, int kb, int lane) {
  const int words = kb / 4;
  for (int o = 0; o < 16 * words; o += 64) {
    const int q = o + lane;
    if (q < 16 * words)
      __builtin_amdgcn_global_load_lds(rows(q / words) + 4 * (q % words),
                                       (lds_ptr_t*)(dst + 4 * o), 4, 0, 0);
  }
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

// Code loads of one K step starting at 32-element block `step` (a multiple
// of 4). Product j of the step covers the 128 elements [step*32 + 128j, +128):
//  - a weight lane (column c16, lane group g) supplies block step + 4j + g,
//    16 contiguous bytes; one load instruction reads the 16 rows' 64-byte
//    pieces of one K piece, a contiguous KiB in the block layout;
//  - an FP4 activation lane does the same on its row;
//  - an FP8 activation lane supplies 16-element halves: the matrix core reads
//    an FP8 lane's bytes 0-15 as K = 16g.. and bytes 16-31 as K = 64 + 16g..
//    of the product's 128 (an FP4 lane's 32 elements are K = 32g..), so it
//    takes elements [16g, 16g+16) and [64+16g, 64+16g+16) of the product;
//  - scales: the scale lane g is block g of the product (block 4j + g).
// Every lane loads (rows past the tile's end read a valid row of the tile;
// their accumulator rows are never stored).
template <int FA, int J, int NB>
__device__ __forceinline__ void frag_codes(Frag<FA, J, NB>& f, const uint8_t* a_row,
                                           const uint8_t* const* b_rows, size_t b_off, int step,
                                           int g, bool av = true) {
  // the step's loads go out as one group, ahead of the products that follow
  // them in program order (the scheduler would otherwise interleave them with
  // those products and leave each load only a few instructions of lead)
  __builtin_amdgcn_sched_barrier(0);
  if (av) {  // lanes of rows past the tile's end skip their activation loads
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if constexpr (FA == 0) {
        const uint8_t* base = a_row + (size_t)step * 32 + 128 * j + 16 * g;
        f.a[2 * j] = ld16<false>(base);
        f.a[2 * j + 1] = ld16<false>(base + 64);
      } else if constexpr (FA == 2) {  // block step + 4j + g: the 32-byte slot
        const uint8_t* base = a_row + (size_t)(step + 4 * j + g) * 32;
        f.a[2 * j] = ld16<false>(base);
        f.a[2 * j + 1] = ld16<false>(base + 16);
      } else {
        f.a[j] = ld16<false>(a_row + (size_t)(step + 4 * j + g) * 16);
      }
    }
  }
  // weights in the block layout (moe_pack_fp4_weights): b_rows[n] is this
  // lane's 64-byte row piece of K piece 0 of its 16-row group; product j of
  // the step is K piece step / 4 + j, one contiguous KiB for the 64 lanes,
  // read with the streaming (non-temporal) policy, which pays for whole
  // contiguous KiB reads
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int j = 0; j < J; ++j)
      f.b[n][j] = ld16<true>(b_rows[n] + b_off + (size_t)(step / 4 + j) * 1024 + 16 * g);
  __builtin_amdgcn_sched_barrier(0);
}

// Byte g of each of the J scale words packed into bytes 0..J-1.
template <int J>
__device__ __forceinline__ uint32_t pick_scales(const uint32_t* w, int g) {
  uint32_t r = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) r |= ((w[j] >> (8 * g)) & 0xffu) << (8 * j);
  return r;
}

// Scales of step `step` into f: activation row at LDS byte offset xa,
// weight rows at wbuf + wo[n].
template <int FA, int J, int NB>
__device__ __forceinline__ void frag_scales(Frag<FA, J, NB>& f, uint32_t xa, uint32_t wbuf,
                                            const uint32_t* wo, int step, int g) {
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  uint32_t w[J];
#pragma unroll
  for (int j = 0; j < J; ++j) w[j] = *reinterpret_cast<const uint32_t*>(lds + xa + step + 4 * j);
  f.as = pick_scales<J>(w, g);
#pragma unroll
  for (int n = 0; n < NB; ++n) {
#pragma unroll
    for (int j = 0; j < J; ++j)
      w[j] = *reinterpret_cast<const uint32_t*>(lds + wbuf + wo[n] + step + 4 * j);
    f.bs[n] = pick_scales<J>(w, g);
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
    } else if constexpr (FA == 2) {  // six words: the 32 codes of the block at 6 bits each
      const v4u lo = f.a[2 * j], hi = f.a[2 * j + 1];
      a = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, 0, 0};
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

// The K loop of one wave: nst steps of 4J blocks, double-buffered in
// registers. pro() runs right after the first step's code loads are issued
// (it stages the scale rows, so both latencies overlap). With nst even
// (EVEN) the loop runs step pairs with no branch around a load; odd nst
// (K/32 not a multiple of 8) takes a plain loop.
// av: this lane's activation row is a row of the tile (lanes past the end
// skip their activation loads and multiply zeros; rows are independent in
// the product, and those accumulator rows are never stored).
template <int FA, int J, int NB, bool EVEN, typename Pro>
__device__ __forceinline__ void stream_k(const uint8_t* a_row, const uint8_t* const* b_rows,
                                         int nst, uint32_t xa, uint32_t wb, const uint32_t* wo,
                                         int g, v4f* acc, Pro pro, bool av = true) {
  constexpr int kc = 4 * J;
  Frag<FA, J, NB> f0, f1;
#pragma unroll
  for (int i = 0; i < Frag<FA, J, NB>::kAV; ++i) f0.a[i] = f1.a[i] = v4u{0u, 0u, 0u, 0u};
  if constexpr (EVEN) {
    frag_codes<FA, J, NB>(f0, a_row, b_rows, 0, 0, g, av);
    pro();
    wait_all_vmem();  // the first step and the scale rows are needed next anyway
    for (int c = 0; c + 2 < nst; c += 2) {  // f0 holds step c
      frag_codes<FA, J, NB>(f1, a_row, b_rows, 0, (c + 1) * kc, g, av);
      frag_scales<FA, J, NB>(f0, xa, wb, wo, c * kc, g);
      frag_mma<FA, J, NB>(f0, acc);
      frag_codes<FA, J, NB>(f0, a_row, b_rows, 0, (c + 2) * kc, g, av);
      frag_scales<FA, J, NB>(f1, xa, wb, wo, (c + 1) * kc, g);
      frag_mma<FA, J, NB>(f1, acc);
    }
    frag_codes<FA, J, NB>(f1, a_row, b_rows, 0, (nst - 1) * kc, g, av);
    frag_scales<FA, J, NB>(f0, xa, wb, wo, (nst - 2) * kc, g);
    frag_mma<FA, J, NB>(f0, acc);
    frag_scales<FA, J, NB>(f1, xa, wb, wo, (nst - 1) * kc, g);
    frag_mma<FA, J, NB>(f1, acc);
  } else {
    pro();
    wait_all_vmem();
    for (int c = 0; c < nst; ++c) {
      frag_codes<FA, J, NB>(f0, a_row, b_rows, 0, c * kc, g, av);
      frag_scales<FA, J, NB>(f0, xa, wb, wo, c * kc, g);
      frag_mma<FA, J, NB>(f0, acc);
    }
  }
}

// The same K loop with three register buffers, for a compile-time step
// count NST: the codes of step c + 2 go out before the products of step c,
// so two steps of loads are in flight while one is multiplied (the
// products and their order are those of stream_k). A third buffer still
// fits the two waves per SIMD the double-buffered loop runs at.
template <int FA, int J, int NB, int NST, typename Pro>
__device__ __forceinline__ void stream_k3(const uint8_t* a_row, const uint8_t* const* b_rows,
                                          uint32_t xa, uint32_t wb, const uint32_t* wo, int g,
                                          v4f* acc, Pro pro, bool av) {
  constexpr int kc = 4 * J;
  Frag<FA, J, NB> f[3];
#pragma unroll
  for (int q = 0; q < 3; ++q)
#pragma unroll
    for (int i = 0; i < Frag<FA, J, NB>::kAV; ++i) f[q].a[i] = v4u{0u, 0u, 0u, 0u};
  frag_codes<FA, J, NB>(f[0], a_row, b_rows, 0, 0, g, av);
  pro();
  wait_all_vmem();
  frag_codes<FA, J, NB>(f[1], a_row, b_rows, 0, kc, g, av);
  static_for<NST>([&](auto C) {
    constexpr int c = decltype(C)::value;
    if constexpr (c + 2 < NST)
      frag_codes<FA, J, NB>(f[(c + 2) % 3], a_row, b_rows, 0, (c + 2) * kc, g, av);
    frag_scales<FA, J, NB>(f[c % 3], xa, wb, wo, c * kc, g);
    frag_mma<FA, J, NB>(f[c % 3], acc);
  });
}

// K loop of a streaming wave: triple-buffered for steps of 8 blocks and K of
// 1024, 2048, 4096 or 8192 (nst = 4 .. 32), double-buffered otherwise.
template <int FA, int J, int NB, bool EVEN, typename Pro>
__device__ __forceinline__ void stream_any(const uint8_t* a_row, const uint8_t* const* b_rows,
                                           int nst, uint32_t xa, uint32_t wb, const uint32_t* wo,
                                           int g, v4f* acc, Pro pro, bool av) {
  if constexpr (EVEN && J == 2) {
    switch (nst) {
      case 4: return stream_k3<FA, J, NB, 4>(a_row, b_rows, xa, wb, wo, g, acc, pro, av);
      case 8: return stream_k3<FA, J, NB, 8>(a_row, b_rows, xa, wb, wo, g, acc, pro, av);
      case 16: return stream_k3<FA, J, NB, 16>(a_row, b_rows, xa, wb, wo, g, acc, pro, av);
      case 32: return stream_k3<FA, J, NB, 32>(a_row, b_rows, xa, wb, wo, g, acc, pro, av);
      default: break;
    }
  }
  stream_k<FA, J, NB, EVEN>(a_row, b_rows, nst, xa, wb, wo, g, acc, pro, av);
}

// Steps s0 .. s0 + NST - 1 of the K loop (one wave's half of a two-wave
// split), triple-buffered like stream_k3; sync() runs once this wave's
// prologue DMA has landed, before any scale is read from LDS.
template <int FA, int J, int NB, int NST, typename Pro, typename Sync>
__device__ __forceinline__ void stream_k3h(const uint8_t* a_row, const uint8_t* const* b_rows,
                                           uint32_t xa, uint32_t wb, const uint32_t* wo, int g,
                                           v4f* acc, Pro pro, Sync sync, bool av, int s0) {
  constexpr int kc = 4 * J;
  Frag<FA, J, NB> f[3];
#pragma unroll
  for (int q = 0; q < 3; ++q)
#pragma unroll
    for (int i = 0; i < Frag<FA, J, NB>::kAV; ++i) f[q].a[i] = v4u{0u, 0u, 0u, 0u};
  frag_codes<FA, J, NB>(f[0], a_row, b_rows, 0, s0 * kc, g, av);
  pro();
  wait_all_vmem();
  sync();
  if constexpr (NST > 1) frag_codes<FA, J, NB>(f[1], a_row, b_rows, 0, (s0 + 1) * kc, g, av);
  static_for<NST>([&](auto C) {
    constexpr int c = decltype(C)::value;
    if constexpr (c + 2 < NST)
      frag_codes<FA, J, NB>(f[(c + 2) % 3], a_row, b_rows, 0, (s0 + c + 2) * kc, g, av);
    frag_scales<FA, J, NB>(f[c % 3], xa, wb, wo, (s0 + c) * kc, g);
    frag_mma<FA, J, NB>(f[c % 3], acc);
  });
}

// Stage 1 with the K extent split over the two waves of a workgroup (steps
// of 8 blocks, NSTH per wave). A streaming launch ends with a last, partly
// filled round of workgroups, whose rate is bound by each wave's own loads
// in flight rather than by HBM; halving a wave's share of K halves that
// tail (measured on the decode layer: stage 1 ~3% faster). Wave 0 stages
// the activation and gate scale rows, wave 1 the up scale rows; wave 1
// hands its fp32 sums over through LDS and wave 0 forms first half + second
// half (a fixed order, so results repeat bit for bit) before the SwiGLU
// epilogue.
template <int FA, int NBW, int NSTH>
__global__ __launch_bounds__(128) void s1_stream2_kernel(S1Args p) {
  constexpr int NB = 2 * NBW, J = 2;
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int kw = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));  // K half of the wave
  const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int kb = p.H / 32;
  const int hc0 = nt * (NBW * 16);  // first h column of the workgroup
  const size_t ebase = (size_t)e * 2 * p.I;

  // LDS: the scale rows as in s1_stream_kernel, then wave 1's sums [NB][64] v4f
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int half = NBW * 16 * kb;
  const int tok = p.sorted[row0 + (c16 < nrows ? c16 : 0)] / p.k_total;
  const uint8_t* a_row = p.xq + (size_t)tok * (p.H / 32) * kAB;
  const uint8_t* b_rows[NB];
  uint32_t wo[NB];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t gr = ebase + hc0 + 16 * b;  // first gate row of the group
    b_rows[b] = p.w13 + gr * (p.H / 2) + 64 * c16;
    b_rows[NBW + b] = p.w13 + (gr + p.I) * (p.H / 2) + 64 * c16;
    wo[b] = (16 * b + c16) * kb;
    wo[NBW + b] = (NBW * 16 + 16 * b + c16) * kb;
  }
  v4f acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k3h<FA, J, NB, NSTH>(a_row, b_rows, c16 * kb, 16 * kb, wo, g, acc, [&]() {
    if (kw == 0) {
      dma_gather16(
          lds,
          [&](int r) {
            const int t = p.sorted[row0 + (r < nrows ? r : 0)] / p.k_total;
            return p.xs + (size_t)t * kb;
          },
          kb, lane);
      dma_rows16(lds + 16 * kb, p.w13s + (ebase + hc0) * kb, half, lane);
    } else {
      dma_rows16(lds + 16 * kb + half, p.w13s + (ebase + p.I + hc0) * kb, half, lane);
    }
  }, [&]() { __syncthreads(); }, c16 < nrows, kw * NSTH);
  v4f* red = reinterpret_cast<v4f*>(lds + (1 + 2 * NBW) * 16 * kb);
  if (kw == 1) {
#pragma unroll
    for (int n = 0; n < NB; ++n) red[n * 64 + lane] = acc[n];
  }
  __syncthreads();
  if (kw == 1) return;
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = acc[n] + red[n * 64 + lane];
  s1_epilogue<FA, NBW>(acc, p, row0, nrows, hc0, g, c16);
}

template <int FA, int J, int NBW, bool EVEN>
__global__ __launch_bounds__(64) void s1_stream_kernel(S1Args p) {
  static_assert(NBW % 2 == 0, "a quantisation block spans two 16-column tiles");
  constexpr int NB = 2 * NBW;
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x, g = lane >> 4, c16 = lane & 15;
  const int kb = p.H / 32;
  const int hc0 = nt * (NBW * 16);  // first h column of the wave
  const size_t ebase = (size_t)e * 2 * p.I;

  // LDS: the tile's 16 activation scale rows, then the wave's 16 NBW gate
  // and 16 NBW up weight scale rows.
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int half = NBW * 16 * kb;  // bytes of the gate (or up) scale rows

  const int tok = p.sorted[row0 + (c16 < nrows ? c16 : 0)] / p.k_total;
  const uint8_t* a_row = p.xq + (size_t)tok * (p.H / 32) * kAB;
  const uint8_t* b_rows[NB];
  uint32_t wo[NB];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t gr = ebase + hc0 + 16 * b;  // first gate row of the group
    b_rows[b] = p.w13 + gr * (p.H / 2) + 64 * c16;
    b_rows[NBW + b] = p.w13 + (gr + p.I) * (p.H / 2) + 64 * c16;
    wo[b] = (16 * b + c16) * kb;
    wo[NBW + b] = (NBW * 16 + 16 * b + c16) * kb;
  }
  v4f acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_any<FA, J, NB, EVEN>(a_row, b_rows, kb / (4 * J), c16 * kb, 16 * kb, wo, g, acc, [&]() {
    dma_gather16(
        lds,
        [&](int r) {
          const int t = p.sorted[row0 + (r < nrows ? r : 0)] / p.k_total;
          return p.xs + (size_t)t * kb;
        },
        kb, lane);
    dma_rows16(lds + 16 * kb, p.w13s + (ebase + hc0) * kb, half, lane);
    dma_rows16(lds + 16 * kb + half, p.w13s + (ebase + p.I + hc0) * kb, half, lane);
  }, c16 < nrows);
  s1_epilogue<FA, NBW>(acc, p, row0, nrows, hc0, g, c16);
}

template <int FA, int J, int NBW, bool EVEN>
__global__ __launch_bounds__(64) void s2_stream_kernel(S2Args p) {
  constexpr int NB = NBW;
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x, g = lane >> 4, c16 = lane & 15;
  const int kb = p.I / 32;
  const int nc0 = nt * (NBW * 16);  // first output column of the wave
  const size_t rbase = (size_t)e * p.H + nc0;

  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const size_t ar = (size_t)row0 + (c16 < nrows ? c16 : 0);
  const uint8_t* a_row = p.hq + ar * (p.I / 32) * kAB;
  const uint8_t* b_rows[NB];
  uint32_t wo[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    b_rows[b] = p.w2 + (rbase + 16 * b) * (p.I / 2) + 64 * c16;
    wo[b] = (16 * b + c16) * kb;
  }
  v4f acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_any<FA, J, NB, EVEN>(a_row, b_rows, kb / (4 * J), c16 * kb, 16 * kb, wo, g, acc, [&]() {
    dma_gather16(
        lds, [&](int r) { return p.hs + ((size_t)row0 + (r < nrows ? r : 0)) * kb; }, kb, lane);
    dma_rows16(lds + 16 * kb, p.w2s + rbase * kb, NB * 16 * kb, lane);
  }, c16 < nrows);
  s2_epilogue<NBW>(acc, p, row0, nrows, nc0, g, c16);
}

// Stage 2 with the K extent split over two waves, as s1_stream2_kernel
// (wave 0 stages the activation scale rows, wave 1 the weight scale rows;
// partial = first half + second half).
template <int FA, int NBW, int NSTH>
__global__ __launch_bounds__(128) void s2_stream2_kernel(S2Args p) {
  constexpr int NB = NBW, J = 2;
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int kw = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));  // K half of the wave
  const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int kb = p.I / 32;
  const int nc0 = nt * (NBW * 16);  // first output column of the workgroup
  const size_t rbase = (size_t)e * p.H + nc0;

  // LDS: the scale rows as in s2_stream_kernel, then wave 1's sums [NB][64] v4f
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const size_t ar = (size_t)row0 + (c16 < nrows ? c16 : 0);
  const uint8_t* a_row = p.hq + ar * (p.I / 32) * kAB;
  const uint8_t* b_rows[NB];
  uint32_t wo[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    b_rows[b] = p.w2 + (rbase + 16 * b) * (p.I / 2) + 64 * c16;
    wo[b] = (16 * b + c16) * kb;
  }
  v4f acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k3h<FA, J, NB, NSTH>(a_row, b_rows, c16 * kb, 16 * kb, wo, g, acc, [&]() {
    if (kw == 0)
      dma_gather16(
          lds, [&](int r) { return p.hs + ((size_t)row0 + (r < nrows ? r : 0)) * kb; }, kb, lane);
    else
      dma_rows16(lds + 16 * kb, p.w2s + rbase * kb, NB * 16 * kb, lane);
  }, [&]() { __syncthreads(); }, c16 < nrows, kw * NSTH);
  v4f* red = reinterpret_cast<v4f*>(lds + (1 + NBW) * 16 * kb);
  if (kw == 1) {
#pragma unroll
    for (int n = 0; n < NB; ++n) red[n * 64 + lane] = acc[n];
  }
  __syncthreads();
  if (kw == 1) return;
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = acc[n] + red[n * 64 + lane];
  s2_epilogue<NBW>(acc, p, row0, nrows, nc0, g, c16);
}

// The streaming stages split K over two waves for K/32 = 32, 64, 128 or 256
// (4 .. 32 steps of 8 blocks); the fused down + combine kernel follows the
// same rule so that both paths add the same two halves.
inline bool split_k(int kb) { return kb == 32 || kb == 64 || kb == 128 || kb == 256; }

// Stage 2 fused with the fixed-order combine, for few rows (decode): the
// paper's small down consumer joined to the reducer (Historical down-consumer
// pilot; Current TP8 native-AR results). A workgroup owns 16 output columns
// and every row: its waves take the row tiles round-robin, stream those 16
// W2 rows of the tile's expert once over the whole K extent with the same
// products in the same order as the unfused stage 2 (so the same fp32
// values; where that splits K over two waves, so do these: waves 2i and
// 2i + 1 take the same tiles, one K half each, and the halves are added in
// the same order), and put each row's result into LDS at the row's
// assignment index. After
// one barrier the workgroup forms out[t, columns] = bf16(acc), acc =
// fmaf(topk_w[t, j], P[t*k_total + j], acc) for j = 0, 1, ... -- the combine
// kernel's arithmetic -- so the output has the bits of s2_stream_kernel +
// combine_kernel while no fp32 partial row reaches global memory.
//
// A wave streams about a dozen tiles one after another, each only a few K
// steps long, so the start of a tile (its scale rows staged in LDS, its
// first codes loaded) must not wait for the memory round trip: the next
// tile's scale rows go out by DMA into the wave's second LDS slot during
// the current tile's first step, and its first codes are loaded during the
// current tile's last step. That DMA is written out (sdma4 / sdma16) so the
// compiler does not turn it into waits for every outstanding load; one
// explicit wait at each tile's first step covers it (see s2c_tiles).
//
// LDS: P [A][16] fp32 (zeroed first, so an assignment whose expert id was
// invalid contributes 0; with the K split, one such array per K half), then
// two slots per wave of 16 activation and 16 weight scale rows.
#ifndef MOE_FUSED_WAVES
#define MOE_FUSED_WAVES 16
#endif
constexpr int kFusedWaves = MOE_FUSED_WAVES;

// Per-tile values of a wave: the tile's activation row of this lane (lane
// c16 multiplies row c16; rows past the end repeat row 0), its W2 row and
// the first W2 scale row.
struct S2CTile {
  int row0, nrows;
  size_t rbase;  // first W2 row: expert * H + first column
};

__device__ __forceinline__ S2CTile s2c_tile(const int4& t, int H, int nc0) {
  const int e = __builtin_amdgcn_readfirstlane(t.x);  // tile values are wave-uniform
  return S2CTile{__builtin_amdgcn_readfirstlane(t.y), __builtin_amdgcn_readfirstlane(t.z),
                 (size_t)e * H + nc0};
}

// Scale rows of a tile into the LDS slot at byte offset `slot`: the 16
// activation scale rows gathered 4 bytes a lane, then the 16 consecutive W2
// scale rows of the workgroup's columns, 16 bytes a lane.
__device__ __forceinline__ void s2c_scales(uint8_t* lds, uint32_t slot, const S2Args& p,
                                           const S2CTile& t, int kb, int lane) {
  const int words = kb / 4;
  const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr(lds) + slot);
  for (int o = 0; o < 16 * words; o += 64) {
    const int q = o + lane;
    if (q < 16 * words) {
      const int r = q / words;
      sdma4(p.hs, (uint32_t)((t.row0 + (r < t.nrows ? r : 0)) * kb + 4 * (q % words)), base + 4 * o);
    }
  }
  const uint8_t* src = p.w2s + t.rbase * kb;
  for (int o = 0; o < 16 * kb; o += 1024)
    if (o + 16 * lane < 16 * kb) sdma16(src, (uint32_t)(o + 16 * lane), base + 16 * kb + o);
}

// The tiles of one wave with the cross-tile prefetch; nst (K steps of 4J
// blocks per tile) is even. fa holds even steps, fb odd steps.
// Waits: the compiler waits for the code registers before each product; the
// scale rows are read from LDS before the products, so the first step of a
// tile waits explicitly for all but the step-1 codes just issued
// (vmcnt(kStepLoads)): the tile's scale DMA was issued earlier (during the
// previous tile, or the prologue, which waits for everything), and the
// step-1 loads are kStepLoads unconditional instructions issued after it,
// so the DMA is complete when at most kStepLoads loads are outstanding
// (loads complete in order).
template <int FA, int J, bool SPLIT>
__device__ __forceinline__ void s2c_tiles(const S2CArgs& c, uint8_t* lds, float* P, int wave,
                                          int lane, int nc0) {
  const S2Args& p = c.s;
  using F = Frag<FA, J, 1>;
  constexpr int kAB = ActBytes<FA>::kBlock;
  constexpr int kc = 4 * J;
  constexpr int kStepLoads = F::kAV + J;  // code load instructions of one step
  const int g = lane >> 4, c16 = lane & 15;
  const int kb = p.I / 32, nst = kb / kc;
  wave = __builtin_amdgcn_readfirstlane(wave);
  const int ntl = *p.t.ntiles;
  // with the K split: wave pairs take the tiles, wave 2i + h steps K half h
  const int W = SPLIT ? kFusedWaves / 2 : kFusedWaves;
  const int kh = SPLIT ? (wave & 1) : 0;
  const int ns = SPLIT ? nst / 2 : nst, s0 = kh * ns;  // this wave's steps s0 .. s0 + ns - 1
  float* const Pw = P + (size_t)kh * c.T * c.k_total * 16;
  int tj = SPLIT ? wave >> 1 : wave;
  if (tj >= ntl) return;
  const uint32_t slot0 = (uint32_t)((SPLIT ? 2 : 1) * c.T * c.k_total * 64 + wave * 64 * kb);
  const uint32_t wo[1] = {(uint32_t)(c16 * kb)};
  auto a_row = [&](const S2CTile& t) {
    return p.hq + ((size_t)t.row0 + (c16 < t.nrows ? c16 : 0)) * (p.I / 32) * kAB;
  };
  auto b_row = [&](const S2CTile& t) { return p.w2 + t.rbase * (p.I / 2) + 64 * c16; };

  S2CTile tc = s2c_tile(p.t.tiles[tj], p.H, nc0);
  int4 tn4 = p.t.tiles[tj + W < ntl ? tj + W : tj];
  uint32_t slot = slot0;
  F fa, fb;
  {
    const uint8_t* br = b_row(tc);
    frag_codes<FA, J, 1>(fa, a_row(tc), &br, 0, s0 * kc, g);
  }
  s2c_scales(lds, slot, p, tc, kb, lane);
  wait_all_vmem();
  for (;;) {
    const bool has_next = tj + W < ntl;
    const S2CTile tn = s2c_tile(tn4, p.H, nc0);
    const int4 tnn4 = p.t.tiles[tj + 2 * W < ntl ? tj + 2 * W : tj];
    int arow[4];  // assignment index of the lane's accumulator rows 4g + i (-1: past the end)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rl = 4 * g + i;
      const int a = p.sorted[tc.row0 + (rl < tc.nrows ? rl : tc.nrows - 1)];
      arow[i] = rl < tc.nrows ? a : -1;
    }
    const uint8_t* ar = a_row(tc);
    const uint8_t* br = b_row(tc);
    // codes of the step after s + 1: step s + 2 of this tile, else the first
    // step (s0) of the next tile (of this tile again when there is none:
    // every step issues the same loads, so the compiler's waits count exactly)
    const uint8_t* arn = has_next ? a_row(tn) : ar;
    const uint8_t* brn = has_next ? b_row(tn) : br;
    const uint32_t xa = slot + c16 * kb, wb = slot + 16 * kb;
    const uint32_t nslot = slot ^ (slot0 ^ (slot0 + 32 * kb));
    v4f acc[1] = {v4f{0.f, 0.f, 0.f, 0.f}};
    auto pair = [&](int s, bool first) {  // steps s0 + s, s0 + s + 1
      frag_codes<FA, J, 1>(fb, ar, &br, 0, (s0 + s + 1) * kc, g);
      if (first) {
        tvmcnt_s<kStepLoads>();
        if (has_next) s2c_scales(lds, nslot, p, tn, kb, lane);
      }
      frag_scales<FA, J, 1>(fa, xa, wb, wo, (s0 + s) * kc, g);
      frag_mma<FA, J, 1>(fa, acc);
      const bool last = s + 2 >= ns;
      const uint8_t* a2 = last ? arn : ar;
      const uint8_t* b2 = last ? brn : br;
      frag_codes<FA, J, 1>(fa, a2, &b2, 0, (last ? s0 : s0 + s + 2) * kc, g);
      frag_scales<FA, J, 1>(fb, xa, wb, wo, (s0 + s + 1) * kc, g);
      frag_mma<FA, J, 1>(fb, acc);
    };
    pair(0, true);
    for (int s = 2; s < ns; s += 2) pair(s, false);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (arow[i] >= 0) Pw[arow[i] * 16 + c16] = acc[0][i];
    if (!has_next) break;
    tj += W;
    tc = tn;
    tn4 = tnn4;
    slot = nslot;
  }
}

template <int FA, int J, bool EVEN, bool SPLIT>
__global__ __launch_bounds__(64 * kFusedWaves) void s2c_stream_kernel(S2CArgs c) {
  const S2Args& p = c.s;
  constexpr int kAB = ActBytes<FA>::kBlock;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  float* P = reinterpret_cast<float*>(lds);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int kb = p.I / 32, kt = c.k_total;
  const int A = c.T * kt;
  const int nc0 = blockIdx.x * 16;  // first output column of the workgroup

  constexpr int kNP = SPLIT ? 2 : 1;  // result arrays (one per K half)
  for (int i = threadIdx.x; i < kNP * A * 4; i += blockDim.x)
    reinterpret_cast<v4f*>(P)[i] = v4f{0.f, 0.f, 0.f, 0.f};
  __syncthreads();

  if constexpr (EVEN) {
    s2c_tiles<FA, J, SPLIT>(c, lds, P, wave, lane, nc0);
  } else {  // odd step counts: one tile at a time
    const uint32_t sb = (uint32_t)(A * 64 + wave * 64 * kb);  // this wave's scale rows
    const int ntl = *p.t.ntiles;
    for (int tj = wave; tj < ntl; tj += kFusedWaves) {
      const int4 tile = p.t.tiles[tj];
      const int row0 = tile.y, nrows = tile.z;
      const size_t rbase = (size_t)tile.x * p.H + nc0;
      int arow[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) arow[i] = 4 * g + i < nrows ? p.sorted[row0 + 4 * g + i] : -1;
      const size_t ar = (size_t)row0 + (c16 < nrows ? c16 : 0);
      const uint8_t* a_row = p.hq + ar * (p.I / 32) * kAB;
      const uint8_t* b_rows[1] = {p.w2 + rbase * (p.I / 2) + 64 * c16};
      const uint32_t wo[1] = {(uint32_t)(c16 * kb)};
      v4f acc[1] = {v4f{0.f, 0.f, 0.f, 0.f}};
      stream_k<FA, J, 1, false>(
          a_row, b_rows, kb / (4 * J), sb + c16 * kb, sb + 16 * kb, wo, g, acc, [&]() {
            dma_gather16(
                lds + sb,
                [&](int r) { return p.hs + ((size_t)row0 + (r < nrows ? r : 0)) * kb; }, kb,
                lane);
            dma_rows16(lds + sb + 16 * kb, p.w2s + rbase * kb, 16 * kb, lane);
          });
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (arow[i] >= 0) P[arow[i] * 16 + c16] = acc[0][i];
    }
  }
  __syncthreads();

  // fixed-order combine of the workgroup's 16 columns, two per thread
  for (int o = threadIdx.x; o < c.T * 8; o += blockDim.x) {
    const int t = o >> 3, cp = 2 * (o & 7);
    const float* wrow = c.topk_w + (size_t)t * kt;
    const float* prow = P + (size_t)t * kt * 16 + cp;
    const float* qrow = prow + (size_t)A * 16;  // second K half (with the split)
    float a0 = 0.f, a1 = 0.f;
    for (int j = 0; j < kt; ++j) {
      const float wj = wrow[j];
      const float p0 = SPLIT ? prow[16 * j] + qrow[16 * j] : prow[16 * j];
      const float p1 = SPLIT ? prow[16 * j + 1] + qrow[16 * j + 1] : prow[16 * j + 1];
      a0 = fmaf(wj, p0, a0);
      a1 = fmaf(wj, p1, a1);
    }
    *reinterpret_cast<uint32_t*>(c.out + (size_t)t * p.H + nc0 + cp) =
        f32_to_bf16_rne(a0) | (f32_to_bf16_rne(a1) << 16);
  }
}

size_t fused_lds_bytes(int T, int k_total, int I) {
  const int kb = I / 32;
  const size_t np = kb % 16 == 0 && split_k(kb) ? 2 : 1;
  return np * T * k_total * 64 + (size_t)kFusedWaves * 64 * kb;
}

template <int FA>
static void launch_s2c(const S2CArgs& p, hipStream_t s) {
  const int kb = p.s.I / 32;
  const size_t lds = fused_lds_bytes(p.T, p.k_total, p.s.I);
  const dim3 grid(p.s.H / 16), block(64 * kFusedWaves);
  if (kb % 16 == 0 && split_k(kb))
    hipLaunchKernelGGL((s2c_stream_kernel<FA, 2, true, true>), grid, block, lds, s, p);
  else if (kb % 16 == 0)
    hipLaunchKernelGGL((s2c_stream_kernel<FA, 2, true, false>), grid, block, lds, s, p);
  else if (kb % 8 == 0)
    hipLaunchKernelGGL((s2c_stream_kernel<FA, 1, true, false>), grid, block, lds, s, p);
  else hipLaunchKernelGGL((s2c_stream_kernel<FA, 1, false, false>), grid, block, lds, s, p);
}

void launch_s2c_stream(const S2CArgs& p, int fa, hipStream_t s) {
  if (fa == 0) launch_s2c<0>(p, s);
  else launch_s2c<4>(p, s);
}

// Kernel instance: steps of 8 blocks (kb = K/32 a multiple of 16), else of
// 4 with an even count (kb % 8 == 0), else a plain loop.
template <typename K2, typename K1, typename K0, typename P>
static void launch_stream(int kb, K2 k2, K1 k1, K0 k0, long mt, int ntl, const P& p0,
                          hipStream_t s, size_t lds) {
  P q = p0;
  q.t.n_ntiles = ntl;
  q.t.ngroup = n_group_of(ntl);
  const long n = mt * ntl;
  const dim3 grid((int)((n + 7) / 8 * 8));
  if (kb % 16 == 0) hipLaunchKernelGGL(k2, grid, dim3(64), lds, s, q);
  else if (kb % 8 == 0) hipLaunchKernelGGL(k1, grid, dim3(64), lds, s, q);
  else hipLaunchKernelGGL(k0, grid, dim3(64), lds, s, q);
}

template <int FA, int NBW1>
static void launch_s1(const S1Args& p, long mt, hipStream_t s) {
  const int kb = p.H / 32;
  if (split_k(kb)) {  // K = 1024 .. 8192: the two-wave split
    S1Args q = p;
    const int ntl = p.I / (NBW1 * 16);
    q.t.n_ntiles = ntl;
    q.t.ngroup = n_group_of(ntl);
    const long n = mt * ntl;
    const dim3 grid((int)((n + 7) / 8 * 8)), block(128);
    const size_t lds = (size_t)(1 + 2 * NBW1) * 16 * kb + (size_t)2 * NBW1 * 64 * 16;
    if (kb == 32) hipLaunchKernelGGL((s1_stream2_kernel<FA, NBW1, 2>), grid, block, lds, s, q);
    else if (kb == 64) hipLaunchKernelGGL((s1_stream2_kernel<FA, NBW1, 4>), grid, block, lds, s, q);
    else if (kb == 128) hipLaunchKernelGGL((s1_stream2_kernel<FA, NBW1, 8>), grid, block, lds, s, q);
    else hipLaunchKernelGGL((s1_stream2_kernel<FA, NBW1, 16>), grid, block, lds, s, q);
    return;
  }
  launch_stream(kb, s1_stream_kernel<FA, 2, NBW1, true>, s1_stream_kernel<FA, 1, NBW1, true>,
                s1_stream_kernel<FA, 1, NBW1, false>, mt, p.I / (NBW1 * 16), p, s,
                (size_t)(1 + 2 * NBW1) * 16 * kb);
}

template <int FA, int NBW2>
static void launch_s2(const S2Args& p, long mt, hipStream_t s) {
  const int kb = p.I / 32;
  if (split_k(kb)) {
    S2Args q = p;
    const int ntl = p.H / (NBW2 * 16);
    q.t.n_ntiles = ntl;
    q.t.ngroup = n_group_of(ntl);
    const long n = mt * ntl;
    const dim3 grid((int)((n + 7) / 8 * 8)), block(128);
    const size_t lds = (size_t)(1 + NBW2) * 16 * kb + (size_t)NBW2 * 64 * 16;
    if (kb == 32) hipLaunchKernelGGL((s2_stream2_kernel<FA, NBW2, 2>), grid, block, lds, s, q);
    else if (kb == 64) hipLaunchKernelGGL((s2_stream2_kernel<FA, NBW2, 4>), grid, block, lds, s, q);
    else if (kb == 128) hipLaunchKernelGGL((s2_stream2_kernel<FA, NBW2, 8>), grid, block, lds, s, q);
    else hipLaunchKernelGGL((s2_stream2_kernel<FA, NBW2, 16>), grid, block, lds, s, q);
    return;
  }
  launch_stream(kb, s2_stream_kernel<FA, 2, NBW2, true>, s2_stream_kernel<FA, 1, NBW2, true>,
                s2_stream_kernel<FA, 1, NBW2, false>, mt, p.H / (NBW2 * 16), p, s,
                (size_t)(1 + NBW2) * 16 * kb);
}

// Steps of 256 K elements (128 when K/32 is not a multiple of 16); stage 1:
// 32 h columns per workgroup, two waves splitting K for K = 1024 .. 8192,
// else one wave; stage 2: one wave per workgroup, 64 output columns.
void launch_s1_stream(const S1Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_s1<0, 2>(p, mt, s);
  else if (fa == 2) launch_s1<2, 2>(p, mt, s);
  else launch_s1<4, 2>(p, mt, s);
}

void launch_s2_stream(const S2Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_s2<0, 4>(p, mt, s);
  else if (fa == 2) launch_s2<2, 4>(p, mt, s);
  else launch_s2<4, 4>(p, mt, s);
}

// ---------------------------------------------------------------------------
// Probe: one 16x16x128 product with the GEMM's operand and scale placement.
// ---------------------------------------------------------------------------
template <int FA>
__global__ void probe_kernel(const uint8_t* a, const uint8_t* sa, const uint8_t* b,
                             const uint8_t* sb, float* d) {
  constexpr int kAB = ActBytes<FA>::kBlock;
  const int lane = threadIdx.x, g = lane >> 4, c16 = lane & 15;
  const uint8_t* ar = a + (size_t)c16 * 4 * kAB;
  const uint8_t* br = b + (size_t)c16 * 64;
  v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
  Frag<FA, 1, 1> f;
  frag_codes<FA, 1, 1>(f, ar, &br, 0, 0, g);
  const uint32_t wa = *reinterpret_cast<const uint32_t*>(sa + 4 * c16);
  const uint32_t wb = *reinterpret_cast<const uint32_t*>(sb + 4 * c16);
  f.as = pick_scales<1>(&wa, g);
  f.bs[0] = pick_scales<1>(&wb, g);
  frag_mma<FA, 1, 1>(f, &acc);
#pragma unroll
  for (int i = 0; i < 4; ++i) d[(4 * g + i) * 16 + c16] = acc[i];
}

hipError_t launch_probe(const uint8_t* a, const uint8_t* sa, int fmt, const uint8_t* b,
                        const uint8_t* sb, float* d, hipStream_t s) {
  if (fmt == 0)
    hipLaunchKernelGGL(probe_kernel<0>, dim3(1), dim3(64), 0, s, a, sa, b, sb, d);
  else if (fmt == 4)
    hipLaunchKernelGGL(probe_kernel<4>, dim3(1), dim3(64), 0, s, a, sa, b, sb, d);
  else
    return hipErrorNotSupported;
  return hipGetLastError();
}

}  // namespace moe
