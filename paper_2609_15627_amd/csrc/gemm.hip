// a5 / a6: the grouped FP4 expert GEMM behind moe_fp4_grouped_gemm --
// activation quantisation, row-tile list, geometry choice, stage launches.
#include "gemm_common.h"
#include "gemm_launch.h"
#include "moe_launch.h"
#include "quant_dev.h"

namespace moe {

// ---------------------------------------------------------------------------
// Tile list: expert e with c rows gets ceil(c / BM) row tiles. One block of
// 1024 threads: tile counts, exclusive scan, then every thread fills tiles
// i = tid, tid + 1024, ... by binary search over the per-expert tile starts.
//
// The work queue of the persistent tiled kernels starts at zero here; each
// of their launches leaves it at zero when it ends.
//
// Chunk list (the tiled geometry launches C row tiles at a time, so that
// they share their weight rows in L2). C = 2 (256-row tiles): an expert's
// tiles pair up among themselves, so its weights are never split across two
// chunks; the odd tile left over by an expert pairs with the next expert's
// leftover. Chunk order: all within-expert pairs (expert order), then the
// leftover pairs. C = 4 (128-row tiles): an expert's tiles in groups of
// four, the last group of each expert padded with empty places (-1).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void build_tiles(const int32_t* __restrict__ offsets, int NE, int BM,
                                            int4* __restrict__ tiles, int* __restrict__ ntiles,
                                            int4* __restrict__ chunks, int* __restrict__ nchunks,
                                            int* __restrict__ queue) {
  const int C = BM == 128 ? 4 : 2;  // row tiles per chunk
  extern __shared__ int start[];  // [NE + 1]
  int m[2], tot[3][2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int e = threadIdx.x + 1024 * q;
    m[q] = e < NE ? (offsets[e + 1] - offsets[e] + BM - 1) / BM : 0;
  }
  // exclusive prefix of: tiles, within-expert chunks (pairs, or groups of
  // four with the last one padded), leftover singles (C = 2 only)
  int p0[3], p1[3];
  auto per_expert = [&](int k, int mv) {
    if (k == 0) return mv;
    if (C == 4) return k == 1 ? (mv + 3) / 4 : 0;
    return k == 1 ? mv / 2 : mv % 2;
  };
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int v0 = per_expert(k, m[0]);
    const int v1 = per_expert(k, m[1]);
    p0[k] = block_exclusive_scan_1024(v0, &tot[k][0]);
    p1[k] = block_exclusive_scan_1024(v1, &tot[k][1]) + tot[k][0];
  }
  const int total = tot[0][0] + tot[0][1];
  const int pairs = tot[1][0] + tot[1][1];
  const int singles = tot[2][0] + tot[2][1];
  if (threadIdx.x < NE) start[threadIdx.x] = p0[0];
  if (threadIdx.x + 1024 < NE) start[threadIdx.x + 1024] = p1[0];
  if (threadIdx.x < kQueueInts) queue[threadIdx.x] = 0;
  if (threadIdx.x == 0) {
    start[NE] = total;
    *ntiles = total;
    *nchunks = pairs + (singles + 1) / 2;
    if (singles & 1) chunks[pairs + singles / 2].y = -1;  // (C = 2; C = 4 has no singles)
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int e = threadIdx.x + 1024 * q;
    if (e >= NE) continue;
    const int ts = q ? p1[0] : p0[0], pr = q ? p1[1] : p0[1], sg = q ? p1[2] : p0[2];
    if (C == 4) {
      const int mq = m[q];
      for (int j = 0; j < (mq + 3) / 4; ++j) {
        const int b = 4 * j;
        chunks[pr + j] = make_int4(ts + b, b + 1 < mq ? ts + b + 1 : -1, b + 2 < mq ? ts + b + 2 : -1,
                                   b + 3 < mq ? ts + b + 3 : -1);
      }
      continue;
    }
    for (int j = 0; j < m[q] / 2; ++j) chunks[pr + j] = make_int4(ts + 2 * j, ts + 2 * j + 1, -1, -1);
    if (m[q] & 1) {
      int* c = reinterpret_cast<int*>(&chunks[pairs + sg / 2]);
      c[sg & 1] = ts + m[q] - 1;
      if ((sg & 1) == 0) c[2] = c[3] = -1;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < total; i += 1024) {
    int lo = 0, hi = NE;  // find e with start[e] <= i < start[e + 1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (start[mid] <= i) lo = mid; else hi = mid;
    }
    const int j = i - start[lo];
    const int r0 = offsets[lo] + j * BM;
    tiles[i] = make_int4(lo, r0, min(BM, offsets[lo + 1] - r0), 0);
  }
}

// The preparation launch: blocks [0, nqb) quantise x (1024 blocks of 32
// elements each), then one block per tile list builds it (the two jobs are
// independent, so they run side by side).
template <int FMT>
__global__ __launch_bounds__(1024) void prep_kernel(const uint16_t* __restrict__ x, long nblk,
                                                    uint8_t* __restrict__ codes,
                                                    uint8_t* __restrict__ scales, int nqb,
                                                    const int32_t* __restrict__ offsets, int NE,
                                                    int BM1, TileArgs t1, int BM2, TileArgs t2) {
  if ((int)blockIdx.x < nqb) {
    if constexpr (FMT >= 0) {
      const long b = (long)blockIdx.x * 1024 + threadIdx.x;
      if (b < nblk) quant_block<FMT, true>(x, b, codes, scales);
    }
    return;
  }
  const bool first = (int)blockIdx.x == nqb;
  const TileArgs& t = first ? t1 : t2;
  build_tiles(offsets, NE, first ? BM1 : BM2, const_cast<int4*>(t.tiles), const_cast<int*>(t.ntiles),
              const_cast<int4*>(t.chunks), const_cast<int*>(t.nchunks), t.queue);
}

static int tile_bound(long A, int NE, int BM) {
  const long nonempty = A < NE ? A : NE;
  return (int)((A + nonempty * (BM - 1)) / BM);
}

// Bytes of one tile list (sized for the smallest row tile, 16 rows).
static size_t tile_list_bytes(long A, int NE) {
  const size_t tb = (size_t)tile_bound(A, NE, 16) + 1;
  return sizeof(int4) * tb + 16 + sizeof(int4) * tb + 16 + 4 * kQueueInts;
}

// The tile list at `base` for row tiles of BM rows.
static TileArgs tile_list(uint8_t* base, long A, int NE, int BM) {
  const int tb = tile_bound(A, NE, 16) + 1;
  int4* tiles = reinterpret_cast<int4*>(base);
  int* ntiles = reinterpret_cast<int*>(tiles + tb);
  int4* chunks = reinterpret_cast<int4*>(ntiles + 4);
  int* nchunks = reinterpret_cast<int*>(chunks + tb);
  return TileArgs{tiles, ntiles, tile_bound(A, NE, BM), 0, 1, chunks, nchunks, nchunks + 4};
}

GemmWorkspace gemm_workspace(int T, int H, int I, int NE, int k_total, int fmt) {
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t A = (size_t)T * k_total;
  const size_t bits = ws_act_bits(fmt);
  GemmWorkspace w;
  size_t o = 0;
  const bool mx = fmt != kFmtBf16;  // the BF16 contract has no x codes and no scales
  w.off[0] = o;  o += mx ? al((size_t)T * H * bits / 8) : 0;
  w.off[1] = o;  o += mx ? al((size_t)T * (H / 32)) : 0;
  w.off[2] = o;  o += al(A * I * bits / 8);
  w.off[3] = o;  o += mx ? al(A * (I / 32)) : 0;
  // two tile lists (stage 1's and, when stage 2 runs another geometry,
  // stage 2's), each: tiles (int4 x bound), count, chunks (int4 x bound),
  // count, work queue
  w.off[4] = o;  o += 2 * al(tile_list_bytes((long)A, NE));
  w.off[5] = o;
  return w;
}

static int max_lds_per_block() {
  static const int v = [] {
    int dev = 0, bytes = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&bytes, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
      return 0;
    return bytes;
  }();
  return v;
}

// Geometry rule (runtime M), per stage: the LDS-tiled geometry when experts
// average at least kTiledMinRows rows and the stage's K is a multiple of the
// tiled K loop's 512 (stage 1: K = H, N tiles of 128 h columns; stage 2:
// K = I, N tiles of 256 output columns); with as many rows but K = I of 128
// or 256, stage 2 runs on the short-K geometry (a tile's whole K extent in
// LDS); the weight-streaming geometry otherwise. So a shape like the TP8
// expert shard (I = 256) runs stage 1 tiled and stage 2 short-K.
constexpr int kTiledMinRows = 64;

struct Geometry {
  bool s1_tiled, s2_tiled;
  bool s2_short;  // stage 2 on the short-K geometry (I = 128 or 256, many rows)
};

static Geometry geometry(const GemmArgs& a) {
  const long A = (long)a.T * a.k_total;
  // the BF16 contract: its LDS-tiled kernel takes any K (a multiple of 128)
  if (a.fmt == kFmtBf16) {
    const bool many_bf = A >= (long)kTiledMinRows * a.NE;
    return Geometry{many_bf, many_bf, false};
  }
  const bool rows = A >= (long)kTiledMinRows * a.NE;
  const bool many =
      rows && (size_t)max_lds_per_block() >= tiled_lds_bytes(a.fmt, tiled_rows(A, a.NE));
  const bool s2_tiled = many && tiled_ok(a.H, a.I);
  const bool s2_short = rows && !s2_tiled && short_k_ok(a.I) && a.H % 256 == 0 &&
                        (size_t)max_lds_per_block() >= short_lds_bytes(a.fmt, a.I);
  return Geometry{many && tiled_k_ok(a.H) && a.I % 128 == 0, s2_tiled, s2_short};
}

bool fused_combine_ok(const GemmArgs& a) {
  const Geometry g = geometry(a);
  return a.fmt != kFmtBf16 && !g.s1_tiled && !g.s2_tiled && !g.s2_short &&
         fused_lds_bytes(a.T, a.k_total, a.I) <= (size_t)max_lds_per_block();
}

static hipError_t launch_geometry(const GemmArgs& a, const GemmWorkspace& w, int stages,
                                  Geometry g, hipStream_t s) {
  const bool bf = a.fmt == kFmtBf16;
  const long A = (long)a.T * a.k_total;
  const int TR = tiled_rows(A, a.NE);
  const int BM1 = g.s1_tiled ? (bf ? bf16_rows() : TR) : (bf ? bf16_stream_rows() : 16);
  const int BM2 = g.s2_tiled ? (bf ? bf16_rows() : TR)
                             : (g.s2_short ? short_rows() : (bf ? bf16_stream_rows() : 16));
  uint8_t* lists = a.ws + w.off[4];
  const TileArgs t1 = tile_list(lists, A, a.NE, BM1);
  const TileArgs t2 = BM2 == BM1 ? t1 : tile_list(lists + (w.off[5] - w.off[4]) / 2, A, a.NE, BM2);
  if (stages & 1) {
    // quantisation of x (none under the BF16 contract) and the tile list(s)
    const long nblk = bf ? 0 : (long)a.T * (a.H / 32);
    const int nqb = (int)((nblk + 1023) / 1024);
    const dim3 grid(nqb + (BM2 == BM1 ? 1 : 2));
    const size_t lds = (a.NE + 1) * sizeof(int);
    uint8_t *codes = a.ws + w.off[0], *scales = a.ws + w.off[1];
    if (bf)
      hipLaunchKernelGGL(prep_kernel<-1>, grid, dim3(1024), lds, s, a.x, nblk, codes, scales, nqb,
                         a.offsets, a.NE, BM1, t1, BM2, t2);
    else if (a.fmt == 0)
      hipLaunchKernelGGL(prep_kernel<0>, grid, dim3(1024), lds, s, a.x, nblk, codes, scales, nqb,
                         a.offsets, a.NE, BM1, t1, BM2, t2);
    else if (a.fmt == 2)
      hipLaunchKernelGGL(prep_kernel<2>, grid, dim3(1024), lds, s, a.x, nblk, codes, scales, nqb,
                         a.offsets, a.NE, BM1, t1, BM2, t2);
    else
      hipLaunchKernelGGL(prep_kernel<4>, grid, dim3(1024), lds, s, a.x, nblk, codes, scales, nqb,
                         a.offsets, a.NE, BM1, t1, BM2, t2);
  }
  if (stages & 2) {
    S1Args p1;
    p1.xq = bf ? reinterpret_cast<const uint8_t*>(a.x) : a.ws + w.off[0];
    p1.xs = a.ws + w.off[1];
    p1.sorted = a.sorted;
    p1.w13 = a.w13;
    p1.w13s = a.w13_s;
    p1.hq = a.ws + w.off[2];
    p1.hs = a.ws + w.off[3];
    p1.H = a.H;
    p1.I = a.I;
    p1.k_total = a.k_total;
    p1.t = t1;
    if (bf) (g.s1_tiled ? launch_s1_bf16 : launch_s1_bf16_stream)(p1, t1.mt_bound, s);
    else if (g.s1_tiled) launch_s1_tiled(p1, t1.mt_bound, a.fmt, TR, s);
    else launch_s1_stream(p1, t1.mt_bound, a.fmt, s);
  }
  if (stages & 4) {
    S2Args p2;
    p2.hq = a.ws + w.off[2];
    p2.hs = a.ws + w.off[3];
    p2.sorted = a.sorted;
    p2.w2 = a.w2;
    p2.w2s = a.w2_s;
    p2.partials = a.partials;
    p2.H = a.H;
    p2.I = a.I;
    p2.t = t2;
    if (a.out) launch_s2c_stream(S2CArgs{p2, a.topk_w, a.out, a.T, a.k_total}, a.fmt, s);
    else if (bf) (g.s2_tiled ? launch_s2_bf16 : launch_s2_bf16_stream)(p2, t2.mt_bound, s);
    else if (g.s2_tiled) launch_s2_tiled(p2, t2.mt_bound, a.fmt, TR, s);
    else if (g.s2_short) launch_s2_short(p2, t2.mt_bound, a.fmt, s);
    else launch_s2_stream(p2, t2.mt_bound, a.fmt, s);
  }
  return hipGetLastError();
}

hipError_t launch_grouped_gemm(const GemmArgs& a, int stages, hipStream_t s, int* variant) {
  const GemmWorkspace w = gemm_workspace(a.T, a.H, a.I, a.NE, a.k_total, a.fmt);
  const Geometry g = geometry(a);
  *variant = a.fmt == kFmtBf16 ? (g.s1_tiled ? 3 : 5)
                               : (g.s2_tiled ? 2 : (g.s2_short ? 6 : (g.s1_tiled ? 4 : 1)));
  if (a.T == 0) return hipSuccess;
  if (a.fmt != 0 && a.fmt != 2 && a.fmt != 4 && a.fmt != kFmtBf16) return hipErrorNotSupported;
  if (a.out && !fused_combine_ok(a)) return hipErrorNotSupported;
  return launch_geometry(a, w, stages, g, s);
}

}  // namespace moe
