// a5 / a6: grouped FP4 expert GEMMs, weight-streaming geometry.
//
// Work item: (row tile of up to 16 sorted rows of one expert, N tile). Every
// workgroup streams its N tile of the expert's packed FP4 weights from HBM
// exactly once, over the whole K extent, and multiplies it with the tile's
// activation rows on the block-scaled matrix cores (16x16x128, FP4 weights
// consumed directly: no unpacking, no offline expansion -- the paper found
// that expanding FP4 to INT8 doubled weight traffic and slowed the gate
// kernel; Rejected or reverted directions).
//
// K placement. The matrix core sums over K, so any permutation of K applied
// to both operands gives the same result. A weight lane (column n = l % 16,
// lane group g = l / 16) takes, per step of KC = 128*J elements, the J
// consecutive 32-element blocks [g*J, g*J + J) of the step: one contiguous
// 16*J-byte run of every weight row it owns (row segments of 64*J bytes per
// wave, fully used). Product j of the step consumes block g*J + j from lane
// group g, and the lane's scale register holds the J block scales in bytes
// 0..J-1, selected per product with the instruction's op_sel field. The
// activation lanes load whatever meets those weight elements (frag_load).
//
// Stage 1 (gate/up): each wave owns 16*NBW h columns; it streams those gate
// rows and the matching up rows, so SwiGLU and the per-32 re-quantisation of
// h (the quantisation block spans two 16-column tiles of the same wave) run in
// registers. Stage 2 (down): each wave owns 16*NBW output columns of H and
// writes fp32 partials to the unique row a = sorted[r] of every assignment.
#include "moe_dev.h"
#include "moe_launch.h"

namespace moe {

template <int FA>
struct ActBytes;  // bytes per 32-element block of the activation operand
template <>
struct ActBytes<0> {
  static constexpr int kBlock = 32;
};
template <>
struct ActBytes<4> {
  static constexpr int kBlock = 16;
};

template <int J>
__device__ __forceinline__ uint32_t load_scales(const uint8_t* p) {
  if constexpr (J == 4) return *reinterpret_cast<const uint32_t*>(p);
  if constexpr (J == 2) return *reinterpret_cast<const uint16_t*>(p);
  return *p;
}

// Registers of one K step: activation run + scales, NB weight rows + scales.
template <int FA, int J, int NB>
struct Frag {
  static constexpr int kAV = J * ActBytes<FA>::kBlock / 16;
  uint4 a[kAV];
  uint32_t as;
  uint4 b[NB][J];
  uint32_t bs[NB];
};

// Loads of one K step starting at 32-element block `step` (a multiple of 4J).
// Weights (FP4) and FP4 activations: lane group g takes the contiguous blocks
// [step + g*J, step + g*J + J). FP8 activations: the matrix core reads an FP8
// lane's 32 bytes as two 16-element halves that sit 64 elements apart in its
// K order (bytes 0-15 at K 16g.., bytes 16-31 at K 64+16g..), while an FP4
// lane's 32 elements are contiguous; so for product j the FP8 lane takes the
// 16-byte pieces that meet the FP4 lanes' elements: pieces (g/2)*J + j and
// (2 + g/2)*J + j of 32-byte blocks, half g%2 of each.
template <int FA, int J, int NB>
__device__ __forceinline__ void frag_load(Frag<FA, J, NB>& f, const uint8_t* a_row,
                                          const uint8_t* as_row, bool a_ok,
                                          const uint8_t* const* b_rows,
                                          const uint8_t* const* bs_rows, int step, int g) {
  constexpr int kAB = ActBytes<FA>::kBlock;
  const int blk0 = step + g * J;
  if (a_ok) {
    if constexpr (FA == 0) {
      const uint8_t* base = a_row + (size_t)step * 32 + 16 * (g & 1);
#pragma unroll
      for (int j = 0; j < J; ++j) {
        f.a[2 * j] = *reinterpret_cast<const uint4*>(base + 32 * ((g >> 1) * J + j));
        f.a[2 * j + 1] = *reinterpret_cast<const uint4*>(base + 32 * ((2 + (g >> 1)) * J + j));
      }
    } else {
#pragma unroll
      for (int v = 0; v < Frag<FA, J, NB>::kAV; ++v)
        f.a[v] = *reinterpret_cast<const uint4*>(a_row + (size_t)blk0 * kAB + 16 * v);
    }
    f.as = load_scales<J>(as_row + blk0);
  } else {
#pragma unroll
    for (int v = 0; v < Frag<FA, J, NB>::kAV; ++v) f.a[v] = make_uint4(0, 0, 0, 0);
    f.as = 0x7f7f7f7fu;  // 2^0: a zero row contributes exact zeros
  }
#pragma unroll
  for (int n = 0; n < NB; ++n) {
#pragma unroll
    for (int j = 0; j < J; ++j)
      f.b[n][j] = *reinterpret_cast<const uint4*>(b_rows[n] + (size_t)blk0 * 16 + 16 * j);
    f.bs[n] = load_scales<J>(bs_rows[n] + blk0);
  }
}

template <int FA, int J, int NB>
__device__ __forceinline__ void frag_mma(const Frag<FA, J, NB>& f, v4f* acc) {
  static_for<J>([&](auto jc) {
    constexpr int j = decltype(jc)::value;
    v8i a;
    if constexpr (FA == 0) {
      const uint4 lo = f.a[2 * j], hi = f.a[2 * j + 1];
      a = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    } else {
      const uint4 lo = f.a[j];
      a = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
    }
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const uint4 bq = f.b[n][j];
      const v8i b = v8i{(int)bq.x, (int)bq.y, (int)bq.z, (int)bq.w, 0, 0, 0, 0};
      acc[n] = mfma_scaled_16x16x128<FA, j, j>(a, b, acc[n], (int)f.as, (int)f.bs[n]);
    }
  });
}

// Full K loop for one wave: NB weight rows (16 each, one per lane column),
// one 16-row activation tile. K = nblk32 * 32 with nblk32 % 4 == 0.
template <int FA, int J, int NB>
__device__ __forceinline__ void stream_k(const uint8_t* a_row, const uint8_t* as_row, bool a_ok,
                                         const uint8_t* const* b_rows,
                                         const uint8_t* const* bs_rows, int nblk32, int g,
                                         v4f* acc) {
  const int kc_blocks = 4 * J;  // 32-element blocks per step
  const int nsteps = nblk32 / kc_blocks;
  if (nsteps > 0) {
    Frag<FA, J, NB> f0, f1;
    frag_load<FA, J, NB>(f0, a_row, as_row, a_ok, b_rows, bs_rows, 0, g);
    for (int c = 0; c < nsteps; c += 2) {
      if (c + 1 < nsteps)
        frag_load<FA, J, NB>(f1, a_row, as_row, a_ok, b_rows, bs_rows, (c + 1) * kc_blocks, g);
      frag_mma<FA, J, NB>(f0, acc);
      if (c + 1 < nsteps) {
        if (c + 2 < nsteps)
          frag_load<FA, J, NB>(f0, a_row, as_row, a_ok, b_rows, bs_rows, (c + 2) * kc_blocks, g);
        frag_mma<FA, J, NB>(f1, acc);
      }
    }
  }
  // K tail: steps of 128 elements (J = 1)
  for (int blk = nsteps * kc_blocks; blk < nblk32; blk += 4) {
    Frag<FA, 1, NB> f;
    frag_load<FA, 1, NB>(f, a_row, as_row, a_ok, b_rows, bs_rows, blk, g);
    frag_mma<FA, 1, NB>(f, acc);
  }
}

struct TileArgs {
  const int4* tiles;    // (expert, first sorted row, rows, 0)
  const int* ntiles;    // number of valid tiles
  int mt_bound;         // tiles the grid was sized for
  int n_ntiles;         // N tiles per expert
};

// Decode the workgroup's (row tile, N tile); false if it has no work.
__device__ __forceinline__ bool tile_of_block(const TileArgs& t, int4* tile, int* nt) {
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = lin % t.mt_bound;
  *nt = lin / t.mt_bound;
  if (*nt >= t.n_ntiles || mt >= *t.ntiles) return false;
  *tile = t.tiles[mt];
  return true;
}

struct S1Args {
  const uint8_t *xq, *xs;      // activation codes [T, H*bits/8], scales [T, H/32]
  const int32_t* sorted;
  const uint8_t *w13, *w13s;   // [NE, 2I, H/2], [NE, 2I, H/32]
  uint8_t *hq, *hs;            // [A, I*bits/8], [A, I/32]
  int H, I, k_total;
  TileArgs t;
};

template <int FA, int J, int NBW>
__global__ __launch_bounds__(256) void s1_stream_kernel(S1Args p) {
  static_assert(NBW % 2 == 0, "a quantisation block spans two 16-column tiles");
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int hc0 = nt * (4 * NBW * 16) + w * (NBW * 16);  // first h column of this wave

  const bool a_ok = c16 < nrows;
  const int tok = a_ok ? p.sorted[row0 + c16] / p.k_total : 0;
  const uint8_t* a_row = p.xq + (size_t)tok * (p.H / 32) * kAB;
  const uint8_t* as_row = p.xs + (size_t)tok * (p.H / 32);

  const uint8_t* b_rows[2 * NBW];
  const uint8_t* bs_rows[2 * NBW];
  const size_t ebase = (size_t)e * 2 * p.I;
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t gr = ebase + hc0 + 16 * b + c16;  // gate row
    const size_t ur = gr + p.I;                    // up row
    b_rows[b] = p.w13 + gr * (p.H / 2);
    bs_rows[b] = p.w13s + gr * (p.H / 32);
    b_rows[NBW + b] = p.w13 + ur * (p.H / 2);
    bs_rows[NBW + b] = p.w13s + ur * (p.H / 32);
  }
  v4f acc[2 * NBW];
#pragma unroll
  for (int n = 0; n < 2 * NBW; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k<FA, J, 2 * NBW>(a_row, as_row, a_ok, b_rows, bs_rows, p.H / 32, g, acc);

  // SwiGLU and per-32 quantisation of h. Lane (g, c16) holds rows 4g+i of
  // columns hc0 + 16b + c16; a quantisation block is columns [32q, 32q+32)
  // of the wave, i.e. tiles b = 2q, 2q+1 across the 16 lanes of group g.
  const int ib = p.I / 32;
#pragma unroll
  for (int q = 0; q < NBW / 2; ++q) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float G0 = acc[2 * q][i], U0 = acc[NBW + 2 * q][i];
      const float G1 = acc[2 * q + 1][i], U1 = acc[NBW + 2 * q + 1][i];
      const float h0 = G0 * U0 / (1.0f + expf(-G0));
      const float h1 = G1 * U1 / (1.0f + expf(-G1));
      float m = fmaxf(fabsf(h0), fabsf(h1));
#pragma unroll
      for (int s = 8; s >= 1; s >>= 1) m = fmaxf(m, shfl_xor_f(m, s));
      const int X = mx_scale_exp<FA>(m);
      const uint32_t c0 = mx_encode<FA>(ldexpf(h0, -X));
      const uint32_t c1 = mx_encode<FA>(ldexpf(h1, -X));
      const int rl = 4 * g + i;
      const size_t r = (size_t)row0 + rl;
      const int col = hc0 + 32 * q + c16;
      if constexpr (FA == 0) {
        if (rl < nrows) {
          p.hq[r * p.I + col] = (uint8_t)c0;
          p.hq[r * p.I + col + 16] = (uint8_t)c1;
        }
      } else {
        // two adjacent columns per byte, low nibble first
        const uint32_t o0 = __shfl_xor((int)c0, 1, kWave), o1 = __shfl_xor((int)c1, 1, kWave);
        if (rl < nrows && (c16 & 1) == 0) {
          p.hq[r * (p.I / 2) + col / 2] = (uint8_t)(c0 | (o0 << 4));
          p.hq[r * (p.I / 2) + (col + 16) / 2] = (uint8_t)(c1 | (o1 << 4));
        }
      }
      if (rl < nrows && c16 == 0) p.hs[r * ib + (hc0 / 32) + q] = (uint8_t)(X + 127);
    }
  }
}

struct S2Args {
  const uint8_t *hq, *hs;     // [A, I*bits/8], [A, I/32] in sorted-row order
  const int32_t* sorted;
  const uint8_t *w2, *w2s;    // [NE, H, I/2], [NE, H, I/32]
  float* partials;            // [A, H] indexed by assignment
  int H, I;
  TileArgs t;
};

template <int FA, int J, int NBW>
__global__ __launch_bounds__(256) void s2_stream_kernel(S2Args p) {
  constexpr int kAB = ActBytes<FA>::kBlock;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int nc0 = nt * (4 * NBW * 16) + w * (NBW * 16);  // first output column of this wave

  const bool a_ok = c16 < nrows;
  const size_t ar = (size_t)row0 + (a_ok ? c16 : 0);
  const uint8_t* a_row = p.hq + ar * (p.I / 32) * kAB;
  const uint8_t* as_row = p.hs + ar * (p.I / 32);

  const uint8_t* b_rows[NBW];
  const uint8_t* bs_rows[NBW];
#pragma unroll
  for (int b = 0; b < NBW; ++b) {
    const size_t rr = (size_t)e * p.H + nc0 + 16 * b + c16;
    b_rows[b] = p.w2 + rr * (p.I / 2);
    bs_rows[b] = p.w2s + rr * (p.I / 32);
  }
  v4f acc[NBW];
#pragma unroll
  for (int n = 0; n < NBW; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  stream_k<FA, J, NBW>(a_row, as_row, a_ok, b_rows, bs_rows, p.I / 32, g, acc);

#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rl = 4 * g + i;
    if (rl < nrows) {
      const size_t a = (size_t)p.sorted[row0 + rl];
      float* dst = p.partials + a * p.H + nc0 + c16;
#pragma unroll
      for (int b = 0; b < NBW; ++b) dst[16 * b] = acc[b][i];
    }
  }
}

// ---------------------------------------------------------------------------
// Tile list: expert e with c rows gets ceil(c / BM) row tiles. One block of
// 1024 threads: tile counts, exclusive scan, then every thread fills tiles
// i = tid, tid + 1024, ... by binary search over the per-expert tile starts.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void build_tiles_kernel(const int32_t* __restrict__ offsets,
                                                           int NE, int BM, int4* __restrict__ tiles,
                                                           int* __restrict__ ntiles) {
  extern __shared__ int start[];  // [NE + 1]
  int m[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int e = threadIdx.x + 1024 * q;
    m[q] = e < NE ? (offsets[e + 1] - offsets[e] + BM - 1) / BM : 0;
  }
  int t0, t1;
  const int p0 = block_exclusive_scan_1024(m[0], &t0);
  const int p1 = block_exclusive_scan_1024(m[1], &t1) + t0;
  if (threadIdx.x < NE) start[threadIdx.x] = p0;
  if (threadIdx.x + 1024 < NE) start[threadIdx.x + 1024] = p1;
  const int total = t0 + t1;
  if (threadIdx.x == 0) {
    start[NE] = total;
    *ntiles = total;
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

static int tile_bound(long A, int NE, int BM) {
  const long nonempty = A < NE ? A : NE;
  return (int)((A + nonempty * (BM - 1)) / BM);
}

GemmWorkspace gemm_workspace(int T, int H, int I, int NE, int k_total, int fmt) {
  auto al = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t A = (size_t)T * k_total;
  const size_t bits = act_bits(fmt);
  GemmWorkspace w;
  size_t o = 0;
  w.off[0] = o;  o += al((size_t)T * H * bits / 8);
  w.off[1] = o;  o += al((size_t)T * (H / 32));
  w.off[2] = o;  o += al(A * I * bits / 8);
  w.off[3] = o;  o += al(A * (I / 32));
  w.off[4] = o;  o += al(sizeof(int4) * ((size_t)tile_bound((long)A, NE, 16) + 1) + 16);
  w.off[5] = o;
  return w;
}

template <int FA>
static hipError_t launch_stream(const GemmArgs& a, const GemmWorkspace& w, int stages,
                                hipStream_t s) {
  constexpr int BM = 16, J = 2, NBW1 = 2, NBW2 = 4;
  const long A = (long)a.T * a.k_total;
  const int mt = tile_bound(A, a.NE, BM);
  int4* tiles = reinterpret_cast<int4*>(a.ws + w.off[4]);
  int* ntiles = reinterpret_cast<int*>(tiles + mt + 1);
  auto grid_of = [](long n) { return (int)((n + 7) / 8 * 8); };
  if (a.I % (4 * NBW1 * 16) != 0) return hipErrorInvalidValue;

  if (stages & 1) {
    hipError_t err = launch_quantize_act(a.x, a.T, a.H, a.fmt, a.ws + w.off[0], a.ws + w.off[1], s);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(build_tiles_kernel, dim3(1), dim3(1024), (a.NE + 1) * sizeof(int), s,
                       a.offsets, a.NE, BM, tiles, ntiles);
  }
  if (stages & 2) {
    S1Args p1;
    p1.xq = a.ws + w.off[0];
    p1.xs = a.ws + w.off[1];
    p1.sorted = a.sorted;
    p1.w13 = a.w13;
    p1.w13s = a.w13_s;
    p1.hq = a.ws + w.off[2];
    p1.hs = a.ws + w.off[3];
    p1.H = a.H;
    p1.I = a.I;
    p1.k_total = a.k_total;
    p1.t = TileArgs{tiles, ntiles, mt, a.I / (4 * NBW1 * 16)};
    hipLaunchKernelGGL((s1_stream_kernel<FA, J, NBW1>), dim3(grid_of((long)mt * p1.t.n_ntiles)),
                       dim3(256), 0, s, p1);
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
    if (a.H % (4 * NBW2 * 16) == 0) {
      p2.t = TileArgs{tiles, ntiles, mt, a.H / (4 * NBW2 * 16)};
      hipLaunchKernelGGL((s2_stream_kernel<FA, J, NBW2>), dim3(grid_of((long)mt * p2.t.n_ntiles)),
                         dim3(256), 0, s, p2);
    } else {
      p2.t = TileArgs{tiles, ntiles, mt, a.H / (4 * 2 * 16)};
      hipLaunchKernelGGL((s2_stream_kernel<FA, J, 2>), dim3(grid_of((long)mt * p2.t.n_ntiles)),
                         dim3(256), 0, s, p2);
    }
  }
  return hipGetLastError();
}

hipError_t launch_grouped_gemm(const GemmArgs& a, int stages, hipStream_t s, int* variant) {
  const GemmWorkspace w = gemm_workspace(a.T, a.H, a.I, a.NE, a.k_total, a.fmt);
  *variant = 1;
  if (a.T == 0) return hipSuccess;
  if (a.fmt == 0) return launch_stream<0>(a, w, stages, s);
  if (a.fmt == 4) return launch_stream<4>(a, w, stages, s);
  return hipErrorNotSupported;
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
  const uint8_t* bsr = sb + c16 * 4;
  v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
  Frag<FA, 1, 1> f;
  frag_load<FA, 1, 1>(f, ar, sa + c16 * 4, true, &br, &bsr, 0, g);
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
