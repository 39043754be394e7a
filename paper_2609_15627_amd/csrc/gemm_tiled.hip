// a5 / a6: grouped FP4 expert GEMMs, LDS-tiled matrix-core geometry for many
// rows per expert (prefill-sized batches).
//
// Workgroup tile: 128 sorted rows of one expert x 256 weight rows (stage 1:
// 128 gate rows and the 128 matching up rows; stage 2: 256 output columns),
// K in steps of 128. Four waves in a 2 x 2 arrangement, each owning 64 rows x
// 128 weight rows = 4 x 8 products of 16x16 per step (16x16x128 block-scaled
// matrix-core instructions), so every activation fragment read from LDS is
// used 8 times and every weight fragment 4 times.
//
// Global -> LDS: direct loads (global_load_lds_dwordx4 writes lane l's 16
// bytes at LDS offset 16*l of the instruction's destination), two stages in
// flight. Each lane picks the global address that lands in the right
// swizzled LDS slot:
//   activation rows (FP8, 128 bytes per row and step): 16-byte chunk c of row
//     r is stored at chunk c ^ ((r >> 1) & 7);
//   weight rows (FP4, 64 bytes per row and step) and FP4 activation rows:
//     chunk c of row r at chunk c ^ ((r >> 2) & 3);
// so the matrix-core operand reads (16 lanes = 16 consecutive rows, one
// chunk each) hit 16 distinct bank groups. Scales: one dword per row and
// step (the 4 block scales of the step), lane group g uses byte g.
//
// Rows past the tile's end load a valid row instead (a product row depends
// only on its own activation row, and those rows are never stored), and
// 16-row blocks that are entirely past the end skip their products.
//
// Work order: chunks of kChunkM consecutive row tiles x all N tiles, N tile
// fastest across chunks of row tiles: the workgroups that run together on an
// XCD share activation rows (across N tiles) and weight tiles (across the row
// tiles of one expert) through that XCD's L2.
#include "gemm_common.h"
#include "gemm_launch.h"

namespace moe {

constexpr int TBM = 128, TBN = 256;
constexpr int kChunkM = 4;

typedef __attribute__((address_space(3))) void lds_ptr_t;

template <int FA>
struct TStage {
  static constexpr int kARow = FA == 0 ? 128 : 64;  // activation bytes per row per step
  static constexpr int kA = 0;
  static constexpr int kB = kA + TBM * kARow;        // 256 weight rows x 64 bytes
  static constexpr int kAS = kB + TBN * 64;          // 128 activation scale dwords
  static constexpr int kBS = kAS + TBM * 4;          // 256 weight scale dwords
  static constexpr int kBytes = kBS + TBN * 4;
  static constexpr int kAInstr = TBM * kARow / 4096;  // activation DMA instructions per wave
  static constexpr int kLoads = kAInstr + 4 + 2;      // DMA instructions per wave per step
};

__device__ __forceinline__ void tdma16(const void* g, uint8_t* l) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr_t*)l, 16, 0, 0);
}
__device__ __forceinline__ void tdma4(const void* g, uint8_t* l) {
  __builtin_amdgcn_global_load_lds(g, (lds_ptr_t*)l, 4, 0, 0);
}

template <int N>
__device__ __forceinline__ void twait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xf00);
}

// Per-lane source rows of the DMA instructions of one wave.
template <int FA>
struct TLoad {
  const uint8_t* a[TStage<FA>::kAInstr];  // activation row of each instruction
  const uint8_t* b[4];                    // weight row of each instruction
  const uint8_t* as;                      // activation scale row (lanes < 32)
  const uint8_t* bs;                      // weight scale row
  uint32_t a_chunk[TStage<FA>::kAInstr];  // logical 16-byte chunk this lane fetches
  uint32_t b_chunk[4];
};

template <int FA>
__device__ __forceinline__ void tissue(uint8_t* st, const TLoad<FA>& L, int w, int lane, int k0) {
  using S = TStage<FA>;
#pragma unroll
  for (int i = 0; i < S::kAInstr; ++i)
    tdma16(L.a[i] + (size_t)k0 * S::kARow / 128 + 16 * L.a_chunk[i],
           st + S::kA + 1024 * (S::kAInstr * w + i));
#pragma unroll
  for (int i = 0; i < 4; ++i)
    tdma16(L.b[i] + (size_t)k0 / 2 + 16 * L.b_chunk[i], st + S::kB + 1024 * (4 * w + i));
  if (lane < 32) tdma4(L.as + k0 / 32, st + S::kAS + 128 * w);  // 32 rows per wave
  tdma4(L.bs + k0 / 32, st + S::kBS + 256 * w);
}

// One K step for one wave: rows [64 wm, +64), weight rows given by brow0[cb].
template <int FA>
__device__ __forceinline__ void tcompute(const uint8_t* st, int wm, const int* brow, int nrb,
                                         int g, int c16, v4f (*acc)[8]) {
  using S = TStage<FA>;
  v4u bop[8];
  int sb[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) {
    const int r = brow[cb] + c16;
    const int ch = g ^ ((r >> 2) & 3);
    bop[cb] = *reinterpret_cast<const v4u*>(st + S::kB + r * 64 + 16 * ch);
    sb[cb] = (int)(*reinterpret_cast<const uint32_t*>(st + S::kBS + 4 * r) >> (8 * g));
  }
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    if (rb < nrb) {
      const int r = 64 * wm + 16 * rb + c16;
      v8i aop;
      if constexpr (FA == 0) {
        const int sw = (r >> 1) & 7;
        const v4u lo = *reinterpret_cast<const v4u*>(st + S::kA + r * 128 + 16 * (g ^ sw));
        const v4u hi = *reinterpret_cast<const v4u*>(st + S::kA + r * 128 + 16 * ((4 + g) ^ sw));
        aop = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z,
                  (int)hi.w};
      } else {
        const v4u lo = *reinterpret_cast<const v4u*>(st + S::kA + r * 64 + 16 * (g ^ ((r >> 2) & 3)));
        aop = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
      }
      const int sa = (int)(*reinterpret_cast<const uint32_t*>(st + S::kAS + 4 * r) >> (8 * g));
#pragma unroll
      for (int cb = 0; cb < 8; ++cb) {
        const v8i b = v8i{(int)bop[cb].x, (int)bop[cb].y, (int)bop[cb].z, (int)bop[cb].w, 0, 0, 0, 0};
        acc[rb][cb] = mfma_scaled_16x16x128<FA, 0, 0>(aop, b, acc[rb][cb], sa, sb[cb]);
      }
    }
  }
}

// Work item of this workgroup: row tile mt, N tile nt.
__device__ __forceinline__ bool ttile(const TileArgs& t, int4* tile, int* nt) {
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int per = kChunkM * t.n_ntiles;
  const int chunk = lin / per, r = lin % per;
  *nt = r / kChunkM;
  const int mt = chunk * kChunkM + r % kChunkM;
  if (mt >= *t.ntiles) return false;
  *tile = t.tiles[mt];
  return true;
}

// The K loop shared by both stages (two-stage DMA ring, barriers around the
// consumption of each stage).
template <int FA>
__device__ __forceinline__ void tk_loop(uint8_t* lds, const TLoad<FA>& L, int nk, int w, int lane,
                                        int wm, const int* brow, int nrb, int g, int c16,
                                        v4f (*acc)[8]) {
  using S = TStage<FA>;
  tissue<FA>(lds, L, w, lane, 0);
  for (int k = 0; k < nk; ++k) {
    uint8_t* cur = lds + (k & 1) * S::kBytes;
    if (k + 1 < nk) {
      tissue<FA>(lds + ((k + 1) & 1) * S::kBytes, L, w, lane, (k + 1) * 128);
      twait_vmcnt<S::kLoads>();
    } else {
      twait_vmcnt<0>();
    }
    __syncthreads();
    tcompute<FA>(cur, wm, brow, nrb, g, c16, acc);
    __syncthreads();
  }
}

template <int FA>
__global__ __launch_bounds__(256, 1) void s1_tiled_kernel(S1Args p) {
  using S = TStage<FA>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int4 tile;
  int nt;
  if (!ttile(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int wm = w & 1, wn = w >> 1;
  const int hc0 = nt * (TBN / 2);  // first h column of the workgroup

  TLoad<FA> L;
#pragma unroll
  for (int i = 0; i < S::kAInstr; ++i) {
    int r, phys, sw;
    if constexpr (FA == 0) {
      r = 8 * (S::kAInstr * w + i) + lane / 8;
      phys = lane % 8;
      sw = (r >> 1) & 7;
    } else {
      r = 16 * (S::kAInstr * w + i) + lane / 4;
      phys = lane % 4;
      sw = (r >> 2) & 3;
    }
    const int rr = r < nrows ? r : 0;
    const int tok = p.sorted[row0 + rr] / p.k_total;
    L.a[i] = p.xq + (size_t)tok * (p.H / 32) * ActBytes<FA>::kBlock;
    L.a_chunk[i] = phys ^ sw;
  }
  const size_t ebase = (size_t)e * 2 * p.I;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 16 * (4 * w + i) + lane / 4;  // weight row of the tile, 0..255
    const size_t wr = ebase + (r < 128 ? hc0 + r : p.I + hc0 + (r - 128));
    L.b[i] = p.w13 + wr * (p.H / 2);
    L.b_chunk[i] = (lane % 4) ^ ((r >> 2) & 3);
  }
  {
    const int ra = 32 * w + (lane & 31);
    const int tok = p.sorted[row0 + (ra < nrows ? ra : 0)] / p.k_total;
    L.as = p.xs + (size_t)tok * (p.H / 32);
    const int rb = 64 * w + lane;
    const size_t wr = ebase + (rb < 128 ? hc0 + rb : p.I + hc0 + (rb - 128));
    L.bs = p.w13s + wr * (p.H / 32);
  }
  // this wave's 8 weight column blocks: 4 gate then 4 up
  int brow[8];
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    brow[cb] = 64 * wn + 16 * cb;
    brow[4 + cb] = 128 + 64 * wn + 16 * cb;
  }
  const int nrb = min(4, max(0, (nrows - 64 * wm + 15) / 16));
  v4f acc[4][8];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) acc[rb][cb] = v4f{0.f, 0.f, 0.f, 0.f};
  tk_loop<FA>(lds, L, p.H / 128, w, lane, wm, brow, nrb, g, c16, acc);
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int off = 64 * wm + 16 * rb;
    if (off < nrows) s1_epilogue<FA, 4>(acc[rb], p, row0 + off, nrows - off, hc0 + 64 * wn, g, c16);
  }
}

template <int FA>
__global__ __launch_bounds__(256, 1) void s2_tiled_kernel(S2Args p) {
  using S = TStage<FA>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int4 tile;
  int nt;
  if (!ttile(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int wm = w & 1, wn = w >> 1;
  const int nc0 = nt * TBN;

  TLoad<FA> L;
#pragma unroll
  for (int i = 0; i < S::kAInstr; ++i) {
    int r, phys, sw;
    if constexpr (FA == 0) {
      r = 8 * (S::kAInstr * w + i) + lane / 8;
      phys = lane % 8;
      sw = (r >> 1) & 7;
    } else {
      r = 16 * (S::kAInstr * w + i) + lane / 4;
      phys = lane % 4;
      sw = (r >> 2) & 3;
    }
    const size_t ar = (size_t)row0 + (r < nrows ? r : 0);
    L.a[i] = p.hq + ar * (p.I / 32) * ActBytes<FA>::kBlock;
    L.a_chunk[i] = phys ^ sw;
  }
  const size_t ebase = (size_t)e * p.H + nc0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 16 * (4 * w + i) + lane / 4;
    L.b[i] = p.w2 + (ebase + r) * (p.I / 2);
    L.b_chunk[i] = (lane % 4) ^ ((r >> 2) & 3);
  }
  {
    const int ra = 32 * w + (lane & 31);
    L.as = p.hs + ((size_t)row0 + (ra < nrows ? ra : 0)) * (p.I / 32);
    L.bs = p.w2s + (ebase + 64 * w + lane) * (p.I / 32);
  }
  int brow[8];
#pragma unroll
  for (int cb = 0; cb < 8; ++cb) brow[cb] = 128 * wn + 16 * cb;
  const int nrb = min(4, max(0, (nrows - 64 * wm + 15) / 16));
  v4f acc[4][8];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < 8; ++cb) acc[rb][cb] = v4f{0.f, 0.f, 0.f, 0.f};
  tk_loop<FA>(lds, L, p.I / 128, w, lane, wm, brow, nrb, g, c16, acc);
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int off = 64 * wm + 16 * rb;
    if (off < nrows) s2_epilogue<8>(acc[rb], p, row0 + off, nrows - off, nc0 + 128 * wn, g, c16);
  }
}

int tiled_rows() { return TBM; }

size_t tiled_lds_bytes(int fa) {
  return 2 * (size_t)(fa == 0 ? TStage<0>::kBytes : TStage<4>::kBytes);
}

bool tiled_ok(int H, int I) { return I % (TBN / 2) == 0 && H % TBN == 0; }

template <int FA>
static void launch_t1(const S1Args& p, long mt, hipStream_t s) {
  S1Args q = p;
  q.t.n_ntiles = p.I / (TBN / 2);
  const long chunks = (mt + kChunkM - 1) / kChunkM;
  const long n = chunks * kChunkM * q.t.n_ntiles;
  hipLaunchKernelGGL((s1_tiled_kernel<FA>), dim3((int)((n + 7) / 8 * 8)), dim3(256),
                     2 * TStage<FA>::kBytes, s, q);
}

template <int FA>
static void launch_t2(const S2Args& p, long mt, hipStream_t s) {
  S2Args q = p;
  q.t.n_ntiles = p.H / TBN;
  const long chunks = (mt + kChunkM - 1) / kChunkM;
  const long n = chunks * kChunkM * q.t.n_ntiles;
  hipLaunchKernelGGL((s2_tiled_kernel<FA>), dim3((int)((n + 7) / 8 * 8)), dim3(256),
                     2 * TStage<FA>::kBytes, s, q);
}

void launch_s1_tiled(const S1Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_t1<0>(p, mt, s);
  else launch_t1<4>(p, mt, s);
}

void launch_s2_tiled(const S2Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_t2<0>(p, mt, s);
  else launch_t2<4>(p, mt, s);
}

}  // namespace moe
