// a5 / a6: grouped FP4 expert GEMMs, LDS-tiled matrix-core geometry for many
// rows per expert (prefill-sized batches).
//
// Workgroup tile: 128 sorted rows of one expert x 256 weight rows (stage 1:
// 128 gate rows and the 128 matching up rows; stage 2: 256 output columns),
// K in steps of 128. NW waves (4 or 8) in a 2 x NW/2 arrangement, each owning
// 64 rows x 512/NW weight rows = 4 x 32/NW products of 16x16 per step
// (16x16x128 block-scaled matrix-core instructions).
//
// Global -> LDS: direct loads (global_load_lds_dwordx4 writes lane l's 16
// bytes at LDS offset 16*l of the instruction's destination), several stages in
// flight (kStages-deep ring). Each lane picks the global address that lands in the right
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

#ifndef TILED_WAVES
#define TILED_WAVES 8
#endif

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
  static constexpr int kAKB = TBM * kARow / 1024;    // activation KiB per step
};

// Work split of the workgroup's NW waves.
template <int FA, int NW>
struct TWaves {
  static constexpr int kAInstr = TStage<FA>::kAKB / NW;   // activation DMA instructions per wave
  static constexpr int kBInstr = 16 / NW;                 // weight DMA instructions per wave
  static constexpr int kASRows = TBM / NW;                // activation scale rows per wave
  static constexpr int kBSRows = TBN / NW;                // weight scale rows per wave
  static constexpr int kLoads = kAInstr + kBInstr + 2;    // DMA instructions per wave per step
  static constexpr int kNCB = 32 / NW;                    // 16-column blocks per wave
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
template <int FA, int NW>
struct TLoad {
  using W = TWaves<FA, NW>;
  const uint8_t* a[W::kAInstr];  // activation row of each instruction
  const uint8_t* b[W::kBInstr];  // weight row of each instruction
  const uint8_t* as;             // activation scale row (lanes < kASRows)
  const uint8_t* bs;             // weight scale row (lanes < kBSRows)
  uint32_t a_chunk[W::kAInstr];  // logical 16-byte chunk this lane fetches
  uint32_t b_chunk[W::kBInstr];
};

// Row of the tile and swizzled chunk for activation DMA instruction i of wave
// w: one instruction fills 1 KiB of the row-major, chunk-swizzled layout.
template <int FA, int NW>
__device__ __forceinline__ void a_slot(int w, int i, int lane, int* row, uint32_t* chunk) {
  const int ci = TWaves<FA, NW>::kAInstr * w + i;
  if constexpr (FA == 0) {
    *row = 8 * ci + lane / 8;
    *chunk = (lane % 8) ^ ((*row >> 1) & 7);
  } else {
    *row = 16 * ci + lane / 4;
    *chunk = (lane % 4) ^ ((*row >> 2) & 3);
  }
}

template <int NW>
__device__ __forceinline__ void b_slot(int w, int i, int lane, int* row, uint32_t* chunk) {
  const int ci = (16 / NW) * w + i;
  *row = 16 * ci + lane / 4;
  *chunk = (lane % 4) ^ ((*row >> 2) & 3);
}

template <int FA, int NW>
__device__ __forceinline__ void tissue(uint8_t* st, const TLoad<FA, NW>& L, int w, int lane,
                                       int k0) {
  using S = TStage<FA>;
  using W = TWaves<FA, NW>;
#pragma unroll
  for (int i = 0; i < W::kAInstr; ++i)
    tdma16(L.a[i] + (size_t)k0 * S::kARow / 128 + 16 * L.a_chunk[i],
           st + S::kA + 1024 * (W::kAInstr * w + i));
#pragma unroll
  for (int i = 0; i < W::kBInstr; ++i)
    tdma16(L.b[i] + (size_t)k0 / 2 + 16 * L.b_chunk[i], st + S::kB + 1024 * (W::kBInstr * w + i));
  if (lane < W::kASRows) tdma4(L.as + k0 / 32, st + S::kAS + 4 * W::kASRows * w);
  if (lane < W::kBSRows) tdma4(L.bs + k0 / 32, st + S::kBS + 4 * W::kBSRows * w);
}

template <int FA>
__device__ __forceinline__ v8i read_a(const uint8_t* st, int r, int g) {
  using S = TStage<FA>;
  if constexpr (FA == 0) {
    const int sw = (r >> 1) & 7;
    const v4u lo = *reinterpret_cast<const v4u*>(st + S::kA + r * 128 + 16 * (g ^ sw));
    const v4u hi = *reinterpret_cast<const v4u*>(st + S::kA + r * 128 + 16 * ((4 + g) ^ sw));
    return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z,
               (int)hi.w};
  } else {
    const v4u lo = *reinterpret_cast<const v4u*>(st + S::kA + r * 64 + 16 * (g ^ ((r >> 2) & 3)));
    return v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
  }
}

// One K step for one wave: rows [64 wm, +64) (the first nrb 16-row blocks
// hold valid rows), weight rows brow[cb] + [0, 16). All fragments of the
// step are read from LDS first, then the 4 x NCB products issue.
template <int FA, int NCB, bool FULL>
__device__ __forceinline__ void tcompute(const uint8_t* st, int wm, const int* brow, int nrb,
                                         int g, int c16, v4f (*acc)[NCB]) {
  using S = TStage<FA>;
  v4u bop[NCB];
  int sb[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int r = brow[cb] + c16;
    bop[cb] = *reinterpret_cast<const v4u*>(st + S::kB + r * 64 + 16 * (g ^ ((r >> 2) & 3)));
    sb[cb] = (int)(*reinterpret_cast<const uint32_t*>(st + S::kBS + 4 * r) >> (8 * g));
  }
  v8i aop[4];
  int sa[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int r = 64 * wm + 16 * rb + c16;
    if (FULL || rb < nrb) {
      aop[rb] = read_a<FA>(st, r, g);
      sa[rb] = (int)(*reinterpret_cast<const uint32_t*>(st + S::kAS + 4 * r) >> (8 * g));
    }
  }
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    if (FULL || rb < nrb) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const v8i b =
            v8i{(int)bop[cb].x, (int)bop[cb].y, (int)bop[cb].z, (int)bop[cb].w, 0, 0, 0, 0};
        acc[rb][cb] = mfma_scaled_16x16x128<FA, 0, 0>(aop[rb], b, acc[rb][cb], sa[rb], sb[cb]);
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

// The K loop shared by both stages: a ring of kStages LDS stages, kStages-1
// of them in flight. Iteration k waits for its own stage-k loads, then one
// barrier makes every wave's stage k visible and guarantees every wave has
// finished reading stage k-1, whose slot is refilled with stage k+kStages-1.
constexpr int kStages = 4;

template <int FA, int NW>
__device__ __forceinline__ void tk_loop(uint8_t* lds, const TLoad<FA, NW>& L, int nk, int w,
                                        int lane, int wm, const int* brow, int nrb, int g, int c16,
                                        v4f (*acc)[TWaves<FA, NW>::kNCB]) {
  using S = TStage<FA>;
  using W = TWaves<FA, NW>;
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s)
    if (s < nk) tissue<FA, NW>(lds + s * S::kBytes, L, w, lane, s * 128);
  for (int k = 0; k < nk; ++k) {
    if (k + kStages - 2 < nk) twait_vmcnt<(kStages - 2) * W::kLoads>();
    else twait_vmcnt<0>();
    // Workgroup barrier without a memory fence: __syncthreads() would make the
    // compiler wait for every outstanding load (the younger stages too). The
    // explicit vmcnt wait above already covers this wave's stage-k loads, and
    // the asm memory clobber keeps LDS accesses on their side of the barrier.
    asm volatile("s_barrier" ::: "memory");
    if (k + kStages - 1 < nk)
      tissue<FA, NW>(lds + ((k + kStages - 1) % kStages) * S::kBytes, L, w, lane,
                     (k + kStages - 1) * 128);
    if (nrb == 4)
      tcompute<FA, W::kNCB, true>(lds + (k % kStages) * S::kBytes, wm, brow, nrb, g, c16, acc);
    else
      tcompute<FA, W::kNCB, false>(lds + (k % kStages) * S::kBytes, wm, brow, nrb, g, c16, acc);
  }
}

template <int FA, int NW>
__global__ __launch_bounds__(64 * NW, 1) void s1_tiled_kernel(S1Args p) {
  using W = TWaves<FA, NW>;
  constexpr int NCB = W::kNCB, NBW = NCB / 2;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int4 tile;
  int nt;
  if (!ttile(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int wm = w & 1, wn = w >> 1;
  const int hc0 = nt * (TBN / 2);  // first h column of the workgroup

  TLoad<FA, NW> L;
#pragma unroll
  for (int i = 0; i < W::kAInstr; ++i) {
    int r;
    a_slot<FA, NW>(w, i, lane, &r, &L.a_chunk[i]);
    const int tok = p.sorted[row0 + (r < nrows ? r : 0)] / p.k_total;
    L.a[i] = p.xq + (size_t)tok * (p.H / 32) * ActBytes<FA>::kBlock;
  }
  const size_t ebase = (size_t)e * 2 * p.I;
  auto wrow = [&](int r) {  // weight row of tile row r: 128 gate rows then 128 up rows
    return ebase + (r < TBN / 2 ? hc0 + r : p.I + hc0 + (r - TBN / 2));
  };
#pragma unroll
  for (int i = 0; i < W::kBInstr; ++i) {
    int r;
    b_slot<NW>(w, i, lane, &r, &L.b_chunk[i]);
    L.b[i] = p.w13 + wrow(r) * (p.H / 2);
  }
  {
    const int ra = W::kASRows * w + lane % W::kASRows;
    const int tok = p.sorted[row0 + (ra < nrows ? ra : 0)] / p.k_total;
    L.as = p.xs + (size_t)tok * (p.H / 32);
    L.bs = p.w13s + wrow(W::kBSRows * w + lane % W::kBSRows) * (p.H / 32);
  }
  // this wave's column blocks: NBW gate blocks then the matching NBW up blocks
  int brow[NCB];
#pragma unroll
  for (int cb = 0; cb < NBW; ++cb) {
    brow[cb] = 16 * (NBW * wn + cb);
    brow[NBW + cb] = TBN / 2 + 16 * (NBW * wn + cb);
  }
  const int nrb = min(4, max(0, (nrows - 64 * wm + 15) / 16));
  v4f acc[4][NCB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = v4f{0.f, 0.f, 0.f, 0.f};
  tk_loop<FA, NW>(lds, L, p.H / 128, w, lane, wm, brow, nrb, g, c16, acc);
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int off = 64 * wm + 16 * rb;
    if (off < nrows)
      s1_epilogue<FA, NBW>(acc[rb], p, row0 + off, nrows - off, hc0 + 16 * NBW * wn, g, c16);
  }
}

template <int FA, int NW>
__global__ __launch_bounds__(64 * NW, 1) void s2_tiled_kernel(S2Args p) {
  using W = TWaves<FA, NW>;
  constexpr int NCB = W::kNCB;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int4 tile;
  int nt;
  if (!ttile(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  const int g = lane >> 4, c16 = lane & 15;
  const int wm = w & 1, wn = w >> 1;
  const int nc0 = nt * TBN;

  TLoad<FA, NW> L;
#pragma unroll
  for (int i = 0; i < W::kAInstr; ++i) {
    int r;
    a_slot<FA, NW>(w, i, lane, &r, &L.a_chunk[i]);
    const size_t ar = (size_t)row0 + (r < nrows ? r : 0);
    L.a[i] = p.hq + ar * (p.I / 32) * ActBytes<FA>::kBlock;
  }
  const size_t ebase = (size_t)e * p.H + nc0;
#pragma unroll
  for (int i = 0; i < W::kBInstr; ++i) {
    int r;
    b_slot<NW>(w, i, lane, &r, &L.b_chunk[i]);
    L.b[i] = p.w2 + (ebase + r) * (p.I / 2);
  }
  {
    const int ra = W::kASRows * w + lane % W::kASRows;
    L.as = p.hs + ((size_t)row0 + (ra < nrows ? ra : 0)) * (p.I / 32);
    L.bs = p.w2s + (ebase + W::kBSRows * w + lane % W::kBSRows) * (p.I / 32);
  }
  int brow[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) brow[cb] = 16 * (NCB * wn + cb);
  const int nrb = min(4, max(0, (nrows - 64 * wm + 15) / 16));
  v4f acc[4][NCB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = v4f{0.f, 0.f, 0.f, 0.f};
  tk_loop<FA, NW>(lds, L, p.I / 128, w, lane, wm, brow, nrb, g, c16, acc);
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) {
    const int off = 64 * wm + 16 * rb;
    if (off < nrows)
      s2_epilogue<NCB>(acc[rb], p, row0 + off, nrows - off, nc0 + 16 * NCB * wn, g, c16);
  }
}

int tiled_rows() { return TBM; }

size_t tiled_lds_bytes(int fa) {
  return kStages * (size_t)(fa == 0 ? TStage<0>::kBytes : TStage<4>::kBytes);
}

bool tiled_ok(int H, int I) { return I % (TBN / 2) == 0 && H % TBN == 0; }

// Waves per workgroup of the tiled kernels (4 or 8).
constexpr int kTiledWaves = TILED_WAVES;

template <int FA>
static void launch_t1(const S1Args& p, long mt, hipStream_t s) {
  S1Args q = p;
  q.t.n_ntiles = p.I / (TBN / 2);
  const long chunks = (mt + kChunkM - 1) / kChunkM;
  const long n = chunks * kChunkM * q.t.n_ntiles;
  hipLaunchKernelGGL((s1_tiled_kernel<FA, kTiledWaves>), dim3((int)((n + 7) / 8 * 8)),
                     dim3(64 * kTiledWaves), kStages * TStage<FA>::kBytes, s, q);
}

template <int FA>
static void launch_t2(const S2Args& p, long mt, hipStream_t s) {
  S2Args q = p;
  q.t.n_ntiles = p.H / TBN;
  const long chunks = (mt + kChunkM - 1) / kChunkM;
  const long n = chunks * kChunkM * q.t.n_ntiles;
  hipLaunchKernelGGL((s2_tiled_kernel<FA, kTiledWaves>), dim3((int)((n + 7) / 8 * 8)),
                     dim3(64 * kTiledWaves), kStages * TStage<FA>::kBytes, s, q);
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
