// a6: the down projection (stage 2) for a short reduction extent and many
// rows per expert -- the tensor-parallel expert shard's shape (I = 256, ~128
// rows per expert), where the fp32 partial stores (H * 4 bytes per row) are
// four times the bytes of the FP4 weights they are computed from, so the
// stage is bound by its stores.
//
// Work item: a row tile of up to 128 sorted rows of one expert x 256 output
// columns. The whole K = I extent of both operands fits in LDS, so one burst
// of DMA (16 bytes a lane, 1 KiB per instruction) brings the tile's
// activation rows (contiguous in the sorted-row h buffer), its 256 W2 rows
// (contiguous in the expert's W2) and both sets of scale rows; then one
// barrier, the products, and the partial stores. Two workgroups share a CU
// (about 67 KiB of LDS each at I = 256), so one's loads and products run
// under the other's stores. Each W2 row of an N tile is fetched once per
// row tile (an expert of up to 128 rows reads its W2 once; the streaming
// geometry's 16-row tiles read it about eight times).
//
// Products: 32x32x64 block-scaled MFMA, activations x weights, four waves in
// a 2 x 2 arrangement of 64 rows x 128 columns. The K order inside a
// 128-element step is the LDS-tiled geometry's: sub-step s, lane half h takes
// the 32-element block 2h + s (FP8 activation lanes: its 16-element halves
// from 16-byte chunks 2s + h and 4 + 2s + h of the step, the matrix core's
// split FP8 layout), so a lane's two scale bytes of a step are adjacent and
// op_sel s picks the byte. Accumulator element i of lane l is row
// 8 (i / 4) + 4 h + i % 4, column l % 32 of the 32 x 32 block: each store
// instruction writes two 128-byte row pieces.
#include "gemm_common.h"
#include "gemm_launch.h"

namespace moe {

typedef float v16f_s __attribute__((ext_vector_type(16)));

constexpr int SBM = 128;  // rows per tile
constexpr int SBN = 256;  // output columns per tile

// Chunk swizzle of rows of nch 16-byte chunks: chunk c of row r sits at
// c ^ key(r), so that the 16 rows one LDS read phase touches hit 16 distinct
// 16-byte bank groups (rows of 64, 128, 256 bytes).
template <int NCH>
__device__ __forceinline__ int s_key(int r) {
  static_assert(NCH == 4 || NCH == 8 || NCH == 16, "row length");
  return (r / (16 / NCH)) & (NCH - 1);
}

// One DMA instruction: this lane's 16 (4) bytes at src go to LDS at
// base + 16 * lane (4 * lane), base wave-uniform.
__device__ __forceinline__ void s_dma16(const uint8_t* src, uint8_t* base) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t*)base, 16, 0, 0);
}
__device__ __forceinline__ void s_dma4(const uint8_t* src, uint8_t* base) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t*)base, 4, 0, 0);
}

template <int FA, int KS>
struct SL {
  static constexpr int K = 128 * KS;
  static constexpr int kARow = FA == 4 ? K / 2 : K;  // activation bytes per row (e2m3: slots)
  static constexpr int kBRow = K / 2;                // weight bytes per row
  static constexpr int kACh = kARow / 16, kBCh = kBRow / 16;
  static constexpr int kSRow = K / 32;               // scale bytes per row
  static constexpr int kA = 0;
  static constexpr int kB = kA + SBM * kARow;
  static constexpr int kAS = kB + SBN * kBRow;
  static constexpr int kBS = kAS + SBM * kSRow;
  static constexpr int kIdx = kBS + SBN * kSRow;     // assignment slot of each row
  static constexpr int kBytes = kIdx + SBM * 4;
};

size_t short_lds_bytes(int fa, int I) {
  const int ks = I / 128;
  if (fa == 4) return ks == 1 ? SL<4, 1>::kBytes : SL<4, 2>::kBytes;
  return ks == 1 ? SL<0, 1>::kBytes : SL<0, 2>::kBytes;
}

bool short_k_ok(int I) { return I == 128 || I == 256; }

template <int FA, int KS>
__global__ __launch_bounds__(256, 2) void s2_short_kernel(S2Args p) {
  using L = SL<FA, KS>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int tid = threadIdx.x, lane = tid % kWave;
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int wm = w & 1, wn = w >> 1;
  const int nc0 = nt * SBN;
  const size_t wr0 = (size_t)e * p.H + nc0;  // first W2 row of the tile

  // ---- one burst of DMA: activation rows, W2 rows, scale rows ----
  {
    const uint8_t* abase = p.hq + (size_t)row0 * L::kARow;
    for (int q = tid; q < SBM * L::kACh; q += 256) {
      const int r = q / L::kACh, c = (q % L::kACh) ^ s_key<L::kACh>(q / L::kACh);
      const int rr = r < nrows ? r : 0;  // rows past the tile's end repeat row 0
      s_dma16(abase + (size_t)rr * L::kARow + 16 * c, lds + L::kA + 16 * (q - lane));
    }
    // W2 in the block layout: chunk c of row r is K piece c / 4 of r's group
    const uint8_t* bbase = p.w2 + wr0 * L::kBRow;
    for (int q = tid; q < SBN * L::kBCh; q += 256) {
      const int r = q / L::kBCh, c = (q % L::kBCh) ^ s_key<L::kBCh>(q / L::kBCh);
      s_dma16(bbase + (size_t)(r & ~15) * L::kBRow + 1024 * (c >> 2) + 64 * (r & 15) + 16 * (c & 3),
              lds + L::kB + 16 * (q - lane));
    }
    const uint8_t* asb = p.hs + (size_t)row0 * L::kSRow;
    for (int q = tid; q < SBM * L::kSRow / 4; q += 256) {
      const int r = q / (L::kSRow / 4);
      const int rr = r < nrows ? r : 0;
      s_dma4(asb + (size_t)rr * L::kSRow + 4 * (q % (L::kSRow / 4)), lds + L::kAS + 4 * (q - lane));
    }
    const uint8_t* bsb = p.w2s + wr0 * L::kSRow;
    for (int q = tid; q < SBN * L::kSRow / 4; q += 256)
      s_dma4(bsb + 4 * (size_t)q, lds + L::kBS + 4 * (q - lane));
    if (tid < SBM)
      reinterpret_cast<int*>(lds + L::kIdx)[tid] = tid < nrows ? p.sorted[row0 + tid] : 0;
  }
  wait_all_vmem();
  __syncthreads();

  // ---- products: wave (wm, wn) owns rows 64 wm .. +63, columns 128 wn .. +127 ----
  const int nmb = __builtin_amdgcn_readfirstlane(min(2, max(0, (nrows - 64 * wm + 31) / 32)));
  if (nmb == 0) return;
  const int r = lane & 31, h = lane >> 5;
  v16f_s acc[2][4];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = v16f_s{};
#pragma unroll
  for (int t = 0; t < KS; ++t) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      v8i a[2], b[4];
      uint32_t sa[2], sb[4];
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        const int ar = 64 * wm + 32 * mb + r;
        const uint8_t* row = lds + L::kA + ar * L::kARow;
        const int key = s_key<L::kACh>(ar);
        if constexpr (FA == 0) {
          const v4u lo = *reinterpret_cast<const v4u*>(row + 16 * ((8 * t + 2 * s + h) ^ key));
          const v4u hi = *reinterpret_cast<const v4u*>(row + 16 * ((8 * t + 4 + 2 * s + h) ^ key));
          a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w,
                      (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
        } else if constexpr (FA == 2) {  // the 32-byte slot of block 4t + 2h + s
          const int b = 4 * t + 2 * h + s;
          const v4u lo = *reinterpret_cast<const v4u*>(row + 16 * ((2 * b) ^ key));
          const v4u hi = *reinterpret_cast<const v4u*>(row + 16 * ((2 * b + 1) ^ key));
          a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, 0, 0};
        } else {
          const v4u lo = *reinterpret_cast<const v4u*>(row + 16 * ((4 * t + 2 * h + s) ^ key));
          a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
        }
        sa[mb] = *reinterpret_cast<const uint16_t*>(lds + L::kAS + ar * L::kSRow + 4 * t + 2 * h);
      }
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int br = 128 * wn + 32 * nb + r;
        const uint8_t* row = lds + L::kB + br * L::kBRow;
        const v4u v = *reinterpret_cast<const v4u*>(
            row + 16 * ((4 * t + 2 * h + s) ^ s_key<L::kBCh>(br)));
        b[nb] = v8i{(int)v.x, (int)v.y, (int)v.z, (int)v.w, 0, 0, 0, 0};
        sb[nb] = *reinterpret_cast<const uint16_t*>(lds + L::kBS + br * L::kSRow + 4 * t + 2 * h);
      }
#pragma unroll
      for (int mb = 0; mb < 2; ++mb) {
        if (mb < nmb) {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            if (s == 0)
              acc[mb][nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                  a[mb], b[nb], acc[mb][nb], FA, 4, 0, (int)sa[mb], 0, (int)sb[nb]);
            else
              acc[mb][nb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                  a[mb], b[nb], acc[mb][nb], FA, 4, 1, (int)sa[mb], 1, (int)sb[nb]);
          }
        }
      }
    }
  }

  // ---- unique-slot fp32 partial stores (non-temporal: read once, much
  // later, by the combine) ----
  const int* sidx = reinterpret_cast<const int*>(lds + L::kIdx);
  float* const col = p.partials + nc0 + 128 * wn + r;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    if (mb < nmb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = 64 * wm + 32 * mb + 8 * (i / 4) + 4 * h + (i % 4);
        if (row < nrows) {
          float* dst = col + (size_t)sidx[row] * p.H;
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) __builtin_nontemporal_store(acc[mb][nb][i], dst + 32 * nb);
        }
      }
    }
  }
}

int short_rows() { return SBM; }

template <int FA, int KS>
static void launch_short(const S2Args& p0, long mt, hipStream_t s) {
  S2Args q = p0;
  q.t.n_ntiles = p0.H / SBN;
  q.t.ngroup = n_group_of(q.t.n_ntiles);
  const long n = mt * q.t.n_ntiles;
  const dim3 grid((int)((n + 7) / 8 * 8));
  constexpr size_t lds = SL<FA, KS>::kBytes;
  hipLaunchKernelGGL((s2_short_kernel<FA, KS>), grid, dim3(256), lds, s, q);
}

void launch_s2_short(const S2Args& p, long mt, int fa, hipStream_t s) {
  const bool one = p.I == 128;
  if (fa == 0) {
    if (one) launch_short<0, 1>(p, mt, s);
    else launch_short<0, 2>(p, mt, s);
  } else if (fa == 2) {
    if (one) launch_short<2, 1>(p, mt, s);
    else launch_short<2, 2>(p, mt, s);
  } else {
    if (one) launch_short<4, 1>(p, mt, s);
    else launch_short<4, 2>(p, mt, s);
  }
}

}  // namespace moe
