// Pieces shared by the grouped-GEMM geometries: operand formats, the row-tile
// list, kernel arguments, and the two epilogues (SwiGLU + h quantisation for
// stage 1, unique-slot fp32 stores for stage 2).
#pragma once

#include "moe_dev.h"

namespace moe {

template <int FA>
struct ActBytes;  // bytes per 32-element block of the activation operand
template <>
struct ActBytes<0> {
  static constexpr int kBlock = 32;
};
template <>
struct ActBytes<2> {
  static constexpr int kBlock = 32;  // a 24-byte e2m3 block in a 32-byte slot
};
template <>
struct ActBytes<4> {
  static constexpr int kBlock = 16;
};

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// 16-byte load; NT marks weight streams that are read exactly once, so they
// are fetched with the non-temporal (streaming) cache policy and do not push
// the re-read activation rows out of L2.
template <bool NT>
__device__ __forceinline__ v4u ld16(const uint8_t* p) {
  const v4u* q = reinterpret_cast<const v4u*>(p);
  if constexpr (NT) return __builtin_nontemporal_load(q);
  return *q;
}

// LDS DMA written out so that the compiler neither waits for it nor orders
// LDS reads behind it: the caller's explicit vmcnt waits (loads complete in
// order) and barriers cover it.
// One 4-byte (sdma4) or 16-byte (sdma16) DMA instruction: lane i's bytes at
// base + voff go to LDS byte lds_base + 4 i (16 i); base and lds_base are
// wave-uniform.
typedef __attribute__((address_space(3))) void lds_ptr_t;

// nbytes (a multiple of 16) of contiguous global memory to LDS by 16-byte
// DMA: 1 KiB of contiguous bytes per instruction (lane = 0 .. 63).
__device__ __forceinline__ void dma_rows16(uint8_t* dst, const uint8_t* src, int nbytes, int lane) {
  for (int o = 0; o < nbytes; o += 1024)
    if (o + 16 * lane < nbytes)
      __builtin_amdgcn_global_load_lds(src + o + 16 * lane, (lds_ptr_t*)(dst + o), 16, 0, 0);
}

// Wait for every outstanding vector memory operation: after a prologue's
// DMA the compiler can no longer count the loads exactly; one explicit wait
// restores exact waits for the step loop that follows.
__device__ __forceinline__ void wait_all_vmem() { __builtin_amdgcn_s_waitcnt(0x0f70); }

// A wave-uniform pointer held in scalar registers.
__device__ __forceinline__ const uint8_t* sptr(const uint8_t* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ void sdma4(const uint8_t* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, %2"
               :
               : "s"(lds_base), "v"(voff), "s"(sptr(base))
               : "m0");
}
__device__ __forceinline__ void sdma16(const uint8_t* base, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds_base), "v"(voff), "s"(sptr(base))
               : "m0");
}

// Wait until at most N vector memory operations are outstanding.
template <int N>
__device__ __forceinline__ void tvmcnt_s() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xf00);
}

__device__ __forceinline__ uint32_t lds_addr(const uint8_t* l) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)l;
}

// Scale bytes of the step's 4J blocks starting at p (4-byte aligned); lane
// group g takes block 4j + g for product j: byte g of word j goes to byte j.
template <int J>
__device__ __forceinline__ uint32_t gather_scales(const uint8_t* p, int g) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(p);
  uint32_t r = 0;
#pragma unroll
  for (int j = 0; j < J; ++j) r |= ((w[j] >> (8 * g)) & 0xffu) << (8 * j);
  return r;
}

constexpr int kQueueInts = 16;  // ints of the persistent geometry's work queue

struct TileArgs {
  const int4* tiles;    // (expert, first sorted row, rows, 0)
  const int* ntiles;    // number of valid tiles
  int mt_bound;         // tiles the grid was sized for
  int n_ntiles;         // N tiles per expert
  int ngroup;           // consecutive N tiles per group (divides n_ntiles)
  const int4* chunks;   // row tiles launched together: 2 (256-row tiles) or 4 (-1: none)
  const int* nchunks;   // number of valid chunks
  int* queue;           // work tickets of the persistent geometry: [8] per XCD, [8] finished
};

// Host side: the largest of 8, 4, 2, 1 that divides n.
inline int n_group_of(int n) { return n % 8 == 0 ? 8 : (n % 4 == 0 ? 4 : (n % 2 == 0 ? 2 : 1)); }

// Decode the workgroup's (row tile, N tile); false if it has no work.
// The grid is n_ntiles * mt_bound workgroups. Each XCD (the dispatcher sends
// workgroup b to XCD b % 8) gets a contiguous range of logical ids; inside
// it, groups of `ngroup` consecutive ids are consecutive N tiles of one row
// tile, so the row tile's activation rows are fetched into that XCD's L2
// once and reused ngroup times while still resident, and the groups sweep
// the row tiles (experts) so concurrent workgroups spread over many experts'
// weights. Logical ids past n_ntiles * mt_bound (grid padding) map to
// nt >= n_ntiles and exit.
__device__ __forceinline__ bool tile_of_block(const TileArgs& t, int4* tile, int* nt) {
  const int lin = xcd_remap(blockIdx.x, gridDim.x);
  const int grp = lin / t.ngroup, within = lin % t.ngroup;
  const int mt = grp % t.mt_bound;
  *nt = (grp / t.mt_bound) * t.ngroup + within;
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

struct S2Args {
  const uint8_t *hq, *hs;     // [A, I*bits/8], [A, I/32] in sorted-row order
  const int32_t* sorted;
  const uint8_t *w2, *w2s;    // [NE, H, I/2], [NE, H, I/32]
  float* partials;            // [A, H] indexed by assignment
  int H, I;
  TileArgs t;
};

// Stage 2 fused with the fixed-order combine (few rows): out[t, :] is formed
// from the topk weights and the down projections of token t's slots.
struct S2CArgs {
  S2Args s;                   // partials unused
  const float* topk_w;        // [T, k_total]
  uint16_t* out;              // bf16 [T, H]
  int T, k_total;
};

// Stage-1 epilogue for one wave holding gate accumulators acc[0..NBW) and up
// accumulators acc[NBW..2NBW) of 16-column tiles hc0 + 16b: SwiGLU and
// per-32 quantisation of h. Lane (g, c16) holds rows 4g+i of columns
// hc0 + 16b + c16; a quantisation block is columns [32q, 32q+32) of the
// wave, i.e. tiles b = 2q, 2q+1 across the 16 lanes of group g.
template <int FA, int NBW>
__device__ __forceinline__ void s1_epilogue(const v4f* acc, const S1Args& p, int row0, int nrows,
                                            int hc0, int g, int c16) {
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
      } else if constexpr (FA == 2) {
        // the block's 32 codes are spread over the 16 lanes of group g (two
        // each, positions c16 and c16 + 16): each lane places its two at bits
        // 6 c16 and 96 + 6 c16 of the 192-bit block, an OR over the 16 lanes
        // joins them, and lanes 0..5 store the six words of the slot
        uint32_t wv[6];
#pragma unroll
        for (int k = 0; k < 6; ++k) wv[k] = 0;
        const int o0 = 6 * c16, o1 = 96 + 6 * c16;
#pragma unroll
        for (int k = 0; k < 6; ++k) {
          if (o0 / 32 == k) wv[k] |= c0 << (o0 % 32);
          if (o0 / 32 + 1 == k && o0 % 32 > 26) wv[k] |= c0 >> (32 - o0 % 32);
          if (o1 / 32 == k) wv[k] |= c1 << (o1 % 32);
          if (o1 / 32 + 1 == k && o1 % 32 > 26) wv[k] |= c1 >> (32 - o1 % 32);
        }
#pragma unroll
        for (int k = 0; k < 6; ++k) {
          static_for<4>([&](auto L) { wv[k] |= (uint32_t)wave_partner<decltype(L)::value>((int)wv[k]); });
        }
        if (rl < nrows && c16 < 6) {
          uint32_t v = wv[0];
#pragma unroll
          for (int k = 1; k < 6; ++k) v = c16 == k ? wv[k] : v;
          *reinterpret_cast<uint32_t*>(p.hq + r * p.I + (hc0 + 32 * q) + 4 * c16) = v;
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

// Stage-2 epilogue: fp32 partial rows to their unique assignment slots.
template <int NBW>
__device__ __forceinline__ void s2_epilogue(const v4f* acc, const S2Args& p, int row0, int nrows,
                                            int nc0, int g, int c16) {
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

}  // namespace moe
