// f2: the grouped expert GEMM under the paper's BF16 contract (Large-M CK and
// the meaning of the earlier 6.42k result; Accepted large-prefill
// configuration): activations are not quantised, FP4 weights are expanded to
// BF16, products accumulate in fp32, the intermediate h is rounded once to
// bf16 before the down projection (Historical down-consumer pilot: the down
// consumer reads the already-rounded BF16 intermediate), and stage 2 keeps
// unique-slot fp32 partials for the fixed-order combine.
//
// The paper materialised the expert shard in BF16 in HBM; here the expansion
// happens in registers at operand-read time (v_cvt_scalef32_pk_bf16_fp4:
// two FP4 codes times the block's E8M0 scale to two bf16, exact), so weights
// still stream as 4.5 bits per value.
//
// Two geometries, chosen by rows per expert. The LDS-tiled one (below; the
// weight-streaming one for few rows per expert follows it): workgroup tile
// 128 sorted rows x 256 weight rows (stage 1: 128 gate rows and the matching
// 128 up rows, so SwiGLU stays in the workgroup), K in steps of 32 (one
// scale block); 8 waves, each one 32-row weight block x all 128 rows = 4
// products of 32x32x16 bf16 per 16 K elements. Measured facts behind the shape: the
// FP4 -> bf16 conversion instruction costs about 16 clocks a wave, as much
// per step as the products, so no two waves convert the same codes (each
// wave's weight block is the one it moves by DMA); and a 128-row weight
// tile re-read the bf16 activation rows twice as often as this one. A tile
// of fewer than 128 rows (decode: a few rows per expert) skips the operand
// reads and products of its empty 32-row blocks; full tiles run a loop
// without those tests (the tests cost full tiles ~10%). The
// product is transposed (weights are the row operand), so a lane's
// accumulator holds 16 weight-row values of one activation row; stage 1's
// up waves hand their accumulators to the gate waves through LDS.
//
// Data movement: activation rows (64 bytes a step) and weight rows (16 bytes
// of FP4 a step) go global -> LDS by DMA through a ring of steps; every
// wave issues exactly 2 DMA instructions per step (rows past the tile's end
// repeat its first row; a stage past the last step reloads the last one), so
// one explicit vmcnt wait per step counts exactly. The tile's weight scale
// rows (K/32 bytes each) are staged once. Activation rows are chunk-swizzled
// (16-byte chunk c of row r at c ^ ((r >> 2) & 3)) so the operand reads do
// not collide in LDS banks.
#include "gemm_common.h"
#include "gemm_launch.h"

namespace moe {

typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int kBM = 128;              // sorted rows per tile
constexpr int kBN = 256;              // weight rows per tile
constexpr int kWaves = 8;
constexpr int kBK = 32;               // K elements per step
#ifndef MOE_BF16_RING
#define MOE_BF16_RING 4
#endif
constexpr int kRingN = MOE_BF16_RING;  // steps in the LDS ring
constexpr int kAS = kBM * kBK * 2;    // activation bytes per step (8 KiB)
constexpr int kBS = kBN * kBK / 2;    // weight bytes per step (4 KiB)
constexpr int kSlot = kAS + kBS;
constexpr int kRingBytes = kRingN * kSlot;
constexpr int kDmaPerStep = 2;        // DMA instructions per wave per step

struct BfArgs {
  const uint8_t* act;       // stage 1: x bf16 [T, K]; stage 2: h bf16 [A, K] in sorted-row order
  const int32_t* sorted;
  const uint8_t *w, *ws;    // FP4 codes [NE, N, K/2], E8M0 scales [NE, N, K/32]
  uint8_t* hout;            // stage 1: h bf16 [A, I] in sorted-row order
  float* partials;          // stage 2: [A, H] indexed by assignment
  int K, N, I, H, k_total;  // N: weight rows per expert (2I or H)
  TileArgs t;
};

// Stage 1 passes the up accumulators [128 rows][128 columns] through LDS
// after the K loop, rows padded to kExStride floats (no bank collisions).
constexpr int kExStride = 132;
constexpr size_t kExBytes = (size_t)kBM * kExStride * 4;

size_t bf16_lds_bytes(int K) {
  const size_t loop = kRingBytes + (size_t)kBN * (K / 32);
  return loop > kExBytes ? loop : kExBytes;
}

// E8M0 byte -> 2^(b - 127) as fp32 (b = 0: the subnormal 2^-127; 255: NaN).
__device__ __forceinline__ float e8m0_f32(uint32_t b) {
  uint32_t bits = b << 23;
  bits = b == 0 ? 0x00400000u : bits;
  bits = b == 255 ? 0x7fc00000u : bits;
  return __uint_as_float(bits);
}

// 8 FP4 codes (one dword, element 2i in the low nibble of byte i) times the
// scale -> 8 bf16 in K order.
__device__ __forceinline__ v8bf fp4x8_bf16(uint32_t d, float s) {
  const v2bf p0 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(d, s, 0);
  const v2bf p1 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(d, s, 1);
  const v2bf p2 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(d, s, 2);
  const v2bf p3 = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(d, s, 3);
  return v8bf{p0[0], p0[1], p1[0], p1[1], p2[0], p2[1], p3[0], p3[1]};
}

__device__ __forceinline__ uint32_t bf16_pair(float a, float b) {
  return f32_to_bf16_rne(a) | (f32_to_bf16_rne(b) << 16);
}

// The K loop over steps of 32: ALL runs the four row blocks; otherwise only
// the first nmb (their reads and products).
template <bool ALL, typename Issue>
__device__ __forceinline__ void bf16_kloop(const uint8_t* lds, const uint8_t* sc_lds, int brow,
                                           const int* arow, int nk, int kb, int h, Issue& issue,
                                           v16f* acc, int nmb) {
  uint32_t scb = sc_lds[brow * kb];  // scale byte of the next step (read one step ahead)
  for (int k = 0; k < nk; ++k) {
    // this wave's DMA of step k landed (later steps may be in flight), and
    // after the barrier every wave's has, and every wave is done with step k-1
    tvmcnt_s<(kRingN - 2) * kDmaPerStep>();
    asm volatile("s_barrier" ::: "memory");
    issue(k + kRingN - 1);  // into the slot of step k - 1
    const uint8_t* as = lds + (k % kRingN) * kSlot;
    const uint8_t* bs = as + kAS;
    const float sc = e8m0_f32(scb);
    scb = sc_lds[brow * kb + (k + 1 < nk ? k + 1 : k)];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const v8bf wa = fp4x8_bf16(*reinterpret_cast<const uint32_t*>(bs + brow * 16 + 8 * ks + 4 * h), sc);
      v8bf xb[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int r = arow[mb];
        if (ALL || mb < nmb)
          xb[mb] = *reinterpret_cast<const v8bf*>(as + r * 64 + 16 * ((2 * ks + h) ^ ((r >> 2) & 3)));
      }
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        if (ALL || mb < nmb) acc[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wa, xb[mb], acc[mb], 0, 0, 0);
    }
  }
}

// ST = 1: gate/up + SwiGLU + bf16 h; ST = 2: down -> fp32 partials.
template <int ST>
__global__ __launch_bounds__(64 * kWaves) void bf16_gemm_kernel(BfArgs p) {
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int e = __builtin_amdgcn_readfirstlane(tile.x);
  const int row0 = __builtin_amdgcn_readfirstlane(tile.y);
  const int nrows = __builtin_amdgcn_readfirstlane(tile.z);
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63, l32 = lane & 31, h = lane >> 5;
  const int kb = p.K / 32, nk = kb;
  const uint32_t ring = __builtin_amdgcn_readfirstlane(lds_addr(lds));
  uint8_t* sc_lds = lds + kRingBytes;  // [kBN][kb] weight scale bytes

  // tile weight row r -> expert weight row (stage 2: rows past H repeat row
  // H - 1; their columns are not stored)
  auto wrow = [&](int r) {
    return ST == 1 ? (r < 128 ? 128 * nt + r : p.I + 128 * nt + r - 128)
                   : (kBN * nt + r < p.H ? kBN * nt + r : p.H - 1);
  };
  const uint8_t* wbase = p.w + (size_t)e * p.N * (p.K / 2);
  const uint8_t* sbase = p.ws + (size_t)e * p.N * kb;

  // DMA sources of this lane: the activation instruction covers tile rows
  // 16 w + lane / 4, chunk slot lane % 4 (global chunk slot ^ f(row)); the
  // weight instruction covers tile row 32 w + lane (lanes < 32).
  uint32_t aoff;
  {
    const int r = 16 * w + (lane >> 2);
    const int rr = row0 + (r < nrows ? r : 0);
    const int src = ST == 1 ? p.sorted[rr] / p.k_total : rr;
    const int c = (lane & 3) ^ ((r >> 2) & 3);
    aoff = (uint32_t)src * (uint32_t)(p.K * 2) + 16 * c;
  }
  // weights in the block layout: step s (16 bytes of a row) is bytes
  // 16 (s % 4) of K piece s / 4 of the row's 16-row group
  const int wr = wrow(32 * w + l32);
  const uint32_t boff = (uint32_t)(wr & ~15) * (uint32_t)(p.K / 2) + 64 * (uint32_t)(wr & 15);
  // step s's slot; past the last step the slot gets the last step again
  auto issue = [&](int s) {
    const uint32_t slot = ring + (uint32_t)((s % kRingN) * kSlot);
    const int step = s < nk ? s : nk - 1;
    sdma16(p.act, aoff + (uint32_t)step * 64, slot + 16 * w * 64);
    if (lane < 32)
      sdma16(wbase, boff + (uint32_t)(step >> 2) * 1024 + 16 * (uint32_t)(step & 3),
             slot + kAS + 32 * w * 16);
  };

  // weight scale rows of the tile (stage 1: the 128 gate rows, then the 128
  // up rows; stage 2: the rows below H)
  {
    const int nblk = ST == 1 ? 2 : 1, rows = kBN / nblk;
    const int vrows = ST == 1 ? rows : (p.H - kBN * nt < rows ? p.H - kBN * nt : rows);
    const int bytes = vrows * kb;
    const uint32_t sl = ring + kRingBytes;
    for (int b = 0; b < nblk; ++b) {
      const uint8_t* src = sbase + (size_t)wrow(b * rows) * kb;
      for (int o = 1024 * w; o < bytes; o += 1024 * kWaves)
        if (o + 16 * lane < bytes) sdma16(src, (uint32_t)(o + 16 * lane), sl + b * rows * kb + o);
    }
  }
#pragma unroll
  for (int s = 0; s < kRingN - 1; ++s) issue(s);
  // every wave's share of the scale rows and of the first stages has landed
  // before any wave reads LDS
  tvmcnt_s<0>();
  asm volatile("s_barrier" ::: "memory");

  // operand rows of this lane: the wave's one weight block (tile rows
  // 32 w .. 32 w + 31, the rows it moves itself, so no two waves convert the
  // same codes) against all four activation blocks
  const int brow = 32 * w + l32;
  int arow[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) arow[mb] = 32 * mb + l32;
  v16f acc[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) acc[mb] = v16f{};

  // row blocks holding tile rows: a tile short of 128 rows skips the reads
  // and products of the others (they stay zero and are not stored); full
  // tiles run the loop without the per-block tests
  const int nmb = __builtin_amdgcn_readfirstlane((nrows + 31) / 32);
  if (nmb >= 4) bf16_kloop<true>(lds, sc_lds, brow, arow, nk, kb, h, issue, acc, 4);
  else bf16_kloop<false>(lds, sc_lds, brow, arow, nk, kb, h, issue, acc, nmb);
  tvmcnt_s<0>();  // the ring's last (repeated) loads

  // D: lane l, element i = weight row 8 (i / 4) + 4 h + i % 4 of the block,
  // activation row l % 32 of the block.
  if constexpr (ST == 1) {
    // waves 0-3 hold gate columns 32 w + .., waves 4-7 the matching up
    // columns: the up waves pass theirs through LDS (the ring is free now)
    asm volatile("s_barrier" ::: "memory");
    float* ex = reinterpret_cast<float*>(lds);  // [128 rows][kExStride]
    if (w >= 4) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<v4f*>(ex + arow[mb] * kExStride + 32 * (w - 4) + 8 * q + 4 * h) =
              v4f{acc[mb][4 * q], acc[mb][4 * q + 1], acc[mb][4 * q + 2], acc[mb][4 * q + 3]};
    }
    asm volatile("s_barrier" ::: "memory");
    if (w < 4) {
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int m = arow[mb];
        if (m >= nrows) continue;
        uint8_t* dst = p.hout + ((size_t)(row0 + m) * p.I + 128 * nt + 32 * w + 4 * h) * 2;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v4f U = *reinterpret_cast<const v4f*>(ex + m * kExStride + 32 * w + 8 * q + 4 * h);
          float hv[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float G = acc[mb][4 * q + j];
            hv[j] = G * U[j] / (1.0f + expf(-G));
          }
          *reinterpret_cast<uint2*>(dst + 16 * q) =
              make_uint2(bf16_pair(hv[0], hv[1]), bf16_pair(hv[2], hv[3]));
        }
      }
    }
  } else {
    if (kBN * nt + 32 * w < p.H) {  // columns past H (H % 256 == 128) are not stored
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const int m = arow[mb];
        if (m >= nrows) continue;
        const size_t a = (size_t)p.sorted[row0 + m];
        float* dst = p.partials + a * p.H + kBN * nt + 32 * w + 4 * h;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<v4f*>(dst + 8 * q) =
              v4f{acc[mb][4 * q], acc[mb][4 * q + 1], acc[mb][4 * q + 2], acc[mb][4 * q + 3]};
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Weight-streaming geometry of the BF16 contract, for few rows per expert
// (decode): a workgroup takes a tile of up to 16 sorted rows and NBW blocks
// of 16 weight rows (stage 1: NBW gate blocks and the matching up blocks),
// so every weight byte is read once, straight into registers, and expanded
// there. With KW = 2 its two waves each stream half of the K steps and wave
// 0 adds wave 1's fp32 sums (first half + second half, through LDS) before
// the epilogue: the last, partly filled round of a streaming launch is
// bound by each wave's own loads in flight, and half the K extent per wave
// halves it. 16x16x32 bf16 products with the weights as the row
// operand: lane l supplies weight row l % 16 and activation row l % 16, and
// its accumulator holds weight rows 4 (l / 16) .. +3 of activation row l % 16.
// K order: in each K step of 128, lane group g = l / 16 takes the physical
// elements [32 g, 32 g + 32) of the step, one scale block, so its 16 bytes of
// FP4 codes expand (with that block's scale) to the four 8-element pieces of
// the step's four products, and its 64 bytes of bf16 activations are the
// matching pieces. Loads run one step ahead in registers, with no branch
// around them inside the loop (the last one or two steps are peeled), so the
// compiler's waits count exactly; the tile's weight scale rows are staged in
// LDS once.
// ---------------------------------------------------------------------------
template <int NB>
struct BfStep {
  v4u a[4];   // 32 bf16 activations: K [32 g, 32 g + 32) of the step
  v4u b[NB];  // 32 FP4 codes of each weight row, same K
};

template <int ST, int NBW, int KW>
__global__ __launch_bounds__(64 * KW) void bf16_stream_kernel(BfArgs p) {
  constexpr int NB = ST == 1 ? 2 * NBW : NBW;
  int4 tile;
  int nt;
  if (!tile_of_block(p.t, &tile, &nt)) return;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int kw = KW == 2 ? __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)) : 0;
  const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
  const int kb = p.K / 32, nst = p.K / 128;
  const int s_lo = kw * (nst / KW), s_hi = s_lo + nst / KW;  // this wave's K steps
  const int c0 = nt * NBW * 16;  // first h column (stage 1) or output column (stage 2)

  // this lane's activation row (rows past the tile's end read its first
  // row; their results are not stored); loads address a wave-uniform base
  // plus a 32-bit lane offset (the host checks that the offsets fit)
  const int rr = row0 + (c16 < nrows ? c16 : 0);
  const uint32_t arow = ST == 1 ? (uint32_t)(p.sorted[rr] / p.k_total) : (uint32_t)rr;
  const uint8_t* abase = p.act;
  const uint32_t aoff = arow * (uint32_t)(p.K * 2) + 64 * g;
  // weight rows (expert-relative): stage 1 gate block n < NBW is h columns
  // c0 + 16 n .., its up block n + NBW the rows I + c0 + 16 n ..
  auto wrow = [&](int n) {
    return ST == 1 ? (n < NBW ? c0 + 16 * n : p.I + c0 + 16 * (n - NBW)) : c0 + 16 * n;
  };
  const uint8_t* wbase = p.w + (size_t)e * p.N * (p.K / 2);
  uint32_t boff[NB];  // this lane's 16 bytes of step 0 (row wrow(n) + c16, block layout)
  uint32_t so[NB];    // LDS byte of this lane's scale of step 0
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    boff[n] = (uint32_t)wrow(n) * (uint32_t)(p.K / 2) + 64 * c16 + 16 * g;  // block layout
    so[n] = (uint32_t)((16 * n + c16) * kb + g);
  }

  // (lanes of rows past the tile's end all load the tile's first row, so
  // their loads coalesce with that lane's; no branch around the loads)
  // a step's loads go out as one group ahead of the products that follow
  // them in program order (interleaved with those products by the scheduler
  // they would have only a few instructions of lead)
  // running lane offsets of the next step to load (advanced in place, so
  // no address register is also a load target)
  uint32_t ao = aoff + 256 * (uint32_t)s_lo;
  uint32_t bo[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) bo[n] = boff[n] + 1024 * (uint32_t)s_lo;
  auto load = [&](BfStep<NB>& f) {
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < 4; ++i) f.a[i] = ld16<false>(abase + ao + 16 * i);
#pragma unroll
    for (int n = 0; n < NB; ++n) f.b[n] = ld16<true>(wbase + bo[n]);  // streamed once
    ao += 256;
#pragma unroll
    for (int n = 0; n < NB; ++n) bo[n] += 1024;  // next K piece of the 16-row group
    __builtin_amdgcn_sched_barrier(0);
  };
  BfStep<NB> f0, f1;
  load(f0);
  // weight scale rows of the tile: [NB * 16 rows][kb bytes] (stage 1: the gate
  // rows, then the up rows)
  // (with KW = 2: wave 0 the first half of them, wave 1 the second)
  const uint8_t* sbase = p.ws + (size_t)e * p.N * kb;
  if constexpr (ST == 1) {
    if (KW == 1 || kw == 0) dma_rows16(lds, sbase + (size_t)wrow(0) * kb, NBW * 16 * kb, lane);
    if (KW == 1 || kw == 1)
      dma_rows16(lds + NBW * 16 * kb, sbase + (size_t)wrow(NBW) * kb, NBW * 16 * kb, lane);
  } else if constexpr (KW == 1) {
    dma_rows16(lds, sbase + (size_t)wrow(0) * kb, NB * 16 * kb, lane);
  } else {
    const int hb = NB * 8 * kb;  // bytes of half the rows
    dma_rows16(lds + kw * hb, sbase + (size_t)wrow(0) * kb + kw * hb, hb, lane);
  }
  wait_all_vmem();
  if constexpr (KW == 2) __syncthreads();  // the other wave's scale rows landed

  v4f acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f{0.f, 0.f, 0.f, 0.f};
  auto mma = [&](const BfStep<NB>& f, int s) {
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const float sc = e8m0_f32(lds[so[n] + 4 * s]);
      const uint32_t w4[4] = {f.b[n].x, f.b[n].y, f.b[n].z, f.b[n].w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const v8bf wb = fp4x8_bf16(w4[i], sc);
        const v8bf xa = __builtin_bit_cast(v8bf, f.a[i]);
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wb, xa, acc[n], 0, 0, 0);
      }
    }
  };
  // f0 holds step s on entry; steps s + 1 and s + 2 exist inside the loop
  int s = s_lo;
  for (; s + 2 < s_hi; s += 2) {
    load(f1);
    mma(f0, s);
    load(f0);
    mma(f1, s + 1);
  }
  if (s + 1 < s_hi) {
    load(f1);
    mma(f0, s);
    mma(f1, s + 1);
  } else {
    mma(f0, s);
  }
  if constexpr (KW == 2) {  // first half + second half, in wave 0
    v4f* red = reinterpret_cast<v4f*>(lds + NB * 16 * kb);
    if (kw == 1) {
#pragma unroll
      for (int n = 0; n < NB; ++n) red[n * 64 + lane] = acc[n];
    }
    __syncthreads();
    if (kw == 1) return;
#pragma unroll
    for (int n = 0; n < NB; ++n) acc[n] = acc[n] + red[n * 64 + lane];
  }

  if (c16 >= nrows) return;
  if constexpr (ST == 1) {
    // h = G * U * sigmoid(G), rounded once to bf16: 4 consecutive h columns
    uint8_t* dst = p.hout + ((size_t)(row0 + c16) * p.I + c0 + 4 * g) * 2;
#pragma unroll
    for (int n = 0; n < NBW; ++n) {
      float hv[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float G = acc[n][j], U = acc[n + NBW][j];
        hv[j] = G * U / (1.0f + expf(-G));
      }
      *reinterpret_cast<uint2*>(dst + 32 * n) =
          make_uint2(bf16_pair(hv[0], hv[1]), bf16_pair(hv[2], hv[3]));
    }
  } else {
    float* dst = p.partials + (size_t)p.sorted[row0 + c16] * p.H + c0 + 4 * g;
#pragma unroll
    for (int n = 0; n < NB; ++n) *reinterpret_cast<v4f*>(dst + 16 * n) = acc[n];
  }
}

int bf16_rows() { return kBM; }

template <int ST>
static void launch_bf(const BfArgs& p0, long mt, int n_ntiles, hipStream_t s) {
  BfArgs p = p0;
  p.t.n_ntiles = n_ntiles;
  p.t.ngroup = n_group_of(n_ntiles);
  const long n = mt * n_ntiles;
  hipLaunchKernelGGL((bf16_gemm_kernel<ST>), dim3((int)((n + 7) / 8 * 8)), dim3(64 * kWaves),
                     bf16_lds_bytes(p.K), s, p);
}

void launch_s1_bf16(const S1Args& a, long mt, hipStream_t s) {
  BfArgs p{a.xq, a.sorted, a.w13, a.w13s, a.hq, nullptr, a.H, 2 * a.I, a.I, a.H, a.k_total, a.t};
  launch_bf<1>(p, mt, a.I / 128, s);
}

void launch_s2_bf16(const S2Args& a, long mt, hipStream_t s) {
  BfArgs p{a.hq, a.sorted, a.w2, a.w2s, nullptr, a.partials, a.I, a.H, a.I, a.H, 1, a.t};
  launch_bf<2>(p, mt, (a.H + kBN - 1) / kBN, s);
}

// Streaming geometry: 32 h columns per wave in stage 1 (2 gate + 2 up
// blocks), 64 output columns in stage 2; tiles of up to 16 rows.
constexpr int kBfS1 = 2, kBfS2 = 4;

int bf16_stream_rows() { return 16; }

// K split over two waves when each gets at least two steps of 128 and the
// same number of them.
static bool bf_split(int K) { return K % 256 == 0 && K >= 512; }

void launch_s1_bf16_stream(const S1Args& a, long mt, hipStream_t s) {
  BfArgs p{a.xq, a.sorted, a.w13, a.w13s, a.hq, nullptr, a.H, 2 * a.I, a.I, a.H, a.k_total, a.t};
  const int ntl = a.I / (kBfS1 * 16);
  p.t.n_ntiles = ntl;
  p.t.ngroup = n_group_of(ntl);
  const long n = mt * ntl;
  const dim3 grid((int)((n + 7) / 8 * 8));
  const size_t lds = (size_t)2 * kBfS1 * 16 * (a.H / 32);
  if (bf_split(a.H))
    hipLaunchKernelGGL((bf16_stream_kernel<1, kBfS1, 2>), grid, dim3(128),
                       lds + (size_t)2 * kBfS1 * 64 * 16, s, p);
  else
    hipLaunchKernelGGL((bf16_stream_kernel<1, kBfS1, 1>), grid, dim3(64), lds, s, p);
}

void launch_s2_bf16_stream(const S2Args& a, long mt, hipStream_t s) {
  BfArgs p{a.hq, a.sorted, a.w2, a.w2s, nullptr, a.partials, a.I, a.H, a.I, a.H, 1, a.t};
  const int ntl = a.H / (kBfS2 * 16);
  p.t.n_ntiles = ntl;
  p.t.ngroup = n_group_of(ntl);
  const long n = mt * ntl;
  const dim3 grid((int)((n + 7) / 8 * 8));
  const size_t lds = (size_t)kBfS2 * 16 * (a.I / 32);
  if (bf_split(a.I))
    hipLaunchKernelGGL((bf16_stream_kernel<2, kBfS2, 2>), grid, dim3(128),
                       lds + (size_t)kBfS2 * 64 * 16, s, p);
  else
    hipLaunchKernelGGL((bf16_stream_kernel<2, kBfS2, 1>), grid, dim3(64), lds, s, p);
}

}  // namespace moe
