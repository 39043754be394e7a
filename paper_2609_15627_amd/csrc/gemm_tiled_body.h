// The LDS-tiled kernels' body, compiled once per row-tile size: the file
// that includes it defines MOE_TILED_ROWS (128 or 256) and a namespace
// around it. Included only by gemm_tiled.hip.

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lds_ptr_t;

constexpr int TBM = MOE_TILED_ROWS;  // sorted rows per tile (128 or 256)
static_assert(TBM == 128 || TBM == 256, "row tile of 128 or 256");
constexpr int kMB = TBM / 64;  // 32-row blocks per wave half
// Workgroups per CU: 256-row tiles fill a CU's LDS; two 128-row workgroups
// share it, so one's epilogue and hand-over run under the other's products.
constexpr int kWGperCU = TBM == 128 ? 2 : 1;
// Row tiles per chunk (launched together so that they share their expert's
// weight rows in one XCD's L2): a chunk covers up to 512 rows either way.
constexpr int kChunk = TBM == 128 ? 4 : 2;
constexpr int TBN = 256;       // weight rows per tile
constexpr int kSG = 4;         // K steps per scale group (16 scale bytes per row)

template <int FA>
struct TL {
  // activation bytes per row per K step (e2m3: four 32-byte slots, like e4m3)
  static constexpr int kARow = FA == 4 ? 64 : 128;
  static constexpr int kB = TBM * kARow;             // weight rows follow the activation rows
  static constexpr int kStage = kB + TBN * 64;
  // K-step stages in the LDS ring. 256-row tiles: 3 of 48 KiB with FP8
  // activations, 4 of 32 KiB with FP4 ones (one more step of DMA lead in the
  // same LDS, and the ring slot of step 4q + J is J). 128-row tiles: 2, so
  // that two workgroups fit a CU.
  static constexpr int kNS = TBM == 128 ? 2 : (FA == 4 ? 4 : 3);
  static constexpr int kS = kNS * kStage;            // two scale buffers follow the stages
  static constexpr int kSBuf = (TBM + TBN) * 16;
  static constexpr int kLoop = kS + 2 * kSBuf;
  static constexpr int kAInstr = TBM * kARow / 4096;  // DMA instructions per wave per step
  static constexpr int kBInstr = TBN * 64 / 4096;
  static constexpr int kStageLoads = kAInstr + kBInstr;
  static constexpr int kScaleLoads = 2;
};

template <int FA>
constexpr int t_lds_s1() {
  return TL<FA>::kLoop;
}

// 16-byte-per-lane DMA global -> LDS (global `base` + 32-bit lane offset
// `voff`, LDS destination `l` for lane 0, 1 KiB per instruction), written
// out so that the compiler neither orders LDS accesses behind it nor waits
// for it: its completion is covered only by the explicit vmcnt waits of the
// K loop, each followed by a workgroup barrier, before any wave reads the
// bytes it wrote.
__device__ __forceinline__ void tdma16_x(const uint8_t* base, uint32_t voff, const uint8_t* l) {
  const uint32_t m = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)l;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(m), "v"(voff), "s"(base)
               : "m0");
}

template <int N>
__device__ __forceinline__ void tvmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xf00);
}
__device__ __forceinline__ void tlgkm0() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// Workgroup barrier without a memory fence: __syncthreads() would also wait
// for every outstanding DMA (the younger stages too). The explicit waits
// before it cover this wave's own loads; the asm memory clobber keeps LDS
// accesses on their side of it.
__device__ __forceinline__ void tbarrier() { asm volatile("s_barrier" ::: "memory"); }

// DMA sources of one wave at K step 0: workgroup-uniform bases plus 32-bit
// per-lane byte offsets (so the loads use the scalar-base addressing form).
template <int FA>
struct TSrc {
  const uint8_t *abase, *bbase, *asbase, *bsbase;
  uint32_t a[TL<FA>::kAInstr];  // activation row + chunk of each instruction
  uint32_t b[TL<FA>::kBInstr];  // weight row + chunk of each instruction
  uint32_t as;                  // activation scale row 64 w + lane
  uint32_t bs;                  // weight scale row 64 w + lane
};

// Tile row and logical 16-byte chunk fetched by lane `lane` of activation
// DMA instruction ci (1 KiB of the chunk-swizzled activation rows).
template <int FA>
__device__ __forceinline__ void t_aslot(int ci, int lane, int* row, int* chunk) {
  if constexpr (FA != 4) {
    *row = 8 * ci + lane / 8;
    *chunk = (lane % 8) ^ ((*row >> 1) & 7);
  } else {
    *row = 16 * ci + lane / 4;
    *chunk = (lane % 4) ^ ((*row >> 2) & 3);
  }
}
__device__ __forceinline__ void t_bslot(int ci, int lane, int* row, int* chunk) {
  *row = 16 * ci + lane / 4;
  *chunk = (lane % 4) ^ ((*row >> 2) & 3);
}

// Activation rows a wave moves by DMA: LDS positions t_arow0(w) ..
// + TBM / 4 - 1, inside the TBM / 2 positions the wave multiplies
// ((TBM / 2) (w & 1) ..), which hold its wave half's row blocks, so a wave
// without rows to multiply (a tile of at most 32 rows, w odd) moves no
// activation data either. Its DMA instruction i fills activation tile chunk
// t_aci.
__device__ __forceinline__ int t_arow0(int w) { return (TBM / 2) * (w & 1) + (TBM / 4) * (w >> 1); }

// DMA of a wave's activation scale pieces (rows t_arow0(w) ..): one per lane,
// 64 rows; with 128-row tiles a wave moves 32 rows, so the upper lanes sit
// the instruction out (never all lanes, so the load count stays uniform).
__device__ __forceinline__ void tdma_ascale(const uint8_t* base, uint32_t voff, const uint8_t* l) {
  if constexpr (TBM == 128) {
    // the base is uniform; say so (sptr, zero-extending both halves) before
    // the branch, whose inside the compiler would otherwise treat as divergent
    const uint8_t* bu = sptr(base);
    if ((threadIdx.x & 63) < 32) tdma16_x(bu, voff, l);
  } else {
    tdma16_x(base, voff, l);
  }
}
template <int FA>
__device__ __forceinline__ int t_aci(int w, int i) {
  return t_arow0(w) * TL<FA>::kARow / 1024 + i;
}

// DMA of stage k; AON: this wave moves activation rows (else only weights).
template <int FA, bool AON>
__device__ __forceinline__ void t_issue_stage(uint8_t* lds, const TSrc<FA>& S, int w, int k) {
  using L = TL<FA>;
  uint8_t* st = lds + (k % L::kNS) * L::kStage;
  const size_t ka = (size_t)k * L::kARow, kb = (size_t)k * 1024;  // K piece k of the weight groups
  if constexpr (AON) {
#pragma unroll
    for (int i = 0; i < L::kAInstr; ++i)
      tdma16_x(S.abase + ka, S.a[i], st + 1024 * t_aci<FA>(w, i));
  }
#pragma unroll
  for (int i = 0; i < L::kBInstr; ++i)
    tdma16_x(S.bbase + kb, S.b[i], st + L::kB + 1024 * (L::kBInstr * w + i));
}

template <int FA, bool AON>
__device__ __forceinline__ void t_issue_scales(uint8_t* lds, const TSrc<FA>& S, int w, int q) {
  using L = TL<FA>;
  uint8_t* sb = lds + L::kS + (q & 1) * L::kSBuf;
  if constexpr (AON) tdma_ascale(S.asbase + 16 * q, S.as, sb + 16 * t_arow0(w));
  tdma16_x(S.bsbase + 16 * q, S.bs, sb + TBM * 16 + 1024 * w);
}

// Per-lane LDS byte offsets of the operand reads (block 0; block b adds a
// compile-time offset).
struct TLane {
  uint32_t a0[2], a1[2];  // activation piece(s) of sub-step s (FP8: bytes 0-15, 16-31)
  uint32_t b[2];          // weight piece of sub-step s
  uint32_t as, bs;        // this lane's scale byte pair of block 0 in a scale buffer
};

// Weight tile row of block nb relative to the wave's first weight row:
// stage 1 pairs gate blocks (rows 64 wn + 32 nb) with the up blocks of the
// same h columns (rows 128 + 64 wn + 32 nb); stage 2 takes 4 consecutive.
template <int ST>
__device__ __forceinline__ constexpr int t_nrow(int nb) {
  return ST == 1 ? (nb < 2 ? 32 * nb : 128 + 32 * (nb - 2)) : 32 * nb;
}

struct TOps {
  v8i a[4];
  v8i b[4];
};

// Operand reads of sub-step S for the wave's first NMB row blocks (none at
// all when the wave has no rows).
template <int FA, int ST, int S, int NMB>
__device__ __forceinline__ void t_read_ops(const uint8_t* st, const TLane& L, TOps& o) {
  using Lo = TL<FA>;
  if constexpr (NMB > 0) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const v4u v = *reinterpret_cast<const v4u*>(st + L.b[S] + t_nrow<ST>(nb) * 64);
      o.b[nb] = v8i{(int)v.x, (int)v.y, (int)v.z, (int)v.w, 0, 0, 0, 0};
    }
  }
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb) {
    const v4u lo = *reinterpret_cast<const v4u*>(st + L.a0[S] + mb * 32 * Lo::kARow);
    if constexpr (FA == 0) {
      const v4u hi = *reinterpret_cast<const v4u*>(st + L.a1[S] + mb * 32 * Lo::kARow);
      o.a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w,
                    (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
    } else if constexpr (FA == 2) {
      const v4u hi = *reinterpret_cast<const v4u*>(st + L.a1[S] + mb * 32 * Lo::kARow);
      o.a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, 0, 0};
    } else {
      o.a[mb] = v8i{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, 0, 0, 0, 0};
    }
  }
}

// Scale byte pairs of step j of a group: byte s of the result is the scale
// of sub-step s for this lane.
template <int ST, int NMB>
__device__ __forceinline__ void t_read_scales(const uint8_t* sbuf, const TLane& L, int j,
                                              uint32_t* sa, uint32_t* sb) {
  if constexpr (NMB > 0) {
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
      sa[mb] = *reinterpret_cast<const uint16_t*>(sbuf + L.as + mb * 32 * 16 + 4 * j);
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      sb[nb] = *reinterpret_cast<const uint16_t*>(sbuf + L.bs + t_nrow<ST>(nb) * 16 + 4 * j);
  }
}

// One 32x32x64 product of activation operand a (format FA) and weight
// operand b (FP4), op_sel OPS picking the sub-step's scale byte. Stage 2
// computes activations x weights (accumulator rows = activation rows);
// stage 1 the transpose, weights x activations, so that a lane's
// accumulator holds 16 h values of one token (rows = weight rows).
template <int FA, int ST, int OPS>
__device__ __forceinline__ v16f t_mfma(const v8i& a, const v8i& b, const v16f& c, uint32_t sa,
                                       uint32_t sb) {
  if constexpr (ST == 1)
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(b, a, c, 4, FA, OPS, (int)sb, OPS,
                                                           (int)sa);
  else
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, FA, 4, OPS, (int)sa, OPS,
                                                           (int)sb);
}

// Products of sub-step S for blocks (mb, nb) with mb in [MB0, MB1).
template <int FA, int ST, int S, int MB0, int MB1>
__device__ __forceinline__ void t_mma(v16f (*acc)[4], const TOps& o, const uint32_t* sa,
                                      const uint32_t* sb) {
#pragma unroll
  for (int mb = MB0; mb < MB1; ++mb)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      acc[mb][nb] = t_mfma<FA, ST, S>(o.a[mb], o.b[nb], acc[mb][nb], sa[mb], sb[nb]);
}

// Interleave hint: M single products, each followed by D LDS reads and V
// DMA instructions (what is left over is scheduled freely).
template <int M, int D, int V>
__device__ __forceinline__ void t_sched() {
#pragma unroll
  for (int i = 0; i < M; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (D > 0) __builtin_amdgcn_sched_group_barrier(0x100, D, 0);
    if constexpr (V > 0) __builtin_amdgcn_sched_group_barrier(0x020, V, 0);
  }
}

constexpr int t_ceil(int a, int b) { return b > 0 ? (a + b - 1) / b : 0; }
constexpr int t_min(int a, int b) { return a < b ? a : b; }

// Interleave hint for the second half of a step: the LDS reads go first (the
// DMA writes that follow them in program order may not pass them), R per
// product, then the DMA instructions spread over the remaining products.
template <int M, int D, int V>
__device__ __forceinline__ void t_sched_b() {
  constexpr int R = M > 0 ? (t_ceil(D, M) > 4 ? t_ceil(D, M) : 4) : 0;
  constexpr int M1 = t_min(M, t_ceil(D, R));
  constexpr int M2 = M - M1;
  t_sched<M1, R, 0>();
  t_sched<M2, 0, t_ceil(V, M2)>();
}

// One K step k = 4q + J (J compile-time) of a wave that owns NMB row blocks
// (0..4, uniform per wave; a wave without rows still moves data and takes
// part in the barriers). Stage k lives in ring slot k % NS, scale group q in
// buffer q % 2. X holds the step's sub-step-0 operands and sa/sb its scales
// on entry; on exit they hold those of step k + 1.
//   1. sub-step-0 products on X while sub-step-1 operands are read into Y;
//   2. one row of sub-step-1 products, then: this wave's loads of stage k + 1
//      landed, workgroup barrier (every wave has left stage k, stage k + 1 is
//      visible);
//   3. reads of step k + 1's operands and scales, then the DMA of stage
//      k + NS into slot k % NS (at J == 0 also scale group q + 1, into the buffer
//      group q - 1 used), interleaved with the remaining sub-step-1 products.
// LAST marks the final group (k = nk - 4 + J), where the ring drains.
#ifndef MOE_TILED_PRE
#define MOE_TILED_PRE 4
#endif
// Sub-step-1 products issued before the barrier (they cover its wait).
constexpr int kPre = MOE_TILED_PRE;

template <int FA, int ST, int NMB, int J, bool LAST>
__device__ __forceinline__ void t_step(uint8_t* lds, const TSrc<FA>& src, const TLane& L,
                                       int k, int w, v16f (*acc)[4], TOps& X, TOps& Y,
                                       uint32_t* sa, uint32_t* sb) {
  using Lo = TL<FA>;
  constexpr int NS = Lo::kNS;
  constexpr bool kNext = !LAST || J < 3;  // step k + 1 exists
  constexpr bool kIssue = !LAST || J + NS < 4;  // stage k + NS exists
  constexpr bool kScales = !LAST && J == 0;  // scale group q + 1 exists
  // Loads this wave issued after stage k + 1's: stages k + 2 .. k + NS - 1
  // (those that exist in the last group) and the scale group issued at the
  // group's first step when that came after stage k + 1 (1 <= J <= NS - 2).
  constexpr int kOutStages = !LAST ? NS - 2 : (NS - 2 < 2 - J ? NS - 2 : 2 - J);
  constexpr int kOutScales = (!LAST && J >= 1 && J <= NS - 2) ? 1 : 0;
  constexpr int kAPieces = FA == 4 ? 1 : 2;
  constexpr int kOpReads = NMB > 0 ? 4 + kAPieces * NMB : 0;
  constexpr int kScaleReads = NMB > 0 ? 4 + NMB : 0;
  constexpr int kPreN = 4 * NMB < kPre ? 4 * NMB : kPre;  // sub-step-1 products before the barrier
  constexpr bool kAOn = NMB > 0;  // this wave moves activation rows
  constexpr int kStageLoads = (kAOn ? Lo::kAInstr : 0) + Lo::kBInstr;
  constexpr int kScaleLoads = kAOn ? 2 : 1;
  // ring slot of step k (compile-time with 4 stages: k = 4q + J)
  const int slot = NS == 4 ? J : k % NS;
  const uint8_t* st = lds + slot * Lo::kStage;

  __builtin_amdgcn_sched_barrier(0);
  t_read_ops<FA, ST, 1, NMB>(st, L, Y);
  t_mma<FA, ST, 0, 0, NMB>(acc, X, sa, sb);
  t_sched<4 * NMB, t_ceil(kOpReads, 4 * NMB), 0>();
  __builtin_amdgcn_sched_barrier(0);
  tlgkm0();
#pragma unroll
  for (int f = 0; f < kPreN; ++f)
    acc[f / 4][f % 4] = t_mfma<FA, ST, 1>(Y.a[f / 4], Y.b[f % 4], acc[f / 4][f % 4], sa[f / 4], sb[f % 4]);
  if constexpr (kNext) tvmcnt<kOutStages * kStageLoads + kOutScales * kScaleLoads>();
  tbarrier();
  __builtin_amdgcn_sched_barrier(0);
  // Second half, in explicit order: after each remaining sub-step-1 product
  // its share of the next step's LDS reads (front-loaded, two per product)
  // and of the DMA instructions (spread over all products).
  uint32_t ra[4], rb[4];
  v4u blo[4], alo[4], ahi[4];
  const int k1 = k + 1;
  const uint8_t* sbuf1 = lds + Lo::kS + ((k1 / kSG) & 1) * Lo::kSBuf;
  const uint8_t* st1 = lds + (NS == 4 ? (J + 1) % 4 : k1 % NS) * Lo::kStage;
  uint8_t* dst = lds + slot * Lo::kStage;  // stage k + NS reuses the slot of step k
  const size_t ka = (size_t)(k + NS) * Lo::kARow, kb = (size_t)(k + NS) * 1024;
  uint8_t* sdst = lds + Lo::kS + ((k / kSG + 1) & 1) * Lo::kSBuf;
  constexpr int kR = kNext ? kOpReads + kScaleReads : 0;
  constexpr int kDS = kScales ? kScaleLoads : 0;
  constexpr int kD = kIssue ? kStageLoads + kDS : 0;
  constexpr int kDA = kAOn ? Lo::kAInstr : 0;
  constexpr int kM = 4 * NMB - kPreN;
  constexpr int kRPer = kM > 0 ? (t_ceil(kR, kM) > 2 ? t_ceil(kR, kM) : 2) : kR;
  auto read_one = [&](int r) {
    if (r < NMB) {
      ra[r] = *reinterpret_cast<const uint16_t*>(sbuf1 + L.as + r * 32 * 16 + 4 * ((J + 1) % kSG));
    } else if (r < NMB + 4) {
      const int nb = r - NMB;
      rb[nb] = *reinterpret_cast<const uint16_t*>(sbuf1 + L.bs + t_nrow<ST>(nb) * 16 + 4 * ((J + 1) % kSG));
    } else if (r < NMB + 8) {
      const int nb = r - NMB - 4;
      blo[nb] = *reinterpret_cast<const v4u*>(st1 + L.b[0] + t_nrow<ST>(nb) * 64);
    } else {
      const int q = r - NMB - 8, mb = q / kAPieces;
      if (q % kAPieces == 0) alo[mb] = *reinterpret_cast<const v4u*>(st1 + L.a0[0] + mb * 32 * Lo::kARow);
      else ahi[mb] = *reinterpret_cast<const v4u*>(st1 + L.a1[0] + mb * 32 * Lo::kARow);
    }
  };
  auto dma_one = [&](int d) {
    if (d < kDS) {
      const int q1 = k / kSG + 1;
      if (kAOn && d == 0) tdma_ascale(src.asbase + 16 * q1, src.as, sdst + 16 * t_arow0(w));
      else tdma16_x(src.bsbase + 16 * q1, src.bs, sdst + TBM * 16 + 1024 * w);
    } else if (d - kDS < kDA) {
      const int i = d - kDS;
      tdma16_x(src.abase + ka, src.a[i], dst + 1024 * t_aci<FA>(w, i));
    } else {
      const int i = d - kDS - kDA;
      tdma16_x(src.bbase + kb, src.b[i], dst + Lo::kB + 1024 * (Lo::kBInstr * w + i));
    }
  };
#pragma unroll
  for (int i = 0; i < (kM > 0 ? kM : 1); ++i) {
    if (kM > 0) {
      const int f = kPreN + i;  // flat product index (row-major) of sub-step 1
      acc[f / 4][f % 4] = t_mfma<FA, ST, 1>(Y.a[f / 4], Y.b[f % 4], acc[f / 4][f % 4], sa[f / 4], sb[f % 4]);
    }
    const int r0 = kM > 0 ? t_min(kR, i * kRPer) : 0, r1 = kM > 0 ? t_min(kR, (i + 1) * kRPer) : kR;
#pragma unroll
    for (int r = r0; r < r1; ++r) read_one(r);
    const int d0 = kM > 0 ? i * kD / kM : 0, d1 = kM > 0 ? (i + 1) * kD / kM : kD;
#pragma unroll
    for (int d = d0; d < d1; ++d) dma_one(d);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (kNext && NMB > 0) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb)
      X.b[nb] = v8i{(int)blo[nb].x, (int)blo[nb].y, (int)blo[nb].z, (int)blo[nb].w, 0, 0, 0, 0};
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
      if constexpr (FA == 0)
        X.a[mb] = v8i{(int)alo[mb].x, (int)alo[mb].y, (int)alo[mb].z, (int)alo[mb].w,
                      (int)ahi[mb].x, (int)ahi[mb].y, (int)ahi[mb].z, (int)ahi[mb].w};
      else if constexpr (FA == 2)
        X.a[mb] = v8i{(int)alo[mb].x, (int)alo[mb].y, (int)alo[mb].z, (int)alo[mb].w,
                      (int)ahi[mb].x, (int)ahi[mb].y, 0, 0};
      else
        X.a[mb] = v8i{(int)alo[mb].x, (int)alo[mb].y, (int)alo[mb].z, (int)alo[mb].w, 0, 0, 0, 0};
    }
  }
  if constexpr (kNext) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sa[i] = ra[i];
      sb[i] = rb[i];
    }
  }
}

template <int FA, int ST, int NMB, bool LAST>
__device__ __forceinline__ void t_group(uint8_t* lds, const TSrc<FA>& src, const TLane& L, int q,
                                        int w, v16f (*acc)[4], TOps& X, TOps& Y, uint32_t* sa,
                                        uint32_t* sb) {
  t_step<FA, ST, NMB, 0, LAST>(lds, src, L, 4 * q + 0, w, acc, X, Y, sa, sb);
  t_step<FA, ST, NMB, 1, LAST>(lds, src, L, 4 * q + 1, w, acc, X, Y, sa, sb);
  t_step<FA, ST, NMB, 2, LAST>(lds, src, L, 4 * q + 2, w, acc, X, Y, sa, sb);
  t_step<FA, ST, NMB, 3, LAST>(lds, src, L, 4 * q + 3, w, acc, X, Y, sa, sb);
}

// The K loop shared by both stages: nk = K / 128 steps, a multiple of 4.
// Scale group 0 and stages 0 .. NS-1 are in flight before the first step.
template <int FA, bool AON>
__device__ __forceinline__ void t_prologue_n(uint8_t* lds, const TSrc<FA>& src, int w) {
  t_issue_scales<FA, AON>(lds, src, w, 0);
#pragma unroll
  for (int s = 0; s < TL<FA>::kNS; ++s) t_issue_stage<FA, AON>(lds, src, w, s);
}

// nmb: the row blocks this wave will multiply in the tile.
template <int FA>
__device__ __forceinline__ void t_prologue(uint8_t* lds, const TSrc<FA>& src, int w, int nmb) {
  if (nmb > 0) t_prologue_n<FA, true>(lds, src, w);
  else t_prologue_n<FA, false>(lds, src, w);
}

// PRO: issue the prologue here (else the caller issued it earlier; loads or
// stores issued after it only make the first wait stricter, since loads
// complete in order).
template <int FA, int ST, int NMB, bool PRO>
__device__ __forceinline__ void t_kloop_n(uint8_t* lds, const TSrc<FA>& src, const TLane& L, int nk,
                                       int w, v16f (*acc)[4]) {
  using Lo = TL<FA>;
  if constexpr (PRO) t_prologue_n<FA, (NMB > 0)>(lds, src, w);
  tvmcnt<(Lo::kNS - 1) * ((NMB > 0 ? Lo::kAInstr : 0) + Lo::kBInstr)>();
  tbarrier();

  TOps X, Y;
  uint32_t sa[4], sb[4];
  t_read_ops<FA, ST, 0, NMB>(lds, L, X);
  t_read_scales<ST, NMB>(lds + Lo::kS, L, 0, sa, sb);
  const int nq = nk / kSG;
  for (int q = 0; q < nq - 1; ++q) t_group<FA, ST, NMB, false>(lds, src, L, q, w, acc, X, Y, sa, sb);
  t_group<FA, ST, NMB, true>(lds, src, L, nq - 1, w, acc, X, Y, sa, sb);
}

// nmb: row blocks of 32 this wave owns in the tile (wave-uniform).
template <int FA, int ST, bool PRO>
__device__ __forceinline__ void t_kloop(uint8_t* lds, const TSrc<FA>& src, const TLane& L, int nk,
                                        int w, int nmb, v16f (*acc)[4]) {
  switch (nmb) {
    case 4: if constexpr (kMB == 4) t_kloop_n<FA, ST, 4, PRO>(lds, src, L, nk, w, acc); break;
    case 3: if constexpr (kMB == 4) t_kloop_n<FA, ST, 3, PRO>(lds, src, L, nk, w, acc); break;
    case 2: t_kloop_n<FA, ST, 2, PRO>(lds, src, L, nk, w, acc); break;
    case 1: t_kloop_n<FA, ST, 1, PRO>(lds, src, L, nk, w, acc); break;
    default: t_kloop_n<FA, ST, 0, PRO>(lds, src, L, nk, w, acc); break;
  }
}

// Work distribution (persistent kernels, kWGperCU workgroups per CU). A work
// item is one row tile x one N tile. A chunk is kChunk row tiles (of one
// expert where it has that many) x all N tiles, row tile fastest; the chunk's items run
// at about the same time on one XCD and share their activation rows and
// weight rows in that XCD's L2. Chunk c belongs to queue c % 8; workgroup b
// takes tickets from queue b % 8 (the dispatcher places workgroup b on XCD
// b % 8) and, once that queue is empty, from the others. Which workgroup
// computes an item does not change any result: every item writes its own
// outputs.
__device__ __forceinline__ int t_queue_items(int nch, int x, int per) {
  return (nch > x ? (nch - x + 7) / 8 : 0) * per;
}

// Next item as 8 * (index within its queue) + queue, or -1 when none is left.
__device__ __forceinline__ int t_grab(const TileArgs& t, int nch, int per) {
  const int x = blockIdx.x & 7;
  for (int v = 0; v < 8; ++v) {
    const int q = (x + v) & 7;
    const int n = t_queue_items(nch, q, per);
    if (n == 0) continue;
    const int i = __hip_atomic_fetch_add(t.queue + q, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (i >= 0 && i < n) return 8 * i + q;
  }
  return -1;
}

// Row tile index of an item (-1 for an empty place of a chunk) and its N tile.
__device__ __forceinline__ int t_item_tile(const TileArgs& t, int item, int per, int* nt) {
  const int q = item & 7, i = item >> 3;
  const int chunk = 8 * (i / per) + q, r = i % per;
  *nt = r / kChunk;
  const int4 c = t.chunks[chunk];
  const int j = r % kChunk;
  return j == 0 ? c.x : (j == 1 ? c.y : (j == 2 ? c.z : c.w));
}

// Called once per workgroup after its last item: the last one to finish
// returns the queue to zero for the next launch (all others have taken
// their final ticket by then).
__device__ __forceinline__ void t_finish(const TileArgs& t) {
  const int done = __hip_atomic_fetch_add(t.queue + 8, 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
  if (done == (int)gridDim.x - 1) {
    for (int q = 0; q <= 8; ++q)
      __hip_atomic_store(t.queue + q, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Barrier for the persistent loop: this wave's LDS accesses are complete,
// then all waves meet (no wait for global memory).
__device__ __forceinline__ void t_sync_lds() {
  tlgkm0();
  tbarrier();
}

// Next work item of the workgroup (false: none left). Thread 0 takes the
// tickets, skipping the empty places of chunks, and hands the item's row
// tile index and N tile to the other waves through the LDS words slot[0..1],
// which nothing else writes between the two barriers.
__device__ __forceinline__ bool t_next(const TileArgs& t, int* slot, int nch, int per,
                                       int4* tile, int* nt) {
  t_sync_lds();  // every wave has read the previous ticket
  if (threadIdx.x == 0) {
    int ti = -1, ntt = 0;
    for (;;) {
      const int it = t_grab(t, nch, per);
      if (it < 0) break;
      ti = t_item_tile(t, it, per, &ntt);
      if (ti >= 0) break;
    }
    slot[0] = ti;
    slot[1] = ntt;
  }
  t_sync_lds();
  const int ti = __builtin_amdgcn_readfirstlane(slot[0]);  // uniform: scalar tile loads
  if (ti < 0) return false;
  *nt = __builtin_amdgcn_readfirstlane(slot[1]);
  *tile = t.tiles[ti];
  return true;
}

// Tile row held at LDS row position pos: positions (TBM / 2) wm + 32 mb + r
// hold row 32 (2 mb + wm) + r, wave half wm's block mb (row blocks alternate
// between the wave halves).
__device__ __forceinline__ int t_row(int pos) {
  return 64 * ((pos >> 5) & (kMB - 1)) + 32 * (pos / (TBM / 2)) + (pos & 31);
}
// Row blocks of 32 that wave half wm multiplies in a tile of nrows rows
// (blocks wm, wm + 2, .. that hold rows; wave-uniform).
__device__ __forceinline__ int t_nmb(int nrows, int wm) {
  const int nb = (nrows + 31) / 32;  // 32-row blocks holding rows
  return __builtin_amdgcn_readfirstlane(min(kMB, max(0, (nb + 1 - wm) / 2)));
}

template <int FA, int ST>
__device__ __forceinline__ TLane t_lane(int w, int lane) {
  const int r = lane & 31, h = lane >> 5;
  const int wm = w & 1, wn = w >> 1;
  TLane L;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int ar = (TBM / 2) * wm + r;
    if constexpr (FA == 0) {
      // bytes 0-15: physical K [32 s + 16 h, +16); bytes 16-31: [64 + 32 s + 16 h, +16)
      const int sw = (ar >> 1) & 7;
      L.a0[s] = ar * 128 + 16 * ((2 * s + h) ^ sw);
      L.a1[s] = ar * 128 + 16 * ((4 + 2 * s + h) ^ sw);
    } else if constexpr (FA == 2) {
      // the 32-byte slot of block 2h + s: chunks 2(2h + s) and 2(2h + s) + 1
      const int sw = (ar >> 1) & 7, b = 2 * h + s;
      L.a0[s] = ar * 128 + 16 * ((2 * b) ^ sw);
      L.a1[s] = ar * 128 + 16 * ((2 * b + 1) ^ sw);
    } else {
      L.a0[s] = ar * 64 + 16 * ((2 * h + s) ^ ((ar >> 2) & 3));
      L.a1[s] = L.a0[s];
    }
    const int br = (ST == 1 ? 64 : 128) * wn + r;
    L.b[s] = TL<FA>::kB + br * 64 + 16 * ((2 * h + s) ^ ((br >> 2) & 3));
  }
  L.as = ((TBM / 2) * wm + r) * 16 + 2 * h;
  L.bs = TBM * 16 + ((ST == 1 ? 64 : 128) * wn + r) * 16 + 2 * h;
  return L;
}

// Stage-1 work item: DMA sources and shape of one tile.
template <int FA>
struct S1Tile {
  TSrc<FA> S;
  int row0, nrows, hc0;
};

template <int FA>
__device__ __forceinline__ S1Tile<FA> s1_setup(const S1Args& p, int4 tile, int nt, int w, int lane) {
  using Lo = TL<FA>;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int hc0 = nt * (TBN / 2);  // first h column of the tile
  const int xrow = (p.H / 32) * ActBytes<FA>::kBlock;
  S1Tile<FA> c;
  c.row0 = row0;
  c.nrows = nrows;
  c.hc0 = hc0;
  c.S.abase = p.xq;
  c.S.asbase = p.xs;
#pragma unroll
  for (int i = 0; i < Lo::kAInstr; ++i) {
    int r, ch;
    t_aslot<FA>(t_aci<FA>(w, i), lane, &r, &ch);
    const int R = t_row(r);
    const int tok = p.sorted[row0 + (R < nrows ? R : 0)] / p.k_total;
    c.S.a[i] = (uint32_t)(tok * xrow + 16 * ch);
  }
  // weight row (within the expert) of tile row r: 128 gate rows, then the 128 up rows
  auto wrow = [&](int r) { return r < TBN / 2 ? hc0 + r : p.I + hc0 + (r - TBN / 2); };
  c.S.bbase = p.w13 + (size_t)e * 2 * p.I * (p.H / 2);
  c.S.bsbase = p.w13s + (size_t)e * 2 * p.I * (p.H / 32);
#pragma unroll
  for (int i = 0; i < Lo::kBInstr; ++i) {
    int r, ch;
    t_bslot(Lo::kBInstr * w + i, lane, &r, &ch);
    const int wr = wrow(r);  // its 16-row group in the block layout, K piece 0
    c.S.b[i] = (uint32_t)((wr & ~15) * (p.H / 2) + 64 * (wr & 15) + 16 * ch);
  }
  const int ra = t_row(t_arow0(w) + lane);
  const int tok = p.sorted[row0 + (ra < nrows ? ra : 0)] / p.k_total;
  c.S.as = (uint32_t)(tok * (p.H / 32));
  c.S.bs = (uint32_t)(wrow(64 * w + lane) * (p.H / 32));
  return c;
}

// SwiGLU h = G * U * sigmoid(G) with the hardware exp2 and reciprocal (about
// one ulp each; G itself carries the much larger accumulation error).
__device__ __forceinline__ float swiglu_fast(float G, float U) {
  const float e = __builtin_amdgcn_exp2f(-G * 1.4426950408889634f);
  return G * U * __builtin_amdgcn_rcpf(1.0f + e);
}

// Value of lane l ^ 32 (the other half of the wave), by a VALU lane swap.
__device__ __forceinline__ uint32_t t_xhalf(uint32_t x, int h) {
  const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return h ? r[0] : r[1];
}

// Stage-1 epilogue, in registers. The accumulators hold the transposed tile:
// block (mb, nb), element i of lane l is weight row t_nrow(nb) + 8 (i / 4) +
// 4 h + i % 4 (h = l / 32) of the wave, token column 64 mb + 32 wm + l % 32
// of the tile (the wave half's row block mb). Gate
// block q and up block q + 2 cover the same 32 h columns, so the 32 values
// of one token's quantisation block are lane l's 16 and lane (l ^ 32)'s 16:
// the block maximum takes one exchange, and two more assemble each lane's
// contiguous half of the block's codes for one 16-byte (FP8) or 8-byte
// (FP4) store per token row.
template <int FA>
__device__ __forceinline__ void s1_epilogue(const S1Args& p, v16f (*acc)[4], int row0, int nrows,
                                            int hc0, int wm, int wn, int lane, int nmb) {
  constexpr int kCB = FA == 4 ? 16 : 32;  // code bytes per 32-element block (e2m3: its slot)
  const int r = lane & 31, h = lane >> 5;
  const size_t crow = (size_t)(p.I / 32) * kCB;  // code bytes per hq row
  const int blk0 = (hc0 + 64 * wn) / 32;         // the wave's two h blocks
#pragma unroll
  for (int mb = 0; mb < kMB; ++mb) {
    if (mb < nmb) {
      const int tr = 64 * mb + 32 * wm + r;  // token row within the tile
      uint8_t* crow_p = p.hq + ((size_t)row0 + tr) * crow;
      uint32_t sc = 0;
      // both blocks' codes first, then the stores: one branch per row block,
      // so the two blocks' arithmetic can be scheduled together
      uint4 v8[2];
      uint32_t v6[2][3];
      uint2 v4[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        float hv[16];
        float m = 0.0f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          hv[i] = swiglu_fast(acc[mb][q][i], acc[mb][q + 2][i]);
          m = fmaxf(m, fabsf(hv[i]));
        }
        m = fmaxf(m, __uint_as_float(t_xhalf(__float_as_uint(m), h)));
        const int X = mx_scale_exp<FA>(m);
        sc |= (uint32_t)(X + 127) << (8 * q);
        // d[k]: positions 8k + 4h .. +3 of the block (four consecutive h columns)
        uint32_t d[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if constexpr (FA == 0) {
            d[k] = e4m3_pack4(ldexpf(hv[4 * k], -X), ldexpf(hv[4 * k + 1], -X),
                              ldexpf(hv[4 * k + 2], -X), ldexpf(hv[4 * k + 3], -X));
          } else if constexpr (FA == 2) {  // one code per byte, packed to 6 bits below
            uint32_t v = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) v |= mx_encode<FA>(ldexpf(hv[4 * k + j], -X)) << (8 * j);
            d[k] = v;
          } else {
            uint32_t v = 0;
#pragma unroll
            for (int j = 0; j < 4; ++j) v |= mx_encode<FA>(ldexpf(hv[4 * k + j], -X)) << (4 * j);
            d[k] = v;
          }
        }
        // lane h = 0 keeps block positions 0-15, lane h = 1 positions 16-31
        const uint32_t s0 = h ? d[0] : d[2], s1 = h ? d[1] : d[3];
        const uint32_t r0 = t_xhalf(s0, h), r1 = t_xhalf(s1, h);
        if constexpr (FA == 0) {
          v8[q] = h ? make_uint4(r0, d[2], r1, d[3]) : make_uint4(d[0], r0, d[1], r1);
        } else if constexpr (FA == 2) {  // 16 codes at 6 bits: 12 bytes of the slot
          const uint32_t wv[4] = {h ? r0 : d[0], h ? d[2] : r0, h ? r1 : d[1], h ? d[3] : r1};
          pack6x16(wv, v6[q]);
        } else {
          v4[q] = h ? make_uint2(r0 | (d[2] << 16), r1 | (d[3] << 16))
                    : make_uint2(d[0] | (r0 << 16), d[1] | (r1 << 16));
        }
      }
      if (tr < nrows) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          if constexpr (FA == 0) {
            *reinterpret_cast<uint4*>(crow_p + (blk0 + q) * kCB + 16 * h) = v8[q];
          } else if constexpr (FA == 2) {
            uint32_t* dst = reinterpret_cast<uint32_t*>(crow_p + (blk0 + q) * kCB + 12 * h);
            dst[0] = v6[q][0];
            dst[1] = v6[q][1];
            dst[2] = v6[q][2];
          } else {
            *reinterpret_cast<uint2*>(crow_p + (blk0 + q) * kCB + 8 * h) = v4[q];
          }
        }
        if (h == 0)
          *reinterpret_cast<uint16_t*>(p.hs + ((size_t)row0 + tr) * (p.I / 32) + blk0) =
              (uint16_t)sc;
      }
    }
  }
}

// Stage-2 work item: DMA sources and shape of one tile.
template <int FA>
struct S2Tile {
  TSrc<FA> S;
  int row0, nrows, nc0;
};

template <int FA>
__device__ __forceinline__ S2Tile<FA> s2_setup(const S2Args& p, int4 tile, int nt, int w, int lane) {
  using Lo = TL<FA>;
  const int e = tile.x, row0 = tile.y, nrows = tile.z;
  const int arow = (p.I / 32) * ActBytes<FA>::kBlock;
  S2Tile<FA> c;
  c.row0 = row0;
  c.nrows = nrows;
  c.nc0 = nt * TBN;  // first output column of the tile
  c.S.abase = p.hq + (size_t)row0 * arow;
  c.S.asbase = p.hs + (size_t)row0 * (p.I / 32);
#pragma unroll
  for (int i = 0; i < Lo::kAInstr; ++i) {
    int r, ch;
    t_aslot<FA>(t_aci<FA>(w, i), lane, &r, &ch);
    const int R = t_row(r);
    c.S.a[i] = (uint32_t)((R < nrows ? R : 0) * arow + 16 * ch);
  }
  const size_t wr0 = (size_t)e * p.H + c.nc0;  // first weight row of the tile
  c.S.bbase = p.w2 + wr0 * (p.I / 2);
  c.S.bsbase = p.w2s + wr0 * (p.I / 32);
#pragma unroll
  for (int i = 0; i < Lo::kBInstr; ++i) {
    int r, ch;
    t_bslot(Lo::kBInstr * w + i, lane, &r, &ch);
    c.S.b[i] = (uint32_t)((r & ~15) * (p.I / 2) + 64 * (r & 15) + 16 * ch);  // block layout
  }
  const int ra = t_row(t_arow0(w) + lane);
  c.S.as = (uint32_t)((ra < nrows ? ra : 0) * (p.I / 32));
  c.S.bs = (uint32_t)((64 * w + lane) * (p.I / 32));
  return c;
}

// Persistent stage-2 kernel. Per tile: K loop; then the next tile's first
// DMA stages go out before this tile's epilogue (fp32 partial rows to their
// unique assignment slots, non-temporal stores: the combine reads them once,
// much later), so the epilogue's stores cover their latency.
// The epilogue only uses the second scale buffer (assignment slots of the
// tile's rows, and the two ticket words), which no prologue writes.
template <int FA>
__global__ __launch_bounds__(256, kWGperCU) void s2_tiled_kernel(S2Args p) {
  using Lo = TL<FA>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int* sidx = reinterpret_cast<int*>(lds + Lo::kS + Lo::kSBuf);
  int* slot = reinterpret_cast<int*>(lds + Lo::kS + Lo::kSBuf + TBM * 16);
  const int per = kChunk * p.t.n_ntiles, nch = *p.t.nchunks;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int wm = w & 1, wn = w >> 1;
  int4 tile;
  int nt;
  bool have = t_next(p.t, slot, nch, per, &tile, &nt);
  if (have) {
    int lane = threadIdx.x % kWave;
    asm volatile("" : "+v"(lane));
    t_prologue<FA>(lds, s2_setup<FA>(p, tile, nt, w, lane).S, w, t_nmb(tile.z, wm));
  }
  while (have) {
    // lane-derived offsets are recomputed per tile rather than held in
    // registers across the persistent loop (the opaque copy blocks hoisting)
    int lane = threadIdx.x % kWave;
    asm volatile("" : "+v"(lane));
    const S2Tile<FA> c = s2_setup<FA>(p, tile, nt, w, lane);
    const TLane L = t_lane<FA, 2>(w, lane);
    const int nrows = c.nrows;
    const int nmb = t_nmb(nrows, wm);
    v16f acc[kMB][4];
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = v16f{};
    t_kloop<FA, 2, false>(lds, c.S, L, p.I / 128, w, nmb, acc);

    const int sv = (int)threadIdx.x < min(nrows, TBM) ? p.sorted[c.row0 + threadIdx.x] : 0;
    int4 tile2;
    int nt2;
    have = t_next(p.t, slot, nch, per, &tile2, &nt2);
    sidx[threadIdx.x] = sv;
    if (have) t_prologue<FA>(lds, s2_setup<FA>(p, tile2, nt2, w, lane).S, w, t_nmb(tile2.z, wm));
    t_sync_lds();

    const int r = lane & 31, g = lane >> 5;
    float* const col = p.partials + c.nc0 + 128 * wn + r;
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb) {
      if (mb < nmb) {
        // the block's 16 slot numbers first, in a few wide LDS reads (rows
        // past nrows read the zero stored for them and are not written)
        int slot16[16];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          slot16[i] = sidx[64 * mb + 32 * wm + 8 * (i / 4) + 4 * g + (i % 4)];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int row = 64 * mb + 32 * wm + 8 * (i / 4) + 4 * g + (i % 4);
          if (row < nrows) {
            float* dst = col + (size_t)slot16[i] * p.H;
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) __builtin_nontemporal_store(acc[mb][nb][i], dst + 32 * nb);
          }
        }
      }
    }
    tile = tile2;
    nt = nt2;
  }
  if (threadIdx.x == 0) t_finish(p.t);
}

// Persistent stage-1 kernel. Per tile: K loop; then the next tile's first
// DMA stages go out before this tile's epilogue, which works in registers
// only. The ticket words lie in the second scale buffer (past its activation
// scales), which no prologue writes.
template <int FA>
__global__ __launch_bounds__(256, kWGperCU) void s1_tiled_kernel(S1Args p) {
  using Lo = TL<FA>;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  int* slot = reinterpret_cast<int*>(lds + Lo::kS + Lo::kSBuf + TBM * 16);
  const int per = kChunk * p.t.n_ntiles, nch = *p.t.nchunks;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int wm = w & 1, wn = w >> 1;
  int lane = threadIdx.x % kWave;
  int4 tile;
  int nt;
  bool have = t_next(p.t, slot, nch, per, &tile, &nt);
  S1Tile<FA> c;
  if (have) {
    c = s1_setup<FA>(p, tile, nt, w, lane);
    t_prologue<FA>(lds, c.S, w, t_nmb(c.nrows, wm));
  }
  while (have) {
    // lane-derived offsets are recomputed per tile rather than held in
    // registers across the persistent loop (the opaque copy blocks hoisting)
    asm volatile("" : "+v"(lane));
    const TLane L = t_lane<FA, 1>(w, lane);
    const int nmb = t_nmb(c.nrows, wm);
    v16f acc[kMB][4];
#pragma unroll
    for (int mb = 0; mb < kMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mb][nb] = v16f{};
    t_kloop<FA, 1, false>(lds, c.S, L, p.H / 128, w, nmb, acc);

    int4 tile2;
    int nt2;
    have = t_next(p.t, slot, nch, per, &tile2, &nt2);
    const int row0 = c.row0, nrows = c.nrows, hc0 = c.hc0;
    if (have) {
      c = s1_setup<FA>(p, tile2, nt2, w, lane);
      t_prologue<FA>(lds, c.S, w, t_nmb(c.nrows, wm));
    }
    s1_epilogue<FA>(p, acc, row0, nrows, hc0, wm, wn, lane, nmb);
  }
  if (threadIdx.x == 0) t_finish(p.t);
}

size_t tiled_lds_bytes(int fa) {
  return fa == 4 ? (size_t)t_lds_s1<4>() : (size_t)t_lds_s1<0>();
}

// Scale groups cover 512 K elements in both stages; N tiles are 128 h
// columns (stage 1) and 256 output columns (stage 2).
bool tiled_ok(int H, int I) { return H % (128 * kSG) == 0 && I % (128 * kSG) == 0; }
bool tiled_k_ok(int K) { return K % (128 * kSG) == 0; }

// kWGperCU workgroups per CU (together they hold a CU's LDS), never more
// than the items.
static int persistent_grid(long mt, int n_ntiles) {
  static const int slots = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    return n * kWGperCU;
  }();
  const long items = mt * n_ntiles;
  return (int)(items < slots ? (items > 0 ? items : 1) : slots);
}

template <int FA>
static void launch_t1(const S1Args& p, long mt, hipStream_t s) {
  S1Args q = p;
  q.t.n_ntiles = p.I / (TBN / 2);
  hipLaunchKernelGGL((s1_tiled_kernel<FA>), dim3(persistent_grid(mt, q.t.n_ntiles)), dim3(256),
                     t_lds_s1<FA>(), s, q);
}

template <int FA>
static void launch_t2(const S2Args& p, long mt, hipStream_t s) {
  S2Args q = p;
  q.t.n_ntiles = p.H / TBN;
  hipLaunchKernelGGL((s2_tiled_kernel<FA>), dim3(persistent_grid(mt, q.t.n_ntiles)), dim3(256),
                     TL<FA>::kLoop, s, q);
}

void launch_s1_tiled(const S1Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_t1<0>(p, mt, s);
  else if (fa == 2) launch_t1<2>(p, mt, s);
  else launch_t1<4>(p, mt, s);
}

void launch_s2_tiled(const S2Args& p, long mt, int fa, hipStream_t s) {
  if (fa == 0) launch_t2<0>(p, mt, s);
  else if (fa == 2) launch_t2<2>(p, mt, s);
  else launch_t2<4>(p, mt, s);
}

