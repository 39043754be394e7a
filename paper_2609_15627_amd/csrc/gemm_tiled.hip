// a5 / a6: grouped FP4 expert GEMMs, LDS-tiled geometry for prefill-sized
// batches (many rows per expert), on the 32x32x64 block-scaled matrix cores.
//
// Workgroup tile: TBM sorted rows of one expert x 256 weight rows (stage 1:
// 128 gate rows and the 128 matching up rows; stage 2: 256 output columns),
// K in steps of 128 = two 64-element sub-steps. Four waves in a 2 x 2
// arrangement; each owns TBM / 64 32-row blocks x 128 weight rows, i.e.
// TBM / 64 x 4 products of 32x32 per sub-step, accumulated in fp32. The wave
// halves take alternate row blocks (wave half wm: blocks wm, wm + 2, ..), so
// a tile of fewer rows still keeps both halves' matrix cores busy; in LDS
// the rows sit in owner order (t_row), so each wave's operand reads and DMA
// stay within one contiguous half.
//
// Two arrangements of the same code (gemm_tiled_body.h, compiled for each
// TBM), chosen per call by the average rows per expert (tiled_rows):
//  - TBM = 128 when experts average at least 192 rows (prefill): two
//    workgroups per CU (76 KiB of LDS each, a ring of two stages, the
//    accumulators in 128 registers), so one workgroup's epilogue, ticket and
//    set-up run under the other's products; a chunk of the work list holds up
//    to four row tiles of one expert, so their weight rows are streamed from
//    DRAM once and shared in L2;
//  - TBM = 256 otherwise (e.g. the TP-shard shape's ~140 rows per expert):
//    one workgroup per CU, 256 accumulator registers per wave, a ring of 3
//    (FP8 activations) or 4 (FP4) stages, chunks of two row tiles.
// Both give the same bits: every output's K reduction is the same sequence
// of products.
//
// Data movement, chosen from measurements on gfx950:
//  - operands travel global -> LDS by DMA (global_load_lds, 16 bytes a lane,
//    1 KiB of contiguous LDS per instruction) through a ring of NS K-step
//    stages; an activation instruction reads whole 64- or 128-byte row
//    segments, a weight instruction one contiguous KiB (16 rows x 64 bytes of
//    the block layout of moe_pack_fp4_weights);
//  - E8M0 scales move in 16-byte row pieces covering four K steps (a
//    separate ring of two scale groups), not one word per row per step: a
//    4-byte gather costs a cache line per lane;
//  - LDS rows are chunk-swizzled (16-byte chunk c of row r stored at
//    c ^ f(r)) so the operand reads of the 32x32x64 layout run at full LDS
//    rate;
//  - matrix-core time is lost to load issue in bursts, not to spread-out
//    issue: each wave reads the next sub-step's operands one read per
//    product, and after the step's one workgroup barrier interleaves the
//    next step's reads (two per product) and DMA instructions with the
//    remaining products in explicit program order.
//
// K order inside a step: the products only need A and B to agree on which
// physical K elements a lane's bytes stand for. Sub-step s, lane half h takes
// the physical 32-element block 2h + s of the step's four, so a lane's two
// scale bytes of a step (blocks 2h and 2h + 1) are adjacent: one aligned
// 16-bit LDS read per row and step, op_sel s picks the byte.
//
// Matrix-core operand layout (32x32x64, measured): lane l supplies row l % 32
// of the row operand and column l % 32 of the column operand. An FP4 lane
// holds K elements [32 h, 32 h + 32) of the 64 (h = l / 32), two per byte,
// low nibble first; an FP8 lane holds K [16 h, 16 h + 16) in bytes 0-15 and
// K [32 + 16 h, +16) in bytes 16-31. The lane's scale register carries the
// scale of 32-element K block h in the byte selected by the instruction's
// op_sel. D: lane l, element i holds row 8 (i / 4) + 4 h + i % 4, column
// l % 32.
//
// Both kernels are persistent (one or two workgroups per CU) and take work
// items from per-XCD queues; the next tile's first DMA stages go out before
// the current tile's epilogue.
#include "gemm_common.h"
#include "gemm_launch.h"
#include "quant_dev.h"
#include "moe_launch.h"

#include <atomic>

namespace moe {

namespace t256 {
#define MOE_TILED_ROWS 256
#include "gemm_tiled_body.h"
#undef MOE_TILED_ROWS
}  // namespace t256

namespace t128 {
#define MOE_TILED_ROWS 128
#include "gemm_tiled_body.h"
#undef MOE_TILED_ROWS
}  // namespace t128

// Rows per expert (on average) from which the 128-row arrangement runs: it
// keeps the matrix cores of two workgroups per CU busy when experts fill
// their tiles, but tiles of fewer rows (the TP-shard shape) run better as
// 256-row tiles with the row blocks split between the wave halves.
constexpr long kRows128 = 192;

// 0: automatic; 128 or 256: forced (moe_set_tiled_rows).
static std::atomic<int> g_tiled_rows{0};

void set_tiled_rows(int rows) { g_tiled_rows.store(rows, std::memory_order_relaxed); }

int tiled_rows(long A, int NE) {
  const int forced = g_tiled_rows.load(std::memory_order_relaxed);
  if (forced) return forced;
  return NE > 0 && A >= kRows128 * NE ? 128 : 256;
}

size_t tiled_lds_bytes(int fa, int rows) {
  return rows == 128 ? t128::tiled_lds_bytes(fa) : t256::tiled_lds_bytes(fa);
}

bool tiled_ok(int H, int I) { return t256::tiled_ok(H, I); }
bool tiled_k_ok(int K) { return t256::tiled_k_ok(K); }

void launch_s1_tiled(const S1Args& p, long mt, int fa, int rows, hipStream_t s) {
  if (rows == 128) t128::launch_s1_tiled(p, mt, fa, s);
  else t256::launch_s1_tiled(p, mt, fa, s);
}

void launch_s2_tiled(const S2Args& p, long mt, int fa, int rows, hipStream_t s) {
  if (rows == 128) t128::launch_s2_tiled(p, mt, fa, s);
  else t256::launch_s2_tiled(p, mt, fa, s);
}

}  // namespace moe
