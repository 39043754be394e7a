// Internal launchers behind the C ABI (host side). Arguments are already
// validated by api.hip; every launcher only enqueues on the given stream.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

hipError_t launch_router_logits(const uint16_t* x, const uint16_t* wr, int T, int H, int E,
                                float* logits, hipStream_t s);
hipError_t launch_route_topk(const float* logits, int T, int E, int k, int n_shared, int32_t* ids,
                             float* w, hipStream_t s);

// Routing variants (scoring, selection bias, group-limited selection,
// renormalisation, scaling); sigmoid: 0 softmax, 1 sigmoid.
struct RouteOpts {
  int sigmoid;
  const float* bias;
  int n_group, topk_group, renorm;
  float scale;
};
hipError_t launch_router_topk(const uint16_t* x, const uint16_t* wr, int T, int H, int E, int k,
                              int n_shared, const RouteOpts& o, float* logits, int32_t* ids,
                              float* w, hipStream_t s);
hipError_t launch_route_topk_ex(const float* logits, int T, int E, int k, int n_shared,
                                const RouteOpts& o, int32_t* ids, float* w, hipStream_t s);

size_t permute_workspace_bytes(int T, int NE, int k_total);
hipError_t launch_permute(const int32_t* ids, int T, int NE, int k_total, int32_t* counts,
                          int32_t* offsets, int32_t* sorted, int32_t* pos, void* ws,
                          hipStream_t s);

// fmt: 0 = e4m3, 2 = e2m3, 4 = e2m1 (matrix-core operand codes)
// Internal activation format codes: 0 MXFP8 e4m3, 2 MXFP6 e2m3, 4 MXFP4
// e2m1, kFmtBf16 the BF16 contract (bf16 activations, no scales).
constexpr int kFmtBf16 = 16;
int act_bits(int fmt);
// Bits per activation element in the grouped GEMM's workspace (e2m3 blocks
// sit in 32-byte slots there).
int ws_act_bits(int fmt);
hipError_t launch_quantize_act(const uint16_t* x, long rows, int K, int fmt, uint8_t* codes,
                               uint8_t* scales, hipStream_t s);

struct GemmWorkspace {
  size_t off[6];  // x codes, x scales, h codes, h scales, tile list, total
};
GemmWorkspace gemm_workspace(int T, int H, int I, int NE, int k_total, int fmt);

struct GemmArgs {
  const uint16_t* x;
  int T, H, I, NE, k_total, fmt;
  const int32_t* offsets;
  const int32_t* sorted;
  const uint8_t *w13, *w13_s, *w2, *w2_s;
  float* partials;
  uint8_t* ws;
  const float* topk_w = nullptr;  // with out: stage 2 fused with the combine
  uint16_t* out = nullptr;
};
// stages: bit 0 = activation quantisation + tile list, bit 1 = gate/up
// (stage 1), bit 2 = down (stage 2). Writes the geometry variant used
// (MOE_VARIANT_*) to *variant.
// Row-tile size of the LDS-tiled geometry: 0 (automatic), 128 or 256.
void set_tiled_rows(int rows);
hipError_t launch_grouped_gemm(const GemmArgs& a, int stages, hipStream_t s, int* variant);
// Whether stage 2 can run fused with the combine for these dims (streaming
// geometry chosen and every row's 16-column result fits one workgroup's LDS).
bool fused_combine_ok(const GemmArgs& a);

hipError_t launch_combine(const float* partials, const float* w, int T, int H, int k_total,
                          uint16_t* out, hipStream_t s);

// Expert weights [rows, K/2] FP4 codes -> the GEMM's layout (pack.hip).
hipError_t launch_pack_fp4(const uint8_t* w, uint8_t* out, long rows, int K, hipStream_t s);

hipError_t launch_probe(const uint8_t* a, const uint8_t* sa, int fmt, const uint8_t* b,
                        const uint8_t* sb, float* d, hipStream_t s);

}  // namespace moe
