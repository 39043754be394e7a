// The C ABI (include/moe.h): host-side argument validation, then the
// launchers. Validation runs before anything is enqueued, so every error path
// can be exercised without a GPU. No exception crosses the boundary.
#include "moe.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "moe_launch.h"

namespace {

// Workspace of moe_fp4_grouped_gemm_noalloc: one static array per GPU. In
// host code `scratch` only stands in for the symbol; its device address on
// the current GPU comes from scratch_address().
constexpr size_t kScratchBytes = MOE_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device, looked up once

// Device address of the current GPU's scratch array (looked up on the first
// call on that device, with that device current).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

thread_local int g_last_variant = MOE_VARIANT_NONE;

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline moe_status launched(hipError_t e) {
  if (e == hipSuccess) return MOE_OK;
  if (e == hipErrorNotSupported) return MOE_ERR_UNSUPPORTED;
  return MOE_ERR_LAUNCH;
}

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int fmt_code(moe_act_format f) {
  switch (f) {
    case MOE_ACT_MXFP8_E4M3: return 0;
    case MOE_ACT_MXFP6_E2M3: return 2;
    case MOE_ACT_MXFP4_E2M1: return 4;
    case MOE_ACT_BF16: return moe::kFmtBf16;
  }
  return -1;
}

bool tokens_ok(int T, int k_total) { return T >= 0 && (long)T * k_total < (1L << 31); }

}  // namespace

extern "C" {

const char* moe_status_string(moe_status s) {
  switch (s) {
    case MOE_OK: return "ok";
    case MOE_ERR_INVALID_ARG: return "invalid argument";
    case MOE_ERR_UNSUPPORTED: return "unsupported";
    case MOE_ERR_WORKSPACE: return "workspace too small or missing";
    case MOE_ERR_LAUNCH: return "kernel launch failed";
  }
  return "unknown status";
}

int moe_last_variant(void) { return g_last_variant; }

moe_status moe_set_tiled_rows(int rows) {
  if (rows != 0 && rows != 128 && rows != 256) return MOE_ERR_INVALID_ARG;
  moe::set_tiled_rows(rows);
  return MOE_OK;
}

moe_status moe_router_logits(const uint16_t* x, const uint16_t* w_router, int T, int H, int E,
                             float* logits, void* stream) {
  if (T < 0 || H <= 0 || H % 8 || E < 1 || E > MOE_MAX_EXPERTS) return MOE_ERR_INVALID_ARG;
  if ((long)T * E >= (1L << 31) / 64) return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!x || !w_router || !logits)) return MOE_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(w_router, 16)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_router_logits(x, w_router, T, H, E, logits, as_stream(stream)));
}

moe_status moe_route_topk(const float* logits, int T, int E, int k, int n_shared, int32_t* topk_ids,
                          float* topk_w, void* stream) {
  if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS || k < 1 || k > E) return MOE_ERR_INVALID_ARG;
  if (n_shared != 0 && n_shared != 1) return MOE_ERR_INVALID_ARG;
  if (k + n_shared > MOE_MAX_K_TOTAL || !tokens_ok(T, k + n_shared)) return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!logits || !topk_ids || !topk_w)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_route_topk(logits, T, E, k, n_shared, topk_ids, topk_w,
                                         as_stream(stream)));
}

// Below this many tokens moe_router_topk computes the logits and routes them
// in two kernels when the caller gives a logits buffer.
constexpr int kRouterFusedMinTokens = 1024;

// Validation shared by moe_route_topk_ex and moe_router_topk (opts not NULL).
static moe_status check_route(int T, int E, int k, int n_shared, const moe_route_opts* opts) {
  if (T < 0 || E < 1 || E > MOE_MAX_EXPERTS || k < 1 || k > E) return MOE_ERR_INVALID_ARG;
  if (n_shared != 0 && n_shared != 1) return MOE_ERR_INVALID_ARG;
  if (k + n_shared > MOE_MAX_K_TOTAL || !tokens_ok(T, k + n_shared)) return MOE_ERR_INVALID_ARG;
  if (opts->score != MOE_SCORE_SOFTMAX && opts->score != MOE_SCORE_SIGMOID)
    return MOE_ERR_INVALID_ARG;
  const int ng = opts->n_group, tg = opts->topk_group;
  if (ng < 1 || ng > 64 || E % ng != 0 || tg < 1 || tg > ng || k > tg * (E / ng))
    return MOE_ERR_INVALID_ARG;
  return MOE_OK;
}

static moe::RouteOpts route_opts(const moe_route_opts* opts) {
  return moe::RouteOpts{opts->score == MOE_SCORE_SIGMOID ? 1 : 0, opts->bias, opts->n_group,
                        opts->topk_group, opts->renorm ? 1 : 0, opts->scale};
}

moe_status moe_router_topk(const uint16_t* x, const uint16_t* w_router, int T, int H, int E, int k,
                           int n_shared, const moe_route_opts* opts, float* logits,
                           int32_t* topk_ids, float* topk_w, void* stream) {
  static const moe_route_opts kDefault{MOE_SCORE_SOFTMAX, nullptr, 1, 1, 1, 1.0f};
  if (!opts) opts = &kDefault;
  const moe_status st = check_route(T, E, k, n_shared, opts);
  if (st != MOE_OK) return st;
  if (H <= 0 || H % 128 != 0) return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!x || !w_router || !topk_ids || !topk_w)) return MOE_ERR_INVALID_ARG;
  // Few tokens: each fused workgroup streams the whole router matrix, which
  // takes longer than computing the logits with many waves and routing them
  // separately; that needs the logits buffer.
  if (logits && T < kRouterFusedMinTokens) {
    hipError_t err = moe::launch_router_logits(x, w_router, T, H, E, logits, as_stream(stream));
    if (err != hipSuccess) return MOE_ERR_LAUNCH;
    return launched(moe::launch_route_topk_ex(logits, T, E, k, n_shared, route_opts(opts),
                                              topk_ids, topk_w, as_stream(stream)));
  }
  return launched(moe::launch_router_topk(x, w_router, T, H, E, k, n_shared, route_opts(opts),
                                          logits, topk_ids, topk_w, as_stream(stream)));
}

moe_status moe_route_topk_ex(const float* logits, int T, int E, int k, int n_shared,
                             const moe_route_opts* opts, int32_t* topk_ids, float* topk_w,
                             void* stream) {
  if (!opts) return MOE_ERR_INVALID_ARG;
  const moe_status st = check_route(T, E, k, n_shared, opts);
  if (st != MOE_OK) return st;
  if (T > 0 && (!logits || !topk_ids || !topk_w)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_route_topk_ex(logits, T, E, k, n_shared, route_opts(opts), topk_ids,
                                            topk_w, as_stream(stream)));
}

size_t moe_permute_workspace_bytes(int T, int n_experts_total, int k_total) {
  if (T < 0 || n_experts_total < 1 || k_total < 1) return 0;
  return moe::permute_workspace_bytes(T, n_experts_total, k_total);
}

moe_status moe_permute(const int32_t* topk_ids, int T, int n_experts_total, int k_total,
                       int32_t* counts, int32_t* offsets, int32_t* sorted, int32_t* pos, void* ws,
                       size_t ws_bytes, void* stream) {
  if (T < 0 || n_experts_total < 1 || n_experts_total > MOE_MAX_EXPERTS_TOTAL) return MOE_ERR_INVALID_ARG;
  if (k_total < 1 || k_total > MOE_MAX_K_TOTAL || !tokens_ok(T, k_total)) return MOE_ERR_INVALID_ARG;
  if (!counts || !offsets) return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!topk_ids || !sorted || !pos)) return MOE_ERR_INVALID_ARG;
  const size_t need = moe::permute_workspace_bytes(T, n_experts_total, k_total);
  if ((long)T * k_total > 1024 && (!ws || ws_bytes < need || !aligned(ws, 256)))
    return MOE_ERR_WORKSPACE;
  return launched(moe::launch_permute(topk_ids, T, n_experts_total, k_total, counts, offsets, sorted,
                                      pos, ws, as_stream(stream)));
}

moe_status moe_quantize_act(const uint16_t* x, int rows, int K, moe_act_format f, uint8_t* codes,
                            uint8_t* scales, void* stream) {
  const int fc = fmt_code(f);
  if (fc < 0 || fc == moe::kFmtBf16 || rows < 0 || K <= 0 || K % 32) return MOE_ERR_INVALID_ARG;
  if (rows > 0 && (!x || !codes || !scales)) return MOE_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(codes, 16)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_quantize_act(x, rows, K, fc, codes, scales, as_stream(stream)));
}

moe_status moe_pack_fp4_weights(const uint8_t* w, uint8_t* out, long rows, int K, void* stream) {
  if (rows < 0 || rows % 16 || K <= 0 || K % 128) return MOE_ERR_INVALID_ARG;
  if (rows == 0) return MOE_OK;
  if (!w || !out || !aligned(w, 16) || !aligned(out, 16)) return MOE_ERR_INVALID_ARG;
  const uintptr_t a = reinterpret_cast<uintptr_t>(w), b = reinterpret_cast<uintptr_t>(out);
  const uintptr_t n = (uintptr_t)rows * (uintptr_t)(K / 2);
  if (a < b + n && b < a + n) return MOE_ERR_INVALID_ARG;  // overlapping buffers
  return launched(moe::launch_pack_fp4(w, out, rows, K, as_stream(stream)));
}

// The GEMM kernels address activation rows (x, h) and one expert's weights
// with 32-bit byte offsets from a base: each must stay below 4 GiB.
static bool offsets_fit(int T, int H, int I, int k_total, int fc) {
  const double bits = moe::ws_act_bits(fc);
  const double lim = 4294967296.0;
  return (double)T * H * bits / 8 < lim && (double)T * k_total * I * bits / 8 < lim &&
         (double)H * I < lim;
}

static bool gemm_dims_ok(int T, int H, int I, int NE, int k_total) {
  return T >= 0 && H > 0 && I > 0 && H % 128 == 0 && I % 128 == 0 && NE >= 1 &&
         NE <= MOE_MAX_EXPERTS_TOTAL && k_total >= 1 && k_total <= MOE_MAX_K_TOTAL &&
         tokens_ok(T, k_total);
}

size_t moe_fp4_grouped_gemm_workspace_bytes(int T, int H, int I, int n_experts_total, int k_total,
                                            moe_act_format f) {
  if (fmt_code(f) < 0 || !gemm_dims_ok(T, H, I, n_experts_total, k_total)) return 0;
  return moe::gemm_workspace(T, H, I, n_experts_total, k_total, fmt_code(f)).off[5];
}

moe_status moe_fp4_grouped_gemm_workspace_layout(int T, int H, int I, int n_experts_total,
                                                 int k_total, moe_act_format f,
                                                 size_t offsets[MOE_WS_REGIONS]) {
  if (!offsets || fmt_code(f) < 0 || !gemm_dims_ok(T, H, I, n_experts_total, k_total))
    return MOE_ERR_INVALID_ARG;
  const moe::GemmWorkspace w = moe::gemm_workspace(T, H, I, n_experts_total, k_total, fmt_code(f));
  for (int i = 0; i < MOE_WS_REGIONS; ++i) offsets[i] = w.off[i];
  return MOE_OK;
}

// fused: stage 2 writes out through the combine (topk_w, out) instead of
// partials. use_scratch: the workspace is the library's static scratch array
// (ws is ignored); shapes that need more return MOE_ERR_WORKSPACE.
static moe_status grouped_gemm(const uint16_t* x, int T, int H, int I, int n_experts_total,
                               int k_total, const int32_t* offsets, const int32_t* sorted,
                               const uint8_t* w13, const uint8_t* w13_s, const uint8_t* w2,
                               const uint8_t* w2_s, moe_act_format f, float* partials,
                               bool fused, const float* topk_w, uint16_t* out, void* ws,
                               size_t ws_bytes, int stages, void* stream,
                               bool use_scratch = false) {
  const int fc = fmt_code(f);
  if (fc < 0 || !gemm_dims_ok(T, H, I, n_experts_total, k_total)) return MOE_ERR_INVALID_ARG;
  if (stages < 1 || stages > 7) return MOE_ERR_INVALID_ARG;
  if (fused && fc == 2) return MOE_ERR_UNSUPPORTED;
  if (T > 0 && (!x || !offsets || !sorted || !w13 || !w13_s || !w2 || !w2_s))
    return MOE_ERR_INVALID_ARG;
  if (T > 0 && (fused ? (!topk_w || !out) : !partials)) return MOE_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(w13, 16) || !aligned(w2, 16) || !aligned(w13_s, 4) ||
      !aligned(w2_s, 4) || !aligned(partials, 16) || !aligned(out, 16) || !aligned(topk_w, 4))
    return MOE_ERR_INVALID_ARG;
  if (!offsets_fit(T, H, I, k_total, fc)) return MOE_ERR_UNSUPPORTED;
  const size_t need = moe::gemm_workspace(T, H, I, n_experts_total, k_total, fc).off[5];
  if (use_scratch) {
    if (need > kScratchBytes) return MOE_ERR_WORKSPACE;
    ws = nullptr;
    ws_bytes = kScratchBytes;
    if (T > 0 && scratch_address(&ws) != hipSuccess) return MOE_ERR_LAUNCH;
  }
  if (T > 0 && (!ws || ws_bytes < need || !aligned(ws, 256))) return MOE_ERR_WORKSPACE;
  moe::GemmArgs a{x, T, H, I, n_experts_total, k_total, fc, offsets, sorted,
                  w13, w13_s, w2, w2_s, partials, static_cast<uint8_t*>(ws), topk_w, out};
  if (fused && T > 0 && !moe::fused_combine_ok(a)) return MOE_ERR_UNSUPPORTED;
  int variant = MOE_VARIANT_NONE;
  const moe_status st = launched(moe::launch_grouped_gemm(a, stages, as_stream(stream), &variant));
  g_last_variant = variant;
  return st;
}

moe_status moe_fp4_grouped_gemm(const uint16_t* x, int T, int H, int I, int n_experts_total,
                                int k_total, const int32_t* offsets, const int32_t* sorted,
                                const uint8_t* w13, const uint8_t* w13_s, const uint8_t* w2,
                                const uint8_t* w2_s, moe_act_format f, float* partials, void* ws,
                                size_t ws_bytes, void* stream) {
  return grouped_gemm(x, T, H, I, n_experts_total, k_total, offsets, sorted, w13, w13_s, w2, w2_s,
                      f, partials, false, nullptr, nullptr, ws, ws_bytes, 7, stream);
}

moe_status moe_fp4_grouped_gemm_stages(const uint16_t* x, int T, int H, int I,
                                       int n_experts_total, int k_total, const int32_t* offsets,
                                       const int32_t* sorted, const uint8_t* w13,
                                       const uint8_t* w13_s, const uint8_t* w2,
                                       const uint8_t* w2_s, moe_act_format f, float* partials,
                                       void* ws, size_t ws_bytes, int stages, void* stream) {
  return grouped_gemm(x, T, H, I, n_experts_total, k_total, offsets, sorted, w13, w13_s, w2, w2_s,
                      f, partials, false, nullptr, nullptr, ws, ws_bytes, stages, stream);
}

moe_status moe_fp4_grouped_gemm_noalloc(const uint16_t* x, int T, int H, int I,
                                        int n_experts_total, int k_total, const int32_t* offsets,
                                        const int32_t* sorted, const uint8_t* w13,
                                        const uint8_t* w13_s, const uint8_t* w2,
                                        const uint8_t* w2_s, moe_act_format f, float* partials,
                                        void* stream) {
  return grouped_gemm(x, T, H, I, n_experts_total, k_total, offsets, sorted, w13, w13_s, w2, w2_s,
                      f, partials, false, nullptr, nullptr, nullptr, 0, 7, stream, true);
}

int moe_fp4_grouped_gemm_combine_supported(int T, int H, int I, int n_experts_total, int k_total,
                                           moe_act_format f) {
  const int fc = fmt_code(f);
  if (fc < 0 || fc == 2 || !gemm_dims_ok(T, H, I, n_experts_total, k_total)) return 0;
  moe::GemmArgs a{nullptr, T, H, I, n_experts_total, k_total, fc, nullptr, nullptr,
                  nullptr, nullptr, nullptr, nullptr, nullptr, nullptr};
  return moe::fused_combine_ok(a) ? 1 : 0;
}

moe_status moe_fp4_grouped_gemm_combine(const uint16_t* x, int T, int H, int I,
                                        int n_experts_total, int k_total, const int32_t* offsets,
                                        const int32_t* sorted, const uint8_t* w13,
                                        const uint8_t* w13_s, const uint8_t* w2,
                                        const uint8_t* w2_s, moe_act_format f,
                                        const float* topk_w, uint16_t* out, void* ws,
                                        size_t ws_bytes, int stages, void* stream) {
  return grouped_gemm(x, T, H, I, n_experts_total, k_total, offsets, sorted, w13, w13_s, w2, w2_s,
                      f, nullptr, true, topk_w, out, ws, ws_bytes, stages, stream);
}

moe_status moe_combine_fixed_order(const float* partials, const float* topk_w, int T, int H,
                                   int k_total, uint16_t* out, void* stream) {
  if (T < 0 || H <= 0 || H % 8 || k_total < 1 || k_total > MOE_MAX_K_TOTAL || !tokens_ok(T, k_total))
    return MOE_ERR_INVALID_ARG;
  if (T > 0 && (!partials || !topk_w || !out)) return MOE_ERR_INVALID_ARG;
  if (!aligned(partials, 16) || !aligned(out, 16)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_combine(partials, topk_w, T, H, k_total, out, as_stream(stream)));
}

moe_status moe_probe_scaled_mfma(const uint8_t* a, const uint8_t* sa, moe_act_format fa,
                                 const uint8_t* b, const uint8_t* sb, float* d, void* stream) {
  const int fc = fmt_code(fa);
  if (fc < 0 || !a || !sa || !b || !sb || !d) return MOE_ERR_INVALID_ARG;
  if (!aligned(a, 16) || !aligned(b, 16)) return MOE_ERR_INVALID_ARG;
  return launched(moe::launch_probe(a, sa, fc, b, sb, d, as_stream(stream)));
}

}  // extern "C"
