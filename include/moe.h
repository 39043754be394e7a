/*
 * moe.h -- C ABI of the routed mixture-of-experts layer for AMD gfx950 (MI355X).
 *
 * The layer (paper: System and model context / Execution structure, Fig.
 * architecture) routes every token to its top-k experts, runs each expert's
 * gate/up projection, SwiGLU and down projection on FP4 e2m1 weights with
 * per-32 E8M0 block scales, runs an always-on shared expert beside them, and
 * sums the weighted partial outputs in a fixed order. A layer forward is:
 *
 *   moe_router_logits   (optional: logits from bf16 router weights)
 *   moe_route_topk      -> topk_ids, topk_w
 *   moe_permute         -> counts, offsets, sorted, pos
 *   moe_fp4_grouped_gemm-> partials (one fp32 row per (token, slot))
 *   moe_combine_fixed_order -> out (bf16)
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every array pointer is a DEVICE pointer owned by the caller. The library
 *    never allocates, frees or synchronises; it only enqueues kernels on
 *    `stream` (a hipStream_t passed as void*; NULL is the default stream).
 *    Buffers must stay alive until the stream has passed the call.
 *  - Arrays are dense row-major and little-endian. bf16 values are passed as
 *    their uint16_t bit patterns.
 *  - FP4 e2m1 weight codes are packed two per byte: element 2i in bits 0-3,
 *    element 2i+1 in bits 4-7. An e2m1 code has bit 3 = sign, bits 2-1 =
 *    exponent (bias 1), bit 0 = mantissa: values 0, .5, 1, 1.5, 2, 3, 4, 6 and
 *    their negatives.
 *  - E8M0 scales are one byte per 32 consecutive elements along the reduction
 *    axis; byte b means 2^(b-127) (255 is NaN and is rejected nowhere: it is a
 *    caller precondition, like finite inputs).
 *  - Scales are passed in their LOGICAL layout ([rows, K/32], unshuffled): the
 *    paper found that packed weights do not imply an unshuffled scale layout
 *    (Correctness recovery / Later numerical and integration repairs).
 *  - Arguments are validated on the host before anything is enqueued; a bad
 *    argument returns MOE_ERR_INVALID_ARG (or MOE_ERR_WORKSPACE) and enqueues
 *    nothing. A failed kernel launch returns MOE_ERR_LAUNCH. No C++ exception
 *    crosses this boundary. Sizes of zero tokens are valid and enqueue only
 *    what is needed to define the outputs.
 *  - Results are deterministic: no call uses floating-point atomics or split
 *    reductions, so repeated calls on the same inputs give identical bits.
 */
#ifndef MOE_H_
#define MOE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOE_OK = 0,
  MOE_ERR_INVALID_ARG = 1, /* null pointer, bad size, unsupported shape */
  MOE_ERR_UNSUPPORTED = 2, /* valid request that the library does not implement */
  MOE_ERR_WORKSPACE = 3,   /* workspace missing or smaller than the query said */
  MOE_ERR_LAUNCH = 4       /* a kernel launch failed (HIP error) */
} moe_status;

/* Element format of the activations fed to the matrix cores (OCP MX v1.0):
 * each block of 32 values shares one E8M0 scale. The paper's gfx90a kernels
 * quantised activations to INT8 per 32 elements (Historical TP4 decode
 * optimization / Parallel decomposition); gfx950's scaled MFMA consumes MX
 * formats instead. */
typedef enum {
  MOE_ACT_MXFP8_E4M3 = 0, /* 1 byte per element */
  MOE_ACT_MXFP6_E2M3 = 1, /* 24 bytes per 32-element block, element j in bits [6j, 6j+6)
                             (the matrix cores' FP6 operand: a lane's 32 elements in six
                             words); in the grouped GEMM's workspace each block's 24 bytes
                             sit in a 32-byte slot. Not available fused with the combine. */
  MOE_ACT_MXFP4_E2M1 = 2, /* 2 elements per byte, low nibble first */
  /* The paper's BF16 contract (Large-M CK and the meaning of the earlier
   * 6.42k result; Accepted large-prefill configuration): x is not quantised,
   * FP4 weights are expanded to bf16 (exactly, for scale bytes <= 252), G and
   * U accumulate in fp32 and h = SwiGLU(G, U) is rounded once to bf16
   * (nearest, ties to even) before the down projection; partials and the
   * combine are unchanged. Grouped GEMM only (not moe_quantize_act). */
  MOE_ACT_BF16 = 3
} moe_act_format;

/* Geometry variants reported by moe_last_variant(). */
enum {
  MOE_VARIANT_NONE = 0,
  MOE_VARIANT_STREAM = 1, /* weight-streaming geometry for few rows per expert (decode) */
  MOE_VARIANT_TILED = 2,  /* LDS-tiled MFMA geometry for many rows per expert (prefill) */
  MOE_VARIANT_BF16 = 3,   /* MOE_ACT_BF16: LDS-tiled bf16 geometry (many rows per expert) */
  MOE_VARIANT_MIXED = 4,  /* tiled stage 1, streaming stage 2 (I not a multiple of 512) */
  MOE_VARIANT_BF16_STREAM = 5, /* MOE_ACT_BF16: weight-streaming bf16 geometry (few rows) */
  MOE_VARIANT_SHORT = 6   /* stage 2 on the short-K geometry (I = 128 or 256, many rows per
                             expert: the whole K extent of a 128-row tile in LDS); stage 1
                             tiled when H is a multiple of 512, else streaming */
};

/* Limits checked by the validators. */
#define MOE_MAX_EXPERTS 1024       /* routed experts E */
#define MOE_MAX_EXPERTS_TOTAL 2048 /* E + shared experts */
#define MOE_MAX_K_TOTAL 32         /* k + n_shared */

/* ---- a1: router projection (optional helper) ----------------------------
 * logits[t,e] = sum_h x[t,h] * w_router[e,h], products accumulated in fp32 in
 * a fixed order. The "Router" box of the paper's layer figure.
 *   x         bf16 [T, H]        w_router  bf16 [E, H]
 *   logits    fp32 [T, E] (written)
 * Requires T >= 0, H > 0 and H % 8 == 0, 1 <= E <= MOE_MAX_EXPERTS. */
moe_status moe_router_logits(const uint16_t* x, const uint16_t* w_router, int T, int H, int E,
                             float* logits, void* stream);

/* ---- a2: top-k routing ----------------------------------------------------
 * For every token: the k largest logits, ordered by (logit descending, expert
 * id ascending) -- ties go to the lower id and positions are in this fixed
 * order (paper: Correctness recovery / Later numerical and integration
 * repairs, deterministic index selection). Weights are the softmax over the k
 * picks, w_j = exp(l_j - l_0) / sum_{i<k} exp(l_i - l_0), in fp32.
 * With n_shared = 1 a last column holds expert id E with weight 1.0 (the
 * shared expert, stacked after the routed ones).
 *   logits    fp32 [T, E]; NaN is read as -inf
 *   topk_ids  int32 [T, k + n_shared] (written)
 *   topk_w    fp32  [T, k + n_shared] (written)
 * Requires 1 <= k <= E <= MOE_MAX_EXPERTS, n_shared in {0, 1},
 * k + n_shared <= MOE_MAX_K_TOTAL. */
moe_status moe_route_topk(const float* logits, int T, int E, int k, int n_shared, int32_t* topk_ids,
                          float* topk_w, void* stream);

/* ---- f1: routing variants -------------------------------------------------
 * moe_route_topk_ex generalises moe_route_topk. The paper fixes the router's
 * top-k (top-6 for the model: System and model context / Execution
 * structure) and a deterministic selection order, and is silent on the
 * scoring. These options follow DeepSeek's published router design; each is
 * a reading, not a statement of the paper:
 *   score      MOE_SCORE_SOFTMAX: s_e = exp(l_e - max l) / sum_e' exp(l_e' - max l)
 *              MOE_SCORE_SIGMOID: s_e = 1 / (1 + exp(-l_e))
 *   bias       fp32 [E] (device) or NULL: the selection key of expert e is
 *              s_e + bias[e]; the bias steers selection only, weights use s_e
 *   n_group,   experts form n_group groups of E / n_group consecutive ids; a
 *   topk_group group's score is the sum of its two largest keys (its only key
 *              when groups have one expert); the topk_group groups with the
 *              largest scores (ties to the lower group) stay and every other
 *              expert is excluded; n_group = 1 disables grouping
 *   renorm     nonzero: the k weights are divided by their sum (in pick order)
 *   scale      multiplies the k weights (routed scaling factor)
 * Picks: the k largest keys among the remaining experts, ordered by (key
 * descending, expert id ascending). Weights: s of each pick, renormalised as
 * asked, times scale; the shared expert's column (n_shared = 1) keeps weight
 * 1.0. Arithmetic in fp32; the softmax denominator is summed in a fixed
 * order. Without a bias, keys are compared as the raw logits (s is
 * increasing in l), so the picks are exact; with a bias or with groups, a
 * key tie within fp32 rounding can resolve either way against a reference.
 * {MOE_SCORE_SOFTMAX, NULL, 1, 1, 1, 1.0f} is exactly moe_route_topk.
 * Requires opts != NULL, 1 <= n_group <= 64, n_group divides E,
 * 1 <= topk_group <= n_group, k <= topk_group * E / n_group, plus the
 * requirements of moe_route_topk. */
typedef enum { MOE_SCORE_SOFTMAX = 0, MOE_SCORE_SIGMOID = 1 } moe_score_fn;
typedef struct {
  moe_score_fn score;
  const float* bias;
  int n_group;
  int topk_group;
  int renorm;
  float scale;
} moe_route_opts;
moe_status moe_route_topk_ex(const float* logits, int T, int E, int k, int n_shared,
                             const moe_route_opts* opts, int32_t* topk_ids, float* topk_w,
                             void* stream);

/* ---- f1: fused router projection and routing ------------------------------
 * One call for logits = x . w_router^T (as moe_router_logits, products
 * accumulated in fp32 by the matrix cores, so the summation order differs
 * from moe_router_logits) followed by the routing of moe_route_topk_ex (opts
 * NULL: the defaults of moe_route_topk), without a logits round trip
 * through memory. A logit tie within fp32 accumulation error can resolve
 * either way against a reference.
 *   x         bf16 [T, H]      w_router  bf16 [E, H]
 *   logits    fp32 [T, E] (written if not NULL)
 *   topk_ids, topk_w as moe_route_topk
 * With a logits buffer and T < 1024 the call runs moe_router_logits and
 * moe_route_topk_ex instead (two kernels; faster for few tokens, where a
 * fused workgroup streams the whole router matrix for a handful of tokens).
 * The fused workgroup holds 32 tokens' logits of all E experts in LDS
 * (32 * (E rounded up to 64, plus 1) * 4 bytes: 131 KB at E = 1024).
 * Requires H % 128 == 0 plus the requirements of moe_route_topk_ex
 * (1 <= E <= MOE_MAX_EXPERTS). */
moe_status moe_router_topk(const uint16_t* x, const uint16_t* w_router, int T, int H, int E, int k,
                           int n_shared, const moe_route_opts* opts, float* logits,
                           int32_t* topk_ids, float* topk_w, void* stream);

/* ---- a3: token -> expert permutation ---------------------------------------
 * Stable counting sort of the A = T * k_total assignments a = t*k_total + j by
 * expert id topk_ids[a] (the paper's expert sorter: Prefill optimization /
 * From per-assignment scalar work to CDNA2 MFMA, item 8).
 *   counts   int32 [NE]      assignments per expert
 *   offsets  int32 [NE + 1]  exclusive prefix sum of counts; offsets[NE] = A
 *   sorted   int32 [A]       assignment indices grouped by expert, increasing
 *                            a inside each expert
 *   pos      int32 [A]       inverse: sorted[pos[a]] == a
 * Ids outside [0, NE) are a precondition violation: they are skipped (never
 * used as an address), so counts then sum to less than A and the entries of
 * sorted past offsets[NE] are left unwritten.
 * ws: device workspace of at least moe_permute_workspace_bytes(...) bytes,
 * 256-byte aligned; contents need not be initialised.
 * Requires T >= 0, 1 <= NE <= MOE_MAX_EXPERTS_TOTAL, 1 <= k_total <= MOE_MAX_K_TOTAL. */
size_t moe_permute_workspace_bytes(int T, int n_experts_total, int k_total);
moe_status moe_permute(const int32_t* topk_ids, int T, int n_experts_total, int k_total,
                       int32_t* counts, int32_t* offsets, int32_t* sorted, int32_t* pos, void* ws,
                       size_t ws_bytes, void* stream);

/* ---- expert weight layout -------------------------------------------------
 * The grouped GEMM reads FP4 e2m1 expert weights (two codes per byte, low
 * nibble first, as the paper packs them: Prefill optimization / From
 * per-assignment scalar work to CDNA2 MFMA) in a block layout of its own:
 * rows in groups of 16, each group's bytes ordered by 64-byte K piece, then
 * by row, so that byte c of K piece q of row 16 g + r of a [rows, K/2] code
 * matrix sits at 16 g * K/2 + 1024 q + 64 r + c (one K piece of 16 rows is
 * 1 KiB of contiguous memory). A group covers the same bytes in both
 * layouts, so expert and row offsets are unchanged; only the bytes inside a
 * group move. The E8M0 scales stay row-major. Weights are packed once, when
 * they are loaded; the values are unchanged.
 *   w    uint8 [rows, K/2] row-major codes (e.g. W13 viewed as [NE * 2I, H/2],
 *        W2 as [NE * H, I/2]); read
 *   out  uint8 [rows, K/2] in the block layout (written); must not overlap w
 * Requires rows >= 0, rows % 16 == 0, K > 0, K % 128 == 0, both pointers
 * 16-byte aligned (else MOE_ERR_INVALID_ARG, nothing enqueued). */
moe_status moe_pack_fp4_weights(const uint8_t* w, uint8_t* out, long rows, int K, void* stream);

/* ---- a4: activation quantisation (standalone) -----------------------------
 * Per block of 32 consecutive elements of each row: X = the smallest integer
 * in [-127, 127] with max|v| <= maxval(format) * 2^X (X = 0 for an all-zero
 * block); scale byte = X + 127; each code = round-to-nearest-even(v / 2^X) on
 * the element grid, subnormals included, sign bit = sign bit of v. The paper
 * quantises activations per 32 elements before each projection (Historical
 * TP4 decode optimization / Parallel decomposition; Historical down-consumer
 * pilot). moe_fp4_grouped_gemm runs the same quantiser internally.
 *   x       bf16 [rows, K] (finite)
 *   codes   [rows, K * bits / 8] bytes, packed as the format says (written)
 *   scales  uint8 [rows, K / 32] (written)
 * Requires rows >= 0, K > 0, K % 32 == 0. */
moe_status moe_quantize_act(const uint16_t* x, int rows, int K, moe_act_format f, uint8_t* codes,
                            uint8_t* scales, void* stream);

/* ---- a5 + a6: grouped FP4 expert GEMMs --------------------------------------
 * The expert FFN of the layer (paper: System and model context / Execution
 * structure, Fig. architecture) on FP4 e2m1 weights with per-32 E8M0 scales,
 * grouped by expert over the rows the expert sorter produced (Prefill
 * optimization / From per-assignment scalar work to CDNA2 MFMA, item 8).
 * Activations are quantised per 32 elements before the gate/up projection
 * (Historical TP4 decode optimization / Parallel decomposition) and the
 * intermediate is quantised per 32 again before the down projection
 * (Historical down-consumer pilot); the down projection stores one FP32
 * partial per (token, slot) in its own row, with no cross-expert atomics
 * (Current TP8 native-AR results / Accepted large-prefill configuration),
 * and the partials stay FP32 (Rejected or reverted directions: BF16
 * partials changed values).
 * For every expert e and every sorted row r in [offsets[e], offsets[e+1]),
 * with a = sorted[r] and t = a / k_total:
 *   xq      = MX-quantised x[t]                     (as moe_quantize_act)
 *   G, U    = xq . W1[e]^T, xq . W3[e]^T            (W13 rows 0..I-1 = gate W1,
 *                                                   rows I..2I-1 = up W3)
 *   h       = G * U / (1 + exp(-G))                 (SwiGLU, fp32)
 *   hq      = MX-quantised h (blocks of 32 along I)
 *   partials[a, :] = hq . W2[e]^T                   (fp32, one unique row per
 *                                                   assignment: no atomics)
 * Products of codes and power-of-two scales are exact; sums are fp32 on the
 * matrix cores in a fixed order (the weight-streaming geometry adds two
 * halves of the K extent, first + second; no atomics, no run-to-run
 * variation).
 *   x         bf16 [T, H]
 *   offsets   int32 [NE + 1], sorted int32 [T * k_total]   (from moe_permute)
 *   w13       uint8 [NE, 2I, H/2]   w13_s uint8 [NE, 2I, H/32]
 *   w2        uint8 [NE, H, I/2]    w2_s  uint8 [NE, H, I/32]
 *             (w13 and w2 in the block layout of moe_pack_fp4_weights; the
 *             scales row-major)
 *   partials  fp32 [T * k_total, H]; row a = t*k_total + j (written for every
 *             assignment with a valid expert id)
 * ws: device workspace of at least moe_fp4_grouped_gemm_workspace_bytes(...)
 * bytes, 256-byte aligned, contents need not be initialised. Its regions are
 * reported by moe_fp4_grouped_gemm_workspace_layout (for inspection by tests).
 * Requires T >= 0, H > 0, I > 0, H % 128 == 0, I % 128 == 0,
 * 1 <= NE <= MOE_MAX_EXPERTS_TOTAL, 1 <= k_total <= MOE_MAX_K_TOTAL.
 * The geometry (MOE_VARIANT_*) is chosen per stage from T * k_total / NE and
 * the stage's K extent (the tiled K loop takes multiples of 512) and reported
 * by moe_last_variant(); under MOE_ACT_BF16 from T * k_total / NE alone
 * (tiled from 64 rows per expert on average, both stages alike).
 * The kernels address activation rows and one expert's weights with 32-bit
 * byte offsets: shapes where x [T, H] or h [T * k_total, I] in the activation
 * format, or H * I bytes, reach 4 GiB return MOE_ERR_UNSUPPORTED. */
size_t moe_fp4_grouped_gemm_workspace_bytes(int T, int H, int I, int n_experts_total, int k_total,
                                            moe_act_format f);

/* Byte offsets of the workspace regions: [0] x codes [T, H*bits/8], [1] x
 * scales [T, H/32], [2] h codes [T*k_total, I*bits/8] in sorted-row order,
 * [3] h scales [T*k_total, I/32], [4] tile list, [5] total bytes. bits is 8
 * for MXFP8 and for MXFP6 (its 24-byte blocks in 32-byte slots), 4 for
 * MXFP4. With MOE_ACT_BF16 regions 0, 1 and 3 are empty and region 2 holds
 * h as bf16. */
#define MOE_WS_REGIONS 6
moe_status moe_fp4_grouped_gemm_workspace_layout(int T, int H, int I, int n_experts_total,
                                                 int k_total, moe_act_format f,
                                                 size_t offsets[MOE_WS_REGIONS]);

moe_status moe_fp4_grouped_gemm(const uint16_t* x, int T, int H, int I, int n_experts_total,
                                int k_total, const int32_t* offsets, const int32_t* sorted,
                                const uint8_t* w13, const uint8_t* w13_s, const uint8_t* w2,
                                const uint8_t* w2_s, moe_act_format f, float* partials, void* ws,
                                size_t ws_bytes, void* stream);

/* The grouped GEMM split into its three steps, for per-step timing and
 * inspection: stages is a bit mask, bit 0 = activation quantisation of x and
 * the row-tile list (into ws), bit 1 = gate/up + SwiGLU + h quantisation
 * (reads x codes and tile list from ws, writes h codes to ws), bit 2 = down
 * projection into partials (reads h codes and tile list from ws). Calling the
 * bits in increasing order, in one call or several on one stream with the
 * same arguments, is exactly moe_fp4_grouped_gemm (stages = 7). */
moe_status moe_fp4_grouped_gemm_stages(const uint16_t* x, int T, int H, int I,
                                       int n_experts_total, int k_total, const int32_t* offsets,
                                       const int32_t* sorted, const uint8_t* w13,
                                       const uint8_t* w13_s, const uint8_t* w2,
                                       const uint8_t* w2_s, moe_act_format f, float* partials,
                                       void* ws, size_t ws_bytes, int stages, void* stream);

/* ---- allocation-free grouped GEMM -------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc. Exactly
 * moe_fp4_grouped_gemm (same kernels, same results, same argument meaning
 * and validation) without a workspace argument: the workspace is a static
 * device array of MOE_NOALLOC_SCRATCH_BYTES bytes inside the library, one per
 * GPU, held until the process ends. The call allocates and frees nothing.
 *  - A shape whose workspace (moe_fp4_grouped_gemm_workspace_bytes) exceeds
 *    MOE_NOALLOC_SCRATCH_BYTES returns MOE_ERR_WORKSPACE and enqueues nothing
 *    (32 MiB holds decode batches of up to about 1400 tokens at H = 4096,
 *    I = 2048, top-8 + shared).
 *  - Every call on one GPU uses that GPU's one array, and each call clears
 *    what must start at zero itself. Calls that overlap on one GPU (on
 *    different streams, or from threads without ordering between them) race
 *    on the array and must not be made; calls ordered on one stream are safe.
 *  - The GPU the stream belongs to must be the current device: the first call
 *    on a device looks up that device's copy of the array. */
#define MOE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
moe_status moe_fp4_grouped_gemm_noalloc(const uint16_t* x, int T, int H, int I,
                                        int n_experts_total, int k_total, const int32_t* offsets,
                                        const int32_t* sorted, const uint8_t* w13,
                                        const uint8_t* w13_s, const uint8_t* w2,
                                        const uint8_t* w2_s, moe_act_format f, float* partials,
                                        void* stream);

/* ---- f3: small-M down projection fused with the combine ---------------------
 * moe_fp4_grouped_gemm followed by moe_combine_fixed_order as one call, for
 * decode-sized batches: the down projection of every row and the
 * fixed-order sum over each token's slots run in one kernel, so no fp32
 * partial row is written to global memory and no combine kernel runs (the
 * paper's small down consumer, Historical down-consumer pilot, joined to its
 * fixed-order reducer, Current TP8 native-AR results / Accepted large-prefill
 * configuration). The output has exactly the bits of the two calls: the same
 * products in the same order, then acc = fmaf(topk_w[t, j], ., acc) for j =
 * 0 .. k_total-1 and one bf16 rounding.
 *   topk_w  fp32 [T, k_total] (from moe_route_topk); out bf16 [T, H]
 *   other arguments as moe_fp4_grouped_gemm_stages; stages bit 2 = the fused
 *   down projection + combine (writes out), 7 = the whole call.
 * An assignment with an invalid expert id contributes 0.
 * Available when moe_fp4_grouped_gemm_combine_supported() returns 1: the
 * weight-streaming geometry is chosen (few rows per expert) and the fp32
 * results of all T * k_total rows for 16 output columns fit one workgroup's
 * LDS (n * T * k_total * 64 + 32 * I bytes, n = 2 where the down projection
 * splits K over two waves -- I = 1024, 2048, 4096 or 8192 -- else 1;
 * T * k_total up to 768 at I = 2048). Otherwise (or without a device)
 * MOE_ERR_UNSUPPORTED, and nothing is enqueued: use the two calls. */
int moe_fp4_grouped_gemm_combine_supported(int T, int H, int I, int n_experts_total, int k_total,
                                           moe_act_format f);
moe_status moe_fp4_grouped_gemm_combine(const uint16_t* x, int T, int H, int I,
                                        int n_experts_total, int k_total, const int32_t* offsets,
                                        const int32_t* sorted, const uint8_t* w13,
                                        const uint8_t* w13_s, const uint8_t* w2,
                                        const uint8_t* w2_s, moe_act_format f,
                                        const float* topk_w, uint16_t* out, void* ws,
                                        size_t ws_bytes, int stages, void* stream);

/* ---- a7: fixed-order combine ------------------------------------------------
 * out[t, :] = bf16_rne(acc), acc = 0; for j = 0 .. k_total-1:
 *   acc = fmaf(topk_w[t, j], partials[t*k_total + j, :], acc)      (fp32)
 * The shared expert's weight is 1.0, so its fma is an exact add. The paper's
 * accepted path keeps one FP32 partial per (token, slot) and reduces them in a
 * fixed order (Current TP8 native-AR results / Accepted large-prefill
 * configuration; Rejected or reverted directions: BF16 partials rejected).
 *   partials fp32 [T * k_total, H]   topk_w fp32 [T, k_total]   out bf16 [T, H]
 * Requires T >= 0, H > 0, H % 8 == 0, 1 <= k_total <= MOE_MAX_K_TOTAL. */
moe_status moe_combine_fixed_order(const float* partials, const float* topk_w, int T, int H,
                                   int k_total, uint16_t* out, void* stream);

/* ---- diagnostics ------------------------------------------------------------ */

/* Human-readable name of a status code (static storage). */
const char* moe_status_string(moe_status s);

/* MOE_VARIANT_* chosen by the calling thread's last moe_fp4_grouped_gemm. */
int moe_last_variant(void);

/* Row-tile size of the LDS-tiled geometry (MOE_VARIANT_TILED and the tiled
 * stage 1 of MOE_VARIANT_MIXED and MOE_VARIANT_SHORT). Not an operation
 * of the paper: a tuning and testing control. rows = 128: tiles of 128 rows,
 * two workgroups per CU; 256: tiles of 256 rows, one workgroup per CU;
 * 0 (the default): 128 when T * k_total / NE >= 192, else 256. Both give the
 * same bits (every output's K reduction is the same sequence of products).
 * Process-wide: it affects every later call on every thread and device; a
 * call that overlaps it may use either size. Other values return
 * MOE_ERR_INVALID_ARG and leave the setting unchanged. */
moe_status moe_set_tiled_rows(int rows);

/* One block-scaled matrix-core product, D = (A * 2^(sa-127)) . (B * 2^(sb-127))^T
 * per 32-element K block, using the same operand and scale placement as the
 * grouped GEMM. Used to check that placement against the oracle.
 *   a   [16, 128] activation codes in format fa (packed like moe_quantize_act)
 *   sa  uint8 [16, 4]      b  uint8 [16, 64] FP4 weight codes   sb uint8 [16, 4]
 *   d   fp32 [16, 16] (written), d[i][j] = sum_k A[i][k] * B[j][k] */
moe_status moe_probe_scaled_mfma(const uint8_t* a, const uint8_t* sa, moe_act_format fa,
                                 const uint8_t* b, const uint8_t* sb, float* d, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* MOE_H_ */
