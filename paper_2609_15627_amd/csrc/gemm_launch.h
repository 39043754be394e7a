// Launchers of the grouped-GEMM kernels of each geometry (host side).
#pragma once

#include <hip/hip_runtime.h>

#include "gemm_common.h"

namespace moe {

// Weight-streaming geometry. mt: row tiles the grid is sized for; fa:
// activation operand format code.
void launch_s1_stream(const S1Args& p, long mt, int fa, hipStream_t s);
void launch_s2_stream(const S2Args& p, long mt, int fa, hipStream_t s);

// Stage 2 + combine in one kernel for the streaming geometry: one workgroup
// per 16 output columns holding every row's fp32 result in LDS.
// fused_lds_bytes: its LDS need (0 when T * k_total rows are too many).
size_t fused_lds_bytes(int T, int k_total, int I);
void launch_s2c_stream(const S2CArgs& p, int fa, hipStream_t s);

// BF16 contract (bf16 activations, FP4 weights expanded to bf16 in
// registers, bf16 intermediate): one LDS-tiled geometry of bf16_rows() rows.
int bf16_rows();
size_t bf16_lds_bytes(int K);
void launch_s1_bf16(const S1Args& p, long mt, hipStream_t s);
void launch_s2_bf16(const S2Args& p, long mt, hipStream_t s);
// ... and its weight-streaming geometry for few rows per expert (tiles of
// bf16_stream_rows() rows).
int bf16_stream_rows();
void launch_s1_bf16_stream(const S1Args& p, long mt, hipStream_t s);
void launch_s2_bf16_stream(const S2Args& p, long mt, hipStream_t s);

// LDS-tiled geometry (many rows per expert): row tiles of tiled_rows(A, NE)
// rows (128 or 256, by the average rows per expert of A assignments over NE
// experts); the launches take the same row count.
int tiled_rows(long A, int NE);
size_t tiled_lds_bytes(int fa, int rows);
bool tiled_ok(int H, int I);  // both stages (K = H and K = I) fit the tiled K loop
bool tiled_k_ok(int K);       // a K extent fits the tiled K loop
void launch_s1_tiled(const S1Args& p, long mt, int fa, int rows, hipStream_t s);
void launch_s2_tiled(const S2Args& p, long mt, int fa, int rows, hipStream_t s);

// Short-K geometry of stage 2 (K = I of 128 or 256, many rows per expert):
// row tiles of short_rows() rows, the whole K extent of a tile in LDS.
int short_rows();
bool short_k_ok(int I);
size_t short_lds_bytes(int fa, int I);
void launch_s2_short(const S2Args& p, long mt, int fa, hipStream_t s);

}  // namespace moe
