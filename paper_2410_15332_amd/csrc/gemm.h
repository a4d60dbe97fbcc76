// Row-set GEMMs of the link step (host side): C[M x N] = A[M x K] . W[N x K]^T
// on MFMA with a fused epilogue.  Shapes are validated by the entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace epic {

enum GemmEpilogue { kStoreF32 = 0, kResidual = 1, kSwiGLU = 2 };

struct GemmArgs {
  const uint16_t* A;   // [M][K] bf16
  const uint16_t* W;   // [N][K] bf16 ([2 ffn][K] for kSwiGLU: gate rows, then up rows)
  float* C;            // [M][N] fp32 output (kStoreF32) or residual stream (kResidual)
  uint16_t* act;       // [M][ffn] bf16 (kSwiGLU)
  int M, N, K, ffn;
  float* partial;      // split-tile partial sums, gemm_workspace_bytes() with tile_count
  int* tile_count;     // arrival counters of split tiles (per wavefront); zero before the first launch
};
// Requirements: K % 32 == 0; N % 128 == 0 (kStoreF32 / kResidual); ffn % 128 == 0
// (kSwiGLU); M * K and N * K below 2^30 (byte offsets of the operands fit 31 bits).

// Bytes of partials + counters that every launch needs (independent of the shape).
size_t gemm_workspace_bytes();
// Carve the workspace: partials first, then the counters.
void gemm_workspace(void* base, float** partial, int** tile_count);
// Zero the arrival counters (a kernel, so it can sit in a captured stream).
void launch_gemm_clear(int* tile_count, hipStream_t stream);
void launch_gemm(const GemmArgs& g, int epi, hipStream_t stream);

}  // namespace epic
