// Row-set GEMMs of the link step (host side): C[M x N] = A[M x K] . W[N x K]^T
// on MFMA with a fused epilogue.  Shapes are validated by the entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace epic {

enum GemmEpilogue { kStoreF32 = 0, kResidual = 1, kSwiGLU = 2, kRope = 3 };

struct GemmArgs {
  const uint16_t* A;   // [M][K] bf16
  const uint16_t* W;   // [N][K] bf16 ([2 ffn][K] for kSwiGLU: gate rows, then up rows)
  float* C;            // [M][N] fp32 output (kStoreF32) or residual stream (kResidual)
  uint16_t* act;       // [M][ffn] bf16 (kSwiGLU)
  int M, N, K, ffn;
  // kRope (the fused Q|K|V projection): columns are heads of head_dim (hq query heads,
  // then hkv key heads, then hkv value heads); q and k heads are rotated by the rotary
  // table cs [M][head_dim / 2] (cos, sin) of each row, v heads are not; outputs bf16
  // q [M][hq][D], k / v [M][hkv][D].
  uint16_t *q, *k, *v;
  const float2* cs;
  int hq, hkv, head_dim;
  float* partial;      // split-tile partial sums, gemm_workspace_bytes() with tile_count
  int* tile_count;     // arrival counters of split tiles (per wavefront); zero before the first launch
};
// Requirements: K % 64 == 0; N % 128 == 0 (kStoreF32 / kResidual / kRope); ffn % 128 == 0
// (kSwiGLU); head_dim 64 or 128 (kRope); M * K and N * K below 2^30 (byte offsets of the
// operands fit 31 bits).

// Bytes of partials + counters that every launch needs (independent of the shape).
size_t gemm_workspace_bytes();
// Carve the workspace: partials first, then the counters.
void gemm_workspace(void* base, float** partial, int** tile_count);
// Zero the arrival counters (a kernel, so it can sit in a captured stream).
void launch_gemm_clear(int* tile_count, hipStream_t stream);
void launch_gemm(const GemmArgs& g, int epi, hipStream_t stream);

}  // namespace epic
