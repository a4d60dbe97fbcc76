// Elementwise parts of a decoder layer for the selected rows: RMSNorm and the
// rotary table at linked positions (the rotation itself runs in the epilogue of
// the fused Q|K|V projection, gemm.hip).
//
// RMSNorm: y = x / sqrt(mean(x^2) + eps) * w, fp32 statistics.
// Rotary embedding: the pair (i, i + D/2) of a head is rotated by angle
// pos * theta^(-2i/D), pos = the row's LINKED position (its place in the
// concatenated sequence), so recomputed chunk tokens see their non-initial
// positions (Sec. 4.2).  Angles are formed in float64: in float32,
// pos * inv_freq at pos ~ 1e5 would be off by ~1e-2 rad.
#include <cmath>

#include "device_common.h"
#include "kernels.h"

namespace epic {

namespace {

constexpr int kNormThreads = 256;

__device__ __forceinline__ float block_sum(float v, float* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float s = 0.0f;
#pragma unroll
  for (int w = 0; w < kNormThreads / 64; ++w) s += red[w];
  return s;
}

// One workgroup per row; hidden % 4 == 0.  out_bf16 or out_f32 receives the row.
__global__ __launch_bounds__(kNormThreads) void rmsnorm_kernel(const float* __restrict__ x, const uint16_t* __restrict__ w,
                                                               uint16_t* __restrict__ out_bf16,
                                                               float* __restrict__ out_f32, int hidden, float eps) {
  // The row stays in registers between the two passes (up to kKeep float4 per
  // thread, hidden <= 8192 at 256 threads); a longer row is read again.  The kept
  // part's loads, and its weights, are issued together from clamped indices (no
  // branch between them, so one wait covers them all); slots past the row add an
  // exact 0 to the sum of squares, which leaves it as the in-order sum of the row.
  constexpr int kKeep = 8;
  __shared__ float red[kNormThreads / 64];
  const int row = blockIdx.x;
  const float4* xr = reinterpret_cast<const float4*>(x + size_t(row) * hidden);
  const int n4 = hidden / 4;
  float4 keep[kKeep];
  uint2 keep_w[kKeep];
#pragma unroll
  for (int k = 0; k < kKeep; ++k) {
    const int i = min(int(threadIdx.x) + k * kNormThreads, n4 - 1);
    keep[k] = xr[i];
    keep_w[k] = *reinterpret_cast<const uint2*>(w + 4 * i);
  }
  float ss = 0.0f;
#pragma unroll
  for (int k = 0; k < kKeep; ++k) {
    const float sq = keep[k].x * keep[k].x + keep[k].y * keep[k].y + keep[k].z * keep[k].z + keep[k].w * keep[k].w;
    ss += int(threadIdx.x) + k * kNormThreads < n4 ? sq : 0.0f;
  }
  for (int i = threadIdx.x + kKeep * kNormThreads; i < n4; i += kNormThreads) {
    const float4 v = xr[i];
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float total = block_sum(ss, red);
  const float inv = 1.0f / sqrtf(total / float(hidden) + eps);
  auto put = [&](int i, const float4& v, const uint2& wb) {
    const float y0 = v.x * inv * bf16_to_f32(uint16_t(wb.x & 0xFFFFu));
    const float y1 = v.y * inv * bf16_to_f32(uint16_t(wb.x >> 16));
    const float y2 = v.z * inv * bf16_to_f32(uint16_t(wb.y & 0xFFFFu));
    const float y3 = v.w * inv * bf16_to_f32(uint16_t(wb.y >> 16));
    if (out_bf16) {
      *reinterpret_cast<uint2*>(out_bf16 + size_t(row) * hidden + 4 * i) =
          make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
    } else {
      *reinterpret_cast<float4*>(out_f32 + size_t(row) * hidden + 4 * i) = make_float4(y0, y1, y2, y3);
    }
  };
#pragma unroll
  for (int k = 0; k < kKeep; ++k) {
    const int i = threadIdx.x + k * kNormThreads;
    if (i < n4) put(i, keep[k], keep_w[k]);
  }
  for (int i = threadIdx.x + kKeep * kNormThreads; i < n4; i += kNormThreads)
    put(i, xr[i], *reinterpret_cast<const uint2*>(w + 4 * i));
}

// cs[row][i] = (cos, sin)(s_pos[row] * theta^(-2i/D)), float64 angle.
__global__ void rope_table_kernel(const int32_t* __restrict__ s_pos, float2* __restrict__ cs, int n_rows, int half_dim,
                                  double log2_theta) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n_rows * half_dim) return;
  const int row = idx / half_dim, i = idx % half_dim;
  const double inv_freq = exp2(-double(2 * i) / double(2 * half_dim) * log2_theta);
  const double ang = double(s_pos[row]) * inv_freq;
  double s, c;
  sincos(ang, &s, &c);
  cs[idx] = make_float2(float(c), float(s));
}

}  // namespace

void launch_rmsnorm(const float* x, const uint16_t* w, uint16_t* out_bf16, float* out_f32, int rows, int hidden,
                    float eps, hipStream_t stream) {
  if (rows == 0) return;
  rmsnorm_kernel<<<rows, kNormThreads, 0, stream>>>(x, w, out_bf16, out_f32, hidden, eps);
}

void launch_rope_table(const int32_t* s_pos, float2* cs, int rows, int head_dim, double theta, hipStream_t stream) {
  const int n = rows * (head_dim / 2);
  if (n == 0) return;
  rope_table_kernel<<<(n + 255) / 256, 256, 0, stream>>>(s_pos, cs, rows, head_dim / 2, std::log2(theta));
}

}  // namespace epic
