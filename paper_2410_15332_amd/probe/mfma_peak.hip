// Matrix-core throughput probe (measurement tooling, not part of the link step):
// every wavefront issues independent v_mfma_f32_32x32x16_bf16 back to back, so the
// launch time gives the bf16 MFMA rate this chip sustains (its clock under a pure
// MFMA load included), a second denominator beside the published dense peak.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef short bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int kChains = 4;    // independent accumulators per wavefront

__global__ __launch_bounds__(512) void mfma_peak_kernel(float* out, int iters) {
  const int t = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {          // small bf16 values (exponent 2^-10), so sums stay finite
    a[i] = short(0x3A80 + ((t + i) & 15));
    b[i] = short(0x3A80 + ((t * 3 + i) & 15));
  }
  f32x16 c[kChains];
#pragma unroll
  for (int k = 0; k < kChains; ++k) c[k] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < kChains; ++k) c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c[k], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kChains; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[k][r];
  out[size_t(blockIdx.x) * blockDim.x + t] = s;   // keeps the products live
}

}  // namespace

// out: device buffer of n_blocks * 512 floats.  Launches n_blocks workgroups of 8
// wavefronts, each wavefront iters x 4 MFMAs of 32 x 32 x 16 (2 * 16384 flops each).
// Returns 0, or the HIP error code of the launch.
extern "C" int epic_probe_mfma_bf16(float* out, int n_blocks, int iters, void* stream) {
  if (out == nullptr || n_blocks <= 0 || iters <= 0) return int(hipErrorInvalidValue);
  mfma_peak_kernel<<<dim3(unsigned(n_blocks)), 512, 0, static_cast<hipStream_t>(stream)>>>(out, iters);
  return int(hipGetLastError());
}

// Flops of one launch.
extern "C" double epic_probe_mfma_bf16_flops(int n_blocks, int iters) {
  return double(n_blocks) * 8.0 * double(iters) * kChains * 2.0 * 32 * 32 * 16;
}
