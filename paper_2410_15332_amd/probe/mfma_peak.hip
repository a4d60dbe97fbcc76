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

// lowbias32 integer hash (Wellons' published constants): well-mixed operand bits
__device__ inline uint32_t mix32(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352du;
  x ^= x >> 15;
  x *= 0x846ca68bu;
  x ^= x >> 16;
  return x;
}

// kVaried = false: one fixed operand pair per lane (small bf16 values, only the low
// mantissa bits differ between lanes).  kVaried = true: eight A and eight B fragments
// per lane with hashed signs and mantissas (exponent fixed at 2^-11, so sums stay
// finite), cycled so that every MFMA of a chain sees new operand bits, as matrix
// products of real data do; iters is then a multiple of 8.
template <bool kVaried>
__global__ __launch_bounds__(512) void mfma_peak_kernel(float* out, int iters) {
  const int t = threadIdx.x;
  constexpr int NF = kVaried ? 8 : 1;
  bf16x8 a[NF], b[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (kVaried) {
        const uint32_t id = ((blockIdx.x * 512u + unsigned(t)) * 16u + unsigned(f)) * 8u + unsigned(i);
        const uint32_t h = mix32(id);
        a[f][i] = short(0x3A00 | (h & 0x807Fu));
        b[f][i] = short(0x3A00 | ((h >> 16) & 0x807Fu));
      } else {                           // small bf16 values (exponent 2^-10), so sums stay finite
        a[f][i] = short(0x3A80 + ((t + i) & 15));
        b[f][i] = short(0x3A80 + ((t * 3 + i) & 15));
      }
    }
  f32x16 c[kChains];
#pragma unroll
  for (int k = 0; k < kChains; ++k) c[k] = f32x16{};
  for (int it = 0; it < iters; it += NF) {
#pragma unroll
    for (int u = 0; u < NF; ++u)
#pragma unroll
      for (int k = 0; k < kChains; ++k)
        c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(u + k) % NF], b[(u + 3 * k) % NF], c[k], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int k = 0; k < kChains; ++k)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[k][r];
  out[size_t(blockIdx.x) * blockDim.x + t] = s;   // keeps the products live
}

// Streaming-read probe: every thread reads 16-byte words at a grid stride, four
// loads in flight per trip, and folds them into one word per workgroup.
__global__ __launch_bounds__(256) void hbm_read_kernel(const uint4* src, size_t n16, uint32_t* out) {
  const size_t stride = size_t(gridDim.x) * 256;
  size_t i = size_t(blockIdx.x) * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = src[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  __shared__ uint32_t red[256];
  red[threadIdx.x] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = 0;
    for (int t = 0; t < 256; ++t) x ^= red[t];
    out[blockIdx.x] = x;                  // keeps the loads live
  }
}

}  // namespace

// out: device buffer of n_blocks * 512 floats.  Launches n_blocks workgroups of 8
// wavefronts, each wavefront iters x 4 MFMAs of 32 x 32 x 16 (2 * 16384 flops each).
// Returns 0, or the HIP error code of the launch.
extern "C" int epic_probe_mfma_bf16(float* out, int n_blocks, int iters, void* stream) {
  if (out == nullptr || n_blocks <= 0 || iters <= 0) return int(hipErrorInvalidValue);
  mfma_peak_kernel<false><<<dim3(unsigned(n_blocks)), 512, 0, static_cast<hipStream_t>(stream)>>>(out, iters);
  return int(hipGetLastError());
}

// The same launch with operands whose bits change from one MFMA to the next (see
// mfma_peak_kernel<true>); iters must be a positive multiple of 8.
extern "C" int epic_probe_mfma_bf16_varied(float* out, int n_blocks, int iters, void* stream) {
  if (out == nullptr || n_blocks <= 0 || iters <= 0 || iters % 8 != 0) return int(hipErrorInvalidValue);
  mfma_peak_kernel<true><<<dim3(unsigned(n_blocks)), 512, 0, static_cast<hipStream_t>(stream)>>>(out, iters);
  return int(hipGetLastError());
}

// Flops of one launch.
extern "C" double epic_probe_mfma_bf16_flops(int n_blocks, int iters) {
  return double(n_blocks) * 8.0 * double(iters) * kChains * 2.0 * 32 * 32 * 16;
}

// src: device buffer of `bytes` bytes (a multiple of 16); out: n_blocks words.
// Launches n_blocks workgroups of 256 threads that read the whole buffer once.
extern "C" int epic_probe_hbm_read(const void* src, size_t bytes, uint32_t* out, int n_blocks, void* stream) {
  if (src == nullptr || out == nullptr || n_blocks <= 0 || bytes == 0 || bytes % 16 != 0)
    return int(hipErrorInvalidValue);
  hbm_read_kernel<<<dim3(unsigned(n_blocks)), 256, 0, static_cast<hipStream_t>(stream)>>>(
      static_cast<const uint4*>(src), bytes / 16, out);
  return int(hipGetLastError());
}
