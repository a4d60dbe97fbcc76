// Co-execution probe (measurement tooling, not part of the link step): how much
// vector-ALU work the matrix cores hide.  Each iteration of a wavefront issues 8
// v_mfma_f32_32x32x16_bf16 (4 independent accumulators) and, after each, NV / 8
// independent vector instructions of one kind (v_fma_f32, v_exp_f32 or a pair of
// v_max_f32), pinned to that slot; variants without the MFMAs give the cost of the
// vector work alone.  One workgroup of 4 wavefronts per CU gives one wavefront per
// SIMD, two workgroups per CU give two.  The kernel times itself with the shader
// clock (s_memtime) and the 100 MHz real-time counter, so the output is cycles per
// iteration and the engine clock.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef float f32x16v __attribute__((ext_vector_type(16)));

namespace {

constexpr int kIters = 4096;

template <int NV, int KIND, bool MF>
__global__ __launch_bounds__(256) void coexec_kernel(float* out, long long* cyc) {
  const int tid = threadIdx.x;
  float x[64];
#pragma unroll
  for (int i = 0; i < 64; ++i) x[i] = float((tid + i) % 17) * 0.01f;
  f32x16v acc[4] = {};
  bf16x8v a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(x[i] * 1e-3f);
    b[i] = (__bf16)(x[8 + i] * 1e-3f);
  }
  const long long t0 = __builtin_amdgcn_s_memtime();
  const long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < kIters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (MF) acc[j & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j & 3], 0, 0, 0);
#pragma unroll
      for (int v = 0; v < NV / 8; ++v) {
        const int k = (j * (NV / 8) + v) & 63;
        if (KIND == 0) x[k] = __builtin_fmaf(x[k], 0.5f, 0.25f);
        else if (KIND == 1) x[k] = __builtin_amdgcn_exp2f(x[k]);
        else x[k] = __builtin_fmaxf(__builtin_fmaxf(x[k], x[(k + 1) & 63]), 0.3f);
      }
      if (MF) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);          // the MFMA, then
      if (NV / 8) __builtin_amdgcn_sched_group_barrier(0x002, NV / 8, 0); // its vector ops
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  const long long t1 = __builtin_amdgcn_s_memtime();
  const long long r1 = __builtin_amdgcn_s_memrealtime();
  float r = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) r += x[i];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) r += acc[j][i];
  out[blockIdx.x * 256 + tid] = r;
  if ((tid & 63) == 0) {
    cyc[2 * (blockIdx.x * 4 + (tid >> 6))] = t1 - t0;
    cyc[2 * (blockIdx.x * 4 + (tid >> 6)) + 1] = r1 - r0;
  }
}

template <int NV, int KIND, bool MF>
void launch(int blocks, float* out, long long* cyc, hipStream_t s) {
  coexec_kernel<NV, KIND, MF><<<blocks, 256, 0, s>>>(out, cyc);
}

}  // namespace

// Variants (mfma, nv, kind): kind 0 = fma, 1 = exp, 2 = max.  out: blocks x 256
// floats; cyc: blocks x 4 x 2 counters (shader cycles, real-time ticks per wavefront).
// Returns 0, 1 for an unknown variant or missing buffers, else the HIP error.
extern "C" int epic_probe_coexec(int mfma, int nv, int kind, int blocks, float* out, long long* cyc, void* stream) {
  if (out == nullptr || cyc == nullptr || blocks <= 0) return 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int key = (mfma ? 1000 : 0) + nv * 10 + kind;
  switch (key) {
    case 1000: launch<0, 0, true>(blocks, out, cyc, s); break;
    case 320: launch<32, 0, false>(blocks, out, cyc, s); break;
    case 321: launch<32, 1, false>(blocks, out, cyc, s); break;
    case 322: launch<32, 2, false>(blocks, out, cyc, s); break;
    case 1160: launch<16, 0, true>(blocks, out, cyc, s); break;
    case 1320: launch<32, 0, true>(blocks, out, cyc, s); break;
    case 1480: launch<48, 0, true>(blocks, out, cyc, s); break;
    case 1640: launch<64, 0, true>(blocks, out, cyc, s); break;
    case 1161: launch<16, 1, true>(blocks, out, cyc, s); break;
    case 1321: launch<32, 1, true>(blocks, out, cyc, s); break;
    case 1481: launch<48, 1, true>(blocks, out, cyc, s); break;
    default: return 1;
  }
  return int(hipGetLastError());
}

extern "C" int epic_probe_coexec_iters(void) { return kIters; }
