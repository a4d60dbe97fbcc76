// Co-execution probe (measurement tooling, not part of the link step): how much
// vector-ALU work the matrix cores hide.  Each iteration of a wavefront issues 8
// MFMA slots.  A slot is one v_mfma_f32_32x32x16_bf16 followed by NV / 8
// independent vector instructions of one kind (v_fma_f32, v_exp_f32 or a pair of
// v_max_f32), and a full scheduling barrier closes it, so the compiler can neither
// cluster the vector work of several slots nor move it past an MFMA.  Variants:
//   mode 0: no MFMA (the vector work alone);
//   mode 1: accumulators where the compiler puts them (the AGPRs here), 4 chains;
//   mode 2: accumulators forced into VGPRs (the MFMA written as inline assembly), 4 chains;
//   mode 3 / 4: as mode 1 with 2 / 1 chains (each MFMA accumulates onto the result of
//   the MFMA 2 / 1 slots earlier).
// One workgroup of 4 wavefronts per CU gives one wavefront per SIMD, two workgroups
// per CU give two.  The kernel times itself with the shader clock (s_memtime) and the
// 100 MHz real-time counter, so the output is cycles per iteration and the engine clock.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8v __attribute__((ext_vector_type(8)));
typedef float f32x16v __attribute__((ext_vector_type(16)));

namespace {

constexpr int kIters = 4096;

template <int NV, int KIND, int MODE>
__global__ __launch_bounds__(256) void coexec_kernel(float* out, long long* cyc) {
  constexpr int NA = MODE == 3 ? 2 : MODE == 4 ? 1 : 4;   // independent accumulator chains
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
      if constexpr (MODE == 2)
        __asm__ volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc[j % NA]) : "v"(a), "v"(b));
      else if constexpr (MODE != 0)
        acc[j % NA] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j % NA], 0, 0, 0);
#pragma unroll
      for (int v = 0; v < NV / 8; ++v) {
        const int k = (j * (NV / 8) + v) & 63;
        if (KIND == 0) x[k] = __builtin_fmaf(x[k], 0.5f, 0.25f);
        else if (KIND == 1) x[k] = __builtin_amdgcn_exp2f(x[k]);
        else x[k] = __builtin_fmaxf(__builtin_fmaxf(x[k], x[(k + 1) & 63]), 0.3f);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const long long t1 = __builtin_amdgcn_s_memtime();
  const long long r1 = __builtin_amdgcn_s_memrealtime();
  // the compiler does not see the inline-assembly MFMA's result latency: wait it out
  // before the vector reads below
  if constexpr (MODE == 2) __asm__ volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
  float r = 0.0f;
#pragma unroll
  for (int i = 0; i < 64; ++i) r += x[i];
#pragma unroll
  for (int j = 0; j < NA; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) r += acc[j][i];
  out[blockIdx.x * 256 + tid] = r;
  if ((tid & 63) == 0) {
    cyc[2 * (blockIdx.x * 4 + (tid >> 6))] = t1 - t0;
    cyc[2 * (blockIdx.x * 4 + (tid >> 6)) + 1] = r1 - r0;
  }
}

template <int NV, int KIND, int MODE>
void launch(int blocks, float* out, long long* cyc, hipStream_t s) {
  coexec_kernel<NV, KIND, MODE><<<blocks, 256, 0, s>>>(out, cyc);
}

}  // namespace

// Variants (mode, nv, kind): mode as above; kind 0 = fma, 1 = exp, 2 = max.  out:
// blocks x 256 floats; cyc: blocks x 4 x 2 counters (shader cycles, real-time ticks
// per wavefront).  Returns 0, 1 for an unknown variant or missing buffers, else the
// HIP error.
extern "C" int epic_probe_coexec(int mode, int nv, int kind, int blocks, float* out, long long* cyc, void* stream) {
  if (out == nullptr || cyc == nullptr || blocks <= 0) return 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  switch (mode * 1000 + nv * 10 + kind) {
#define EPIC_COEXEC_VARIANT(M, NV, K) \
  case M * 1000 + NV * 10 + K: launch<NV, K, M>(blocks, out, cyc, s); break;
    EPIC_COEXEC_VARIANT(0, 32, 0) EPIC_COEXEC_VARIANT(0, 32, 1) EPIC_COEXEC_VARIANT(0, 32, 2)
    EPIC_COEXEC_VARIANT(1, 0, 0) EPIC_COEXEC_VARIANT(1, 16, 0) EPIC_COEXEC_VARIANT(1, 32, 0)
    EPIC_COEXEC_VARIANT(1, 48, 0) EPIC_COEXEC_VARIANT(1, 64, 0)
    EPIC_COEXEC_VARIANT(1, 8, 1) EPIC_COEXEC_VARIANT(1, 16, 1) EPIC_COEXEC_VARIANT(1, 32, 1)
    EPIC_COEXEC_VARIANT(1, 16, 2) EPIC_COEXEC_VARIANT(1, 32, 2)
    EPIC_COEXEC_VARIANT(2, 0, 0) EPIC_COEXEC_VARIANT(2, 32, 0) EPIC_COEXEC_VARIANT(2, 48, 0)
    EPIC_COEXEC_VARIANT(2, 16, 1) EPIC_COEXEC_VARIANT(2, 32, 1)
    EPIC_COEXEC_VARIANT(3, 0, 0) EPIC_COEXEC_VARIANT(3, 32, 0)
    EPIC_COEXEC_VARIANT(4, 0, 0) EPIC_COEXEC_VARIANT(4, 32, 0)
#undef EPIC_COEXEC_VARIANT
    default: return 1;
  }
  return int(hipGetLastError());
}

extern "C" int epic_probe_coexec_iters(void) { return kIters; }
