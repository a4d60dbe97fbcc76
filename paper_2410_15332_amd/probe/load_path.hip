// Load-path probe: how many bytes per cycle a CU pulls through buffer loads, by
// access shape, prefetch depth and how the data is shared between CUs.  Measurement
// tooling beside the product library (never linked into it).
//
// Every workgroup (one per CU, 8 wavefronts) streams a 4 MB region: 512 rows of
// 8192 bytes (a bf16 operand with K = 4096), one stage of 8 * LPW KB at a time, each
// wavefront issuing LPW 1 KB load instructions per stage.  Stages go through NB LDS
// buffers with one barrier per stage and the loads of a stage issued NB - 1 stages
// ahead of use, as in the GEMM.  Access shapes of one 1 KB load instruction:
//   kRows64  : 16 rows x 64 bytes (half a cache line per row)
//   kRows128 : 8 rows x 128 bytes (one whole line per row)
//   kContig  : 1 KB contiguous
//   kPair    : 16 rows x 64 bytes, the next instruction the other half of the same
//              16 lines (both halves issued back to back)
// kVgpr variants load the same shapes into registers instead of LDS.
// Region of workgroup w: regions > 0 gives each XCD its own `regions` regions
// (w % 8 is taken as the XCD, round-robin dispatch), so 32 / regions CUs of one XCD
// share a region; regions < 0 gives -regions regions shared by all XCDs.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((address_space(3))) void lds_void;
typedef float f32x4 __attribute__((ext_vector_type(4)));
constexpr int kBufWord3 = 0x00020000;
constexpr int kRowBytes = 8192, kRows = 512, kRegion = kRowBytes * kRows;   // 4 MB

enum { kRows64 = 0, kRows128 = 1, kContig = 2, kPair = 3 };

template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}
__device__ __forceinline__ void barrier_lds() { __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, char* dst, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 16, voff, 0, 0, 0);
}

// Byte offset in the region of lane `lane` of load instruction i of wavefront v in
// stage s (stage = 8 * LPW KB; a pass over the region is 4 MB / stage bytes stages,
// and every 16-byte unit of the region is loaded once per pass).
template <int LPW, int PAT>
__device__ __forceinline__ int offset(int s, int v, int i, int lane) {
  constexpr int kStage = 8 * LPW * 1024;
  constexpr int kStageRows = kStage / 128;             // rows per stage at 128 bytes per row
  const int g = v * LPW + i;                           // 1 KB unit of the stage
  if constexpr (PAT == kContig) return s * kStage + g * 1024 + lane * 16;
  if constexpr (PAT == kRows64) {                      // 64-byte half rows: twice the rows, half the width
    constexpr int kHalfRows = kStage / 64;
    const int rb = s % (kRows / kHalfRows), kk = s / (kRows / kHalfRows);
    return (rb * kHalfRows + g * 16 + (lane >> 2)) * kRowBytes + kk * 64 + (lane & 3) * 16;
  }
  const int rb = s % (kRows / kStageRows), kk = s / (kRows / kStageRows);
  if constexpr (PAT == kRows128) return (rb * kStageRows + g * 8 + (lane >> 3)) * kRowBytes + kk * 128 + (lane & 7) * 16;
  return (rb * kStageRows + (g >> 1) * 16 + (lane >> 2)) * kRowBytes + kk * 128 + (g & 1) * 64 + (lane & 3) * 16;
}

template <int NB, int LPW>
struct ProbeLds {
  char b[NB][8 * LPW * 1024];
};

template <int NB, int LPW, int PAT, bool VGPR>
__global__ __launch_bounds__(512, 1) void load_path_kernel(const char* src, int regions, int steps, float* sink) {
  constexpr int kStages = kRegion / (8 * LPW * 1024);  // stages per pass over the region
  const int w = blockIdx.x, lane = threadIdx.x & 63;
  const int v = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int region = regions > 0 ? (w % 8) * regions + (w / 8) % regions : (w / 8) % (-regions);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(src) + size_t(region) * kRegion, 0, kRegion, kBufWord3);
  float x = 0.0f;
  if constexpr (!VGPR) {
    __shared__ __attribute__((aligned(1024))) ProbeLds<NB, LPW> sh;
    for (int s = 0; s < NB; ++s)
#pragma unroll
      for (int i = 0; i < LPW; ++i) dma16(rs, sh.b[s] + (v * LPW + i) * 1024, offset<LPW, PAT>(s % kStages, v, i, lane));
    for (int s = 0; s < steps; ++s) {
      wait_vmem<(NB - 1) * LPW>();                     // stage s of this wavefront
      barrier_lds();                                   // ... of every wavefront; buffer s % NB free
      const int t = (s + NB) % kStages;
#pragma unroll
      for (int i = 0; i < LPW; ++i) dma16(rs, sh.b[s % NB] + (v * LPW + i) * 1024, offset<LPW, PAT>(t, v, i, lane));
    }
    wait_vmem<0>();
    barrier_lds();
    x = *reinterpret_cast<const float*>(sh.b[0] + threadIdx.x * 4);
  } else {
    static_assert(NB == 4, "register variants keep four stages");
    f32x4 r[4][LPW];
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int i = 0; i < LPW; ++i)
        r[s][i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, offset<LPW, PAT>(s, v, i, lane), 0, 0));
    for (int s = 0; s < steps; s += 4) {
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        wait_vmem<3 * LPW>();
#pragma unroll
        for (int i = 0; i < LPW; ++i) acc += r[b][i];
        const int t = (s + b + 4) % kStages;
#pragma unroll
        for (int i = 0; i < LPW; ++i)
          r[b][i] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, offset<LPW, PAT>(t, v, i, lane), 0, 0));
      }
    }
    wait_vmem<0>();
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int i = 0; i < LPW; ++i) acc += r[b][i];
    x = acc[0] + acc[1] + acc[2] + acc[3];
  }
  if (x == 1234.5f) sink[w] = x;                       // keeps the loads; never true for the probe's data
}

struct Variant {
  int nb, lpw, pat, vgpr;
};
constexpr Variant kVariants[] = {
    {4, 4, kRows64, 0}, {4, 4, kRows128, 0}, {4, 4, kContig, 0}, {4, 4, kPair, 0},   // 0..3 shape
    {4, 4, kRows64, 1}, {4, 4, kRows128, 1},                                        // 4..5 into registers
    {2, 2, kRows128, 0}, {2, 4, kRows128, 0}, {2, 8, kRows128, 0}, {1, 8, kRows128, 0},   // 6..9 depth
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

template <int NB, int LPW, int PAT, bool VGPR>
void launch(const void* src, int regions, int steps, float* sink, hipStream_t st) {
  load_path_kernel<NB, LPW, PAT, VGPR><<<256, 512, 0, st>>>(static_cast<const char*>(src), regions, steps, sink);
}

}  // namespace

// Stage bytes of a variant (per workgroup), or -1 if there is no such variant.
extern "C" int epic_probe_load_path_stage_bytes(int variant) {
  if (variant < 0 || variant >= kNumVariants) return -1;
  return 8 * kVariants[variant].lpw * 1024;
}

// Run variant `variant` on 256 workgroups for `steps` stages each (a multiple of 4).
// src: device buffer of at least 8 * regions * 4 MB (regions > 0) or -regions * 4 MB
// bytes (regions < 0); sink: 256 floats of device memory (written only for data the
// probe never sees).  Returns 0 after the enqueue, nonzero on a bad argument.
extern "C" int epic_probe_load_path(int variant, const void* src, size_t src_bytes, int regions, int steps,
                                    float* sink, void* stream) {
  if (variant < 0 || variant >= kNumVariants || src == nullptr || sink == nullptr) return 1;
  if (regions == 0 || regions > 32 || regions < -256 || steps <= 0 || steps % 4 != 0) return 2;
  const size_t need = size_t(regions > 0 ? 8 * regions : -regions) * kRegion;
  if (src_bytes < need) return 3;
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (variant) {
    case 0: launch<4, 4, kRows64, false>(src, regions, steps, sink, st); break;
    case 1: launch<4, 4, kRows128, false>(src, regions, steps, sink, st); break;
    case 2: launch<4, 4, kContig, false>(src, regions, steps, sink, st); break;
    case 3: launch<4, 4, kPair, false>(src, regions, steps, sink, st); break;
    case 4: launch<4, 4, kRows64, true>(src, regions, steps, sink, st); break;
    case 5: launch<4, 4, kRows128, true>(src, regions, steps, sink, st); break;
    case 6: launch<2, 2, kRows128, false>(src, regions, steps, sink, st); break;
    case 7: launch<2, 4, kRows128, false>(src, regions, steps, sink, st); break;
    case 8: launch<2, 8, kRows128, false>(src, regions, steps, sink, st); break;
    default: launch<1, 8, kRows128, false>(src, regions, steps, sink, st); break;
  }
  return hipGetLastError() == hipSuccess ? 0 : 4;
}
