// Row-set GEMMs of the link step on MFMA: C[M x N] = A[M x K] . W[N x K]^T.
//
// A holds the selected rows' activations (bf16, K contiguous), W a weight
// matrix in [out][in] layout (bf16), so both MFMA operands are read along K.
// Epilogues are fused:
//   kStoreF32 : C -> fp32 [M][N]                     (Q/K/V projections, Sec. 4.2)
//   kResidual : h[M][N] += C                         (W_O and W_down; fp32 residual stream)
//   kSwiGLU   : act[M][N/2] = silu(gate) * up, bf16  (W_gate_up; gate rows [0, F), up rows [F, 2F))
//
// Tiling: 256 threads = 4 wavefronts, workgroup tile 128 x 128 (or 128 x 64 for
// narrow outputs), each wavefront 64 x 64 (64 x 32) as 2 x 2 (2 x 1)
// v_mfma_f32_32x32x16_bf16 tiles, K in steps of 64 staged in
// LDS (rows padded to 144 bytes so the 16 rows one ds_read_b128 pass touches
// fall in distinct banks).  Global loads run two K steps ahead through two
// register stages, so each load has two steps of MFMA work to arrive.  Tiles
// are ordered so that the M tiles sharing one weight tile are launched together
// on one XCD (workgroups are dealt round-robin to the 8 XCDs), which then reads
// that weight tile from HBM once and from its L2 afterwards.  For kSwiGLU the
// 128 weight rows of a tile are gate/up in 32-row groups (gate j.., up j..,
// gate j+32.., up j+32..), so each wavefront's two 32-column MFMA tiles hold
// gate and up of the same 32 outputs in the same registers.
// Rows past M are computed from a clamped row and never stored.
#include "device_common.h"
#include "kernels.h"

namespace epic {

namespace {

constexpr int kBM = 128, kBK = 64;
constexpr int kLdsRow = kBK + 8;   // elements per LDS row (144 bytes)
constexpr int kGemmThreads = 256;
constexpr int kChunks = kBM * kBK / 8 / kGemmThreads;   // 16-byte A chunks per thread (4)

// kBN = 128 (wavefront tile 64 x 64) or 64 (64 x 32, for narrow outputs whose
// 128-wide tiles would leave CUs idle).
template <int EPI, int kBN>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_kernel(GemmArgs g) {
  constexpr int NJ = kBN / 64;                          // 32-column MFMA tiles per wavefront
  constexpr int kBChunks = kBN * kBK / 8 / kGemmThreads; // 16-byte B chunks per thread
  __shared__ __attribute__((aligned(16))) uint16_t lds_a[2][kBM * kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t lds_b[2][kBN * kLdsRow];

  const int m_tiles = (g.M + kBM - 1) / kBM;
  const int n_tiles = EPI == kSwiGLU ? g.ffn / 64 : g.N / kBN;
  const int total = m_tiles * n_tiles;
  int tile_id = blockIdx.x;
  if (total % 8 == 0) tile_id = (blockIdx.x % 8) * (total / 8) + blockIdx.x / 8;   // XCD-contiguous ranges
  const int mt = tile_id % m_tiles;
  const int nt = tile_id / m_tiles;
  const int m0 = mt * kBM;
  const int tid = threadIdx.x & (kGemmThreads - 1);
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int col = lane & 31, half = lane >> 5;

  // weight row of tile column c
  auto wrow = [&](int c) -> int {
    if constexpr (EPI == kSwiGLU) {
      const int grp = c >> 5;                // 0: gate, 1: up, 2: gate, 3: up
      return (grp & 1) * g.ffn + nt * 64 + (grp >> 1) * 32 + (c & 31);
    } else {
      return nt * kBN + c;
    }
  };

  // global -> register staging: chunk i of a thread = row ld_row + 32 i, 8 k at ld_kc
  const int ld_row = tid >> 3, ld_kc = (tid & 7) * 8;
  const uint16_t* a_ptr[kChunks];
  const uint16_t* b_ptr[kBChunks];
#pragma unroll
  for (int i = 0; i < kChunks; ++i) a_ptr[i] = g.A + size_t(min(m0 + ld_row + 32 * i, g.M - 1)) * g.K + ld_kc;
#pragma unroll
  for (int i = 0; i < kBChunks; ++i) b_ptr[i] = g.W + size_t(wrow(ld_row + 32 * i)) * g.K + ld_kc;
  typedef uint32_t stage_t __attribute__((ext_vector_type(4 * (kChunks + kBChunks))));   // A then B chunks
  stage_t st0, st1;
  auto load = [&](int kt, stage_t& st) {
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
      const uint4 a = *reinterpret_cast<const uint4*>(a_ptr[i] + kt * kBK);
      st[4 * i + 0] = a.x; st[4 * i + 1] = a.y; st[4 * i + 2] = a.z; st[4 * i + 3] = a.w;
    }
#pragma unroll
    for (int i = 0; i < kBChunks; ++i) {
      const uint4 b = *reinterpret_cast<const uint4*>(b_ptr[i] + kt * kBK);
      st[4 * kChunks + 4 * i + 0] = b.x; st[4 * kChunks + 4 * i + 1] = b.y;
      st[4 * kChunks + 4 * i + 2] = b.z; st[4 * kChunks + 4 * i + 3] = b.w;
    }
  };
  auto store = [&](int buf, const stage_t& st) {
#pragma unroll
    for (int i = 0; i < kChunks; ++i)
      *reinterpret_cast<uint4*>(&lds_a[buf][(ld_row + 32 * i) * kLdsRow + ld_kc]) =
          make_uint4(st[4 * i + 0], st[4 * i + 1], st[4 * i + 2], st[4 * i + 3]);
#pragma unroll
    for (int i = 0; i < kBChunks; ++i)
      *reinterpret_cast<uint4*>(&lds_b[buf][(ld_row + 32 * i) * kLdsRow + ld_kc]) =
          make_uint4(st[4 * kChunks + 4 * i + 0], st[4 * kChunks + 4 * i + 1], st[4 * kChunks + 4 * i + 2],
                     st[4 * kChunks + 4 * i + 3]);
  };

  f32x16 acc[2][NJ];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x16{};

  auto compute = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      bf16x8 af[2], bfr[NJ];
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&lds_a[buf][(wm * 64 + i * 32 + col) * kLdsRow + ks * 16 + half * 8]);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(
            &lds_b[buf][(wn * (kBN / 2) + j * 32 + col) * kLdsRow + ks * 16 + half * 8]);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[i][j] = mfma_32x32x16(af[i], bfr[j], acc[i][j]);
    }
  };

  // Pipeline: LDS buffer kt % 2 holds step kt; registers carry steps kt + 1 and kt + 2.
  const int nk = g.K / kBK;
  load(0, st0);
  store(0, st0);
  if (nk > 1) load(1, st0);
  if (nk > 2) load(2, st1);
  __syncthreads();
  for (int kt = 0; kt < nk; kt += 2) {
    compute(0);                                // step kt
    if (kt + 1 < nk) {
      store(1, st0);                           // step kt + 1
      if (kt + 3 < nk) load(kt + 3, st0);
    }
    __syncthreads();
    if (kt + 1 >= nk) break;
    compute(1);                                // step kt + 1
    if (kt + 2 < nk) {
      store(0, st1);                           // step kt + 2
      if (kt + 4 < nk) load(kt + 4, st1);
    }
    __syncthreads();
  }

  // Epilogue.  acc[i][j] register r: row wm*64 + i*32 + (r/4)*8 + half*4 + r%4,
  // column wn*(kBN/2) + j*32 + col.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + half * 4 + (r & 3);
      if (m >= g.M) continue;
      if constexpr (EPI == kSwiGLU) {
        const float gt = acc[i][0][r], up = acc[i][1][r];
        const float act = gt / (1.0f + __expf(-gt)) * up;
        const int n = nt * 64 + wn * 32 + col;
        g.act[size_t(m) * g.ffn + n] = uint16_t(pack_bf16x2(act, 0.0f) & 0xFFFFu);
      } else {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          const int n = nt * kBN + wn * (kBN / 2) + j * 32 + col;
          if constexpr (EPI == kStoreF32)
            g.C[size_t(m) * g.N + n] = acc[i][j][r];
          else
            g.C[size_t(m) * g.N + n] += acc[i][j][r];
        }
      }
    }
}

}  // namespace

void launch_gemm(const GemmArgs& g, int epi, hipStream_t stream) {
  if (g.M == 0) return;
  const int m_tiles = (g.M + kBM - 1) / kBM;
  if (epi == kSwiGLU) {
    gemm_kernel<kSwiGLU, 128><<<dim3(unsigned(m_tiles) * unsigned(g.ffn / 64)), kGemmThreads, 0, stream>>>(g);
    return;
  }
  // narrow outputs: 64-column tiles when 128-column ones would not give every CU a tile
  const bool narrow = int64_t(m_tiles) * (g.N / 128) < 256;
  const dim3 grid(unsigned(m_tiles) * unsigned(g.N / (narrow ? 64 : 128)));
  if (epi == kStoreF32) {
    if (narrow) gemm_kernel<kStoreF32, 64><<<grid, kGemmThreads, 0, stream>>>(g);
    else gemm_kernel<kStoreF32, 128><<<grid, kGemmThreads, 0, stream>>>(g);
  } else {
    if (narrow) gemm_kernel<kResidual, 64><<<grid, kGemmThreads, 0, stream>>>(g);
    else gemm_kernel<kResidual, 128><<<grid, kGemmThreads, 0, stream>>>(g);
  }
}

}  // namespace epic
