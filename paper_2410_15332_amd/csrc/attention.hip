// Scattered-query causal attention over the paged linked cache (Eq. 1).
//
// Each S row at linked position p, query head h, attends to the linked keys at
// positions <= p of KV head h / G (MASK of Eq. 1, read as additive -inf with the
// diagonal included), scale 1/sqrt(D).  The linked cache is a list of blocks
// (physical id, first position, valid slots), so chunk caches are read in place
// and recomputed rows come from the private blocks written just before.
//
// Work decomposition (built by the host planner):
//   tile  = 128 query rows = (S rows of one request) x (G query heads of one KV head),
//           row t -> S row t % (128/G), head t / (128/G);
//   item  = (tile, range of linked blocks); rows whose key range spans several
//           items get partial results (O / l, log2 l + m) merged by the combine kernel.
// Grid = items x Hkv with blockIdx % Hkv = KV head: with 8 KV heads each XCD
// (workgroups are dealt round-robin to the 8 XCDs) serves one head, and the
// planner orders items key-segment first, so concurrent workgroups on an XCD
// read the same KV blocks through its L2.
//
// Per workgroup: 4 wavefronts x 32 rows.  Per iteration 64 keys (4 blocks) are
// staged in LDS (double-buffered through registers).  S^T = K Q^T and
// O^T += V^T P^T run on v_mfma_f32_32x32x16_bf16: each lane owns one query row
// (its MFMA column), so the row max / sum need a single lane swap (l <-> l^32).
// P is rounded to bf16 for the second product; softmax runs in base 2 with
// scale*log2(e) applied inside the exponent's FMA; the running output is
// rescaled only when some row's maximum grew; accumulation is fp32.
#include "device_common.h"
#include "kernels.h"

namespace epic {

namespace {

constexpr int kKT = 64;    // keys per iteration (4 blocks of 16)
constexpr int kThreads = 256;

// LDS stage: K as [64 keys][D + 8] (16-byte pad: the 16 rows one ds_read_b128
// pass reads fall in distinct banks); V as the four blocks' [D][16] slabs
// copied as they are, each 32-byte row's two 16-byte halves swapped when bit
// 2 xor bit 3 of the row index is set, so that 16 consecutive rows read at the
// same half hit distinct banks.
template <int D>
struct AttnLds {
  static constexpr int KS = D + 8;
  uint16_t k[2][kKT * KS];
  uint16_t v[2][4 * D * 16];
};

__device__ __forceinline__ int v_swz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

// S^T row rho (0..31 inside a 32-key subtile) holds key (rho>>4)*16 + ((rho>>2)&1)*8 + ((rho>>3)&1)*4 + (rho&3).
// With this order a lane's accumulator registers 8*st .. 8*st+7 hold the 8
// consecutive keys st*16 + half*8 + [0, 8): exactly the B operand of the PV step
// over those 16 keys, and the matching V^T operand is one 16-byte read.
__device__ __forceinline__ int srow_key(int rho) {
  return (rho >> 4) * 16 + ((rho >> 2) & 1) * 8 + ((rho >> 3) & 1) * 4 + (rho & 3);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void link_attention_kernel(AttnArgs a) {
  constexpr int NDS = D / 16;                 // k-steps of S^T = K Q^T
  constexpr int NDT = D / 32;                 // 32-row tiles of O^T
  constexpr int CH = kKT * D / 8 / kThreads;  // 16-byte chunks per thread per operand
  constexpr int KS = AttnLds<D>::KS;
  __shared__ __attribute__((aligned(16))) AttnLds<D> lds;

  const int hkv = a.hkv;
  const int g = blockIdx.x % hkv;
  const int item = blockIdx.x / hkv;
  const int tile = a.work[4 * item + 0];
  const int b0 = a.work[4 * item + 1];
  const int b1 = a.work[4 * item + 2];
  const int part = a.work[4 * item + 3];
  const int row0 = a.tiles[4 * tile + 0];
  const int nrows = a.tiles[4 * tile + 1];
  const int32_t* __restrict__ lblk = a.linked_blocks;
  const int32_t* __restrict__ bpos = a.block_pos0;
  const int32_t* __restrict__ blenp = a.block_len;

  const int tid = threadIdx.x & (kThreads - 1);   // blockDim.x == kThreads
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;
  const int t = wave * 32 + col;               // tile row of this lane
  const int R = a.rows_per_tile;
  const int srl = t % R, h = g * a.G + t / R;
  const bool row_ok = srl < nrows;
  const int srow = row0 + (row_ok ? srl : nrows - 1);
  const int qpos = a.s_pos[srow];
  const int min_qpos = a.s_pos[row0];          // S rows ascend within a request

  bf16x8 qreg[NDS];
  {
    const uint16_t* qp = a.q + (size_t(srow) * a.hq + h) * D + half * 8;
#pragma unroll
    for (int s = 0; s < NDS; ++s) {
      qreg[s] = *reinterpret_cast<const bf16x8*>(qp + s * 16);
      if (!row_ok) qreg[s] = bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  const int nkv = (b1 - b0 + 3) / 4;
  const size_t head_k = size_t(hkv) * 16 * D;   // elements per block (all heads)
  const uint16_t* kbase = a.k_cache + size_t(g) * 16 * D;
  const uint16_t* vbase = a.v_cache + size_t(g) * 16 * D;
  // staging registers as SSA vectors (an array here ends up in scratch memory)
  typedef uint32_t stage_t __attribute__((ext_vector_type(4 * CH)));
  stage_t kreg, vreg;

  // Global -> registers for KV tile `it`.  Block ids and lengths are uniform
  // (scalar loads); blocks past b1 read block b1-1 and are masked later.
  // Chunk i of a thread: K key kkey0 + i*KPT (block (kkey0 + i*KPT) / 16,
  // compile-time for D = 128), 8 dims at kdc; V block vbeta0 + i*VPB, dim vd,
  // 8-slot half vhf.
  constexpr int KPT = kThreads / (D / 8);       // keys covered by one chunk index (16 or 32)
  constexpr int VPB = kThreads / (2 * D);       // V blocks covered by one chunk index (1 or 2)
  const int kkey0 = tid / (D / 8), kdc = tid % (D / 8);
  const int vbeta0 = tid / (2 * D), vd = (tid % (2 * D)) >> 1, vhf = tid & 1;
  auto load_tile = [&](int it) {
    const int bb = b0 + it * 4;
    int phys[4], len[4];
#pragma unroll
    for (int beta = 0; beta < 4; ++beta) {
      const int blk = min(bb + beta, b1 - 1);
      phys[beta] = lblk[blk];
      len[beta] = bb + beta < b1 ? blenp[blk] : 0;
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int key = kkey0 + i * KPT;
      int pb;
      if constexpr (KPT == 16) pb = phys[i];
      else pb = (key >> 4) == 2 * i ? phys[2 * i] : phys[2 * i + 1];
      const uint4 x = *reinterpret_cast<const uint4*>(kbase + size_t(pb) * head_k + (key & 15) * D + kdc * 8);
      kreg[4 * i + 0] = x.x;
      kreg[4 * i + 1] = x.y;
      kreg[4 * i + 2] = x.z;
      kreg[4 * i + 3] = x.w;
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      int pb, ln;
      if constexpr (VPB == 1) {
        pb = phys[i];
        ln = len[i];
      } else {
        pb = vbeta0 == 0 ? phys[2 * i] : phys[2 * i + 1];
        ln = vbeta0 == 0 ? len[2 * i] : len[2 * i + 1];
      }
      uint4 x = *reinterpret_cast<const uint4*>(vbase + size_t(pb) * head_k + vd * 16 + vhf * 8);
      const int valid = ln - vhf * 8;            // valid slots in this 8-slot half
      if (valid < 8) {                           // zero slots past the block's end (never NaN garbage)
        x.x = valid <= 0 ? 0u : valid == 1 ? (x.x & 0xFFFFu) : x.x;
        x.y = valid <= 2 ? 0u : valid == 3 ? (x.y & 0xFFFFu) : x.y;
        x.z = valid <= 4 ? 0u : valid == 5 ? (x.z & 0xFFFFu) : x.z;
        x.w = valid <= 6 ? 0u : valid == 7 ? (x.w & 0xFFFFu) : x.w;
      }
      vreg[4 * i + 0] = x.x;
      vreg[4 * i + 1] = x.y;
      vreg[4 * i + 2] = x.z;
      vreg[4 * i + 3] = x.w;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CH; ++i)
      *reinterpret_cast<uint4*>(&lds.k[buf][(kkey0 + i * KPT) * KS + kdc * 8]) =
          make_uint4(kreg[4 * i + 0], kreg[4 * i + 1], kreg[4 * i + 2], kreg[4 * i + 3]);
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int beta = vbeta0 + i * VPB;
      *reinterpret_cast<uint4*>(&lds.v[buf][(beta * D + vd) * 16 + (vhf ^ v_swz(vd)) * 8]) =
          make_uint4(vreg[4 * i + 0], vreg[4 * i + 1], vreg[4 * i + 2], vreg[4 * i + 3]);
    }
  };

  f32x16 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;
  float m = -INFINITY, lsum = 0.0f;            // m in the scaled log2 domain
  const float sl2 = a.scale_log2;
  const int krow = srow_key(col);              // K row this lane feeds into S^T

  if (nkv > 0) {
    load_tile(0);
    store_tile(0);
  }
  __syncthreads();

  for (int it = 0; it < nkv; ++it) {
    const int cur = it & 1;
    if (it + 1 < nkv) load_tile(it + 1);

    // S^T (64 keys x 32 rows per wave) = K Q^T
    f32x16 sacc[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[ks][r] = 0.0f;
      const uint16_t* kp = &lds.k[cur][(ks * 32 + krow) * KS + half * 8];
#pragma unroll
      for (int s = 0; s < NDS; ++s)
        sacc[ks] = mfma_32x32x16(*reinterpret_cast<const bf16x8*>(kp + s * 16), qreg[s], sacc[ks]);
    }

    // Mask (only tiles that reach past the first row, or hold partial blocks).
    // Register r = i*4 + j of subtile ks holds key ks*32 + (i>>1)*16 + half*8 + (i&1)*4 + j.
    const int bb = b0 + it * 4;
    int bpos0[4], blen[4];
#pragma unroll
    for (int beta = 0; beta < 4; ++beta) {
      const int blk = min(bb + beta, b1 - 1);
      bpos0[beta] = bpos[blk];
      blen[beta] = bb + beta < b1 ? blenp[blk] : 0;
    }
    const bool full = blen[0] == 16 && blen[1] == 16 && blen[2] == 16 && blen[3] == 16 &&
                      bpos0[3] + 15 <= min_qpos;
    if (!full) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = r >> 2, j = r & 3;
          const int beta = ks * 2 + (i >> 1);
          const int slot = half * 8 + (i & 1) * 4 + j;
          const bool ok = slot < blen[beta] && bpos0[beta] + slot <= qpos;
          sacc[ks][r] = ok ? sacc[ks][r] : -INFINITY;
        }
    }
    float mt = sacc[0][0];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, sacc[ks][r]);
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m, mt * sl2);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    if (__ballot(m_new > m)) {                 // some row's max moved: rescale
      const float alpha = fast_exp2(m - m_use);
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    m = m_new;
    float ls = 0.0f;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(sacc[ks][r], sl2, -m_use));
        sacc[ks][r] = p;
        ls += p;
      }
    lsum += ls;

    // P^T as bf16 B operands: registers 8st .. 8st+7 of subtile ks = keys ks*32 + st*16 + half*8 + [0, 8).
    bf16x8 pb[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int r0 = st * 8;
        uint4 u = make_uint4(pack_bf16x2(sacc[ks][r0 + 0], sacc[ks][r0 + 1]),
                             pack_bf16x2(sacc[ks][r0 + 2], sacc[ks][r0 + 3]),
                             pack_bf16x2(sacc[ks][r0 + 4], sacc[ks][r0 + 5]),
                             pack_bf16x2(sacc[ks][r0 + 6], sacc[ks][r0 + 7]));
        pb[ks][st] = __builtin_bit_cast(bf16x8, u);
      }

    // O^T (D x 32 rows) += V^T (D x 64 keys) P^T: one 16-byte LDS read per MFMA.
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int d = dt * 32 + col;
      const uint16_t* vp = &lds.v[cur][d * 16 + (half ^ v_swz(d)) * 8];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int st = 0; st < 2; ++st)
          o[dt] = mfma_32x32x16(*reinterpret_cast<const bf16x8*>(vp + (ks * 2 + st) * D * 16), pb[ks][st],
                                o[dt]);
    }

    if (it + 1 < nkv) store_tile(cur ^ 1);
    __syncthreads();
  }

  const float ltot = lsum + __shfl_xor(lsum, 32);
  if (!row_ok) return;
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
  if (part < 0) {
    uint16_t* op = a.out + (size_t(srow) * a.hq + h) * D + half * 4;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint2 u;
        u.x = pack_bf16x2(o[dt][i * 4 + 0] * inv, o[dt][i * 4 + 1] * inv);
        u.y = pack_bf16x2(o[dt][i * 4 + 2] * inv, o[dt][i * 4 + 3] * inv);
        *reinterpret_cast<uint2*>(op + dt * 32 + i * 8) = u;
      }
    if (a.lse && half == 0) a.lse[size_t(srow) * a.hq + h] = (m + fast_log2(ltot)) * kLn2;
  } else {
    float* pp = a.part_o + ((size_t(part) * hkv + g) * 128 + t) * D + half * 4;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 f = make_float4(o[dt][i * 4 + 0] * inv, o[dt][i * 4 + 1] * inv, o[dt][i * 4 + 2] * inv,
                               o[dt][i * 4 + 3] * inv);
        *reinterpret_cast<float4*>(pp + dt * 32 + i * 8) = f;
      }
    if (half == 0)
      a.part_lse[(size_t(part) * hkv + g) * 128 + t] = ltot > 0.0f ? m + fast_log2(ltot) : -INFINITY;
  }
}

// Merge the split-KV partials of a tile: lse = log2 sum_i 2^lse_i, out = sum_i 2^(lse_i - lse) O_i.
template <int D>
__global__ __launch_bounds__(kThreads) void link_combine_kernel(AttnArgs a) {
  const int hkv = a.hkv;
  const int g = blockIdx.x % hkv;
  const int tile = blockIdx.x / hkv;
  const int p0 = a.tiles[4 * tile + 2];
  const int ns = a.tiles[4 * tile + 3];
  if (p0 < 0) return;
  const int row0 = a.tiles[4 * tile + 0], nrows = a.tiles[4 * tile + 1];
  const int t = threadIdx.x >> 1, hf = threadIdx.x & 1;
  const int R = a.rows_per_tile;
  const int srl = t % R, h = g * a.G + t / R;
  if (srl >= nrows) return;
  const int srow = row0 + srl;
  float mx = -INFINITY;
  for (int i = 0; i < ns; ++i) mx = fmaxf(mx, a.part_lse[(size_t(p0 + i) * hkv + g) * 128 + t]);
  float acc[D / 2];
#pragma unroll
  for (int d = 0; d < D / 2; ++d) acc[d] = 0.0f;
  float wsum = 0.0f;
  for (int i = 0; i < ns; ++i) {
    const float l = a.part_lse[(size_t(p0 + i) * hkv + g) * 128 + t];
    const float w = fast_exp2(l - mx);
    wsum += w;
    const float* pp = a.part_o + ((size_t(p0 + i) * hkv + g) * 128 + t) * D + hf * (D / 2);
#pragma unroll
    for (int d = 0; d < D / 2; d += 4) {
      const float4 f = *reinterpret_cast<const float4*>(pp + d);
      acc[d + 0] += w * f.x;
      acc[d + 1] += w * f.y;
      acc[d + 2] += w * f.z;
      acc[d + 3] += w * f.w;
    }
  }
  const float inv = 1.0f / wsum;
  uint16_t* op = a.out + (size_t(srow) * a.hq + h) * D + hf * (D / 2);
#pragma unroll
  for (int d = 0; d < D / 2; d += 8) {
    uint4 u;
    u.x = pack_bf16x2(acc[d + 0] * inv, acc[d + 1] * inv);
    u.y = pack_bf16x2(acc[d + 2] * inv, acc[d + 3] * inv);
    u.z = pack_bf16x2(acc[d + 4] * inv, acc[d + 5] * inv);
    u.w = pack_bf16x2(acc[d + 6] * inv, acc[d + 7] * inv);
    *reinterpret_cast<uint4*>(op + d) = u;
  }
  if (a.lse && hf == 0) a.lse[size_t(srow) * a.hq + h] = (mx + fast_log2(wsum)) * kLn2;
}

}  // namespace

void launch_link_attention(const AttnArgs& a, int head_dim, int n_work, hipStream_t stream) {
  if (n_work == 0) return;
  const dim3 grid(unsigned(n_work) * unsigned(a.hkv));
  if (head_dim == 128)
    link_attention_kernel<128><<<grid, kThreads, 0, stream>>>(a);
  else
    link_attention_kernel<64><<<grid, kThreads, 0, stream>>>(a);
}

void launch_link_combine(const AttnArgs& a, int head_dim, int n_tiles, hipStream_t stream) {
  if (n_tiles == 0) return;
  const dim3 grid(unsigned(n_tiles) * unsigned(a.hkv));
  if (head_dim == 128)
    link_combine_kernel<128><<<grid, kThreads, 0, stream>>>(a);
  else
    link_combine_kernel<64><<<grid, kThreads, 0, stream>>>(a);
}

}  // namespace epic
