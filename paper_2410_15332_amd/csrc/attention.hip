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
// scale*log2(e) folded into the logits; accumulation is fp32.
#include "device_common.h"
#include "kernels.h"

namespace epic {

namespace {

constexpr int kKT = 64;    // keys per iteration
constexpr int kThreads = 256;

template <int D>
struct AttnLds {
  static constexpr int KS = D + 8;     // K row stride (elements), 16 B aligned
  static constexpr int VS = kKT + 8;   // V^T row stride
  uint16_t k[2][kKT * KS];
  uint16_t v[2][D * VS];
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void link_attention_kernel(AttnArgs a) {
  constexpr int NDS = D / 16;                 // k-steps of S^T = K Q^T
  constexpr int NDT = D / 32;                 // 32-row tiles of O^T
  constexpr int CH = kKT * D / 8 / kThreads;  // 16-byte chunks per thread per operand
  constexpr int KS = AttnLds<D>::KS, VS = AttnLds<D>::VS;
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

  const int tid = threadIdx.x;
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
  uint4 kreg[CH], vreg[CH];

  auto load_tile = [&](int it) {
    const int bb = b0 + it * 4;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + kThreads * i;
      const int key = c / (D / 8), dc = c % (D / 8);
      const int blk = bb + key / 16, slot = key % 16;
      uint4 x = make_uint4(0, 0, 0, 0);
      if (blk < b1 && slot < a.block_len[blk]) {
        const int phys = a.linked_blocks[blk];
        x = *reinterpret_cast<const uint4*>(a.k_cache + ((size_t(phys) * hkv + g) * 16 + slot) * D + dc * 8);
      }
      kreg[i] = x;
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + kThreads * i;
      const int beta = c / (2 * D), rem = c % (2 * D);
      const int d = rem >> 1, hf = rem & 1;
      const int blk = bb + beta;
      uint4 x = make_uint4(0, 0, 0, 0);
      if (blk < b1) {
        const int phys = a.linked_blocks[blk];
        x = *reinterpret_cast<const uint4*>(a.v_cache + ((size_t(phys) * hkv + g) * D + d) * 16 + hf * 8);
        const int len = a.block_len[blk] - hf * 8;   // valid slots in this 8-slot half
        if (len < 8) {                               // zero slots past the block's end
          uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (2 * e >= len) w[e] = 0;
            else if (2 * e + 1 >= len) w[e] &= 0xFFFFu;
          }
          x = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
      vreg[i] = x;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + kThreads * i;
      const int key = c / (D / 8), dc = c % (D / 8);
      *reinterpret_cast<uint4*>(&lds.k[buf][key * KS + dc * 8]) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = tid + kThreads * i;
      const int beta = c / (2 * D), rem = c % (2 * D);
      const int d = rem >> 1, hf = rem & 1;
      *reinterpret_cast<uint4*>(&lds.v[buf][d * VS + beta * 16 + hf * 8]) = vreg[i];
    }
  };

  f32x16 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;
  float m = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale_log2;

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
      const uint16_t* kp = &lds.k[cur][(ks * 32 + col) * KS + half * 8];
#pragma unroll
      for (int s = 0; s < NDS; ++s)
        sacc[ks] = mfma_32x32x16(*reinterpret_cast<const bf16x8*>(kp + s * 16), qreg[s], sacc[ks]);
    }

    // Mask and scale.  Register r = i*4 + j of subtile ks holds key ks*32 + i*8 + half*4 + j.
    const int bb = b0 + it * 4;
    int bpos0[4], blen[4];
#pragma unroll
    for (int beta = 0; beta < 4; ++beta) {
      const int blk = bb + beta;
      const bool in = blk < b1;
      bpos0[beta] = in ? a.block_pos0[blk] : 0;
      blen[beta] = in ? a.block_len[blk] : 0;
    }
    const bool full = blen[0] == 16 && blen[1] == 16 && blen[2] == 16 && blen[3] == 16 &&
                      bpos0[3] + 15 <= min_qpos;
    float mt = -INFINITY;
    if (full) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          sacc[ks][r] *= sl2;
          mt = fmaxf(mt, sacc[ks][r]);
        }
    } else {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = r >> 2, j = r & 3;
          const int beta = ks * 2 + (i >> 1);
          const int slot = (i & 1) * 8 + half * 4 + j;
          const bool ok = slot < blen[beta] && bpos0[beta] + slot <= qpos;
          const float x = ok ? sacc[ks][r] * sl2 : -INFINITY;
          sacc[ks][r] = x;
          mt = fmaxf(mt, x);
        }
    }
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m, mt);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = fast_exp2(m - m_use);
    float ls = 0.0f;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(sacc[ks][r] - m_use);
        sacc[ks][r] = p;
        ls += p;
      }
    lsum = lsum * alpha + ls;
    m = m_new;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;

    // P^T as bf16 B operands: step st of subtile ks = registers (2st)*4.. and (2st+1)*4..,
    // i.e. keys st*16 + half*4 + [0,4) then st*16 + 8 + half*4 + [0,4).
    bf16x8 pb[2][2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        const int r0 = st * 8;
        uint32_t w0 = pack_bf16x2(sacc[ks][r0 + 0], sacc[ks][r0 + 1]);
        uint32_t w1 = pack_bf16x2(sacc[ks][r0 + 2], sacc[ks][r0 + 3]);
        uint32_t w2 = pack_bf16x2(sacc[ks][r0 + 4], sacc[ks][r0 + 5]);
        uint32_t w3 = pack_bf16x2(sacc[ks][r0 + 6], sacc[ks][r0 + 7]);
        uint4 u = make_uint4(w0, w1, w2, w3);
        pb[ks][st] = __builtin_bit_cast(bf16x8, u);
      }

    // O^T (D x 32 rows) += V^T (D x 64 keys) P^T, V^T read with the same key order.
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const uint16_t* vp = &lds.v[cur][(dt * 32 + col) * VS + half * 4];
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          const uint16_t* p = vp + ks * 32 + st * 16;
          uint2 lo = *reinterpret_cast<const uint2*>(p);
          uint2 hi = *reinterpret_cast<const uint2*>(p + 8);
          uint4 u = make_uint4(lo.x, lo.y, hi.x, hi.y);
          o[dt] = mfma_32x32x16(__builtin_bit_cast(bf16x8, u), pb[ks][st], o[dt]);
        }
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
