// Causal attention (Eq. 1) for tiles of 16 query rows: the decode-shaped case, where
// a request brings one or a few new tokens (G query heads each) and attends over
// its whole linked cache.  The 128-row kernel would spend almost all its matrix-core
// work on empty rows here; this one streams K/V at HBM rate instead.
//
// Workgroup = (work item, KV head g), 4 wavefronts.  Tile row t (0..15) is S row
// t % R, query head g G + t / R (R = 16 / G).  Wavefront w takes the item's linked
// blocks b0 + w, b0 + w + 4, ... (16 keys each), loaded into a ring of registers a
// few blocks ahead of their use:
//   S^T (16 keys x 16 rows) = K Q^T by v_mfma_f32_16x16x32_bf16 (D / 32 of them);
//     lane l holds the scores of row l % 16 for keys 4 (l / 16) + i, i < 4;
//   online softmax per row in the scaled log2 domain (the 4 lanes of a row combine
//     by two lane exchanges);
//   O^T (D x 16) += V^T P^T by v_mfma_f32_16x16x16bf16_1k (D / 16 of them): the P
//     operand of lane l is exactly its own 4 probabilities.
// The four wavefronts' (max, sum, O) are merged through LDS at the end; the item
// writes the output rows and lse, or its split-KV partial (O / l and log2 l + m).
#include <cmath>

#include "decode_attention.h"
#include "device_common.h"
#include "plan_internal.h"

namespace epic {

namespace {

typedef short bf16x4 __attribute__((ext_vector_type(4)));

constexpr int kDecRows = 16;
constexpr int kDecWaves = 4;
constexpr int kRing = 3;      // blocks in flight per wavefront

template <int D>
struct DecodeLds {
  float m[kDecWaves][kDecRows];
  float l[kDecWaves][kDecRows];
  float o[kDecWaves][D][kDecRows];
};

template <int D>
__global__ __launch_bounds__(64 * kDecWaves, 3) void link_decode_kernel(AttnArgs a) {
  constexpr int NKS = D / 32;                 // k-steps of the QK product
  constexpr int NDT = D / 16;                 // 16-dim tiles of O^T
  __shared__ DecodeLds<D> lds;

  const int hkv = a.hkv;
  const int g = blockIdx.x % hkv;
  const int item = blockIdx.x / hkv;
  const int32_t* wk = a.work + kWorkInts * item;
  const int tile = wk[0], b0 = wk[1], b1 = wk[2], part = wk[3];
  const int row0 = a.tiles[4 * tile + 0];
  const int nrows = a.tiles[4 * tile + 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 15;                    // tile row of this lane
  const int qd = lane >> 4;                   // its quarter: keys 4 qd .., dims 8 qd .. of a k-step
  const int R = a.rows_per_tile;
  const int srl = r % R;
  const int h = g * a.G + r / R;
  const bool row_ok = srl < nrows;
  const int srow = row0 + (row_ok ? srl : nrows - 1);
  const int qpos = a.s_pos[srow];

  bf16x8 qf[NKS];                             // Q^T operand: row r, dims 32 ks + 8 qd ..
  {
    const uint16_t* qp = a.q + (size_t(srow) * a.hq + h) * D + qd * 8;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) {
      bf16x8 x = *reinterpret_cast<const bf16x8*>(qp + ks * 32);
      qf[ks] = row_ok ? x : bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
    }
  }

  const float sl2 = a.scale_log2;
  const size_t blk_elems = size_t(hkv) * 16 * D;      // one physical block, all heads
  const uint16_t* kbase = a.k_cache + size_t(g) * 16 * D;
  const uint16_t* vbase = a.v_cache + size_t(g) * 16 * D;
  // this lane's K operand: key r, dims 8 qd + 32 ks; V operand: dim 16 dt + r, keys 4 qd ..
  auto load_kv = [&](int b, bf16x8 (&kf)[NKS], bf16x4 (&vf)[NDT]) __attribute__((always_inline)) {
    const int phys = a.linked_blocks[b];
    const uint16_t* kp = kbase + size_t(phys) * blk_elems + r * D + qd * 8;
    const uint16_t* vp = vbase + size_t(phys) * blk_elems + size_t(r) * 16 + qd * 4;
#pragma unroll
    for (int ks = 0; ks < NKS; ++ks) kf[ks] = *reinterpret_cast<const bf16x8*>(kp + ks * 32);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) vf[dt] = *reinterpret_cast<const bf16x4*>(vp + dt * 16 * 16);
  };

  f32x4 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) o[dt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m = -INFINITY, lsum = 0.0f;

  // The wavefront's blocks b0 + w + 4 j stream through a ring of kRing register
  // slots: slot j % kRing is refilled with block j + kRing as soon as block j is used,
  // so kRing blocks (kRing x 8 KB at D = 128) are in flight per wavefront; the
  // compiler's per-load waits then only cover the slot about to be used.
  bf16x8 kr[kRing][NKS];
  bf16x4 vr[kRing][NDT];
  // loads are issued unconditionally, past the item's end with the block index
  // clamped to its last block, so every slot always has the same loads in flight
  const int first = b0 + wave;
  auto clampb = [&](int x) __attribute__((always_inline)) { return x < b1 ? x : b1 - 1; };
#pragma unroll
  for (int j = 0; j < kRing; ++j) load_kv(clampb(first + kDecWaves * j), kr[j], vr[j]);
  for (int base = first; base < b1; base += kDecWaves * kRing) {
#pragma unroll
    for (int j = 0; j < kRing; ++j) {
      const int b = base + kDecWaves * j;
      if (b < b1) {
        const int pos0 = a.block_pos0[b], len = a.block_len[b];
        f32x4 s = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) s = mfma_16x16x32(kr[j][ks], qf[ks], s);
        // keys 4 qd + i of the block: masked past the block's end, after the row, or for empty rows
        float x[4], mb = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = qd * 4 + i;
          const bool ok = row_ok && key < len && pos0 + key <= qpos;
          x[i] = ok ? s[i] * sl2 : -INFINITY;
          mb = fmaxf(mb, x[i]);
        }
        mb = fmaxf(mb, __shfl_xor(mb, 16));
        mb = fmaxf(mb, __shfl_xor(mb, 32));
        const float m_new = fmaxf(m, mb);
        const float m_use = m_new == -INFINITY ? 0.0f : m_new;
        const float alpha = fast_exp2(m - m_use);         // 0 while nothing was seen
        float p[4], ps = 0.0f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          p[i] = fast_exp2(x[i] - m_use);
          ps += p[i];
        }
        ps += __shfl_xor(ps, 16);
        ps += __shfl_xor(ps, 32);
        lsum = lsum * alpha + ps;
        m = m_new;
        bf16x4 pb;
        {
          const uint32_t lo = pack_bf16x2(p[0], p[1]), hi = pack_bf16x2(p[2], p[3]);
          pb = __builtin_bit_cast(bf16x4, (uint64_t(hi) << 32) | lo);
        }
        const bool partial_block = len < 16;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          bf16x4 v = vr[j][dt];
          if (partial_block) {                  // slots past the block's end may hold any bits
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = qd * 4 + i < len ? v[i] : short(0);
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) o[dt][i] *= alpha;
          o[dt] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(v, pb, o[dt], 0, 0, 0);
        }
      }
      load_kv(clampb(b + kDecWaves * kRing), kr[j], vr[j]);   // refill this slot
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);          // vmcnt(0): the ring's last loads land before the exit

  // merge the wavefronts: O^T of lane l holds dims 16 dt + 4 qd + i of row r
  if (qd == 0) {
    lds.m[wave][r] = m;
    lds.l[wave][r] = lsum;
  }
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int i = 0; i < 4; ++i) lds.o[wave][dt * 16 + qd * 4 + i][r] = o[dt][i];
  __syncthreads();
  // thread -> (row rr, dims dd, dd + 16, ...): 16 rows x 16 dim groups
  const int rr = tid & 15, d0 = tid >> 4;
  float mw[kDecWaves], M = -INFINITY;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) {
    mw[w] = lds.m[w][rr];
    M = fmaxf(M, mw[w]);
  }
  const float Mu = M == -INFINITY ? 0.0f : M;
  float wt[kDecWaves], L = 0.0f;
#pragma unroll
  for (int w = 0; w < kDecWaves; ++w) {
    wt[w] = fast_exp2(mw[w] - Mu);
    L += lds.l[w][rr] * wt[w];
  }
  const int s2 = rr % R;
  if (s2 >= nrows) return;
  const int srow2 = row0 + s2, h2 = g * a.G + rr / R;
  const float inv = L > 0.0f ? 1.0f / L : 0.0f;
  for (int d = d0; d < D; d += 16) {
    float acc = 0.0f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) acc += lds.o[w][d][rr] * wt[w];
    acc *= inv;
    if (part < 0)
      a.out[(size_t(srow2) * a.hq + h2) * D + d] = uint16_t(pack_bf16x2(acc, 0.0f) & 0xFFFFu);
    else
      a.part_o[((size_t(part) * hkv + g) * kDecRows + rr) * D + d] = acc;
  }
  if (d0 == 0) {
    if (part < 0) {
      if (a.lse) a.lse[size_t(srow2) * a.hq + h2] = (M + fast_log2(L)) * kLn2;
    } else {
      a.part_lse[(size_t(part) * hkv + g) * kDecRows + rr] = L > 0.0f ? M + fast_log2(L) : -INFINITY;
    }
  }
}

}  // namespace

void launch_link_decode(const AttnArgs& a, int head_dim, int n_work, hipStream_t stream) {
  if (n_work == 0) return;
  const dim3 grid{unsigned(n_work) * unsigned(a.hkv)};
  if (head_dim == 128)
    link_decode_kernel<128><<<grid, 64 * kDecWaves, 0, stream>>>(a);
  else
    link_decode_kernel<64><<<grid, 64 * kDecWaves, 0, stream>>>(a);
}

}  // namespace epic
