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
#include "plan_internal.h"

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

// Both halves of the wavefront exchange: lane l gets op(x[l], x[l ^ 32]).
__device__ __forceinline__ float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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
  const int32_t* wk = a.work + kWorkInts * item;
  const int tile = wk[0];
  const int b0 = wk[1];
  const int b1 = wk[2];
  const int part = wk[3];
  const int n_fast = wk[4];                    // leading KV tiles that need no mask
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
  // staging registers as SSA vectors (an array here ends up in scratch memory):
  // kreg holds K of a tile two ahead, vreg V of the next tile
  typedef uint32_t stage_t __attribute__((ext_vector_type(4 * CH)));
  stage_t kreg, vreg;

  // Chunk i of a thread: K key kkey0 + i*KPT (block (kkey0 + i*KPT) / 16,
  // compile-time for D = 128), 8 dims at kdc; V block vbeta0 + i*VPB, dim vd,
  // 8-slot half vhf.
  constexpr int KPT = kThreads / (D / 8);       // keys covered by one chunk index (16 or 32)
  constexpr int VPB = kThreads / (2 * D);       // V blocks covered by one chunk index (1 or 2)
  const int kkey0 = tid / (D / 8), kdc = tid % (D / 8);
  const int vbeta0 = tid / (2 * D), vd = (tid % (2 * D)) >> 1, vhf = tid & 1;

  // Physical ids of the 4 blocks of KV tile `it` (uniform scalar loads; blocks
  // past b1 repeat block b1-1, whose keys are masked).
  auto tile_phys = [&](int it, int (&ph)[4]) {
    const int bb = b0 + it * 4;
#pragma unroll
    for (int beta = 0; beta < 4; ++beta) ph[beta] = lblk[min(bb + beta, b1 - 1)];
  };
  // Global -> registers: K of tile `it` (block ids ph).
  auto load_k = [&](const int (&ph)[4]) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int key = kkey0 + i * KPT;
      int pb;
      if constexpr (KPT == 16) pb = ph[i];
      else pb = (key >> 4) == 2 * i ? ph[2 * i] : ph[2 * i + 1];
      const uint4 x = *reinterpret_cast<const uint4*>(kbase + size_t(pb) * head_k + (key & 15) * D + kdc * 8);
      kreg[4 * i + 0] = x.x;
      kreg[4 * i + 1] = x.y;
      kreg[4 * i + 2] = x.z;
      kreg[4 * i + 3] = x.w;
    }
  };
  // Global -> registers: V of tile `it`.  A masked tile zeroes V slots past each
  // block's end, so stale or NaN bits there never meet a zero softmax weight.
  auto load_v = [&](int it, const int (&ph)[4]) {
    const bool fast = it < n_fast;
    int len[4] = {16, 16, 16, 16};
    if (!fast) {
      const int bb = b0 + it * 4;
#pragma unroll
      for (int beta = 0; beta < 4; ++beta) len[beta] = bb + beta < b1 ? blenp[min(bb + beta, b1 - 1)] : 0;
    }
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      int pb, ln;
      if constexpr (VPB == 1) {
        pb = ph[i];
        ln = len[i];
      } else {
        pb = vbeta0 == 0 ? ph[2 * i] : ph[2 * i + 1];
        ln = vbeta0 == 0 ? len[2 * i] : len[2 * i + 1];
      }
      uint4 x = *reinterpret_cast<const uint4*>(vbase + size_t(pb) * head_k + vd * 16 + vhf * 8);
      if (!fast) {
        const int valid = ln - vhf * 8;          // valid slots in this 8-slot half
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
  auto store_k_chunk = [&](int buf, int i) {
    *reinterpret_cast<uint4*>(&lds.k[buf][(kkey0 + i * KPT) * KS + kdc * 8]) =
        make_uint4(kreg[4 * i + 0], kreg[4 * i + 1], kreg[4 * i + 2], kreg[4 * i + 3]);
  };
  auto store_v_chunk = [&](int buf, int i) {
    const int beta = vbeta0 + i * VPB;
    *reinterpret_cast<uint4*>(&lds.v[buf][(beta * D + vd) * 16 + (vhf ^ v_swz(vd)) * 8]) =
        make_uint4(vreg[4 * i + 0], vreg[4 * i + 1], vreg[4 * i + 2], vreg[4 * i + 3]);
  };

  f32x16 o[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[dt][r] = 0.0f;
  // Running max m (scaled log2 domain) is allowed to lag the true row max by up
  // to kLag: the output and the sum share it, so the result is exact, P stays
  // below 2^kLag, and O is rescaled only when some row's max jumps past it.
  constexpr float kLag = 8.0f;
  float m = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale_log2;
  const int krow = srow_key(col);              // K row this lane feeds into S^T

  // S^T (64 keys x 32 rows per wave) = K Q^T from LDS stage `buf`; the two
  // 32-key subtiles alternate so that consecutive MFMAs are independent.
  const uint16_t* kp_lane = &lds.k[0][krow * KS + half * 8];
  auto qk = [&](int buf, f32x16 (&sc)[2]) {
    const uint16_t* kp = kp_lane + buf * (kKT * KS);
#pragma unroll
    for (int q = 0; q < 2 * NDS; ++q) {
      const int ks = q & 1, s = q >> 1;
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kp + ks * 32 * KS + s * 16);
      sc[ks] = mfma_32x32x16(kf, qreg[s], s == 0 ? f32x16{} : sc[ks]);
    }
  };
  // V^T operand of lane: row d = dt*32 + col, 16-byte half (half ^ swz(col)) of the row.
  const uint16_t* vp_lane = &lds.v[0][col * 16 + (half ^ v_swz(col)) * 8];

  // Software pipeline over KV tiles.  K runs one tile ahead of V: during
  // iteration it the waves read K(it + 1) (buffer (it + 1) % 2, for S(it + 1))
  // and V(it) (buffer it % 2), and store K(it + 2) into K buffer it % 2 and
  // V(it + 1) into V buffer (it + 1) % 2 -- buffers nobody reads in iteration
  // it, because their last readers ran before the barrier ending iteration
  // it - 1.  One barrier per iteration; the stores overlap the PV MFMAs.  The
  // MFMAs of S(it + 1) are interleaved with the exponentials of tile it.
  int phk[4], phv[4];
  tile_phys(0, phk);
  load_k(phk);
#pragma unroll
  for (int i = 0; i < CH; ++i) store_k_chunk(0, i);
  load_v(0, phk);
#pragma unroll
  for (int i = 0; i < CH; ++i) store_v_chunk(0, i);
  if (nkv > 1) {
    tile_phys(1, phk);
    load_k(phk);
#pragma unroll
    for (int i = 0; i < CH; ++i) store_k_chunk(1, i);
    load_v(1, phk);                            // V(1): stored during iteration 0
  }
  tile_phys(2, phk);
  tile_phys(2, phv);
  if (nkv > 2) load_k(phk);                    // K(2): stored during iteration 0
  tile_phys(3, phk);
  __syncthreads();

  f32x16 sacc[2];
  qk(0, sacc);
  __syncthreads();                             // K buffer 0 is rewritten in iteration 0

  for (int it = 0; it < nkv; ++it) {
    const int cur = it & 1;

    // Mask: only tiles past the item's unmasked prefix (diagonal, partial blocks).
    // Register r = i*4 + j of subtile ks holds key ks*32 + (i>>1)*16 + half*8 + (i&1)*4 + j.
    if (it >= n_fast) {
      const int bb = b0 + it * 4;
      int bpos0[4], blen[4];
#pragma unroll
      for (int beta = 0; beta < 4; ++beta) {
        const int blk = min(bb + beta, b1 - 1);
        bpos0[beta] = bpos[blk];
        blen[beta] = bb + beta < b1 ? blenp[blk] : 0;
      }
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

    // row max: independent partial maxima, then one lane swap across halves
    float mx[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
      mx[c] = fmaxf(fmaxf(sacc[c >> 2][(c & 3) * 4 + 0], sacc[c >> 2][(c & 3) * 4 + 1]),
                    fmaxf(sacc[c >> 2][(c & 3) * 4 + 2], sacc[c >> 2][(c & 3) * 4 + 3]));
    const float mt = xhalf_max(fmaxf(fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3])),
                                     fmaxf(fmaxf(mx[4], mx[5]), fmaxf(mx[6], mx[7]))));
    const float m_cand = fmaxf(m, mt * sl2);
    const bool grow = m_cand > m + kLag;       // also true on the first finite max
    if (__ballot(grow)) {
      const float alpha = grow ? fast_exp2(m - m_cand) : 1.0f;
      m = grow ? m_cand : m;
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    const float m_use = m == -INFINITY ? 0.0f : m;

    // Exponentials of tile it, interleaved with the S(it + 1) MFMAs.
    f32x16 snext[2];
    uint32_t pw[16];                           // P(it) packed to bf16 pairs
    float ps[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    auto softmax_step = [&](int q) {
      constexpr int VPS = 32 / (2 * NDS);      // scores per MFMA step
#pragma unroll
      for (int v = 0; v < VPS; ++v) {
        const int idx = q * VPS + v;           // flattened register (ks = idx / 16, r = idx % 16)
        const float p = fast_exp2(__builtin_fmaf(sacc[idx >> 4][idx & 15], sl2, -m_use));
        sacc[idx >> 4][idx & 15] = p;
        ps[idx & 3] += p;
        if (idx & 1) pw[idx >> 1] = pack_bf16x2(sacc[idx >> 4][(idx & 15) - 1], p);
      }
    };
    if (it + 1 < nkv) {
      const uint16_t* kp = kp_lane + (cur ^ 1) * (kKT * KS);
      bf16x8 kf[2];                            // K fragments, read one step ahead
      kf[0] = *reinterpret_cast<const bf16x8*>(kp);
#pragma unroll
      for (int q = 0; q < 2 * NDS; ++q) {
        const int ks = q & 1, s = q >> 1;
        if (q + 1 < 2 * NDS)
          kf[(q + 1) & 1] = *reinterpret_cast<const bf16x8*>(kp + ((q + 1) & 1) * 32 * KS + ((q + 1) >> 1) * 16);
        snext[ks] = mfma_32x32x16(kf[q & 1], qreg[s], s == 0 ? f32x16{} : snext[ks]);
        softmax_step(q);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 2 * NDS; ++q) softmax_step(q);
    }
    lsum += (ps[0] + ps[1]) + (ps[2] + ps[3]);

    // O^T (D x 32 rows) += V^T (D x 64 keys) P^T.  B operand of step (ks, st) =
    // keys ks*32 + st*16 + half*8 + [0, 8) = packed words 8ks + 4st .. +3; the
    // V^T operand is one 16-byte LDS read; the D/32 accumulators alternate.
    const uint16_t* vp = vp_lane + cur * (4 * D * 16);
    const bool st_k = it + 2 < nkv, st_v = it + 1 < nkv;
    bf16x8 vf[2];                              // V^T fragments, read one MFMA ahead
    vf[0] = *reinterpret_cast<const bf16x8*>(vp);
#pragma unroll
    for (int kst = 0; kst < 4; ++kst) {
      const bf16x8 pbk = __builtin_bit_cast(
          bf16x8, make_uint4(pw[4 * kst + 0], pw[4 * kst + 1], pw[4 * kst + 2], pw[4 * kst + 3]));
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const int n = kst * NDT + dt + 1;      // next fragment
        if (n < 4 * NDT)
          vf[n & 1] = *reinterpret_cast<const bf16x8*>(vp + (n / NDT) * D * 16 + (n % NDT) * 32 * 16);
        o[dt] = mfma_32x32x16(vf[(n - 1) & 1], pbk, o[dt]);
        // LDS stores of K(it + 2) and V(it + 1), spread over the PV MFMAs
        const int c = n - 1;
        if (c < CH) {
          if (st_k) store_k_chunk(cur, c);
        } else if (c < 2 * CH) {
          if (st_v) store_v_chunk(cur ^ 1, c - CH);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // next global loads: K(it + 3), V(it + 2)
    if (it + 3 < nkv) load_k(phk);
    tile_phys(it + 4, phk);
    if (it + 2 < nkv) {
      tile_phys(it + 2, phv);
      load_v(it + 2, phv);
    }

    if (it + 1 < nkv) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) sacc[ks] = snext[ks];
      __syncthreads();                         // stores of this iteration visible; buffers free
    }
  }

  const float ltot = xhalf_sum(lsum);
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
// Workgroup = (tile, KV head, quarter of the head dim); thread = (tile row, 16 dims).
constexpr int kCombineParts = 4;
template <int D>
__global__ __launch_bounds__(kThreads) void link_combine_kernel(AttnArgs a) {
  constexpr int DQ = D / kCombineParts;       // dims per workgroup
  constexpr int DT = DQ / 2;                  // dims per thread (16 or 8)
  const int hkv = a.hkv;
  const int dq = blockIdx.x % kCombineParts;
  const int g = (blockIdx.x / kCombineParts) % hkv;
  const int tile = blockIdx.x / (kCombineParts * hkv);
  const int p0 = a.tiles[4 * tile + 2];
  const int ns = a.tiles[4 * tile + 3];
  if (p0 < 0) return;
  const int row0 = a.tiles[4 * tile + 0], nrows = a.tiles[4 * tile + 1];
  const int t = threadIdx.x >> 1, hf = threadIdx.x & 1;
  const int R = a.rows_per_tile;
  const int srl = t % R, h = g * a.G + t / R;
  if (srl >= nrows) return;
  const int srow = row0 + srl;
  const int d0 = dq * DQ + hf * DT;
  float mx = -INFINITY;
  for (int i = 0; i < ns; ++i) mx = fmaxf(mx, a.part_lse[(size_t(p0 + i) * hkv + g) * 128 + t]);
  float acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) acc[d] = 0.0f;
  float wsum = 0.0f;
  for (int i = 0; i < ns; ++i) {
    const float l = a.part_lse[(size_t(p0 + i) * hkv + g) * 128 + t];
    const float w = fast_exp2(l - mx);
    wsum += w;
    const float* pp = a.part_o + ((size_t(p0 + i) * hkv + g) * 128 + t) * D + d0;
#pragma unroll
    for (int d = 0; d < DT; d += 4) {
      const float4 f = *reinterpret_cast<const float4*>(pp + d);
      acc[d + 0] += w * f.x;
      acc[d + 1] += w * f.y;
      acc[d + 2] += w * f.z;
      acc[d + 3] += w * f.w;
    }
  }
  const float inv = 1.0f / wsum;
  uint16_t* op = a.out + (size_t(srow) * a.hq + h) * D + d0;
#pragma unroll
  for (int d = 0; d < DT; d += 8) {
    uint4 u;
    u.x = pack_bf16x2(acc[d + 0] * inv, acc[d + 1] * inv);
    u.y = pack_bf16x2(acc[d + 2] * inv, acc[d + 3] * inv);
    u.z = pack_bf16x2(acc[d + 4] * inv, acc[d + 5] * inv);
    u.w = pack_bf16x2(acc[d + 6] * inv, acc[d + 7] * inv);
    *reinterpret_cast<uint4*>(op + d) = u;
  }
  if (a.lse && hf == 0 && dq == 0) a.lse[size_t(srow) * a.hq + h] = (mx + fast_log2(wsum)) * kLn2;
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
  const dim3 grid(unsigned(n_tiles) * unsigned(a.hkv) * kCombineParts);
  if (head_dim == 128)
    link_combine_kernel<128><<<grid, kThreads, 0, stream>>>(a);
  else
    link_combine_kernel<64><<<grid, kThreads, 0, stream>>>(a);
}

}  // namespace epic
