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
// staged in LDS by direct global->LDS loads (two buffers each for K and V).  S^T = K Q^T and
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

// LDS stage: K as [64 keys][D] and V as the four blocks' [D][16] slabs, both
// written by direct global->LDS loads (each wavefront instruction fills 1 KB,
// lane l at byte 16 l), so instead of padding the 16-byte chunks are permuted
// within a row: K chunk c of key row r sits at c ^ kswz(r), and the two halves
// of a V row d are swapped when v_swz(d) is set.  The 16 rows one ds_read_b128
// pass touches then fall in distinct banks.
template <int D>
struct AttnLds {
  uint16_t k[2][kKT * D];
  uint16_t v[2][4 * D * 16];
};

template <int D>
__device__ __forceinline__ int kswz(int r) { return D == 128 ? (r & 15) : ((r >> 1) & 7); }
__device__ __forceinline__ int v_swz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from global memory straight into LDS at lds_base + 16 * lane.
__device__ __forceinline__ void dma16(const uint16_t* src, uint16_t* lds_base) {
  __builtin_amdgcn_global_load_lds((global_void*)src, (lds_void*)lds_base, 16, 0, 0);
}
// wait until this wavefront's outstanding global loads (hence its LDS DMA) are done
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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
  // Wavefront w stages block w of each KV tile: its 16 K rows (D/32 instructions
  // of 1 KB) and its [D][16] V slab (D/32 instructions).
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  constexpr int NI = D / 32;                  // 1 KB instructions per operand per wavefront
  constexpr int KRI = 1024 / (2 * D);         // K rows per instruction (4 or 8)
  const int k_rl = lane / (D / 8);            // row within an instruction
  const int k_p = lane % (D / 8);             // chunk position written by this lane
  const int v_d = lane >> 1, v_p = lane & 1;  // V row within an instruction, half position

  // Block metadata of iteration t, gathered one iteration ahead into lanes of
  // one register (a vector load that lands with that iteration's DMA, so the
  // loop never waits on it separately):
  //   lanes  0..3 : physical ids of tile t + 2 (K DMA in iteration t)
  //   lanes  4..7 : physical ids of tile t + 1 (V DMA in iteration t)
  //   lanes  8..11: first positions of tile t's blocks (mask of tile t)
  //   lanes 12..15: valid slots of tile t's blocks, 0 past b1 (mask of tile t)
  //   lanes 16..19: valid slots of tile t + 1's blocks (V fix-up in iteration t)
  auto load_meta = [&](int t) -> int {
    const int j = lane & 31;
    int tile_i, kind;
    if (j < 4) { tile_i = t + 2; kind = 0; }
    else if (j < 8) { tile_i = t + 1; kind = 0; }
    else if (j < 12) { tile_i = t; kind = 1; }
    else if (j < 16) { tile_i = t; kind = 2; }
    else { tile_i = t + 1; kind = 2; }
    const int blk = b0 + tile_i * 4 + (j & 3);
    const int cb = max(b0, min(blk, b1 - 1));    // tile -1 (prologue) and tiles past b1 stay in range
    const int32_t* arr = kind == 0 ? lblk : kind == 1 ? bpos : blenp;
    const int x = arr[cb];
    return (kind == 2 && blk >= b1) ? 0 : x;
  };
  auto meta_at = [&](int meta, int k) -> int { return __builtin_amdgcn_readlane(meta, k); };

  auto dma_k = [&](int buf, int phys) {
    const uint16_t* src = kbase + size_t(phys) * head_k;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = KRI * i + k_rl;           // slot (row) inside the block
      dma16(src + r * D + ((k_p ^ kswz<D>(r)) * 8), &lds.k[buf][(16 * wv + KRI * i) * D]);
    }
  };
  auto dma_v = [&](int buf, int phys) {
    const uint16_t* src = vbase + size_t(phys) * head_k;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int d = 32 * i + v_d;
      dma16(src + d * 16 + ((v_p ^ v_swz(d)) * 8), &lds.v[buf][(wv * D + 32 * i) * 16]);
    }
  };
  // After this wavefront's V DMA of tile `it` landed: zero the slots past its
  // block's end (partial or absent block), so stale or NaN bits never meet a
  // zero softmax weight.  Tiles in the unmasked prefix need nothing.
  auto fix_v = [&](int buf, int it, int len) {
    if (it < n_fast || len >= 16) return;
#pragma unroll
    for (int i = 0; i < D / 64; ++i) {
      const int d = lane + 64 * i;
      uint16_t* row = &lds.v[buf][(wv * D + d) * 16];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        uint4* q = reinterpret_cast<uint4*>(row + (hf ^ v_swz(d)) * 8);
        uint4 x = *q;
        const int valid = len - hf * 8;
        x.x = valid <= 0 ? 0u : valid == 1 ? (x.x & 0xFFFFu) : x.x;
        x.y = valid <= 2 ? 0u : valid == 3 ? (x.y & 0xFFFFu) : x.y;
        x.z = valid <= 4 ? 0u : valid == 5 ? (x.z & 0xFFFFu) : x.z;
        x.w = valid <= 6 ? 0u : valid == 7 ? (x.w & 0xFFFFu) : x.w;
        *q = x;
      }
    }
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
  // 32-key subtiles alternate so that consecutive MFMAs are independent.  The
  // lane reads key row krow (+32 ks), logical chunk 2s + half (dims 16s + 8 half ..).
  const uint16_t* kp_lane = &lds.k[0][krow * D];
  int koff[NDS];
#pragma unroll
  for (int s = 0; s < NDS; ++s) koff[s] = ((2 * s + half) ^ kswz<D>(krow)) * 8;
  auto qk = [&](int buf, f32x16 (&sc)[2]) {
    const uint16_t* kp = kp_lane + buf * (kKT * D);
#pragma unroll
    for (int q = 0; q < 2 * NDS; ++q) {
      const int ks = q & 1, s = q >> 1;
      const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kp + ks * 32 * D + koff[s]);
      sc[ks] = mfma_32x32x16(kf, qreg[s], s == 0 ? f32x16{} : sc[ks]);
    }
  };
  // V^T operand of lane: row d = dt*32 + col, 16-byte half (half ^ swz(col)) of the row.
  const uint16_t* vp_lane = &lds.v[0][col * 16 + (half ^ v_swz(col)) * 8];

  // Software pipeline over KV tiles.  K runs one tile ahead of V: during
  // iteration it the waves read K(it + 1) (buffer (it + 1) % 2, for S(it + 1))
  // and V(it) (buffer it % 2), while the DMA fills K buffer it % 2 with K(it + 2)
  // and V buffer (it + 1) % 2 with V(it + 1) -- buffers nobody reads in
  // iteration it, because their last readers ran before the barrier ending
  // iteration it - 1.  Each wavefront waits for its own DMA before that
  // barrier.  The MFMAs of S(it + 1) are interleaved with the exponentials of
  // tile it.
  int meta;                                    // metadata of the current iteration
  {
    const int pro = load_meta(-1);               // lanes 0..3: tile 1; 4..7: tile 0; 16..19: lengths of tile 0
    meta = load_meta(0);
    wait_vmem();
    const int p0 = meta_at(pro, 4 + wv);
    dma_k(0, p0);
    dma_v(0, p0);
    if (nkv > 1) dma_k(1, meta_at(pro, wv));
    wait_vmem();
    fix_v(0, 0, meta_at(pro, 16 + wv));
  }
  __syncthreads();

  f32x16 sa[2], sb[2];                         // scores of the current / next tile
  qk(0, sa);
  __syncthreads();                             // K buffer 0 is rewritten in iteration 0

  // One KV tile.  sacc holds S(it) on entry; snext receives S(it + 1).
  auto iteration = [&](const int it, f32x16 (&sacc)[2], f32x16 (&snext)[2]) {
    const int cur = it & 1;
    if (it + 2 < nkv) dma_k(cur, meta_at(meta, wv));
    if (it + 1 < nkv) dma_v(cur ^ 1, meta_at(meta, 4 + wv));
    const int meta_next = load_meta(it + 1);   // lands with this iteration's DMA

    // Mask: only tiles past the item's unmasked prefix (diagonal, partial blocks).
    // Register r = i*4 + j of subtile ks holds key ks*32 + (i>>1)*16 + half*8 + (i&1)*4 + j.
    if (it >= n_fast) {
      int bpos0[4], blen[4];
#pragma unroll
      for (int beta = 0; beta < 4; ++beta) {
        bpos0[beta] = meta_at(meta, 8 + beta);
        blen[beta] = meta_at(meta, 12 + beta);
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

    // row max: four chains of three-input maxima, then one lane swap across halves
    float mx[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int ks = c >> 1, r0 = (c & 1) * 8;
      float v = fmaxf(sacc[ks][r0], sacc[ks][r0 + 1]);
#pragma unroll
      for (int r = r0 + 2; r < r0 + 8; r += 2) v = fmaxf(fmaxf(v, sacc[ks][r]), sacc[ks][r + 1]);
      mx[c] = v;
    }
    const float mt = xhalf_max(fmaxf(fmaxf(fmaxf(mx[0], mx[1]), mx[2]), mx[3]));
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
    uint32_t pw[16];                           // P(it) packed to bf16 pairs
    float ps[4];
    auto softmax_step = [&](int q) {
      constexpr int VPS = 32 / (2 * NDS);      // scores per MFMA step
#pragma unroll
      for (int v = 0; v < VPS; ++v) {
        const int idx = q * VPS + v;           // flattened register (ks = idx / 16, r = idx % 16)
        const float p = fast_exp2(__builtin_fmaf(sacc[idx >> 4][idx & 15], sl2, -m_use));
        sacc[idx >> 4][idx & 15] = p;
        ps[idx & 3] = idx < 4 ? p : ps[idx & 3] + p;
        if (idx & 1) pw[idx >> 1] = pack_bf16x2(sacc[idx >> 4][(idx & 15) - 1], p);
      }
    };
    if (it + 1 < nkv) {
      const uint16_t* kp = kp_lane + (cur ^ 1) * (kKT * D);
      constexpr int NQ = 2 * NDS;
      bf16x8 kf[3];                            // K fragments, read two steps ahead
      auto kfrag = [&](int q) {
        return *reinterpret_cast<const bf16x8*>(kp + (q & 1) * 32 * D + koff[q >> 1]);
      };
      kf[0] = kfrag(0);
      kf[1] = kfrag(1);
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int ks = q & 1, s = q >> 1;
        if (q + 2 < NQ) kf[(q + 2) % 3] = kfrag(q + 2);
        snext[ks] = mfma_32x32x16(kf[q % 3], qreg[s], s == 0 ? f32x16{} : snext[ks]);
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
    constexpr int NV = 4 * NDT;                // PV MFMAs
    bf16x8 vf[3];                              // V^T fragments, read two MFMAs ahead
    auto vfrag = [&](int n) {
      return *reinterpret_cast<const bf16x8*>(vp + (n / NDT) * D * 16 + (n % NDT) * 32 * 16);
    };
    vf[0] = vfrag(0);
    vf[1] = vfrag(1);
#pragma unroll
    for (int n = 0; n < NV; ++n) {
      const int kst = n / NDT, dt = n % NDT;
      if (n + 2 < NV) vf[(n + 2) % 3] = vfrag(n + 2);
      const bf16x8 pbk = __builtin_bit_cast(
          bf16x8, make_uint4(pw[4 * kst + 0], pw[4 * kst + 1], pw[4 * kst + 2], pw[4 * kst + 3]));
      o[dt] = mfma_32x32x16(vf[n % 3], pbk, o[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (it + 1 < nkv) {
      wait_vmem();                             // this wavefront's DMA of K(it + 2), V(it + 1) landed
      fix_v(cur ^ 1, it + 1, meta_at(meta, 16 + wv));
      __syncthreads();                         // ... and everybody's: visible, buffers free
    }
    meta = meta_next;
  };

  // two tiles per trip, so the score buffers swap roles without copies
  for (int it = 0; it < nkv; it += 2) {
    iteration(it, sa, sb);
    if (it + 1 < nkv) iteration(it + 1, sb, sa);
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
