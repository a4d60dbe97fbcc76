// Scattered-query causal attention over the paged linked cache (Eq. 1).
//
// Each S row at linked position p, query head h, attends to the linked keys at
// positions <= p of KV head h / G (MASK of Eq. 1, read as additive -inf with the
// diagonal included), scale 1/sqrt(D).  The linked cache is a list of blocks
// (physical id, first position, valid slots), so chunk caches are read in place
// and recomputed rows come from the private blocks written just before.
//
// Work decomposition (built by the host planner):
//   tile  = T query rows (T = 128 or 256, chosen per plan) = (S rows of one
//           request) x (G query heads of one KV head), row t -> S row t % (T/G),
//           head t / (T/G);
//   item  = (tile, range of linked blocks); rows whose key range spans several
//           items get partial results (O / l, log2 l + m) merged by the combine kernel.
// Grid = items x Hkv with blockIdx % Hkv = KV head: with 8 KV heads each XCD
// (workgroups are dealt round-robin to the 8 XCDs) serves one head, and the
// planner orders items key-segment first, so concurrent workgroups on an XCD
// read the same KV blocks through its L2.
//
// Per workgroup: T / 32 wavefronts x 32 rows sharing each K/V stage.  Per step
// 64 keys (4 blocks) are staged in LDS by direct buffer->LDS loads:
//   T = 256: one workgroup per CU, 8 wavefronts -- 0..3 load the four K blocks,
//            4..7 the four V blocks -- three buffers each, loads issued two
//            steps before their use;
//   T = 128: two workgroups per CU, 4 wavefronts each loading one K and one V
//            block, two buffers each, loads issued one step before their use.
// S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_32x32x16_bf16: each lane
// owns one query row (its MFMA column), so the row max / sum need a single lane
// swap (l <-> l^32).  P is rounded to bf16 for the second product; softmax runs
// in base 2 with scale*log2(e) applied inside the exponent's FMA; the running
// output is rescaled only when some row's maximum grew; accumulation is fp32.
//
// Software pipeline: step i issues the PV product of tile i-1 and the QK
// product of tile i+1, alternating, and spreads the softmax of tile i (row
// maximum, then the 32 exponentials per lane) and the step's buffer->LDS loads
// over those 32 MFMAs, so the matrix cores always have independent work beside
// the vector ALU work.
#include <utility>

#include "device_common.h"
#include "kernels.h"
#include "plan_internal.h"

namespace epic {

namespace {

constexpr int kKT = 64;     // keys per step (4 blocks of 16)
// LDS buffers per operand for W wavefronts per workgroup
template <int W>
constexpr int kStages = W == 8 ? 3 : 2;
// Word 3 of a gfx9-family raw buffer descriptor (32-bit data format, no swizzle).
constexpr int kBufWord3 = 0x00020000;

// LDS stage, written by direct buffer->LDS loads (each wavefront instruction
// fills 1 KB, lane l at byte 16 l):
//   K as [block][row group g = row / 8][chunk c ^ g][row % 8] in 16-byte units
//     (c = 16-byte chunk of the head dim) -- each load instruction reads 8 whole
//     rows of a block; the 16 lanes of one ds_read_b128 group read chunk c of 16
//     consecutive keys as two 128-byte runs half a bank-row apart (the ^ g),
//     and every K operand sits at a fixed offset from the lane's base;
//   V as the four blocks' [D][16] slabs with the two halves of row d swapped
//     when v_swz(d) is set, so the 16 rows one group touches fall in distinct banks.
//   Q: the last kQl<D> 16-dim slices of every lane's query row (16 bytes per
//     lane each), which would not fit in registers beside the rest.
template <int D>
constexpr int kQl = D == 128 ? 2 : 0;
template <int D, int W>
struct AttnLds {
  uint16_t k[kStages<W>][kKT * D];
  uint16_t v[kStages<W>][4 * D * 16];
  uint16_t q[kQl<D> > 0 ? kQl<D> : 1][64 * W * 8];
};

__device__ __forceinline__ int v_swz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

typedef __attribute__((address_space(3))) void lds_void;

// One wavefront's share of a block: D/32 loads of 16 bytes per lane from the
// block's descriptor into LDS.  Load I lands lane l at LDS byte dst + 1024 I + 16 l
// and reads block byte voff(I) + GOFF(I); the instruction offset GOFF(I) moves
// both addresses, so the LDS base handed to load I is dst + 1024 I - GOFF(I).
template <class GOFF, int... I>
__device__ __forceinline__ void dma_block(__amdgpu_buffer_rsrc_t rs, char* dst, int voff_even, int voff_odd,
                                          std::integer_sequence<int, I...>) {
#if defined(__HIP_DEVICE_COMPILE__)   // the host pass only parses kernel bodies
  (__builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + 1024 * I - GOFF::template at<I>()), 16,
                                            GOFF::template odd<I>() ? voff_odd : voff_even, 0,
                                            GOFF::template at<I>(), 0),
   ...);
#endif
}
// One 16-byte-per-lane buffer->LDS load (lane l's 16 bytes land at dst + 16 l, the
// lane offset moving the memory address only).  A plain function, so that a call
// from a kernel template is never a template-dependent expression (the host pass
// cannot check the builtin there and would drop the kernel).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, char* dst, int voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 16, voff, 0, 0, 0);
}
// K load I of a D-wide block: row group rb = 64 I / (8 NCH), chunk base v0 = (64 I % (8 NCH)) / 8;
// lane l reads row 8 rb + l % 8, chunk (v0 + l / 8) ^ rb.
template <int D>
struct KLoads {
  static constexpr int NCH = D / 8;
  template <int I> static constexpr int rb() { return 64 * I / (8 * NCH); }
  template <int I> static constexpr int at() { return 16 * rb<I>() * D + 16 * ((64 * I % (8 * NCH)) / 8); }
  template <int I> static constexpr bool odd() { return rb<I>() & 1; }
};
// V load I: rows 32 I .. 32 I + 31 of the [D][16] slab, 1 KB contiguous.
struct VLoads {
  template <int I> static constexpr int at() { return 1024 * I; }
  template <int I> static constexpr bool odd() { return false; }
};
// Workgroup barrier ordering LDS accesses only: the wavefront's own LDS reads
// and writes complete (lgkmcnt(0)) before it, and the memory clobber keeps the
// compiler from moving or forwarding memory accesses across it, while the
// wavefront's buffer->LDS loads still in flight stay in flight (a fence would
// wait for them too, since they write LDS).
__device__ __forceinline__ void barrier_lds() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// f(integral_constant<int, I>) for I = 0 .. N-1, every index a compile-time constant
template <class F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// wait until at most N of this wavefront's vector memory loads (hence LDS DMA
// writes) are outstanding; they complete in issue order
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

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

template <int D, int W>
__global__ __launch_bounds__(64 * W, W == 8 ? 1 : 2) void link_attention_kernel(AttnArgs a) {
  constexpr int kThreads = 64 * W;
  constexpr int S = kStages<W>;               // LDS buffers per operand
  constexpr int TR = 32 * W;                  // tile rows
  constexpr int NDS = D / 16;                 // k-steps of S^T = K Q^T
  constexpr int NDT = D / 32;                 // 32-row tiles of O^T
  constexpr int NSLOT = 2 * NDS;              // QK MFMAs per tile (= PV MFMAs, 4 * NDT)
  static_assert(NSLOT == 4 * NDT, "QK and PV MFMA counts pair up");
  __shared__ __attribute__((aligned(16))) AttnLds<D, W> lds;

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

  const int tid = threadIdx.x & (kThreads - 1);   // blockDim.x == kThreads
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, half = lane >> 5;
  const int t = wave * 32 + col;               // tile row of this lane
  const int R = a.rows_per_tile;
  const int srl = t % R, h = g * a.G + t / R;
  const bool row_ok = srl < nrows;
  const int srow = row0 + (row_ok ? srl : nrows - 1);
  const int qpos = a.s_pos[srow];

  // Q operand of k-step s (dims 16 s + 8 half ..): registers for s < NQR, LDS above
  constexpr int NQR = NDS - kQl<D>;
  bf16x8 qreg[NQR];
  {
    const uint16_t* qp = a.q + (size_t(srow) * a.hq + h) * D + half * 8;
#pragma unroll
    for (int s = 0; s < NDS; ++s) {
      bf16x8 x = *reinterpret_cast<const bf16x8*>(qp + s * 16);
      if (!row_ok) x = bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
      if (s < NQR) qreg[s < NQR ? s : 0] = x;
      else *reinterpret_cast<bf16x8*>(&lds.q[s - NQR][tid * 8]) = x;
    }
  }
  auto qfrag = [&](int s) -> bf16x8 {
    return s < NQR ? qreg[s < NQR ? s : 0] : *reinterpret_cast<const bf16x8*>(&lds.q[s - NQR][tid * 8]);
  };

  const int nkv = (b1 - b0 + 3) / 4;
  // Block dw of each KV tile is staged by this wavefront: its 16 K rows (k_wave)
  // and / or its [D][16] V slab (v_wave), D/32 loads of 1 KB each through a
  // descriptor over that block.  W = 8: wavefronts 0..3 K, 4..7 V; W = 4: both.
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int dw = wv & 3;
  const bool k_wave = W == 4 || wv < 4;
  const bool v_wave = W == 4 || wv >= 4;
  constexpr int NI = D / 32;                  // 1 KB loads per operand per wavefront
  constexpr int NCH = D / 8;                  // 16-byte chunks per K row
  const char* kbase = reinterpret_cast<const char*>(a.k_cache + size_t(g) * 16 * D);
  const char* vbase = reinterpret_cast<const char*>(a.v_cache + size_t(g) * 16 * D);
  const size_t blk_bytes = size_t(hkv) * 16 * D * 2;   // one physical block, all heads
  // Lane byte offsets in the block, the per-load constant part left to the
  // instruction offset: K load i reads row 8 rb + l % 8, chunk (v0 + l / 8) ^ rb,
  // block byte (l % 8) 2D + ((l / 8) ^ rb) 16 + [16 rb D + 16 v0]; V load i reads
  // row d = 32 i + l / 2, half (l & 1) ^ v_swz(d) = (l & 1) ^ v_swz(l / 2), block
  // byte 32 (l / 2) + 16 ((l & 1) ^ v_swz(l / 2)) + [1024 i].
  const int kvo = (lane & 7) * 2 * D + (lane >> 3) * 16;
  const int vvo = (lane >> 1) * 32 + ((lane & 1) ^ v_swz(lane >> 1)) * 16;
  auto dma_k = [&](int buf, int phys) {
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kbase) + size_t(phys) * blk_bytes, 0,
                                                      16 * D * 2, kBufWord3);
    dma_block<KLoads<D>>(rs, reinterpret_cast<char*>(&lds.k[buf][16 * dw * D]), kvo, kvo ^ 16,
                         std::make_integer_sequence<int, NI>{});
  };
  auto dma_v = [&](int buf, int phys) {
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(vbase) + size_t(phys) * blk_bytes, 0,
                                                      16 * D * 2, kBufWord3);
    dma_block<VLoads>(rs, reinterpret_cast<char*>(&lds.v[buf][dw * D * 16]), vvo, vvo,
                      std::make_integer_sequence<int, NI>{});
  };
  // The same loads one at a time (load I of the block), from a descriptor made once.
  auto rsrc_k = [&](int phys) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(kbase) + size_t(phys) * blk_bytes, 0, 16 * D * 2,
                                             kBufWord3);
  };
  auto rsrc_v = [&](int phys) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(vbase) + size_t(phys) * blk_bytes, 0, 16 * D * 2,
                                             kBufWord3);
  };
  auto dma_k1 = [&](auto ic, int buf, __amdgpu_buffer_rsrc_t rs) __attribute__((always_inline)) {
    dma_block<KLoads<D>>(rs, reinterpret_cast<char*>(&lds.k[buf][16 * dw * D]), kvo, kvo ^ 16,
                         std::integer_sequence<int, decltype(ic)::value>{});
  };
  auto dma_v1 = [&](auto ic, int buf, __amdgpu_buffer_rsrc_t rs) __attribute__((always_inline)) {
    dma_block<VLoads>(rs, reinterpret_cast<char*>(&lds.v[buf][dw * D * 16]), vvo, vvo,
                      std::integer_sequence<int, decltype(ic)::value>{});
  };
  // W = 8: a wavefront loads K or V, so one pair of lane offsets serves either
  const int so_even = !k_wave ? vvo : kvo;
  const int so_odd = !k_wave ? vvo : kvo ^ 16;

  // Block metadata, read with scalar loads: the tables are read-only while the
  // kernel runs, and scalar loads are counted by lgkmcnt, so waiting for them
  // never waits for the buffer->LDS loads in flight.  Indices are clamped into
  // the item's range [b0, b1).
  typedef __attribute__((address_space(4))) const int32_t cint32;
  const cint32* lb_c = (const cint32*)a.linked_blocks;
  const cint32* pos_c = (const cint32*)a.block_pos0;
  const cint32* len_c = (const cint32*)a.block_len;
  auto blk_at = [&](const cint32* arr, int i) -> int { return arr[max(b0, min(i, b1 - 1))]; };
  // physical ids this wavefront stages in step ts: K(ts + S) and V(ts + S - 2), block dw
  auto phys_k = [&](int ts) -> int { return blk_at(lb_c, b0 + 4 * (ts + S) + dw); };
  auto phys_v = [&](int ts) -> int { return blk_at(lb_c, b0 + 4 * (ts + S - 2) + dw); };
  // W = 8 reads the ids of later steps ahead with a vector load (every lane loads
  // the same word), two steps before their use: a scalar load in the step had its
  // reply waited for at once (an LDS wait behind a scalar load must be a full wait,
  // since scalar loads may return out of order).  Vector loads complete in issue
  // order with the buffer->LDS loads, so the step's closing wait covers them.  The
  // index is clamped into [b0, b1) as above.
  const auto lb_rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.linked_blocks), 0, b1 * 4, kBufWord3);
  auto id_index = [&](int ts) -> int {
    return max(b0, min(b0 + 4 * (ts + (k_wave ? S : S - 2)) + dw, b1 - 1));
  };
  int idr[2] = {0, 0};                         // ids of steps of either parity, in flight (W = 8)
  // first position / valid slots of block beta of tile ts (0 slots past b1)
  auto blk_pos = [&](int ts, int beta) -> int { return blk_at(pos_c, b0 + 4 * ts + beta); };
  auto blk_len = [&](int ts, int beta) -> int {
    return b0 + 4 * ts + beta < b1 ? blk_at(len_c, b0 + 4 * ts + beta) : 0;
  };

  // After this wavefront's V DMA of tile `it` landed: zero the slots past its
  // block's end (partial or absent block), so stale or NaN bits never meet a
  // zero softmax weight.  Tiles in the unmasked prefix need nothing.
  auto fix_v = [&](int buf, int it, int len) {
    if (it < n_fast || len >= 16) return;
#pragma unroll
    for (int i = 0; i < D / 64; ++i) {
      const int d = lane + 64 * i;
      uint16_t* row = &lds.v[buf][(dw * D + d) * 16];
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
  // A step of the fast form keeps m if no lane's sum of P passes kFastSum, just
  // under 2^kLag.  Then no P passed it, so no row maximum rose past m + kLag
  // (the margin, log2(256 / 255) = 0.0056, covers the roundings of the exponent
  // and of the full step's test), and the full step would have kept m too:
  // both forms give the same bits.
  constexpr float kFastSum = 255.0f;
  constexpr int kFastMin = 16;                 // unmasked tiles an item needs to take the fast form
  static_assert(kLag == 8.0f, "kFastSum sits just under 2^kLag");
  float m = -INFINITY, lsum = 0.0f;
  const float sl2 = a.scale_log2;
  const int krow = srow_key(col);              // K row this lane feeds into S^T

  // S^T (64 keys x 32 rows per wave) = K Q^T: MFMA q = (subtile q & 1, k-step
  // q >> 1); the lane reads key krow + 32 subtile (block 2 subtile + krow / 16,
  // row r = krow % 16, group r / 8), chunk c = 2 s + half, stored at chunk
  // position c ^ (r / 8) = 2 s + (half ^ (r / 8)).
  const int kr = krow & 15;
  const uint16_t* kp_lane =
      &lds.k[0][((krow >> 4) * 16 * NCH + (kr >> 3) * 8 * NCH + (half ^ (kr >> 3)) * 8 + (kr & 7)) * 8];
  // V^T operand of lane: row d = dt*32 + col, 16-byte half (half ^ swz(col)) of the row.
  const uint16_t* vp_lane = &lds.v[0][col * 16 + (half ^ v_swz(col)) * 8];
  auto kfrag = [&](int buf, int q) {
    return *reinterpret_cast<const bf16x8*>(kp_lane + buf * (kKT * D) + (q & 1) * (2 * 16 * NCH * 8) +
                                            (q >> 1) * (2 * 8 * 8));
  };
  // PV MFMA n = (16-key step n / NDT, O^T tile n % NDT)
  auto vfrag = [&](int buf, int n) {
    return *reinterpret_cast<const bf16x8*>(vp_lane + buf * (4 * D * 16) + (n / NDT) * D * 16 + (n % NDT) * 32 * 16);
  };
  // P of a tile as 4 MFMA B operands: operand kst = keys kst*16 + half*8 + [0, 8)
  // as bf16 pairs (score registers 8 kst .. 8 kst + 7 of the S^T layout)
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  auto pfrag = [&](const u32x4 (&p)[4], int kst) { return __builtin_bit_cast(bf16x8, p[kst]); };

  // Pipeline: K(t) and V(t) live in LDS buffer t % S.  Step t reads K(t + 1)
  // and V(t - 1), and issues K(t + S) and V(t + S - 2) into the buffers whose
  // last readers ran in step t - 1; at its end every wavefront waits for its
  // loads of K(t + 2) and V(t) -- with S = 3 those were issued a step earlier,
  // and the loads of this step stay in flight -- and the barrier publishes
  // them.  The loads are issued every step (past the item's end with clamped
  // block ids), so each step leaves exactly NI loads outstanding (S = 3).
  if (k_wave) {                                // K(0) .. K(S - 1)
#pragma unroll
    for (int j = 0; j < S; ++j) dma_k(j, phys_k(j - S));
  }
  if (v_wave) {                                // V(0) .. V(S - 3)
#pragma unroll
    for (int j = 0; j < S - 2; ++j) dma_v(j, phys_v(j - S + 2));
  }
  int pk = phys_k(0), pv = phys_v(0);          // blocks this wavefront stages in the current step
  if constexpr (W == 8) idr[1] = __builtin_amdgcn_raw_buffer_load_b32(lb_rs, 0, id_index(1) * 4, 0);
  wait_vmem<0>();
  if (S == 3 && v_wave) fix_v(0, 0, blk_len(0, dw));
  __syncthreads();

  f32x16 s0[2], s1[2];                         // scores of even / odd tiles
  u32x4 p0[4], p1[4];                          // P of even / odd tiles, packed bf16 pairs
#pragma unroll
  for (int q = 0; q < NSLOT; ++q) {
    const int ks = q & 1, s = q >> 1;
    s0[ks] = mfma_32x32x16(kfrag(0, q), qfrag(s), s == 0 ? f32x16{} : s0[ks]);
  }
  __syncthreads();                             // K buffer 0 is rewritten in step 0 (K(S))

  // One step over tile it.  sc = S(it) on entry (complete); pp = P(it - 1) (PV
  // only); the step leaves P(it) in pc and S(it + 1) in sn (QK only).
  auto step = [&](auto pv_tag, auto qk_tag, auto fast_tag, auto par_tag, const int it, f32x16 (&sc)[2],
                  f32x16 (&sn)[2], const u32x4 (&pp)[4], u32x4 (&pc)[4]) __attribute__((always_inline)) {
    constexpr bool PV = decltype(pv_tag)::value;
    constexpr bool QK = decltype(qk_tag)::value;
    constexpr int PAR = decltype(par_tag)::value;   // it % 2
    // FAST: an unmasked tile after the first, all scores finite and m finite in
    // every row; the exponentials use the current m without a row maximum, and
    // the step is redone as a full one only if some lane's sum of P passes
    // kFastSum (a row maximum that may have risen past m + kLag).
    constexpr bool FAST = decltype(fast_tag)::value;
    const int b3 = it % S;                     // buffer of K(it), V(it), K(it + S)
    const int b3n = b3 == S - 1 ? 0 : b3 + 1;  // buffer of K(it + 1) (and V(it + 1) when S = 3)
    const int b3p = b3 == 0 ? S - 1 : b3 - 1;  // buffer of V(it - 1)
    // K(it + S) into b3 (its buffer held K(it)) and V(it + S - 2) into the buffer of
    // V(it - 2): both buffers are free for the whole step, so the step's loads are
    // spread over its MFMA slots rather than issued together after the barrier, where
    // the eight wavefronts' loads queued behind each other.  W = 8: load I at slot
    // I * KSP + (I odd ? KSP / 2 : 0).  W = 4: K load I at slot I * KSP, V load I half
    // a spacing later, all within the first half of the step (S = 2: the loads must
    // land by the step's end).
    const auto rk = rsrc_k(pk);
    const auto rv = rsrc_v(pv);
    const int vbuf = S == 3 ? b3n : b3;
    char* const dma_dst = k_wave ? reinterpret_cast<char*>(&lds.k[b3][16 * dw * D])
                                 : reinterpret_cast<char*>(&lds.v[vbuf][dw * D * 16]);
    int pk_next = 0, pv_next = 0;
    if constexpr (W == 4) {
      pk_next = phys_k(it + 1);
      pv_next = phys_v(it + 1);
    }

    // Mask: only tiles past the item's unmasked prefix (diagonal, partial blocks).
    // Register r = i*4 + j of subtile ks holds key ks*32 + (i>>1)*16 + half*8 + (i&1)*4 + j.
    if (!FAST && it >= n_fast) {
      int bpos0[4], blen[4];
#pragma unroll
      for (int beta = 0; beta < 4; ++beta) {
        bpos0[beta] = blk_pos(it, beta);
        blen[beta] = blk_len(it, beta);
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = r >> 2, j = r & 3;
          const int beta = ks * 2 + (i >> 1);
          const int slot = half * 8 + (i & 1) * 4 + j;
          const bool ok = slot < blen[beta] && bpos0[beta] + slot <= qpos;
          sc[ks][r] = ok ? sc[ks][r] : -INFINITY;
        }
    }

    bf16x8 kf[3], vf[3], qf[2];                // operands, read two MFMAs ahead
    if (PV) { vf[0] = vfrag(b3p, 0); vf[1] = vfrag(b3p, 1); }
    if (!PV && QK) {
      kf[0] = kfrag(b3n, 0);
      kf[1] = kfrag(b3n, 1);
    }

    float mx[4], m_cand = 0.0f, alpha = 1.0f, m_use = FAST ? m : 0.0f;
    bool grow = false;
    float ps[4];
    // MFMA slots: 0 .. NSLOT-1 the PV product of tile it - 1, NSLOT .. 2 NSLOT-1
    // the QK product of tile it + 1 (so S(it + 1) fills while S(it) drains).
    // Softmax work of tile it per slot: slots 0..3 the row maximum and the
    // rescale decision, slots 4.. the exponentials (unit u = score u).
    constexpr int kMaxSlots = 4;
    constexpr int NS2 = 2 * NSLOT;
    float pe = 0.0f;                           // P of the even unit of the pair being packed
    auto exp_unit = [&](auto uc) __attribute__((always_inline)) {
      constexpr int u = decltype(uc)::value;
      const float p = fast_exp2(__builtin_fmaf(sc[u >> 4][u & 15], sl2, -m_use));
      ps[u & 3] = u < 4 ? p : ps[u & 3] + p;
      // Keep this unit's work in its slot: P is only read in the next step and
      // the sums at its end, and the compiler would otherwise move all the
      // exponentials to those first uses (and hold 32 of them live).  The
      // scores stay as they are, for the redo of a fast step.
      __asm__ volatile("" ::"v"(ps[u & 3]));
      if constexpr (u & 1) {
        pc[u >> 3][(u >> 1) & 3] = pack_bf16x2(pe, p);
        __asm__ volatile("" ::"v"(pc[u >> 3][(u >> 1) & 3]));
      } else {
        pe = p;
      }
    };
    static_for<NS2>([&](auto qc) __attribute__((always_inline)) {
      constexpr int q = decltype(qc)::value;
      constexpr int KSP = (S == 3 ? NS2 : NS2 / 2) / NI;     // slots between a wavefront's K loads
      if constexpr (W == 8 && q == 1) {
        // id of step it + 2 (same parity), after this step's first buffer->LDS load
        idr[PAR] = __builtin_amdgcn_raw_buffer_load_b32(lb_rs, 0, id_index(it + 2) * 4, 0);
      }
      static_for<NI>([&](auto ic) __attribute__((always_inline)) {
        constexpr int I = decltype(ic)::value;
        if constexpr (W == 8) {
          // one load per wavefront and slot, K or V by uniform selects (no branch
          // among the MFMAs); the K / V offset of load I rides in the lane offset,
          // which moves the memory address only
          if constexpr (q == I * KSP + (I & 1) * (KSP / 2)) {
            const int voff = (KLoads<D>::template odd<I>() ? so_odd : so_even) +
                             (k_wave ? KLoads<D>::template at<I>() : VLoads::template at<I>());
            dma16(k_wave ? rk : rv, dma_dst + 1024 * I, voff);
          }
        } else {
          if constexpr (q == I * KSP) dma_k1(ic, b3, rk);
          if constexpr (q == I * KSP + KSP / 2) dma_v1(ic, vbuf, rv);
        }
      });
      if constexpr (q + 2 < NSLOT) {
        if constexpr (PV) vf[(q + 2) % 3] = vfrag(b3p, q + 2);
      } else if constexpr (q + 2 < NS2) {
        constexpr int k2 = q + 2 - NSLOT;
        if constexpr (QK && (PV || k2 >= 2)) {
          kf[k2 % 3] = kfrag(b3n, k2);
          if constexpr ((k2 & 1) == 0 && (k2 >> 1) >= NQR) qf[((k2 >> 1) - NQR) & 1] = qfrag(k2 >> 1);
        }
      }
      if constexpr (q < NSLOT) {
        if constexpr (PV) o[q % NDT] = mfma_32x32x16(vf[q % 3], pfrag(pp, q / NDT), o[q % NDT]);
      } else {
        constexpr int k = q - NSLOT;
        if constexpr (QK) {
          bf16x8 qo;
          if constexpr ((k >> 1) < NQR) qo = qreg[(k >> 1) < NQR ? (k >> 1) : 0];
          else qo = qf[((k >> 1) - NQR) & 1];
          sn[k & 1] = mfma_32x32x16(kf[k % 3], qo, (k >> 1) == 0 ? f32x16{} : sn[k & 1]);
        }
      }
      // row max over the 32 scores: four chains of three-input maxima (7 + 8 + 8
      // + 8 scores), each step max3(running, a, b), then the chains and the lane swap
      if constexpr (FAST) {                    // no maximum: one exponential unit per slot share
        static_for<32>([&](auto uc) __attribute__((always_inline)) {
          if constexpr ((decltype(uc)::value * NS2) / 32 == q) exp_unit(uc);
        });
      } else if constexpr (q == 0) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int ks = c >> 1, r0 = (c & 1) * 8;
          mx[c] = c == 0 ? fmaxf(fmaxf(sc[0][0], sc[0][1]), sc[0][2])
                         : fmaxf(fmaxf(mx[0], sc[ks][r0]), sc[ks][r0 + 1]);
          if (c == 0) continue;
          mx[c] = fmaxf(fmaxf(mx[c], sc[ks][r0 + 2]), sc[ks][r0 + 3]);
        }
      } else if constexpr (q == 1) {
        mx[0] = fmaxf(fmaxf(mx[0], sc[0][3]), sc[0][4]);
        mx[0] = fmaxf(fmaxf(mx[0], sc[0][5]), sc[0][6]);
#pragma unroll
        for (int c = 1; c < 4; ++c) {
          const int ks = c >> 1, r0 = (c & 1) * 8;
          mx[c] = fmaxf(fmaxf(mx[c], sc[ks][r0 + 4]), sc[ks][r0 + 5]);
          mx[c] = fmaxf(fmaxf(mx[c], sc[ks][r0 + 6]), sc[ks][r0 + 7]);
        }
        mx[0] = fmaxf(fmaxf(mx[0], sc[0][7]), mx[1]);
      } else if constexpr (q == 2) {
        const float mt = xhalf_max(fmaxf(fmaxf(mx[0], mx[2]), mx[3]));
        m_cand = fmaxf(m, mt * sl2);
      } else if constexpr (q == 3) {
        grow = m_cand > m + kLag;              // also true on the first finite max
        alpha = grow ? fast_exp2(m - m_cand) : 1.0f;
        m = grow ? m_cand : m;
        m_use = m == -INFINITY ? 0.0f : m;
      } else {
        static_for<32>([&](auto uc) __attribute__((always_inline)) {
          if constexpr (kMaxSlots + (decltype(uc)::value * (NS2 - kMaxSlots)) / 32 == q) exp_unit(uc);
        });
      }
      __builtin_amdgcn_sched_barrier(0);
    });
    float ssum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
    if constexpr (FAST) {
      if (__ballot(ssum > kFastSum)) {         // redo as the full step: same maximum, same sums
        float mr = sc[0][0];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int r = 0; r < 16; ++r) mr = fmaxf(mr, sc[ks][r]);
        m_cand = fmaxf(m, xhalf_max(mr) * sl2);
        grow = m_cand > m + kLag;
        alpha = grow ? fast_exp2(m - m_cand) : 1.0f;
        m = grow ? m_cand : m;
        m_use = m;
        static_for<32>([&](auto uc) __attribute__((always_inline)) {
          constexpr int u = decltype(uc)::value;
          const float p = fast_exp2(__builtin_fmaf(sc[u >> 4][u & 15], sl2, -m_use));
          ps[u & 3] = u < 4 ? p : ps[u & 3] + p;
          if constexpr (u & 1) pc[u >> 3][(u >> 1) & 3] = pack_bf16x2(pe, p);
          else pe = p;
        });
        ssum = (ps[0] + ps[1]) + (ps[2] + ps[3]);
        if (PV && __ballot(grow)) {
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
        }
      }
    }
    lsum = lsum * alpha + ssum;
    if (!FAST && PV && __ballot(grow)) {       // O holds PV(it - 1): move it to the new maximum
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[dt][r] *= alpha;
    }
    // this wavefront's loads of K(it + 2), V(it) (W = 8: and the id of step it + 1)
    wait_vmem<S == 3 ? NI + 1 : 0>();
    if (v_wave) fix_v(b3, it, blk_len(it, dw));
    barrier_lds();                             // ... of every wavefront: visible, buffers free
    if constexpr (W == 8) {
      const int id = __builtin_amdgcn_readfirstlane(idr[PAR ^ 1]);
      pk = id;
      pv = id;
    } else {
      pk = pk_next;
      pv = pv_next;
    }
  };
  // PV of the last tile (nothing left to overlap it with).
  auto last_pv = [&](const u32x4 (&pp)[4], int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NSLOT; ++q) o[q % NDT] = mfma_32x32x16(vfrag(buf, q), pfrag(pp, q / NDT), o[q % NDT]);
  };

  using T = std::true_type;
  using F = std::false_type;
  using E = std::integral_constant<int, 0>;   // even step
  using O = std::integral_constant<int, 1>;   // odd step
  if (nkv == 1) {
    step(F{}, F{}, F{}, E{}, 0, s0, s1, p1, p0);
    last_pv(p0, 0);
  } else {
    // tile 0 sets m: unmasked (n_fast > 0), it gives every row a finite maximum
    step(F{}, T{}, F{}, E{}, 0, s0, s1, p1, p0);
    int it = 1;
    // two steps per trip while both tiles have a successor; odd tiles keep
    // their scores / P in s1 / p1, even tiles in s0 / p0.  Pairs of unmasked
    // tiles take the fast form.
    for (; n_fast >= kFastMin && it + 2 < nkv && it + 1 < n_fast; it += 2) {
      step(T{}, T{}, T{}, O{}, it, s1, s0, p0, p1);
      step(T{}, T{}, T{}, E{}, it + 1, s0, s1, p1, p0);
    }
    for (; it + 2 < nkv; it += 2) {
      step(T{}, T{}, F{}, O{}, it, s1, s0, p0, p1);
      step(T{}, T{}, F{}, E{}, it + 1, s0, s1, p1, p0);
    }
    if (it + 1 < nkv) {                        // tiles it (odd) and it + 1 (last) remain
      step(T{}, T{}, F{}, O{}, it, s1, s0, p0, p1);
      step(T{}, F{}, F{}, E{}, it + 1, s0, s1, p1, p0);
      last_pv(p0, (it + 1) % S);
    } else {                                   // tile it (odd) is the last
      step(T{}, F{}, F{}, O{}, it, s1, s0, p0, p1);
      last_pv(p1, it % S);
    }
  }
  wait_vmem<0>();                              // the last step's loads land before the LDS is released

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
    float* pp = a.part_o + ((size_t(part) * hkv + g) * TR + t) * D + half * 4;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float4 f = make_float4(o[dt][i * 4 + 0] * inv, o[dt][i * 4 + 1] * inv, o[dt][i * 4 + 2] * inv,
                               o[dt][i * 4 + 3] * inv);
        *reinterpret_cast<float4*>(pp + dt * 32 + i * 8) = f;
      }
    if (half == 0)
      a.part_lse[(size_t(part) * hkv + g) * TR + t] = ltot > 0.0f ? m + fast_log2(ltot) : -INFINITY;
  }
}

// Merge the split-KV partials of a tile: lse = log2 sum_i 2^lse_i, out = sum_i 2^(lse_i - lse) O_i.
// Workgroup = (tile, KV head, quarter of the head dim).  Each (valid tile row, half
// of that quarter) gets P lanes of one wavefront (P a power of two, at most 64, the
// number of partials, and 512 / (2 x valid rows)); lane j takes partials j, j + P, ..., and the lanes
// combine their (max, weight sum, weighted sums) by butterfly exchanges.  A tile
// of few rows (decode: one row per head) with many partials so gets the whole
// workgroup's memory parallelism.
constexpr int kCombineParts = 4;
constexpr int kCombineThreads = 512;
template <int D>
__global__ __launch_bounds__(kCombineThreads) void link_combine_kernel(AttnArgs a) {
  constexpr int DQ = D / kCombineParts;       // dims per workgroup
  constexpr int DT = DQ / 2;                  // dims per (row, half)
  const int hkv = a.hkv;
  const int dq = blockIdx.x % kCombineParts;
  const int g = (blockIdx.x / kCombineParts) % hkv;
  const int tile = blockIdx.x / (kCombineParts * hkv);
  const int p0 = a.tiles[4 * tile + 2];
  const int ns = a.tiles[4 * tile + 3];
  if (p0 < 0) return;
  const int nrows = a.tiles[4 * tile + 1];
  const int R = a.rows_per_tile, TR = a.tile_rows;
  const int n_valid = nrows * a.G;            // tile rows t = head * R + s, s < nrows
  const int pairs = 2 * n_valid;
  int P = 64;                                 // lanes per (row, half): no more than partials
  while (P > 1 && (P * pairs > kCombineThreads || P > ns)) P >>= 1;
  const int pair = threadIdx.x / P, j = threadIdx.x % P;
  if (pair >= pairs) return;                  // whole groups of P lanes leave together
  const int vr = pair >> 1, hf = pair & 1;
  const int hh = vr / nrows, srl = vr % nrows;
  const int t = hh * R + srl;
  const int srow = a.tiles[4 * tile + 0] + srl;
  const int h = g * a.G + hh;
  const int d0 = dq * DQ + hf * DT;
  auto lse_of = [&](int i) { return a.part_lse[(size_t(p0 + i) * hkv + g) * TR + t]; };
  float mx = -INFINITY;
  for (int i = j; i < ns; i += P) mx = fmaxf(mx, lse_of(i));
  for (int o = 1; o < P; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  float acc[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d) acc[d] = 0.0f;
  float wsum = 0.0f;
  for (int i = j; i < ns; i += P) {
    const float w = fast_exp2(lse_of(i) - mx);
    wsum += w;
    const float* pp = a.part_o + ((size_t(p0 + i) * hkv + g) * TR + t) * D + d0;
#pragma unroll
    for (int d = 0; d < DT; d += 4) {
      const float4 f = *reinterpret_cast<const float4*>(pp + d);
      acc[d + 0] += w * f.x;
      acc[d + 1] += w * f.y;
      acc[d + 2] += w * f.z;
      acc[d + 3] += w * f.w;
    }
  }
  for (int o = 1; o < P; o <<= 1) {
    wsum += __shfl_xor(wsum, o);
#pragma unroll
    for (int d = 0; d < DT; ++d) acc[d] += __shfl_xor(acc[d], o);
  }
  if (j != 0) return;
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
  if (a.tile_rows == 256) {
    if (head_dim == 128)
      link_attention_kernel<128, 8><<<grid, 512, 0, stream>>>(a);
    else
      link_attention_kernel<64, 8><<<grid, 512, 0, stream>>>(a);
  } else {
    if (head_dim == 128)
      link_attention_kernel<128, 4><<<grid, 256, 0, stream>>>(a);
    else
      link_attention_kernel<64, 4><<<grid, 256, 0, stream>>>(a);
  }
}

void launch_link_combine(const AttnArgs& a, int head_dim, int n_tiles, hipStream_t stream) {
  if (n_tiles == 0) return;
  const dim3 grid(unsigned(n_tiles) * unsigned(a.hkv) * kCombineParts);
  if (head_dim == 128)
    link_combine_kernel<128><<<grid, kCombineThreads, 0, stream>>>(a);
  else
    link_combine_kernel<64><<<grid, kCombineThreads, 0, stream>>>(a);
}

}  // namespace epic
