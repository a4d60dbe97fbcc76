// Row-set GEMMs of the link step on MFMA: C[M x N] = A[M x K] . W[N x K]^T.
//
// A holds the selected rows' activations (bf16, K contiguous), W a weight
// matrix in [out][in] layout (bf16), so both MFMA operands are read along K.
// Epilogues are fused:
//   kStoreF32 : C -> fp32 [M][N]                     (the plain projection of epic_gemm)
//   kResidual : h[M][N] += C                         (W_O and W_down; fp32 residual stream)
//   kSwiGLU   : act[M][N/2] = silu(gate) * up, bf16  (W_gate_up; gate rows [0, F), up rows [F, 2F))
//   kRope     : the fused Q|K|V projection: q and k heads rotated at each row's linked
//               position (rotary pairs (i, i + D/2)), v heads as they are; bf16 q, k, v
//
// Tiling: workgroup tile TM x TN (256 x 256, 192 x 256, 256 x 128, 128 x 128 or
// 96 x 128), 8 wavefronts of 64 columns each (TN = 256: 2 x 4 wavefronts of TM/2 x 64,
// i.e. 4 x 2 or 3 x 2 v_mfma_f32_32x32x16_bf16 tiles; TN = 128: 4 x 2 wavefronts of
// TM/4 x 64, and at TM = 96 3 x 2 of 32 x 64 while the other two only stage
// operands).  K runs in stages of 64 staged in LDS by direct buffer->LDS loads, NS
// stages in LDS (2 at TN = 256, 3 at TN = 128; loads issued NS - 1 stages ahead of
// use).  An operand stage is groups of 8 rows of 128 bytes
// (one whole cache line per row: a load instruction that covers 16 half lines moves
// about 0.6x the bytes per cycle of one that covers 8 whole lines); row r sits at byte
// 128 r with its eight 16-byte chunks XOR-swizzled by (r / 2) % 8, so one load
// instruction fills one group (1 KB) and the 16 lanes of each ds_read_b128 group
// touch distinct banks.  For kSwiGLU the TN weight rows of a tile are gate/up in
// 32-row groups (gate j.., up j.., gate j+32.., ...), so a wavefront's two
// 32-column MFMA tiles hold gate and up of the same 32 outputs.  For kRope the two
// 32-column MFMA tiles of a wavefront hold the two halves of rotary pairs: with
// D = 64 that is the natural order (a wavefront's 64 columns are one head); with
// D = 128 each 128-column head is staged as (i.., i+64.., i+32.., i+96..) in
// 32-row groups, i = 0.., so lane column c of tile 0 and tile 1 are head
// columns ip and ip + 64.
//
// Scheduling: at most one workgroup per CU (G of them), persistent.  With at least
// a round of 256 x 256 tiles, whole 256-wide tiles (256 or 192 rows) are dealt in
// rounds of G, G chosen so the rounds are (nearly) full; 256-wide tiles are never
// cut.  With fewer tiles (short row sets): whole 96 x 128 or 128 x 128 tiles in one
// round where they fill at least 3/4 of the CUs and K is short; else 256 x 128 tiles,
// and the ones that do not fill whole rounds
// (the last partial round plus one full round, or all of them) are cut along K into
// G equal shares of K stages, one per workgroup, so every CU gets the same work.  A
// share runs its last segment (the one that starts a tile) first.
// A tile cut across workgroups: each wavefront part of it has an arrival counter.
// The owner of the tile's last K stage polls it (a bounded number of times) until
// the other parts have written their fp32 partials, then adds them to its own
// accumulators and runs the epilogue; if the polls run out it writes its partial
// too, and the last wavefront to arrive finishes.  Either way the parts are summed
// in one fixed order, so the result does not depend on arrival order.  Workgroups
// are dealt round-robin to the 8 XCDs; worker indices are arranged so that each XCD
// works on a contiguous run of tiles, and tiles are ordered in groups of up to 8 row
// tiles per weight tile, so concurrent workgroups on an XCD share operands through
// its L2.
// Rows past M and columns past N are computed from clamped rows and never stored.
#include <algorithm>
#include <cstdlib>

#include "device_common.h"
#include "gemm.h"

namespace epic {

namespace {

constexpr int kTM = 256, kBK = 64;
constexpr int kThreads = 512;
constexpr int kBufWord3 = 0x00020000;                   // gfx9 raw buffer descriptor word 3
constexpr int kMaxWorkers = 256;                        // one workgroup per CU
constexpr int kPartialFloats = kTM * 256;               // fp32 partial sums of the largest tile
constexpr int kMaxSplitTiles = 2 * kMaxWorkers;
constexpr int kCounters = kMaxSplitTiles * (kThreads / 64);   // one per (cut tile, wavefront)
constexpr int kMinUnits = 4;                            // K stages per workgroup, at least

template <int TM, int TN>
struct Shape {
  static_assert((TM == 256 && (TN == 128 || TN == 256)) || (TM == 192 && TN == 256) ||
                    ((TM == 128 || TM == 96) && TN == 128),
                "tile shape");
  static constexpr int NS = TN == 256 ? 2 : 3;          // LDS stages (128 / 112 / 144 / 96 / 84 KB)
  // wavefronts along M (TM = 96: 3 x 2 wavefronts compute, the other two only stage
  // operands and meet the barriers)
  static constexpr int WAVES_M = TN == 256 ? 2 : TM >= 128 ? 4 : TM / 32;
  static constexpr int WM = TM / WAVES_M;               // rows per wavefront
  static constexpr int I = WM / 32;                     // 32-row MFMA tiles per wavefront
  static constexpr int J = 2;                           // 32-column MFMA tiles per wavefront
  static constexpr int A_STAGE = TM * kBK * 2;          // bytes per stage
  static constexpr int B_STAGE = TN * kBK * 2;
  static constexpr int NLA = TM / 32;                   // A row groups (8 rows) per loading wavefront
  static constexpr int NLB = TN / 32;                   // W row groups per loading wavefront
  static constexpr int NL = NLA > NLB ? NLA : NLB;
};

struct GemmPlan {
  int m_tiles, n_tiles, ks;    // tiles along M and N, K stages per tile
  int gm;                      // row tiles per ordering group
  int G;                       // workgroups
  int dp_rounds, dp_tiles;     // whole-tile rounds and the tiles they cover (tiles 0 .. dp_tiles-1)
  int sk_units;                // K stages of the cut tiles (tiles dp_tiles ..)
  int polls;                   // counter polls of a cut tile's last-stage owner before it falls back
};

template <int TM, int TN>
struct GemmLds {
  char a[Shape<TM, TN>::NS][Shape<TM, TN>::A_STAGE];
  char b[Shape<TM, TN>::NS][Shape<TM, TN>::B_STAGE];
};

typedef __attribute__((address_space(3))) void lds_void;

// One 16-byte-per-lane buffer->LDS load (1 KB per wavefront: lane l's 16 bytes land
// at dst + 16 l).  A plain function, so the call is never a template-dependent
// expression (the host pass cannot check this builtin inside a template).
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, char* dst, int voff, int soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)dst, 16, voff, soff, 0, 0);
}

// Workgroup barrier ordering LDS accesses only (waits for this wavefront's LDS
// reads, not for its buffer->LDS loads still in flight).
__device__ __forceinline__ void barrier_lds() {
  __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// At most N of this wavefront's vector memory operations outstanding (they
// complete in issue order); gfx9 encoding: vmcnt bits [3:0] and [15:14].
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt field");
  __builtin_amdgcn_s_waitcnt((N & 15) | (0x7 << 4) | (0xF << 8) | ((N >> 4) << 14));
}

// Position in a workgroup's sequence of K stages: tile, stage, and the stage range
// [kbeg, kend) of the current segment (the part of the tile this workgroup owns).
struct Cursor {
  int u, tile, kt, kbeg, kend;
};

template <int EPI, int TM, int TN>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(GemmArgs g, GemmPlan p) {
  using SH = Shape<TM, TN>;
  constexpr int NS = SH::NS, I = SH::I, J = SH::J, NLA = SH::NLA, NLB = SH::NLB, NL = SH::NL;
  __shared__ __attribute__((aligned(1024))) GemmLds<TM, TN> lds;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  // wavefront tile: rows wm*WM.., columns wn*64..  At TN = 128 the two wavefronts of
  // each SIMD (wavefronts w and w + 4) take different row halves, so a tile whose
  // rows past M leave half the wavefronts idle still keeps every SIMD busy.  Wavefronts
  // with wm >= WAVES_M (TM = 96: wavefronts 6 and 7) compute and store nothing.
  const int wm = TN == 128 ? wv >> 1 : wv % SH::WAVES_M;
  const int wn = TN == 128 ? wv & 1 : wv / SH::WAVES_M;
  const int w = blockIdx.x;
  const int wr = p.G % 8 == 0 ? (w % 8) * (p.G / 8) + w / 8 : w;   // XCD-contiguous worker index
  const int64_t su = p.sk_units;
  const int s0 = int(int64_t(wr) * su / p.G), s1 = int(int64_t(wr + 1) * su / p.G);
  // whole tiles wr, wr + G, .. below dp_tiles (the last round may be short), then the K share
  const int dp_units = (wr < p.dp_tiles ? (p.dp_tiles - wr + p.G - 1) / p.G : 0) * p.ks;
  const int n_units = dp_units + (s1 - s0);
  if (n_units == 0) return;             // (no such workgroup is launched; kept as a guard)
  // The K share runs its last segment first: that segment starts a tile (K stage 0)
  // and the rest ends one (the last stage), so the workgroups of an XCD that cross a
  // tile boundary sit at two K offsets at any time instead of one each, and their
  // operand stages are shared in the L2.  sh: first unit of the last segment.
  const int sh = max(s0, s1 > s0 ? (s1 - 1) / p.ks * p.ks : s0);

  auto tile_mn = [&](int t, int& mt, int& nt) __attribute__((always_inline)) {
    const int per_group = p.gm * p.n_tiles;
    const int grp = t / per_group;
    const int first = grp * p.gm;
    const int gsz = min(p.m_tiles - first, p.gm);
    const int r = t - grp * per_group;
    mt = first + r % gsz;
    nt = r / gsz;
  };
  auto seek = [&](Cursor& c, int u) __attribute__((always_inline)) {   // u: first unit of a segment
    c.u = u;
    if (u < dp_units) {
      c.tile = (u / p.ks) * p.G + wr;
      c.kbeg = 0;
      c.kend = p.ks;
    } else {
      const int i = u - dp_units;           // position in the share's processing order
      const bool first = i < s1 - sh;       // in the last segment, run first
      const int v = first ? sh + i : s0 + (i - (s1 - sh));
      const int q = v / p.ks;
      c.tile = p.dp_tiles + q;
      c.kbeg = v - q * p.ks;
      c.kend = min(p.ks, (first ? s1 : sh) - q * p.ks);
    }
    c.kt = c.kbeg;
  };
  auto advance = [&](Cursor& c) __attribute__((always_inline)) {      // to the next unit; stays on the last one
    if (c.u + 1 >= n_units) return;
    ++c.u;
    if (++c.kt == c.kend) seek(c, c.u);
  };

  // ---- buffer->LDS loads: wavefronts 0..3 stage the TM / 8 A row groups (NLA each),
  // 4..7 the TN / 8 W row groups (NLB each).
  const bool a_wave = wv < 4;
  // With M <= 128 (one row tile) the A row groups 16..31 hold no row of A: their
  // loading wavefronts issue nothing (none of their waits then has anything to wait for).
  const bool dma_idle = TM == 256 && TN == 128 && a_wave && g.M <= 128 && wv >= 2;
  const int nl = a_wave ? NLA : NLB;                   // loads per stage of this wavefront
  const int grp0 = nl * (wv & 3);
  const int lrow = lane >> 3;                              // row within an 8-row group
  const int row_bytes = g.K * 2;
  const int w_rows = EPI == kSwiGLU ? 2 * g.ffn : g.N;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(a_wave ? g.A : g.W), 0, (a_wave ? g.M : w_rows) * row_bytes, kBufWord3);
  int vo[NL];                                           // lane byte offsets of the row groups (nl)
  // load i of a stage: issued by this wavefront (i < nl; the bound is a constant for
  // the i below both counts)
  auto has_load = [&](int i) __attribute__((always_inline)) { return a_wave ? i < NLA : i < NLB; };
  auto dma_setup = [&](int tile) __attribute__((always_inline)) {
    int mt, nt;
    tile_mn(tile, mt, nt);
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int row = (grp0 + i) * 8 + lrow;               // row of the operand tile
      const int lchunk = (lane & 7) ^ ((row >> 1) & 7);    // 16-byte chunk of that row this lane loads
      int gr;
      if (a_wave) gr = min(mt * TM + row, g.M - 1);
      else if constexpr (EPI == kSwiGLU)
        gr = ((row >> 5) & 1) * g.ffn + nt * (TN / 2) + (row >> 6) * 32 + (row & 31);
      else if constexpr (EPI == kRope) {
        // D = 128: LDS row p = wn' * 64 + j * 32 + r of a head holds head column
        // j * 64 + wn' * 32 + r (wn' = wavefront column half within the head)
        const int hc = g.head_dim == 128 ? (row & ~127) + ((row >> 5) & 1) * 64 + ((row >> 6) & 1) * 32 + (row & 31)
                                         : row;
        gr = min(nt * TN + hc, g.N - 1);
      } else gr = min(nt * TN + row, g.N - 1);
      vo[i] = gr * row_bytes + lchunk * 16;
    }
  };
  char* const dma_base = a_wave ? lds.a[0] + grp0 * 1024 : lds.b[0] + grp0 * 1024;
  const int dma_stage = a_wave ? SH::A_STAGE : SH::B_STAGE;
  auto dma = [&](int buf, int kt) __attribute__((always_inline)) {
    if (dma_idle) return;
    char* dst = dma_base + buf * dma_stage;
#pragma unroll
    for (int i = 0; i < NL; ++i)
      if (has_load(i)) dma16(rs, dst + i * 1024, vo[i], kt * (kBK * 2));
  };

  // ---- MFMA operands: for k-slice ks (16 wide, 4 per stage) lane l reads row l % 32
  // of a 32-row tile, 16-byte chunk 2 ks + l / 32, stored at chunk position
  // chunk ^ ((l % 32) / 2 % 8).
  const int lrow32 = (lane & 31) * 128;
  const int lsw = (lane >> 1) & 7;
  const int lb0 = lrow32 + (((0 + (lane >> 5)) ^ lsw) * 16);
  const int lb1 = lrow32 + (((2 + (lane >> 5)) ^ lsw) * 16);
  const int lb2 = lrow32 + (((4 + (lane >> 5)) ^ lsw) * 16);
  const int lb3 = lrow32 + (((6 + (lane >> 5)) ^ lsw) * 16);
  const char* const pa = lds.a[0] + wm * SH::WM * 128;
  const char* const pb = lds.b[0] + wn * 64 * 128;
  struct Frags {
    bf16x8 a[I], b[J];
  };
  auto read = [&](Frags& f, int buf, int ks) __attribute__((always_inline)) {
    const int lb = ks == 0 ? lb0 : ks == 1 ? lb1 : ks == 2 ? lb2 : lb3;
    const char* a = pa + buf * SH::A_STAGE + lb;
    const char* b = pb + buf * SH::B_STAGE + lb;
#pragma unroll
    for (int i = 0; i < I; ++i) f.a[i] = *reinterpret_cast<const bf16x8*>(a + i * 4096);
#pragma unroll
    for (int j = 0; j < J; ++j) f.b[j] = *reinterpret_cast<const bf16x8*>(b + j * 4096);
  };

  f32x16 acc[I][J];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j) acc[i][j] = f32x16{};
  };
  auto mma = [&](const Frags& f) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < I; ++i)
#pragma unroll
      for (int j = 0; j < J; ++j) acc[i][j] = mfma_32x32x16(f.a[i], f.b[j], acc[i][j]);
  };
  // mma(f) with the loads of unit kt into buffer buf between its MFMAs (NL / (I J)
  // after each, same MFMA order as mma): issued together after the barrier, the
  // workgroup's 64 loads of 1 KB queued behind each other while no MFMA was issued.
  auto mma_dma = [&](const Frags& f, int buf, int kt) __attribute__((always_inline)) {
    constexpr int NM = I * J;
    char* const dst = dma_base + buf * dma_stage;
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      acc[m / J][m % J] = mfma_32x32x16(f.a[m / J], f.b[m % J], acc[m / J][m % J]);
#pragma unroll
      for (int i = m * NL / NM; i < (m + 1) * NL / NM; ++i)
        if (!dma_idle && has_load(i)) dma16(rs, dst + i * 1024, vo[i], kt * (kBK * 2));
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // ---- epilogue through buffer descriptors: rows past M fall outside the
  // descriptor's range (loads read 0, stores are dropped).  Accumulator tile
  // t = i*J + j, register r: row wm*WM + i*32 + (r/4)*8 + half*4 + r%4, column
  // wn*64 + j*32 + col of the workgroup tile.  Written CT = 2 tiles (one row block)
  // at a time, so the fixup below holds two tiles of sums and one partial's two tiles
  // in flight (with four, the 128-wide kernels ran out of registers and the compiler
  // reloaded each 1 KB of a partial into the same registers, one round trip each).
  constexpr int NT = I * J, CT = 2, NCH = NT / CT;
  const int col = lane & 31, half = lane >> 5;
  auto epilogue_part = [&](int mt, int nt, int h, const f32x16 (&v)[CT]) __attribute__((always_inline)) {
    const int m0 = mt * TM + wm * SH::WM + half * 4;
    if constexpr (EPI == kSwiGLU) {
      const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(g.act, 0, g.M * g.ffn * 2, kBufWord3);
      const int n = nt * (TN / 2) + wn * 32 + col;
#pragma unroll
      for (int ii = 0; ii < CT / J; ++ii)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + (h * (CT / J) + ii) * 32 + (r >> 2) * 8 + (r & 3);
          const float gt = v[ii * J + 0][r], up = v[ii * J + 1][r];
          const float act = gt * __builtin_amdgcn_rcpf(1.0f + fast_exp2(-gt * kLog2e)) * up;
          __builtin_amdgcn_raw_buffer_store_b16(uint16_t(pack_bf16x2(act, 0.0f) & 0xFFFFu), ro, (m * g.ffn + n) * 2,
                                                0, 0);
        }
    } else if constexpr (EPI == kRope) {
      // this wavefront's 64 columns: one head (D = 64) or half of one (D = 128, the
      // pairs ip, ip + 64 with ip in [32 (wn % 2), + 32))
      const int D = g.head_dim, half = D >> 1;
      const int head = D == 128 ? (nt * TN >> 7) + (wn >> 1) : (nt * TN >> 6) + wn;
      if (head >= g.hq + 2 * g.hkv) return;               // columns past N
      const int ip = (D == 128 ? (wn & 1) * 32 : 0) + col;
      uint16_t* base;
      int heads, hd;
      bool rotate = true;
      if (head < g.hq) {
        base = g.q, heads = g.hq, hd = head;
      } else if (head < g.hq + g.hkv) {
        base = g.k, heads = g.hkv, hd = head - g.hq;
      } else {
        base = g.v, heads = g.hkv, hd = head - g.hq - g.hkv, rotate = false;
      }
      const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(base, 0, g.M * heads * D * 2, kBufWord3);
      const __amdgpu_buffer_rsrc_t rc =
          __builtin_amdgcn_make_buffer_rsrc(const_cast<float2*>(g.cs), 0, g.M * half * 8, kBufWord3);
#pragma unroll
      for (int ii = 0; ii < CT / J; ++ii) {
        // the row block's cos / sin first, so the 16 loads are in flight together (a
        // load is not moved above an earlier buffer store)
        float2 t[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + (h * (CT / J) + ii) * 32 + (r >> 2) * 8 + (r & 3);
          t[r] = rotate ? __builtin_bit_cast(float2, __builtin_amdgcn_raw_buffer_load_b64(rc, (m * half + ip) * 8, 0, 0))
                        : make_float2(1.0f, 0.0f);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + (h * (CT / J) + ii) * 32 + (r >> 2) * 8 + (r & 3);
          const float x1 = v[ii * J + 0][r], x2 = v[ii * J + 1][r];
          float y1 = x1, y2 = x2;
          if (rotate) {
            y1 = x1 * t[r].x - x2 * t[r].y;
            y2 = x2 * t[r].x + x1 * t[r].y;
          }
          const int e = ((m * heads + hd) * D + ip) * 2;
          __builtin_amdgcn_raw_buffer_store_b16(uint16_t(pack_bf16x2(y1, 0.0f) & 0xFFFFu), ro, e, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b16(uint16_t(pack_bf16x2(y2, 0.0f) & 0xFFFFu), ro, e + half * 2, 0, 0);
        }
      }
    } else {
      if (nt * TN + wn * 64 >= g.N) return;                // this wavefront's columns are past N
      const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(g.C, 0, g.M * g.N * 4, kBufWord3);
      const int n = nt * TN + wn * 64 + col;
#pragma unroll
      for (int ii = 0; ii < CT / J; ++ii) {
        // residual: every load of the row block first, so they are in flight together
        // (a load may not move above an earlier store through the same descriptor)
        float cin[16][J];
        if constexpr (EPI == kResidual) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = m0 + (h * (CT / J) + ii) * 32 + (r >> 2) * 8 + (r & 3);
#pragma unroll
            for (int j = 0; j < J; ++j)
              cin[r][j] = __builtin_bit_cast(float,
                                             __builtin_amdgcn_raw_buffer_load_b32(ro, (m * g.N + n + j * 32) * 4, 0, 0));
          }
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + (h * (CT / J) + ii) * 32 + (r >> 2) * 8 + (r & 3);
#pragma unroll
          for (int j = 0; j < J; ++j) {
            float x = v[ii * J + j][r];
            if constexpr (EPI == kResidual) x += cin[r][j];
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), ro, (m * g.N + n + j * 32) * 4, 0, 0);
          }
        }
      }
    }
  };

  // End of a segment: a whole tile goes straight to the epilogue; a cut tile
  // through the partial buffers and its arrival counter.
  constexpr int kWaveFloats = NT * 16 * 64;
  auto finish = [&](const Cursor& c) __attribute__((always_inline)) {
    int mt, nt;
    tile_mn(c.tile, mt, nt);
    // no rows of this part (past the tile, or every row past M): nothing to write
    if (TN == 128 && (wm >= SH::WAVES_M || mt * TM + wm * SH::WM >= g.M)) return;
    if (c.kbeg == 0 && c.kend == p.ks) {
#pragma unroll
      for (int h = 0; h < NCH; ++h) {
        f32x16 v[CT];
#pragma unroll
        for (int t = 0; t < CT; ++t) v[t] = acc[(h * CT + t) / J][(h * CT + t) % J];
        epilogue_part(mt, nt, h, v);
      }
      return;
    }
    // Only 128-wide tiles are ever cut (the planner deals 256-wide tiles whole), so the
    // 256-wide instantiations carry no partial protocol (and its registers).
    if constexpr (TN == 256) return;
    const int q = c.tile - p.dp_tiles;
    const int64_t U = p.sk_units;
    auto owner = [&](int64_t v) __attribute__((always_inline)) { return int(((v + 1) * p.G + U - 1) / U - 1); };
    const int wf = owner(int64_t(q) * p.ks), wl = owner(int64_t(q + 1) * p.ks - 1);
    // worker x's partial of this tile (this wavefront's part): its last segment if
    // it owns the tile's first stage (slot 2x + 1), else its first segment (slot 2x).
    // Layout: [wavefront][tile t][register quad][lane][4] floats, so each access is
    // 16 bytes per lane, 1 KB per instruction.  Partials are written and read with
    // agent-scope accesses (cache policy sc1 = device scope on gfx950), which go past
    // the XCD's L2, so no cache-wide write-back or invalidate is needed.
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
        g.partial, 0, 2 * kMaxWorkers * kPartialFloats * 4, kBufWord3);
    auto slot_off = [&](int x) __attribute__((always_inline)) {   // bytes
      return int((2 * x + (x == wf ? 1 : 0)) * kPartialFloats + wv * kWaveFloats) * 4 + lane * 16;
    };
    constexpr int kSc1 = 16;             // cache policy sc1 alone: agent (device) scope
    typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
    int* cnt = g.tile_count + q * (kThreads / 64) + wv;
    // The tile's sum in a fixed order: the part of the owner of the tile's last
    // stage (worker wl) first, then the partials of workers wf .. wl - 1 in K order;
    // then the epilogue.  own: this wavefront is that owner and starts from its
    // accumulators, else it starts from the owner's partial.  Each partial's loads
    // are issued together, so a partial costs one round trip.
    auto fixup = [&](bool own) __attribute__((always_inline)) {
#pragma unroll
      for (int h = 0; h < NCH; ++h) {
        f32x16 v[CT];
        auto load_part = [&](int x, f32x4 (&p4)[CT * 4]) __attribute__((always_inline)) {
          const int off = slot_off(x);
#pragma unroll
          for (int c = 0; c < CT * 4; ++c)
            p4[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rp, off + (h * CT * 4 + c) * 1024, 0, kSc1));
        };
        if (own) {
#pragma unroll
          for (int t = 0; t < CT; ++t) v[t] = acc[(h * CT + t) / J][(h * CT + t) % J];
        } else {
          f32x4 p4[CT * 4];
          load_part(wl, p4);
#pragma unroll
          for (int c = 0; c < CT * 4; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[c >> 2][4 * (c & 3) + e] = p4[c][e];
        }
        for (int x = wf; x < wl; ++x) {
          f32x4 p4[CT * 4];
          load_part(x, p4);
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int c = 0; c < CT * 4; ++c)
#pragma unroll
            for (int e = 0; e < 4; ++e) v[c >> 2][4 * (c & 3) + e] += p4[c][e];
        }
        epilogue_part(mt, nt, h, v);
      }
      if (lane == 0) __hip_atomic_exchange(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);   // ready for the next launch
    };
    // The owner of the tile's last stage runs that segment last (its K share runs the
    // segment that starts a tile first), so the others' partials are usually written
    // by then: it polls the counter, a bounded number of times, until the other
    // wl - wf parts have arrived, and finishes from its registers without writing its
    // own partial.  The others never see the count reach wl - wf before it, so none of
    // them finishes the tile.  If they are not all there in time it falls back to the
    // protocol below (write, count, the last to arrive finishes); the sums are the same
    // on both paths.
    if (wr == wl) {
      int seen = 0;
      for (int it = 0; it < p.polls; ++it) {
        if (lane == 0) seen = __hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        seen = __builtin_amdgcn_readfirstlane(seen);
        if (seen == wl - wf) break;
        __builtin_amdgcn_s_sleep(2);
      }
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      if (seen == wl - wf) {
        fixup(true);
        return;
      }
    }
    const int mine = slot_off(wr);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const f32x16& a16 = acc[t / J][t % J];
        const f32x4 v4 = {a16[4 * qd], a16[4 * qd + 1], a16[4 * qd + 2], a16[4 * qd + 3]};
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4v, v4), rp, mine + (t * 4 + qd) * 1024, 0,
                                               kSc1);
      }
    // Each wavefront keeps its own arrival counter for the tile (its part of the
    // tile depends only on the same wavefront's part of the other partials), so no
    // workgroup barrier is needed: the last wavefront to arrive finishes that part.
    // The counter bump is an agent-scope atomic.  The hardware wait orders it after this
    // wavefront's partial stores; the compiler-only fences on both sides keep the
    // compiler from moving the stores below it or the partial loads above it (they
    // emit no instruction, so no L2 write-back).
    wait_vmem<0>();                      // this wavefront's partial has landed
    int before = 0;
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (lane == 0) before = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    before = __builtin_amdgcn_readfirstlane(before);
    if (before != wl - wf) return;       // not the last to arrive
    fixup(false);                        // the last to arrive: every part from the partials
  };

  // ---- pipeline: unit u (one K stage of one tile) lives in LDS buffer u % NS.
  // Step u reads each k-slice while the previous one runs on the matrix cores,
  // waits for this wavefront's loads of unit u + 1, and after the barrier (all
  // loads of u + 1 visible, every read of buffer u % NS done) refills that buffer
  // with unit u + NS and reads the first k-slice of u + 1.  Loads past the last
  // unit repeat it, so every step leaves the same number in flight.  (One barrier
  // per two units measured slower at TN = 128.)
  Cursor cc, dc;
  seek(cc, 0);
  dc = cc;
  int dtile = dc.tile;
  dma_setup(dtile);
  auto dma_advance = [&]() __attribute__((always_inline)) {
    advance(dc);
    if (dc.tile != dtile) {
      dtile = dc.tile;
      dma_setup(dtile);
    }
  };
  auto dma_next = [&](int buf) __attribute__((always_inline)) {
    dma(buf, dc.kt);
    dma_advance();
  };
#pragma unroll
  for (int b = 0; b < NS; ++b) dma_next(b);
  if (a_wave) wait_vmem<(NS - 1) * NLA>();      // unit 0 of this wavefront
  else wait_vmem<(NS - 1) * NLB>();
  barrier_lds();                                    // ... of every wavefront
  Frags f0, f1;
  read(f0, 0, 0);
  zero_acc();
  // rows of this wavefront's part of the current tile exist (else it only stages and
  // syncs); only the 128-column tiles of short row sets skip (256-column tiles run
  // when there are many row tiles, where the saving is small)
  auto live_in = [&](int tile) __attribute__((always_inline)) {
    if constexpr (TN != 128) return true;
    int mt, nt;
    tile_mn(tile, mt, nt);
    return __builtin_amdgcn_readfirstlane(int(wm < SH::WAVES_M && mt * TM + wm * SH::WM < g.M)) != 0;
  };
  bool live = live_in(cc.tile);
  int u = 0, buf = 0;
  while (true) {
    // the units of one segment (the epilogue stays out of the hot loop)
    for (const int ue = u + (cc.kend - cc.kt); u < ue; ++u) {
      const int nbuf = buf + 1 == NS ? 0 : buf + 1;
      if (live) {
        read(f1, buf, 1);
        mma(f0);
        read(f0, buf, 2);
        mma(f1);
        read(f1, buf, 3);
        mma(f0);
      }
      if (a_wave) wait_vmem<(NS - 2) * NLA>();  // this wavefront's loads of unit u + 1
      else wait_vmem<(NS - 2) * NLB>();
      barrier_lds();
      if (live) {
        read(f0, nbuf, 0);
        mma_dma(f1, buf, dc.kt);                  // unit u + NS into buf, between the MFMAs
      } else {
        dma(buf, dc.kt);
      }
      dma_advance();
      buf = nbuf;
    }
    finish(cc);
    if (u >= n_units) break;
    zero_acc();
    seek(cc, u);
    const bool was_live = live;
    live = live_in(cc.tile);
    // f0 (first k-slice of unit u, in buffer buf: loaded and published at the last
    // barrier) was only prefetched if the previous segment was live
    if (live && !was_live) read(f0, buf, 0);
  }
  wait_vmem<0>();                       // no load may land in LDS after the workgroup ends
}

__global__ void gemm_clear_kernel(int* cnt) {
  for (int i = threadIdx.x; i < kCounters; i += blockDim.x) cnt[i] = 0;
}

int cdiv(int a, int b) { return (a + b - 1) / b; }

// Counter polls of a cut tile's last-stage owner (about 0.3 ms at the default).  The
// environment variable EPIC_GEMM_FINISH_POLLS overrides it (0 forces the fallback
// protocol: a test hook); read at every launch.
int finish_polls() {
  const char* e = std::getenv("EPIC_GEMM_FINISH_POLLS");
  if (e == nullptr || *e == 0) return 4096;
  const long v = std::strtol(e, nullptr, 10);
  return int(std::min<long>(std::max<long>(v, 0), 1 << 20));
}

template <int EPI, int TM, int TN>
void launch_tn(const GemmArgs& g, bool whole_tiles, hipStream_t stream) {
  static_assert(TN == 128 || TN == 256, "tile width");
  if (TN == 256) whole_tiles = true;                 // the 256-wide kernels finish whole tiles only
  GemmPlan p{};
  p.m_tiles = cdiv(g.M, TM);
  p.n_tiles = EPI == kSwiGLU ? g.ffn / (TN / 2) : cdiv(g.N, TN);
  p.ks = g.K / kBK;
  p.gm = p.m_tiles < 8 ? p.m_tiles : 8;
  const int64_t tiles = int64_t(p.m_tiles) * p.n_tiles;
  if (whole_tiles) {
    // rounds of whole tiles, as few workgroups as keep the rounds full
    const int64_t rounds = (tiles + kMaxWorkers - 1) / kMaxWorkers;
    p.G = int((tiles + rounds - 1) / rounds);
    p.dp_rounds = int(rounds);
    p.dp_tiles = int(tiles);                         // a short last round leaves some workgroups idle
    p.sk_units = 0;
  } else {
    const int64_t units = tiles * p.ks;
    p.G = int(std::min<int64_t>(kMaxWorkers, std::max<int64_t>(1, units / kMinUnits)));
    const int64_t full = tiles / p.G, rem = tiles % p.G;
    p.dp_rounds = int(rem == 0 ? full : std::max<int64_t>(full - 1, 0));
    p.dp_tiles = p.dp_rounds * p.G;
    p.sk_units = int((tiles - p.dp_tiles) * p.ks);
  }
  p.polls = finish_polls();
  gemm_kernel<EPI, TM, TN><<<dim3(p.G), kThreads, 0, stream>>>(g, p);
}

template <int EPI>
void launch_epi(const GemmArgs& g, hipStream_t stream) {
  // At least a round of 256 x 256 tiles: whole tiles only (measured: cutting tiles
  // along K costs about one tile time in partial traffic, more than a short last
  // round).  The tiles are 256 or 192 rows high, whichever takes less time: a round
  // of 192-row tiles takes about 15/16 of the time of one of 256-row tiles
  // (measured; a stage streams the same 256 weight rows), so 192 rows win where
  // they save a round or more of the short last round: at 736 rows, 448 tiles of
  // 192 rows in 2 rounds of 224 workgroups instead of 336 of 256 rows in 2 rounds
  // of 168.
  const int m_tiles = cdiv(g.M, kTM);
  const int n256 = EPI == kSwiGLU ? (g.ffn % 128 == 0 ? g.ffn / 128 : 0) : cdiv(g.N, 256);
  if (int64_t(m_tiles) * n256 >= kMaxWorkers) {
    const int64_t r256 = (int64_t(m_tiles) * n256 + kMaxWorkers - 1) / kMaxWorkers;
    const int64_t r192 = (int64_t(cdiv(g.M, 192)) * n256 + kMaxWorkers - 1) / kMaxWorkers;
    if (r192 * 15 < r256 * 16) return launch_tn<EPI, 192, 256>(g, true, stream);
    return launch_tn<EPI, 256, 256>(g, true, stream);
  }
  // Fewer: with a short K and one round of 96 x 128 or 128 x 128 tiles that fills at
  // least 3/4 of the CUs, those tiles whole (96 rows where they make such a round: more
  // CUs, fewer bytes each); else 256 x 128 tiles cut along K so that every CU gets a
  // share.  Measured at 736 rows, N = 4096: whole 128 x 128 tiles take about 0.57 us per
  // K stage on 192 CUs, the cut tiles about 0.45 us per stage of a tile's K plus about
  // 15 us of partial traffic and fixup, so whole tiles win up to about 100 stages (W_O,
  // K = 4096: 48.0 -> 40.2 us; W_down, K = 14336: 103.8 -> 127.7 us).  96 x 128 tiles on
  // 256 CUs took W_O about 1 us further (the c3 link step 0.3% faster on one box).
  const int64_t n128 = EPI == kSwiGLU ? g.ffn / 64 : cdiv(g.N, 128);
  const int64_t t128 = int64_t(cdiv(g.M, 128)) * n128, t96 = int64_t(cdiv(g.M, 96)) * n128;
  auto one_round = [](int64_t t) { return t >= 3 * kMaxWorkers / 4 && t <= kMaxWorkers; };
  if (g.K / kBK <= 96) {
    if (one_round(t96)) return launch_tn<EPI, 96, 128>(g, true, stream);
    if (one_round(t128)) return launch_tn<EPI, 128, 128>(g, true, stream);
  }
  launch_tn<EPI, 256, 128>(g, false, stream);
}

}  // namespace

size_t gemm_workspace_bytes() {
  return size_t(2 * kMaxWorkers) * kPartialFloats * sizeof(float) + kCounters * sizeof(int);
}

void gemm_workspace(void* base, float** partial, int** tile_count) {
  *partial = static_cast<float*>(base);
  *tile_count = reinterpret_cast<int*>(static_cast<char*>(base) + size_t(2 * kMaxWorkers) * kPartialFloats * 4);
}

void launch_gemm_clear(int* tile_count, hipStream_t stream) {
  gemm_clear_kernel<<<1, 256, 0, stream>>>(tile_count);
}

void launch_gemm(const GemmArgs& g, int epi, hipStream_t stream) {
  if (g.M == 0) return;
  if (epi == kStoreF32)
    launch_epi<kStoreF32>(g, stream);
  else if (epi == kRope)
    launch_epi<kRope>(g, stream);
  else if (epi == kResidual)
    launch_epi<kResidual>(g, stream);
  else
    launch_epi<kSwiGLU>(g, stream);
}

}  // namespace epic
