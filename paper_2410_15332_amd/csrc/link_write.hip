// Link write: build every request-private block of the linked cache.
//
// Sec. 4.2 forms K_exp / V_exp from the cached vectors of the unselected tokens
// plus the recomputed vectors, each at its own linked position.  Shared chunk blocks are
// immutable, so a block that receives a recomputed row is private: its cached
// rows are copied from the shared block (copy-on-write) and its selected rows
// take k_s / v_s.  Each private block is written exactly once, by one
// workgroup per (block, KV head); copies are bit-exact.
//
// Layouts: K [blocks][Hkv][16][D], V [blocks][Hkv][D][16].
#include <cmath>

#include "device_common.h"
#include "kernels.h"
#include "link_write.h"

namespace epic {

template <int D>
__global__ __launch_bounds__(2 * D) void link_write_kernel(const int32_t* __restrict__ priv_block,
                                                          const int32_t* __restrict__ priv_src,
                                                          const int32_t* __restrict__ priv_rows,
                                                          const uint16_t* __restrict__ k_s,
                                                          const uint16_t* __restrict__ v_s,
                                                          uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                          int hkv) {
  const int pv = blockIdx.x / hkv;
  const int g = blockIdx.x % hkv;
  const int tid = threadIdx.x;
  const int dst = priv_block[pv];
  const int src = priv_src[pv];
  const int32_t* rows = priv_rows + pv * 16;

  // K: thread -> (slot, 8-wide chunk of the head dim); 16 slots x D/8 chunks = 2D threads.
  {
    const int o = tid / (D / 8), dc = tid % (D / 8);
    const int r = rows[o];
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r >= 0)
      val = *reinterpret_cast<const uint4*>(k_s + (size_t(r) * hkv + g) * D + dc * 8);
    else if (src >= 0)
      val = *reinterpret_cast<const uint4*>(kc + ((size_t(src) * hkv + g) * 16 + o) * D + dc * 8);
    *reinterpret_cast<uint4*>(kc + ((size_t(dst) * hkv + g) * 16 + o) * D + dc * 8) = val;
  }
  // V: thread -> (dim d, 8 consecutive slots); D dims x 2 halves = 2D threads.
  {
    const int d = tid >> 1, hf = tid & 1;
    uint16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int o = hf * 8 + i;
      const int r = rows[o];
      uint16_t x = 0;
      if (r >= 0)
        x = v_s[(size_t(r) * hkv + g) * D + d];
      else if (src >= 0)
        x = vc[((size_t(src) * hkv + g) * D + d) * 16 + o];
      e[i] = x;
    }
    uint4 val;
    val.x = uint32_t(e[0]) | (uint32_t(e[1]) << 16);
    val.y = uint32_t(e[2]) | (uint32_t(e[3]) << 16);
    val.z = uint32_t(e[4]) | (uint32_t(e[5]) << 16);
    val.w = uint32_t(e[6]) | (uint32_t(e[7]) << 16);
    *reinterpret_cast<uint4*>(vc + ((size_t(dst) * hkv + g) * D + d) * 16 + hf * 8) = val;
  }
}

// The same write for plans that re-rotate cached rows: a block with priv_rot = off
// != 0 gets its cached K rows rotated by off (R(off) R(t) = R(off + t)): pairs
// (i, i + D/2), angle off * theta^(-2i/D) in float64, rotation in fp32, RNE to bf16.
// A thread's K chunk (8 dims) and its pair partner's chunk sit D/16 lanes apart in
// the same wavefront.  V is copied unchanged.  A block with priv_rot = 0 is
// written exactly as by link_write_kernel.  One workgroup per private block walks
// its KV heads kHeads at a time: the heads' loads are issued first, so the angles
// (computed once per block) are evaluated while they are in flight.
template <int D>
__global__ __launch_bounds__(2 * D) void link_write_rotate_kernel(const int32_t* __restrict__ priv_block,
                                                                 const int32_t* __restrict__ priv_src,
                                                                 const int32_t* __restrict__ priv_rows,
                                                                 const int32_t* __restrict__ priv_rot,
                                                                 const uint16_t* __restrict__ k_s,
                                                                 const uint16_t* __restrict__ v_s,
                                                                 uint16_t* __restrict__ kc, uint16_t* __restrict__ vc,
                                                                 int hkv, double log2_theta) {
  constexpr int kHeads = 8;
  __shared__ float2 cs[D / 2];
  const int pv = blockIdx.x;
  const int tid = threadIdx.x;
  const int dst = priv_block[pv];
  const int src = priv_src[pv];
  const int rot = priv_rot[pv];
  const int32_t* rows = priv_rows + pv * 16;
  const int o = tid / (D / 8), dc = tid % (D / 8);        // K: slot, 8-dim chunk
  const int rk = rows[o];
  const int vd = tid >> 1, vh = tid & 1;                  // V: dim, half of the slots
  int rv[8];
  bool v_whole = src >= 0;                                // these 8 slots all come from src
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    rv[i] = rows[vh * 8 + i];
    v_whole = v_whole && rv[i] < 0;
  }
  const bool first = dc < D / 16;                         // dims [0, D/2): x1' = x1 c - x2 s
  const int i0 = (first ? dc : dc - D / 16) * 8;          // pair index of element 0
  for (int g0 = 0; g0 < hkv; g0 += kHeads) {
    const int nh = min(kHeads, hkv - g0);
    uint4 kv[kHeads], vv[kHeads];
#pragma unroll
    for (int h = 0; h < kHeads; ++h) {
      if (h >= nh) break;
      const int g = g0 + h;
      kv[h] = make_uint4(0, 0, 0, 0);
      if (rk >= 0)
        kv[h] = *reinterpret_cast<const uint4*>(k_s + (size_t(rk) * hkv + g) * D + dc * 8);
      else if (src >= 0)
        kv[h] = *reinterpret_cast<const uint4*>(kc + ((size_t(src) * hkv + g) * 16 + o) * D + dc * 8);
      if (v_whole) {
        vv[h] = *reinterpret_cast<const uint4*>(vc + ((size_t(src) * hkv + g) * D + vd) * 16 + vh * 8);
      } else {
        uint16_t e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int r = rv[i];
          uint16_t x = 0;
          if (r >= 0)
            x = v_s[(size_t(r) * hkv + g) * D + vd];
          else if (src >= 0)
            x = vc[((size_t(src) * hkv + g) * D + vd) * 16 + vh * 8 + i];
          e[i] = x;
        }
        vv[h].x = uint32_t(e[0]) | (uint32_t(e[1]) << 16);
        vv[h].y = uint32_t(e[2]) | (uint32_t(e[3]) << 16);
        vv[h].z = uint32_t(e[4]) | (uint32_t(e[5]) << 16);
        vv[h].w = uint32_t(e[6]) | (uint32_t(e[7]) << 16);
      }
    }
    if (rot != 0 && g0 == 0) {                            // uniform over the workgroup
      if (tid < D / 2) {
        const double inv_freq = exp2(-double(2 * tid) / double(D) * log2_theta);
        double sn, cn;
        sincos(double(rot) * inv_freq, &sn, &cn);
        cs[tid] = make_float2(float(cn), float(sn));
      }
      __syncthreads();
    }
#pragma unroll
    for (int h = 0; h < kHeads; ++h) {
      if (h >= nh) break;
      const int g = g0 + h;
      uint4 val = kv[h];
      if (rot != 0) {
        // partner chunk: the other half of each rotation pair (all lanes take part)
        uint4 pr;
        pr.x = __shfl_xor(val.x, D / 16);
        pr.y = __shfl_xor(val.y, D / 16);
        pr.z = __shfl_xor(val.z, D / 16);
        pr.w = __shfl_xor(val.w, D / 16);
        if (rk < 0 && src >= 0) {
          const uint32_t mine[4] = {val.x, val.y, val.z, val.w};
          const uint32_t other[4] = {pr.x, pr.y, pr.z, pr.w};
          uint32_t res[4];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            float y[2];
#pragma unroll
            for (int e = 0; e < 2; ++e) {
              const float x = bf16_to_f32(uint16_t(mine[w] >> (16 * e)));
              const float z = bf16_to_f32(uint16_t(other[w] >> (16 * e)));
              const float2 t = cs[i0 + 2 * w + e];
              y[e] = first ? x * t.x - z * t.y : x * t.x + z * t.y;
            }
            res[w] = pack_bf16x2(y[0], y[1]);
          }
          val = make_uint4(res[0], res[1], res[2], res[3]);
        }
      }
      *reinterpret_cast<uint4*>(kc + ((size_t(dst) * hkv + g) * 16 + o) * D + dc * 8) = val;
      *reinterpret_cast<uint4*>(vc + ((size_t(dst) * hkv + g) * D + vd) * 16 + vh * 8) = vv[h];
    }
  }
}

void launch_link_write_rotated(const epic_plan* plan, int n_private, int hkv, int head_dim, float rope_theta,
                               const uint16_t* k_s, const uint16_t* v_s, uint16_t* k_cache, uint16_t* v_cache,
                               hipStream_t stream) {
  if (n_private == 0) return;
  const dim3 grid{unsigned(n_private)};
  const double l2t = std::log2(double(rope_theta));
  if (head_dim == 128)
    link_write_rotate_kernel<128><<<grid, 256, 0, stream>>>(plan->priv_block, plan->priv_src, plan->priv_rows,
                                                            plan->priv_rot, k_s, v_s, k_cache, v_cache, hkv, l2t);
  else
    link_write_rotate_kernel<64><<<grid, 128, 0, stream>>>(plan->priv_block, plan->priv_src, plan->priv_rows,
                                                           plan->priv_rot, k_s, v_s, k_cache, v_cache, hkv, l2t);
}

void launch_link_write(const epic_plan* plan, int n_private, int hkv, int head_dim, const uint16_t* k_s,
                       const uint16_t* v_s, uint16_t* k_cache, uint16_t* v_cache, hipStream_t stream) {
  if (n_private == 0) return;
  const dim3 grid(unsigned(n_private) * unsigned(hkv));
  if (head_dim == 128)
    link_write_kernel<128><<<grid, 256, 0, stream>>>(plan->priv_block, plan->priv_src, plan->priv_rows, k_s,
                                                     v_s, k_cache, v_cache, hkv);
  else
    link_write_kernel<64><<<grid, 128, 0, stream>>>(plan->priv_block, plan->priv_src, plan->priv_rows, k_s,
                                                    v_s, k_cache, v_cache, hkv);
}

}  // namespace epic
