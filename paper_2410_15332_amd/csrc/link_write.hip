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
#include "device_common.h"
#include "kernels.h"

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
