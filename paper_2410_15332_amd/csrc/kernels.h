// Host-callable launchers of the gfx950 kernels (defined in the .hip sources).
// Shapes are validated by the entry points before any launcher is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "epic_link.h"

namespace epic {

// Private blocks of the linked cache: copy-on-write source, then the S rows.
void launch_link_write(const epic_plan* plan, int n_private, int hkv, int head_dim,
                       const uint16_t* k_s, const uint16_t* v_s, uint16_t* k_cache, uint16_t* v_cache,
                       hipStream_t stream);

struct AttnArgs {
  const int32_t* s_pos;
  const int32_t* linked_blocks;
  const int32_t* block_pos0;
  const int32_t* block_len;
  const int32_t* tiles;
  const int32_t* work;
  const uint16_t* q;        // [n_s][hq][D]
  const uint16_t* k_cache;
  const uint16_t* v_cache;
  uint16_t* out;            // [n_s][hq][D]
  float* lse;               // [n_s][hq] or null
  float* part_o;            // [n_partials][hkv][tile_rows][D]
  float* part_lse;          // [n_partials][hkv][tile_rows], log2 domain
  int hq, hkv, G, rows_per_tile;
  int tile_rows;            // 128 or 256 (selects the kernel)
  float scale_log2;         // softmax scale * log2(e)
};

// Scattered-query causal attention over the paged linked cache.
void launch_link_attention(const AttnArgs& a, int head_dim, int n_work, hipStream_t stream);
// Merge split-KV partials (tiles whose key range spans several work items).
void launch_link_combine(const AttnArgs& a, int head_dim, int n_tiles, hipStream_t stream);

void launch_rmsnorm(const float* x, const uint16_t* w, uint16_t* out_bf16, float* out_f32, int rows, int hidden,
                    float eps, hipStream_t stream);
void launch_rope_table(const int32_t* s_pos, float2* cs, int rows, int head_dim, double theta, hipStream_t stream);

}  // namespace epic
