// Constants and helpers shared by the host sources (planner and entry points).
#pragma once

#include "epic_link.h"

namespace epic {

constexpr int kBlock = 16;         // token slots per KV block
// (S row, query head) pairs per attention tile: 128 (two 4-wavefront workgroups per
// CU) or 256 (one 8-wavefront workgroup per CU), chosen per plan by the planner
constexpr int kTileRowsSmall = 128;
constexpr int kTileRowsLarge = 256;
// 16-row tiles: decode-shaped plans (a few S rows per request), own kernel
constexpr int kTileRowsTiny = 16;
inline bool valid_tile_rows(int r) { return r == kTileRowsTiny || r == kTileRowsSmall || r == kTileRowsLarge; }
constexpr int kKvTileBlocks = 4;   // KV blocks staged per attention iteration (64 keys)
constexpr int kWorkInts = 8;       // int32 per attention work item
constexpr float kLog2eHost = 1.442695040888963407f;

epic_status validate_attn_cfg(const epic_attn_cfg* cfg);

// Link write + attention (+ split-KV combine) for one layer, arguments already validated.
epic_status run_link_attention(const epic_attn_cfg* cfg, const epic_plan_sizes* s, const epic_plan* p,
                               const uint16_t* q_s, const uint16_t* k_s, const uint16_t* v_s,
                               uint16_t* k_cache, uint16_t* v_cache, uint16_t* out, float* lse,
                               void* workspace, void* stream);

}  // namespace epic
