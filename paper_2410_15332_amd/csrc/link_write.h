// Host launcher of the link write for plans with re-rotated cached rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "epic_link.h"

namespace epic {

// As launch_link_write, plus: rows copied from priv_src into a block with
// priv_rot != 0 have their K rotated by that linked offset (rotary base rope_theta).
void launch_link_write_rotated(const epic_plan* plan, int n_private, int hkv, int head_dim, float rope_theta,
                               const uint16_t* k_s, const uint16_t* v_s, uint16_t* k_cache, uint16_t* v_cache,
                               hipStream_t stream);

}  // namespace epic
