// Host launcher of the attention kernel for 16-row tiles (decode-shaped plans).
#pragma once

#include <hip/hip_runtime.h>

#include "kernels.h"

namespace epic {

// Same contract as launch_link_attention for a plan with tile_rows == 16: one
// workgroup per (work item, KV head); outputs, or split-KV partials that the
// combine kernel merges.
void launch_link_decode(const AttnArgs& a, int head_dim, int n_work, hipStream_t stream);

}  // namespace epic
