// Device entry points of libepic_link: argument validation on the host, then
// kernel launches on the caller's stream.  Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "decode_attention.h"
#include "kernels.h"
#include "link_write.h"
#include "plan_internal.h"
#include "status.h"

using namespace epic;

namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t round_up(size_t n, size_t a) { return (n + a - 1) / a * a; }

// Workspace of the attention step: split-KV partial outputs and their log-sum-exps.
size_t attn_partials_bytes(const epic_attn_cfg* cfg, const epic_plan_sizes* s) {
  const size_t rows = size_t(s->n_partials) * cfg->num_kv_heads * s->tile_rows;
  return round_up(rows * cfg->head_dim * sizeof(float), 256) + round_up(rows * sizeof(float), 256);
}

epic_status check_plan(const epic_plan_sizes* s, const epic_plan* p) {
  EPIC_CHECK_ARG(s != nullptr, "plan sizes are NULL");
  EPIC_CHECK_ARG(p != nullptr, "device plan is NULL");
  EPIC_CHECK_ARG(s->n_s >= 0 && s->n_work >= 0 && s->n_partials >= 0 && s->n_private >= 0, "bad plan sizes");
  EPIC_CHECK_ARG(valid_tile_rows(s->tile_rows), "plan tile rows %d (expected %d, %d or %d)", s->tile_rows,
                 kTileRowsTiny, kTileRowsSmall, kTileRowsLarge);
  if (s->n_s > 0)
    EPIC_CHECK_ARG(p->s_pos && p->linked_blocks && p->block_pos0 && p->block_len && p->tiles && p->work,
                   "device plan arrays are NULL");
  if (s->n_private > 0) EPIC_CHECK_ARG(p->priv_block && p->priv_src && p->priv_rows, "private block arrays are NULL");
  EPIC_CHECK_ARG(s->n_rerotated >= 0 && s->n_rerotated <= s->n_private, "bad plan sizes (re-rotated blocks)");
  if (s->n_rerotated > 0) EPIC_CHECK_ARG(p->priv_rot != nullptr, "priv_rot is NULL");
  return EPIC_OK;
}

// Optional profiling events of the calling thread (see epic_set_profile_events).
thread_local hipEvent_t g_prof_events[4] = {nullptr, nullptr, nullptr, nullptr};

void record_event(int i, hipStream_t stream) {
  if (g_prof_events[i]) (void)hipEventRecord(g_prof_events[i], stream);
}

epic_status hip_status(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(EPIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return EPIC_OK;
}

}  // namespace

extern "C" epic_status epic_set_profile_events(void* const* events) {
  clear_error();
  for (int i = 0; i < 4; ++i) g_prof_events[i] = events ? static_cast<hipEvent_t>(events[i]) : nullptr;
  return EPIC_OK;
}

extern "C" size_t epic_link_workspace_bytes(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes) {
  if (!cfg || !sizes || validate_attn_cfg(cfg) != EPIC_OK) return 0;
  return attn_partials_bytes(cfg, sizes);
}

namespace epic {

// Shared by epic_link_attention and the layer driver: link write, attention, combine.
epic_status run_link_attention(const epic_attn_cfg* cfg, const epic_plan_sizes* s, const epic_plan* p,
                               const uint16_t* q_s, const uint16_t* k_s, const uint16_t* v_s,
                               uint16_t* k_cache, uint16_t* v_cache, uint16_t* out, float* lse,
                               void* workspace, void* stream_ptr) {
  hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  record_event(0, stream);
  if (s->n_rerotated > 0)
    launch_link_write_rotated(p, s->n_private, cfg->num_kv_heads, cfg->head_dim, cfg->rope_theta, k_s, v_s, k_cache,
                              v_cache, stream);
  else
    launch_link_write(p, s->n_private, cfg->num_kv_heads, cfg->head_dim, k_s, v_s, k_cache, v_cache, stream);
  if (s->n_s == 0) return hip_status("link write launch");   // re-rotated copies only
  AttnArgs a{};
  a.s_pos = p->s_pos;
  a.linked_blocks = p->linked_blocks;
  a.block_pos0 = p->block_pos0;
  a.block_len = p->block_len;
  a.tiles = p->tiles;
  a.work = p->work;
  a.q = q_s;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.out = out;
  a.lse = lse;
  const size_t rows = size_t(s->n_partials) * cfg->num_kv_heads * s->tile_rows;
  a.part_o = static_cast<float*>(workspace);
  a.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                        round_up(rows * cfg->head_dim * sizeof(float), 256));
  a.hq = cfg->num_q_heads;
  a.hkv = cfg->num_kv_heads;
  a.G = cfg->num_q_heads / cfg->num_kv_heads;
  a.tile_rows = s->tile_rows;
  a.rows_per_tile = s->tile_rows / a.G;
  const float scale = cfg->softmax_scale > 0.0f ? cfg->softmax_scale : 1.0f / std::sqrt(float(cfg->head_dim));
  a.scale_log2 = scale * kLog2eHost;
  record_event(1, stream);
  if (s->tile_rows == kTileRowsTiny)
    launch_link_decode(a, cfg->head_dim, s->n_work, stream);
  else
    launch_link_attention(a, cfg->head_dim, s->n_work, stream);
  record_event(2, stream);
  if (s->n_partials > 0) launch_link_combine(a, cfg->head_dim, s->n_tiles, stream);
  record_event(3, stream);
  return hip_status("link attention launch");
}

}  // namespace epic

extern "C" epic_status epic_link_attention(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes,
                                           const epic_plan* plan_dev, const uint16_t* q_s, const uint16_t* k_s,
                                           const uint16_t* v_s, uint16_t* k_cache, uint16_t* v_cache,
                                           uint16_t* out, float* lse, void* workspace, size_t workspace_bytes,
                                           void* stream) {
  clear_error();
  epic_status st = validate_attn_cfg(cfg);
  if (st != EPIC_OK) return st;
  st = check_plan(sizes, plan_dev);
  if (st != EPIC_OK) return st;
  if (sizes->n_rerotated > 0 && !(cfg->rope_theta > 1.0f))
    return fail(EPIC_ERR_INVALID_ARG, "plan re-rotates cached K: rope_theta %g must be > 1", cfg->rope_theta);
  if (sizes->n_s == 0 && sizes->n_private == 0) return EPIC_OK;
  EPIC_CHECK_ARG(k_cache && v_cache && aligned16(k_cache) && aligned16(v_cache), "KV caches NULL or unaligned");
  if (sizes->n_s == 0)
    return run_link_attention(cfg, sizes, plan_dev, nullptr, nullptr, nullptr, k_cache, v_cache, nullptr, nullptr,
                              nullptr, stream);
  EPIC_CHECK_ARG(q_s && k_s && v_s && k_cache && v_cache && out, "NULL tensor argument");
  EPIC_CHECK_ARG(aligned16(q_s) && aligned16(k_s) && aligned16(v_s) && aligned16(k_cache) && aligned16(v_cache) &&
                     aligned16(out),
                 "tensors must be 16-byte aligned");
  const size_t need = attn_partials_bytes(cfg, sizes);
  if (need > 0 && (workspace == nullptr || workspace_bytes < need))
    return fail(EPIC_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes, need);
  if (need > 0) EPIC_CHECK_ARG(aligned16(workspace), "workspace must be 16-byte aligned");
  return run_link_attention(cfg, sizes, plan_dev, q_s, k_s, v_s, k_cache, v_cache, out, lse, workspace, stream);
}
