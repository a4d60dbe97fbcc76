// Model-level entry points: one decoder layer (or all of them) for the S rows.
//
// Per layer (Sec. 4.2 recipe inside a Llama-style pre-norm block):
//   x = RMSNorm(h) w_attn                       bf16
//   q, k, v = x Wqkv^T, q and k rotated at the     bf16   (Q = E W_Q, K = E W_K, V = E W_V;
//             rows' linked positions                   one GEMM, rotation in its epilogue)
//   link write + attention over K_exp / V_exp    bf16   (Eq. 1)
//   h += o Wo^T                                  fp32   (O = A V_exp W_O, residual)
//   x = RMSNorm(h) w_mlp;  h += (silu(x Wg^T) * (x Wu^T)) Wd^T
// and after the last layer out = RMSNorm(h) w_final.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "gemm.h"
#include "link_write.h"
#include "kernels.h"
#include "plan_internal.h"
#include "status.h"

using namespace epic;

namespace {

size_t align256(size_t n) { return (n + 255) & ~size_t(255); }

struct LayerWs {
  uint16_t* x;       // [n_s][hidden]
  uint16_t* q;       // [n_s][hq][D]
  uint16_t* k;       // [n_s][hkv][D]
  uint16_t* v;       // [n_s][hkv][D]
  uint16_t* o;       // [n_s][hq D]
  uint16_t* act;     // [n_s][ffn]
  float2* cs;        // [n_s][D/2]
  void* attn;        // split-KV partials
  float* gemm_partial;   // GEMM tiles cut along K: partial sums
  int* gemm_count;       // ... and their arrival counters
  size_t total;
};

LayerWs carve(const epic_model_cfg* c, const epic_plan_sizes* s, char* base) {
  const size_t n = size_t(s->n_s);
  const int hq = c->attn.num_q_heads, hkv = c->attn.num_kv_heads, D = c->attn.head_dim;
  LayerWs w{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  };
  w.x = reinterpret_cast<uint16_t*>(take(n * c->hidden * 2));
  w.q = reinterpret_cast<uint16_t*>(take(n * size_t(hq) * D * 2));
  w.k = reinterpret_cast<uint16_t*>(take(n * size_t(hkv) * D * 2));
  w.v = reinterpret_cast<uint16_t*>(take(n * size_t(hkv) * D * 2));
  w.o = reinterpret_cast<uint16_t*>(take(n * size_t(hq) * D * 2));
  w.act = reinterpret_cast<uint16_t*>(take(n * size_t(c->ffn) * 2));
  w.cs = reinterpret_cast<float2*>(take(n * size_t(D / 2) * 8));
  w.attn = take(epic_link_workspace_bytes(&c->attn, s));
  char* gw = take(gemm_workspace_bytes());
  if (gw) gemm_workspace(gw, &w.gemm_partial, &w.gemm_count);
  w.total = off;
  return w;
}

epic_status validate_model(const epic_model_cfg* c) {
  EPIC_CHECK_ARG(c != nullptr, "model config is NULL");
  epic_status st = validate_attn_cfg(&c->attn);
  if (st != EPIC_OK) return st;
  const int hq = c->attn.num_q_heads, hkv = c->attn.num_kv_heads, D = c->attn.head_dim;
  if (c->hidden <= 0 || c->hidden % 128 != 0)
    return fail(EPIC_ERR_UNSUPPORTED, "hidden %d must be a positive multiple of 128", c->hidden);
  if (c->ffn <= 0 || c->ffn % 128 != 0)
    return fail(EPIC_ERR_UNSUPPORTED, "ffn %d must be a positive multiple of 128", c->ffn);
  if (((hq + 2 * hkv) * D) % 128 != 0 || (hq * D) % 64 != 0)
    return fail(EPIC_ERR_UNSUPPORTED, "(Hq + 2 Hkv) * D must be a multiple of 128");
  EPIC_CHECK_ARG(c->n_layers >= 1, "n_layers %d < 1", c->n_layers);
  EPIC_CHECK_ARG(c->rope_theta > 0.0f && c->rms_eps > 0.0f, "rope_theta and rms_eps must be > 0");
  return EPIC_OK;
}

epic_status check_weights(const epic_layer_weights* w) {
  EPIC_CHECK_ARG(w != nullptr, "layer weights are NULL");
  EPIC_CHECK_ARG(w->attn_norm && w->wqkv && w->wo && w->mlp_norm && w->w_gate_up && w->w_down,
                 "a layer weight pointer is NULL");
  auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  EPIC_CHECK_ARG(al(w->attn_norm) && al(w->wqkv) && al(w->wo) && al(w->mlp_norm) && al(w->w_gate_up) && al(w->w_down),
                 "weights must be 16-byte aligned");
  return EPIC_OK;
}

epic_status hip_ok(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(EPIC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return EPIC_OK;
}

// One layer; the rotary table ws.cs is already filled.
epic_status run_layer(const epic_model_cfg* c, const epic_layer_weights* w, const epic_plan_sizes* s,
                      const epic_plan* p, float* h, uint16_t* kc, uint16_t* vc, const LayerWs& ws,
                      hipStream_t stream) {
  const int n = s->n_s, H = c->hidden, F = c->ffn;
  const int hq = c->attn.num_q_heads, hkv = c->attn.num_kv_heads, D = c->attn.head_dim;
  launch_rmsnorm(h, w->attn_norm, ws.x, nullptr, n, H, c->rms_eps, stream);
  GemmArgs g{};
  g.A = ws.x;
  g.W = w->wqkv;
  g.M = n;
  g.N = (hq + 2 * hkv) * D;
  g.K = H;
  g.q = ws.q;
  g.k = ws.k;
  g.v = ws.v;
  g.cs = ws.cs;
  g.hq = hq;
  g.hkv = hkv;
  g.head_dim = D;
  g.partial = ws.gemm_partial;
  g.tile_count = ws.gemm_count;
  launch_gemm(g, kRope, stream);
  epic_attn_cfg ac = c->attn;
  ac.rope_theta = c->rope_theta;            // cached K was rotated with the model's base
  epic_status st = run_link_attention(&ac, s, p, ws.q, ws.k, ws.v, kc, vc, ws.o, nullptr, ws.attn, stream);
  if (st != EPIC_OK) return st;
  g = GemmArgs{};
  g.A = ws.o;
  g.W = w->wo;
  g.C = h;
  g.M = n;
  g.N = H;
  g.K = hq * D;
  g.partial = ws.gemm_partial;
  g.tile_count = ws.gemm_count;
  launch_gemm(g, kResidual, stream);
  launch_rmsnorm(h, w->mlp_norm, ws.x, nullptr, n, H, c->rms_eps, stream);
  g = GemmArgs{};
  g.A = ws.x;
  g.W = w->w_gate_up;
  g.act = ws.act;
  g.M = n;
  g.N = 2 * F;
  g.K = H;
  g.ffn = F;
  g.partial = ws.gemm_partial;
  g.tile_count = ws.gemm_count;
  launch_gemm(g, kSwiGLU, stream);
  g = GemmArgs{};
  g.A = ws.act;
  g.W = w->w_down;
  g.C = h;
  g.M = n;
  g.N = H;
  g.K = F;
  g.partial = ws.gemm_partial;
  g.tile_count = ws.gemm_count;
  launch_gemm(g, kResidual, stream);
  return hip_ok("decoder layer launch");
}

epic_status check_common(const epic_model_cfg* c, const epic_plan_sizes* s, const epic_plan* p, const float* h,
                         void* ws, size_t ws_bytes) {
  epic_status st = validate_model(c);
  if (st != EPIC_OK) return st;
  EPIC_CHECK_ARG(s && p, "plan is NULL");
  EPIC_CHECK_ARG(valid_tile_rows(s->tile_rows), "plan tile rows %d unsupported", s->tile_rows);
  EPIC_CHECK_ARG(s->n_rerotated >= 0 && s->n_rerotated <= s->n_private, "bad plan sizes (re-rotated blocks)");
  if (s->n_private > 0) EPIC_CHECK_ARG(p->priv_block && p->priv_src && p->priv_rows, "private block arrays are NULL");
  if (s->n_rerotated > 0) EPIC_CHECK_ARG(p->priv_rot != nullptr, "priv_rot is NULL");
  if (s->n_s == 0) return EPIC_OK;
  EPIC_CHECK_ARG(p->s_pos && p->tiles && p->work && p->linked_blocks, "device plan arrays are NULL");
  EPIC_CHECK_ARG(h != nullptr && (reinterpret_cast<uintptr_t>(h) & 15u) == 0, "hidden_s must be 16-byte aligned");
  // GEMM byte offsets are 31-bit: every operand and output (rows padded to a whole
  // 256-row tile) below 2^31 bytes
  const int64_t rows = int64_t(s->n_s) + 256;
  const int64_t qkv_n = int64_t(c->attn.num_q_heads + 2 * c->attn.num_kv_heads) * c->attn.head_dim;
  const int64_t kmax = std::max<int64_t>(std::max(c->hidden, c->ffn), int64_t(c->attn.num_q_heads) * c->attn.head_dim);
  const int64_t lim = int64_t(1) << 31;
  if (rows * kmax * 2 >= lim || rows * std::max<int64_t>(qkv_n, c->hidden) * 4 >= lim ||
      int64_t(4) * c->ffn * c->hidden >= lim)
    return fail(EPIC_ERR_UNSUPPORTED, "%d rows or the weights exceed the 2^31-byte GEMM operand limit", s->n_s);
  const size_t need = carve(c, s, nullptr).total;
  if (ws == nullptr || ws_bytes < need)
    return fail(EPIC_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed", ws_bytes, need);
  EPIC_CHECK_ARG((reinterpret_cast<uintptr_t>(ws) & 255u) == 0, "workspace must be 256-byte aligned");
  return EPIC_OK;
}

}  // namespace

extern "C" size_t epic_model_workspace_bytes(const epic_model_cfg* cfg, const epic_plan_sizes* sizes) {
  if (!cfg || !sizes || validate_model(cfg) != EPIC_OK) return 0;
  return carve(cfg, sizes, nullptr).total;
}

extern "C" epic_status epic_link_layer(const epic_model_cfg* cfg, const epic_layer_weights* w,
                                       const epic_plan_sizes* sizes, const epic_plan* plan_dev, float* hidden_s,
                                       uint16_t* k_cache, uint16_t* v_cache, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  clear_error();
  epic_status st = check_common(cfg, sizes, plan_dev, hidden_s, workspace, workspace_bytes);
  if (st != EPIC_OK) return st;
  if (sizes->n_s == 0) {                    // no rows: only the re-rotated copies, if any
    if (sizes->n_rerotated == 0) return EPIC_OK;
    EPIC_CHECK_ARG(k_cache && v_cache, "KV cache pointers are NULL");
    launch_link_write_rotated(plan_dev, sizes->n_private, cfg->attn.num_kv_heads, cfg->attn.head_dim,
                              cfg->rope_theta, nullptr, nullptr, k_cache, v_cache, static_cast<hipStream_t>(stream));
    return hip_ok("link write launch");
  }
  st = check_weights(w);
  if (st != EPIC_OK) return st;
  EPIC_CHECK_ARG(k_cache && v_cache, "KV cache pointers are NULL");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const LayerWs ws = carve(cfg, sizes, static_cast<char*>(workspace));
  launch_rope_table(plan_dev->s_pos, ws.cs, sizes->n_s, cfg->attn.head_dim, cfg->rope_theta, s);
  launch_gemm_clear(ws.gemm_count, s);
  return run_layer(cfg, w, sizes, plan_dev, hidden_s, k_cache, v_cache, ws, s);
}

extern "C" epic_status epic_link_model(const epic_model_cfg* cfg, const epic_layer_weights* layers,
                                       const uint16_t* final_norm, const epic_plan_sizes* sizes,
                                       const epic_plan* plan_dev, float* hidden_s, uint16_t* const* k_caches,
                                       uint16_t* const* v_caches, float* out_hidden, void* workspace,
                                       size_t workspace_bytes, void* stream) {
  clear_error();
  epic_status st = check_common(cfg, sizes, plan_dev, hidden_s, workspace, workspace_bytes);
  if (st != EPIC_OK) return st;
  if (sizes->n_s == 0) {                    // no rows: only the re-rotated copies, if any
    if (sizes->n_rerotated == 0) return EPIC_OK;
    EPIC_CHECK_ARG(k_caches && v_caches, "KV cache pointers are NULL");
    for (int l = 0; l < cfg->n_layers; ++l) {
      EPIC_CHECK_ARG(k_caches[l] && v_caches[l], "layer %d: KV cache pointers are NULL", l);
      launch_link_write_rotated(plan_dev, sizes->n_private, cfg->attn.num_kv_heads, cfg->attn.head_dim,
                                cfg->rope_theta, nullptr, nullptr, k_caches[l], v_caches[l],
                                static_cast<hipStream_t>(stream));
    }
    return hip_ok("link write launch");
  }
  EPIC_CHECK_ARG(layers && k_caches && v_caches && final_norm && out_hidden, "NULL model argument");
  for (int l = 0; l < cfg->n_layers; ++l) {
    st = check_weights(&layers[l]);
    if (st != EPIC_OK) return st;
    EPIC_CHECK_ARG(k_caches[l] && v_caches[l], "layer %d: KV cache pointers are NULL", l);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const LayerWs ws = carve(cfg, sizes, static_cast<char*>(workspace));
  launch_rope_table(plan_dev->s_pos, ws.cs, sizes->n_s, cfg->attn.head_dim, cfg->rope_theta, s);
  launch_gemm_clear(ws.gemm_count, s);
  for (int l = 0; l < cfg->n_layers; ++l) {
    st = run_layer(cfg, &layers[l], sizes, plan_dev, hidden_s, k_caches[l], v_caches[l], ws, s);
    if (st != EPIC_OK) return st;
  }
  launch_rmsnorm(hidden_s, final_norm, nullptr, out_hidden, sizes->n_s, cfg->hidden, cfg->rms_eps, s);
  return hip_ok("final norm launch");
}

extern "C" size_t epic_gemm_workspace_bytes(void) { return gemm_workspace_bytes(); }

extern "C" epic_status epic_gemm(int32_t epilogue, const uint16_t* a, const uint16_t* w, int32_t m, int32_t n,
                                 int32_t k, float* c, uint16_t* act, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  clear_error();
  EPIC_CHECK_ARG(epilogue >= EPIC_GEMM_STORE && epilogue <= EPIC_GEMM_SWIGLU, "unknown epilogue %d", epilogue);
  EPIC_CHECK_ARG(m >= 0 && n > 0 && k > 0, "m, n, k = %d, %d, %d", m, n, k);
  if (k % 64 != 0 || n % 128 != 0)
    return fail(EPIC_ERR_UNSUPPORTED, "k %% 64 == 0 and n %% 128 == 0 required (k = %d, n = %d)", k, n);
  const int64_t rows = int64_t(m) + 256, lim = int64_t(1) << 31;
  const int64_t out_row_bytes = epilogue == EPIC_GEMM_SWIGLU ? int64_t(n / 2) * 2 : int64_t(n) * 4;
  if (rows * k * 2 >= lim || int64_t(n) * k * 2 >= lim || rows * out_row_bytes >= lim)
    return fail(EPIC_ERR_UNSUPPORTED, "operands of %d x %d x %d exceed the 2^31-byte limit", m, n, k);
  if (m == 0) return EPIC_OK;
  auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  EPIC_CHECK_ARG(a && w && al(a) && al(w), "a and w must be non-NULL and 16-byte aligned");
  if (epilogue == EPIC_GEMM_SWIGLU)
    EPIC_CHECK_ARG(act && al(act), "act must be non-NULL and 16-byte aligned");
  else
    EPIC_CHECK_ARG(c && al(c), "c must be non-NULL and 16-byte aligned");
  if (workspace == nullptr || workspace_bytes < gemm_workspace_bytes())
    return fail(EPIC_ERR_WORKSPACE, "workspace of %zu bytes given, %zu needed", workspace_bytes,
                gemm_workspace_bytes());
  EPIC_CHECK_ARG((reinterpret_cast<uintptr_t>(workspace) & 255u) == 0, "workspace must be 256-byte aligned");
  GemmArgs g{};
  g.A = a;
  g.W = w;
  g.M = m;
  g.N = n;
  g.K = k;
  if (epilogue == EPIC_GEMM_SWIGLU) {
    g.ffn = n / 2;
    g.act = act;
  } else {
    g.C = c;
  }
  gemm_workspace(workspace, &g.partial, &g.tile_count);
  hipStream_t s = static_cast<hipStream_t>(stream);
  launch_gemm_clear(g.tile_count, s);
  launch_gemm(g, epilogue, s);
  return hip_ok("projection GEMM launch");
}
