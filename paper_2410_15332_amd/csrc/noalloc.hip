// The attention step of the link without a caller workspace, for callers that
// cannot allocate device memory (code under HIP graph capture, tight serving
// loops, harnesses that forbid hipMalloc).  The split-KV partials that
// epic_link_attention keeps in the caller's workspace go to a fixed device-global
// array instead; every kernel is the one epic_link_attention launches.
//
// The array is a device global: each GPU the library runs on holds its own copy,
// at its own address, from the time the library's code is loaded on that GPU
// until the process ends.  The host never passes the array's name to a kernel
// (in host code that name is a host-side stand-in, not a device address); the
// device address is looked up once per device with hipGetSymbolAddress, with
// that device current, and kept.
#include <hip/hip_runtime.h>

#include <mutex>

#include "plan_internal.h"
#include "status.h"

using namespace epic;

namespace {

static __device__ __align__(256) unsigned char scratch[EPIC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (looked up on first use).
epic_status scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxDevices)
    return fail(EPIC_ERR_UNSUPPORTED, "device %d: at most %d devices are supported", device, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (g_scratch_ptr[device] == nullptr) {
    int current = -1;
    hipError_t e = hipGetDevice(&current);
    if (e != hipSuccess) return fail(EPIC_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (current != device && (e = hipSetDevice(device)) != hipSuccess)
      return fail(EPIC_ERR_HIP, "hipSetDevice(%d): %s", device, hipGetErrorString(e));
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (current != device) (void)hipSetDevice(current);
    if (e != hipSuccess || p == nullptr)
      return fail(EPIC_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", device, hipGetErrorString(e));
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return EPIC_OK;
}

}  // namespace

extern "C" epic_status epic_link_attention_noalloc(const epic_attn_cfg* cfg, const epic_plan_sizes* sizes,
                                                   const epic_plan* plan_dev, const uint16_t* q_s,
                                                   const uint16_t* k_s, const uint16_t* v_s, uint16_t* k_cache,
                                                   uint16_t* v_cache, uint16_t* out, float* lse, void* stream) {
  clear_error();
  epic_status st = validate_attn_cfg(cfg);
  if (st != EPIC_OK) return st;
  const size_t need = epic_link_workspace_bytes(cfg, sizes);
  if (sizes != nullptr && need > size_t(EPIC_NOALLOC_SCRATCH_BYTES))
    return fail(EPIC_ERR_WORKSPACE,
                "plan needs %zu bytes of split-KV partials, above the fixed %zu-byte scratch array "
                "(a larger kv_split_blocks gives fewer partials)",
                need, size_t(EPIC_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  if (need > 0) {
    int device = -1;                    // the device the work is enqueued on
    hipError_t e = stream == nullptr ? hipGetDevice(&device)
                                     : hipStreamGetDevice(static_cast<hipStream_t>(stream), &device);
    if (e != hipSuccess) return fail(EPIC_ERR_HIP, "device of the stream: %s", hipGetErrorString(e));
    st = scratch_address(device, &ws);
    if (st != EPIC_OK) return st;
  }
  // every argument check of the entry point with a caller workspace, then the same kernels
  return epic_link_attention(cfg, sizes, plan_dev, q_s, k_s, v_s, k_cache, v_cache, out, lse, ws, need, stream);
}
