// Model-level entry points (decoder layers for the S rows).
#include "plan_internal.h"
#include "status.h"

using namespace epic;

extern "C" size_t epic_model_workspace_bytes(const epic_model_cfg*, const epic_plan_sizes*) { return 0; }

extern "C" epic_status epic_link_layer(const epic_model_cfg*, const epic_layer_weights*, const epic_plan_sizes*,
                                       const epic_plan*, float*, uint16_t*, uint16_t*, void*, size_t, void*) {
  return fail(EPIC_ERR_UNSUPPORTED, "epic_link_layer: not built yet");
}

extern "C" epic_status epic_link_model(const epic_model_cfg*, const epic_layer_weights*, const uint16_t*,
                                       const epic_plan_sizes*, const epic_plan*, float*, uint16_t* const*,
                                       uint16_t* const*, float*, void*, size_t, void*) {
  return fail(EPIC_ERR_UNSUPPORTED, "epic_link_model: not built yet");
}
