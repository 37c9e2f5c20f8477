// GPU entry points in the host-only build: they exist so that the same
// symbol set is exported, and report FLUID_E_UNSUPPORTED.
#include "fluid.h"
#include "handles.h"

using namespace fluid;

namespace {
fluid_status unsupported(const char* what) {
  set_last_error(std::string(what) + ": not available in the host-only library (no GPU code)");
  return FLUID_E_UNSUPPORTED;
}
}  // namespace

extern "C" {

fluid_status fluid_run(const fluid_graph*, const fluid_layout_plan*, const fluid_arena_plan*, void*, uint64_t,
                       const void* const*, const void* const*, void* const*, void*) {
  return unsupported("fluid_run");
}

fluid_status fluid_run_static(const fluid_graph*, const fluid_layout_plan*, const fluid_arena_plan*, const void* const*,
                              const void* const*, void* const*, void*) {
  return unsupported("fluid_run_static");
}

fluid_status fluid_pack_constant(const fluid_graph*, const fluid_layout_plan*, int32_t, const void*, void*, void*) {
  return unsupported("fluid_pack_constant");
}

fluid_status fluid_run_nodes(const fluid_graph*, const fluid_layout_plan*, const fluid_arena_plan*, void*, uint64_t,
                             const void* const*, const void* const*, void* const*, const int32_t*, int32_t, int32_t,
                             void*) {
  return unsupported("fluid_run_nodes");
}

fluid_status fluid_measure_costs(const fluid_graph*, uint32_t, void*, uint64_t, void*, fluid_cost_table**) {
  return unsupported("fluid_measure_costs");
}

fluid_status fluid_trace_enable(const fluid_graph*, const uint8_t*, int32_t) { return unsupported("fluid_trace_enable"); }

fluid_status fluid_trace_collect(const fluid_graph*, double*, int32_t*) { return unsupported("fluid_trace_collect"); }

}  // extern "C"
