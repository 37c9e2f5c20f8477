// Opaque handle types behind the C ABI, and the error-to-status wrapper.
#pragma once

#include <new>
#include <string>

#include "costtable.h"
#include "graph.h"
#include "planner.h"

struct fluid_graph {
  fluid::Graph g;
  uint64_t serial = 0;
};
struct fluid_cost_table {
  fluid::CostTable t;
  uint64_t serial = 0;  // graph the table was bound to
};
struct fluid_layout_plan {
  fluid::LayoutPlan p;
  uint64_t serial = 0;  // identity of this plan object (never reused)
};
struct fluid_arena_plan {
  fluid::ArenaPlan a;
  uint64_t serial = 0;
};

namespace fluid {

uint64_t next_serial();

template <class F>
fluid_status call_guarded(F&& f) {
  try {
    f();
    set_last_error("");
    return FLUID_OK;
  } catch (const Error& e) {
    set_last_error(e.what());
    return e.status;
  } catch (const std::bad_alloc&) {
    set_last_error("host allocation failed");
    return FLUID_E_NOMEM;
  } catch (const std::exception& e) {
    set_last_error(std::string("internal error: ") + e.what());
    return FLUID_E_INVALID;
  }
}

// Device-scratch bytes needed to measure every node signature of g.
uint64_t measure_scratch_bytes(const Graph& g);

}  // namespace fluid
