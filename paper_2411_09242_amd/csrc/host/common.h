// Shared host-side types and error plumbing of the fluid library.
#pragma once

#include <cstdint>
#include <stdexcept>
#include <string>
#include <vector>

#include "fluid.h"

namespace fluid {

using Shape = std::vector<int64_t>;
using Perm = std::vector<int>;

constexpr int64_t kInf = int64_t(1) << 62;

// Saturating add of two non-negative costs bounded by kInf.
inline int64_t sat_add(int64_t a, int64_t b) {
  if (a >= kInf || b >= kInf) return kInf;
  int64_t s = a + b;  // both < 2^62: no overflow
  return s >= kInf ? kInf : s;
}

// Errors raised inside the library; converted to a status at the ABI.
struct Error : std::runtime_error {
  fluid_status status;
  Error(fluid_status s, const std::string& msg) : std::runtime_error(msg), status(s) {}
};

[[noreturn]] inline void fail(fluid_status s, const std::string& msg) { throw Error(s, msg); }
inline void require(bool ok, const std::string& msg) {
  if (!ok) fail(FLUID_E_INVALID, msg);
}

void set_last_error(const std::string& msg);

inline int64_t numel(const Shape& s) {
  int64_t n = 1;
  for (int64_t d : s) n *= d;
  return n;
}

inline int dtype_bytes(int dt) { return dt == FLUID_BF16 ? 2 : 4; }

std::string shape_str(const Shape& s);

}  // namespace fluid
