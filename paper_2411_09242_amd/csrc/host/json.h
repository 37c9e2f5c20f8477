// Minimal JSON reader for the cost-table file (objects, arrays, numbers,
// strings, true/false/null).  Numbers are kept as int64 when integral.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <vector>

namespace fluid {

struct Json {
  enum Kind { Null, Bool, Int, Float, Str, Arr, Obj } kind = Null;
  bool b = false;
  int64_t i = 0;
  double f = 0.0;
  std::string s;
  std::vector<Json> a;
  std::map<std::string, Json> o;

  const Json& at(const std::string& k) const;   // throws FLUID_E_INVALID if absent
  bool has(const std::string& k) const { return kind == Obj && o.count(k); }
  int64_t as_int() const;
  const std::vector<Json>& arr() const;
};

Json json_parse(const std::string& text);  // throws fluid::Error(FLUID_E_INVALID)

}  // namespace fluid
