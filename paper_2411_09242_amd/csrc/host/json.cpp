#include "json.h"

#include <cmath>
#include <cstdlib>

#include "common.h"

namespace fluid {

namespace {

struct Parser {
  const std::string& t;
  size_t p = 0;
  explicit Parser(const std::string& s) : t(s) {}

  [[noreturn]] void bad(const char* what) {
    fail(FLUID_E_INVALID, std::string("json: ") + what + " at offset " + std::to_string(p));
  }
  void ws() {
    while (p < t.size() && (t[p] == ' ' || t[p] == '\n' || t[p] == '\r' || t[p] == '\t')) ++p;
  }
  bool lit(const char* w) {
    size_t n = std::char_traits<char>::length(w);
    if (t.compare(p, n, w) == 0) { p += n; return true; }
    return false;
  }
  Json value(int depth) {
    if (depth > 64) bad("nesting too deep");
    ws();
    if (p >= t.size()) bad("unexpected end");
    Json v;
    char c = t[p];
    if (c == '{') {
      v.kind = Json::Obj;
      ++p; ws();
      if (p < t.size() && t[p] == '}') { ++p; return v; }
      for (;;) {
        ws();
        if (p >= t.size() || t[p] != '"') bad("expected key");
        std::string k = str();
        ws();
        if (p >= t.size() || t[p] != ':') bad("expected ':'");
        ++p;
        v.o[k] = value(depth + 1);
        ws();
        if (p < t.size() && t[p] == ',') { ++p; continue; }
        if (p < t.size() && t[p] == '}') { ++p; return v; }
        bad("expected ',' or '}'");
      }
    }
    if (c == '[') {
      v.kind = Json::Arr;
      ++p; ws();
      if (p < t.size() && t[p] == ']') { ++p; return v; }
      for (;;) {
        v.a.push_back(value(depth + 1));
        ws();
        if (p < t.size() && t[p] == ',') { ++p; continue; }
        if (p < t.size() && t[p] == ']') { ++p; return v; }
        bad("expected ',' or ']'");
      }
    }
    if (c == '"') { v.kind = Json::Str; v.s = str(); return v; }
    if (lit("true")) { v.kind = Json::Bool; v.b = true; return v; }
    if (lit("false")) { v.kind = Json::Bool; return v; }
    if (lit("null")) return v;
    return number();
  }
  std::string str() {
    ++p;  // opening quote
    std::string r;
    while (p < t.size() && t[p] != '"') {
      if (t[p] == '\\') {
        ++p;
        if (p >= t.size()) bad("bad escape");
        char e = t[p];
        if (e == 'n') r += '\n';
        else if (e == 't') r += '\t';
        else if (e == 'u') { r += '?'; p += 4; }
        else r += e;
        ++p;
      } else {
        r += t[p++];
      }
    }
    if (p >= t.size()) bad("unterminated string");
    ++p;
    return r;
  }
  Json number() {
    size_t s = p;
    if (p < t.size() && (t[p] == '-' || t[p] == '+')) ++p;
    bool isf = false;
    while (p < t.size()) {
      char c = t[p];
      if (c >= '0' && c <= '9') { ++p; continue; }
      if (c == '.' || c == 'e' || c == 'E' || c == '-' || c == '+') { isf = true; ++p; continue; }
      break;
    }
    if (p == s) bad("unexpected character");
    std::string tok = t.substr(s, p - s);
    Json v;
    if (!isf) {
      char* end = nullptr;
      long long x = std::strtoll(tok.c_str(), &end, 10);
      if (*end) bad("bad integer");
      v.kind = Json::Int;
      v.i = x;
      v.f = (double)x;
    } else {
      char* end = nullptr;
      v.f = std::strtod(tok.c_str(), &end);
      if (*end) bad("bad number");
      v.kind = Json::Float;
    }
    return v;
  }
};

}  // namespace

const Json& Json::at(const std::string& k) const {
  if (kind != Obj) fail(FLUID_E_INVALID, "json: expected an object with key '" + k + "'");
  auto it = o.find(k);
  if (it == o.end()) fail(FLUID_E_INVALID, "json: missing key '" + k + "'");
  return it->second;
}

int64_t Json::as_int() const {
  if (kind == Int) return i;
  if (kind == Float && std::floor(f) == f) return (int64_t)f;
  fail(FLUID_E_INVALID, "json: expected an integer");
}

const std::vector<Json>& Json::arr() const {
  if (kind != Arr) fail(FLUID_E_INVALID, "json: expected an array");
  return a;
}

Json json_parse(const std::string& text) {
  Parser ps(text);
  Json v = ps.value(0);
  ps.ws();
  if (ps.p != text.size()) ps.bad("trailing characters");
  return v;
}

}  // namespace fluid
