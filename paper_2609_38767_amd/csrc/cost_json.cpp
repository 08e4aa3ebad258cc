// Reads the routing cost model from a calibration file (JSON): the object
// under the top-level member "model", whose members name the fields of
// dattri_cost_model.  A small recursive-descent reader of RFC 8259 JSON that
// keeps only numbers inside that object and skips everything else.
#include <cctype>
#include <cerrno>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

#include "api_common.h"
#include "dattri.h"
#include "runtime.h"

namespace dattri {
namespace {

struct Reader {
  const char* p;
  const char* end;
  std::string err;

  bool fail_at(const char* what) {
    if (err.empty()) {
      char buf[96];
      std::snprintf(buf, sizeof(buf), "%s at byte %zu", what, (size_t)(p - begin));
      err = buf;
    }
    return false;
  }
  const char* begin;

  void ws() {
    while (p < end && (*p == ' ' || *p == '\t' || *p == '\n' || *p == '\r')) ++p;
  }
  bool lit(const char* word) {
    const size_t n = std::strlen(word);
    if ((size_t)(end - p) < n || std::strncmp(p, word, n) != 0) return fail_at("bad literal");
    p += n;
    return true;
  }
  bool string(std::string* out) {
    if (p >= end || *p != '"') return fail_at("expected a string");
    ++p;
    while (p < end && *p != '"') {
      if ((unsigned char)*p < 0x20) return fail_at("control character in a string");
      if (*p == '\\') {
        if (++p >= end) break;
        const char e = *p;
        if (e == 'u') {  // the field names are ASCII: keep escapes as '?'
          if (end - p < 5) return fail_at("short \\u escape");
          for (int i = 1; i <= 4; ++i)
            if (!std::isxdigit((unsigned char)p[i])) return fail_at("bad \\u escape");
          p += 4;
          if (out) out->push_back('?');
        } else if (std::strchr("\"\\/bfnrt", e)) {
          if (out) out->push_back(e == 'n' ? '\n' : e == 't' ? '\t' : e);
        } else {
          return fail_at("bad escape");
        }
        ++p;
        continue;
      }
      if (out) out->push_back(*p);
      ++p;
    }
    if (p >= end) return fail_at("unterminated string");
    ++p;
    return true;
  }
  bool number(double* out) {
    // JSON grammar: -? (0 | [1-9][0-9]*) (. [0-9]+)? ([eE] [+-]? [0-9]+)?
    const char* s = p;
    if (p < end && *p == '-') ++p;
    if (p >= end || !std::isdigit((unsigned char)*p)) return fail_at("bad number");
    if (*p == '0') ++p;
    else while (p < end && std::isdigit((unsigned char)*p)) ++p;
    if (p < end && *p == '.') {
      ++p;
      if (p >= end || !std::isdigit((unsigned char)*p)) return fail_at("bad fraction");
      while (p < end && std::isdigit((unsigned char)*p)) ++p;
    }
    if (p < end && (*p == 'e' || *p == 'E')) {
      ++p;
      if (p < end && (*p == '+' || *p == '-')) ++p;
      if (p >= end || !std::isdigit((unsigned char)*p)) return fail_at("bad exponent");
      while (p < end && std::isdigit((unsigned char)*p)) ++p;
    }
    const std::string text(s, p);
    errno = 0;
    const double v = std::strtod(text.c_str(), nullptr);
    if (errno == ERANGE && std::isinf(v)) return fail_at("number out of range");
    if (out) *out = v;
    return true;
  }
  // Any value; when `model` is set and the value is an object, its numeric
  // members are offered to `take`.
  template <class Take>
  bool value(int depth, bool model, Take& take) {
    if (depth > 64) return fail_at("nesting too deep");
    ws();
    if (p >= end) return fail_at("unexpected end");
    switch (*p) {
      case '{': {
        ++p;
        ws();
        if (p < end && *p == '}') { ++p; return true; }
        for (;;) {
          ws();
          std::string key;
          if (!string(&key)) return false;
          ws();
          if (p >= end || *p != ':') return fail_at("expected ':'");
          ++p;
          ws();
          if (model && p < end && (*p == '-' || std::isdigit((unsigned char)*p))) {
            double v;
            if (!number(&v)) return false;
            take(key, v);
          } else if (!value(depth + 1, !model && depth == 0 && key == "model", take)) {
            return false;
          }
          if (depth == 0 && key == "model") take.saw_model = true;
          ws();
          if (p < end && *p == ',') { ++p; continue; }
          if (p < end && *p == '}') { ++p; return true; }
          return fail_at("expected ',' or '}'");
        }
      }
      case '[': {
        ++p;
        ws();
        if (p < end && *p == ']') { ++p; return true; }
        for (;;) {
          if (!value(depth + 1, false, take)) return false;
          ws();
          if (p < end && *p == ',') { ++p; continue; }
          if (p < end && *p == ']') { ++p; return true; }
          return fail_at("expected ',' or ']'");
        }
      }
      case '"': return string(nullptr);
      case 't': return lit("true");
      case 'f': return lit("false");
      case 'n': return lit("null");
      default: return number(nullptr);
    }
  }
};

struct Fields {
  static constexpr int kN = 9;
  const char* names[kN] = {"factored_tflops", "factored_gbs", "gradient_tflops", "gradient_gbs",
                           "gproject_tflops", "gproject_gbs", "launch_us", "call_us", "round_us"};
  double v[kN];
  bool got[kN] = {};
  bool saw_model = false;
  void operator()(const std::string& key, double x) {
    for (int i = 0; i < kN; ++i)
      if (key == names[i]) {
        v[i] = x;
        got[i] = true;
      }
  }
};

}  // namespace

dattri_status read_cost_calibration(const char* path, dattri_cost_model* out) {
  FILE* f = std::fopen(path, "rb");
  if (!f) return fail(DATTRI_E_INVALID_ARG, "cannot open calibration file '%s': %s", path, std::strerror(errno));
  std::string text;
  char buf[65536];
  size_t got;
  while ((got = std::fread(buf, 1, sizeof(buf), f)) > 0) {
    text.append(buf, got);
    if (text.size() > ((size_t)64 << 20)) {
      std::fclose(f);
      return fail(DATTRI_E_INVALID_ARG, "calibration file '%s' is larger than 64 MiB", path);
    }
  }
  const bool read_error = std::ferror(f) != 0;
  std::fclose(f);
  if (read_error) return fail(DATTRI_E_INVALID_ARG, "cannot read calibration file '%s'", path);
  Reader r{text.data(), text.data() + text.size(), {}, text.data()};
  Fields fields;
  r.ws();
  if (r.p >= r.end || *r.p != '{')
    return fail(DATTRI_E_INVALID_ARG, "calibration file '%s' is not a JSON object", path);
  if (!r.value(0, false, fields)) return fail(DATTRI_E_INVALID_ARG, "calibration file '%s': %s", path, r.err.c_str());
  r.ws();
  if (r.p != r.end) return fail(DATTRI_E_INVALID_ARG, "calibration file '%s': trailing data", path);
  if (!fields.saw_model) return fail(DATTRI_E_INVALID_ARG, "calibration file '%s' has no \"model\" object", path);
  for (int i = 0; i < Fields::kN; ++i)
    if (!fields.got[i])
      return fail(DATTRI_E_INVALID_ARG, "calibration file '%s': model.%s missing or not a number", path,
                  fields.names[i]);
  out->factored_tflops = fields.v[0];
  out->factored_gbs = fields.v[1];
  out->gradient_tflops = fields.v[2];
  out->gradient_gbs = fields.v[3];
  out->gproject_tflops = fields.v[4];
  out->gproject_gbs = fields.v[5];
  out->launch_us = fields.v[6];
  out->call_us = fields.v[7];
  out->round_us = fields.v[8];
  return DATTRI_OK;
}

}  // namespace dattri
