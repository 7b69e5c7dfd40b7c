// Minimal JSON reader for the plan specification (objects, arrays, numbers,
// strings, true/false/null).  Parse errors throw dycl::SpecError with the
// byte offset; nothing here touches the GPU.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <stdexcept>
#include <string>
#include <vector>

namespace dycl {

struct SpecError : std::runtime_error {
  explicit SpecError(const std::string& m) : std::runtime_error(m) {}
};

class Json {
 public:
  enum Kind { Null, Bool, Number, String, Array, Object };

  Kind kind = Null;
  bool b = false;
  double num = 0.0;
  std::string str;
  std::vector<Json> arr;
  std::map<std::string, Json> obj;

  static Json parse(const std::string& text);

  bool is_null() const { return kind == Null; }
  bool has(const std::string& k) const { return kind == Object && obj.count(k) != 0; }
  const Json& at(const std::string& k) const;
  const Json& at(size_t i) const;
  size_t size() const { return kind == Array ? arr.size() : obj.size(); }

  int64_t as_int(const char* what = "value") const;
  double as_num(const char* what = "value") const;
  const std::string& as_str(const char* what = "value") const;
  bool as_bool(const char* what = "value") const;

  // convenience accessors with defaults
  int64_t get_int(const std::string& k, int64_t dflt) const {
    return has(k) && !at(k).is_null() ? at(k).as_int(k.c_str()) : dflt;
  }
  double get_num(const std::string& k, double dflt) const {
    return has(k) && !at(k).is_null() ? at(k).as_num(k.c_str()) : dflt;
  }
  std::string get_str(const std::string& k, const std::string& dflt) const {
    return has(k) && !at(k).is_null() ? at(k).as_str(k.c_str()) : dflt;
  }
  bool get_bool(const std::string& k, bool dflt) const {
    return has(k) && !at(k).is_null() ? at(k).as_bool(k.c_str()) : dflt;
  }
};

}  // namespace dycl
