#include "json.hpp"

#include <cmath>
#include <cstdlib>

namespace dycl {

namespace {

struct Parser {
  const std::string& s;
  size_t i = 0;
  int depth = 0;

  explicit Parser(const std::string& t) : s(t) {}

  [[noreturn]] void fail(const std::string& m) const {
    throw SpecError("JSON parse error at byte " + std::to_string(i) + ": " + m);
  }
  void ws() {
    while (i < s.size() && (s[i] == ' ' || s[i] == '\n' || s[i] == '\t' || s[i] == '\r')) ++i;
  }
  bool eat(char c) {
    ws();
    if (i < s.size() && s[i] == c) {
      ++i;
      return true;
    }
    return false;
  }
  void expect(char c) {
    if (!eat(c)) fail(std::string("expected '") + c + "'");
  }

  Json value() {
    if (++depth > 64) fail("nesting too deep");
    ws();
    if (i >= s.size()) fail("unexpected end");
    Json v;
    char c = s[i];
    if (c == '{') {
      ++i;
      v.kind = Json::Object;
      if (!eat('}')) {
        do {
          ws();
          std::string k = string_lit();
          expect(':');
          v.obj[k] = value();
        } while (eat(','));
        expect('}');
      }
    } else if (c == '[') {
      ++i;
      v.kind = Json::Array;
      if (!eat(']')) {
        do {
          v.arr.push_back(value());
        } while (eat(','));
        expect(']');
      }
    } else if (c == '"') {
      v.kind = Json::String;
      v.str = string_lit();
    } else if (s.compare(i, 4, "true") == 0) {
      i += 4;
      v.kind = Json::Bool;
      v.b = true;
    } else if (s.compare(i, 5, "false") == 0) {
      i += 5;
      v.kind = Json::Bool;
    } else if (s.compare(i, 4, "null") == 0) {
      i += 4;
    } else if (c == '-' || (c >= '0' && c <= '9')) {
      const char* start = s.c_str() + i;
      char* end = nullptr;
      v.num = std::strtod(start, &end);
      if (end == start) fail("bad number");
      i += static_cast<size_t>(end - start);
      v.kind = Json::Number;
    } else {
      fail(std::string("unexpected character '") + c + "'");
    }
    --depth;
    return v;
  }

  std::string string_lit() {
    if (i >= s.size() || s[i] != '"') fail("expected string");
    ++i;
    std::string out;
    while (i < s.size() && s[i] != '"') {
      char c = s[i++];
      if (c == '\\') {
        if (i >= s.size()) fail("bad escape");
        char e = s[i++];
        switch (e) {
          case '"': out += '"'; break;
          case '\\': out += '\\'; break;
          case '/': out += '/'; break;
          case 'n': out += '\n'; break;
          case 't': out += '\t'; break;
          case 'r': out += '\r'; break;
          case 'b': out += '\b'; break;
          case 'f': out += '\f'; break;
          default: fail("unsupported escape");
        }
      } else {
        out += c;
      }
    }
    if (i >= s.size()) fail("unterminated string");
    ++i;
    return out;
  }
};

}  // namespace

Json Json::parse(const std::string& text) {
  Parser p(text);
  Json v = p.value();
  p.ws();
  if (p.i != text.size()) p.fail("trailing characters");
  return v;
}

const Json& Json::at(const std::string& k) const {
  if (kind != Object) throw SpecError("expected an object when looking up '" + k + "'");
  auto it = obj.find(k);
  if (it == obj.end()) throw SpecError("missing key '" + k + "'");
  return it->second;
}

const Json& Json::at(size_t idx) const {
  if (kind != Array || idx >= arr.size()) throw SpecError("array index out of range");
  return arr[idx];
}

int64_t Json::as_int(const char* what) const {
  if (kind != Number || std::floor(num) != num || std::fabs(num) > 9.0e15)
    throw SpecError(std::string("'") + what + "' must be an integer");
  return static_cast<int64_t>(num);
}

double Json::as_num(const char* what) const {
  if (kind != Number) throw SpecError(std::string("'") + what + "' must be a number");
  return num;
}

const std::string& Json::as_str(const char* what) const {
  if (kind != String) throw SpecError(std::string("'") + what + "' must be a string");
  return str;
}

bool Json::as_bool(const char* what) const {
  if (kind != Bool) throw SpecError(std::string("'") + what + "' must be true or false");
  return b;
}

}  // namespace dycl
