// Minimal JSON reader for the serialized subgraph (objects, arrays, strings,
// numbers, booleans, null).  Errors carry the byte offset.
#pragma once

#include <cstddef>
#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <vector>

namespace byoc {

struct JsonValue {
  enum Kind { Null, Bool, Number, String, Array, Object } kind = Null;
  bool b = false;
  double num = 0.0;
  bool is_integer = false;  // the literal had no fraction or exponent
  int64_t inum = 0;
  std::string str;
  std::vector<JsonValue> arr;
  std::vector<std::pair<std::string, JsonValue>> obj;  // keeps document order

  const JsonValue* get(const std::string& key) const {
    for (const auto& kv : obj)
      if (kv.first == key) return &kv.second;
    return nullptr;
  }
};

// Parses text[0:len).  On error returns false and fills err.
bool json_parse(const char* text, size_t len, JsonValue* out, std::string* err);

}  // namespace byoc
