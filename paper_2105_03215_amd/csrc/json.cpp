#include "json.h"

#include <cerrno>
#include <cstdlib>
#include <cstring>

namespace byoc {
namespace {

struct Reader {
  const char* p;
  const char* end;
  const char* begin;
  std::string err;
  int depth = 0;

  bool fail(const char* msg) {
    if (err.empty()) err = std::string("JSON: ") + msg + " at byte " + std::to_string(p - begin);
    return false;
  }
  void ws() {
    while (p < end && (*p == ' ' || *p == '\t' || *p == '\n' || *p == '\r')) ++p;
  }
  bool lit(const char* s) {
    size_t n = std::strlen(s);
    if ((size_t)(end - p) < n || std::memcmp(p, s, n) != 0) return false;
    p += n;
    return true;
  }
  static void put_utf8(std::string& o, unsigned cp) {
    if (cp < 0x80) {
      o += (char)cp;
    } else if (cp < 0x800) {
      o += (char)(0xC0 | (cp >> 6));
      o += (char)(0x80 | (cp & 0x3F));
    } else if (cp < 0x10000) {
      o += (char)(0xE0 | (cp >> 12));
      o += (char)(0x80 | ((cp >> 6) & 0x3F));
      o += (char)(0x80 | (cp & 0x3F));
    } else {
      o += (char)(0xF0 | (cp >> 18));
      o += (char)(0x80 | ((cp >> 12) & 0x3F));
      o += (char)(0x80 | ((cp >> 6) & 0x3F));
      o += (char)(0x80 | (cp & 0x3F));
    }
  }
  bool hex4(unsigned* v) {
    if (end - p < 4) return fail("truncated \\u escape");
    unsigned x = 0;
    for (int i = 0; i < 4; ++i) {
      char c = *p++;
      x <<= 4;
      if (c >= '0' && c <= '9') x |= c - '0';
      else if (c >= 'a' && c <= 'f') x |= c - 'a' + 10;
      else if (c >= 'A' && c <= 'F') x |= c - 'A' + 10;
      else return fail("bad \\u escape");
    }
    *v = x;
    return true;
  }
  bool string(std::string* o) {
    if (p >= end || *p != '"') return fail("expected string");
    ++p;
    while (p < end && *p != '"') {
      char c = *p++;
      if ((unsigned char)c < 0x20) return fail("control character in string");
      if (c != '\\') {
        *o += c;
        continue;
      }
      if (p >= end) return fail("truncated escape");
      char e = *p++;
      switch (e) {
        case '"': *o += '"'; break;
        case '\\': *o += '\\'; break;
        case '/': *o += '/'; break;
        case 'b': *o += '\b'; break;
        case 'f': *o += '\f'; break;
        case 'n': *o += '\n'; break;
        case 'r': *o += '\r'; break;
        case 't': *o += '\t'; break;
        case 'u': {
          unsigned cp;
          if (!hex4(&cp)) return false;
          if (cp >= 0xD800 && cp < 0xDC00) {
            unsigned lo;
            if (!lit("\\u") || !hex4(&lo) || lo < 0xDC00 || lo >= 0xE000)
              return fail("bad surrogate pair");
            cp = 0x10000 + ((cp - 0xD800) << 10) + (lo - 0xDC00);
          }
          put_utf8(*o, cp);
          break;
        }
        default: return fail("bad escape");
      }
    }
    if (p >= end) return fail("unterminated string");
    ++p;
    return true;
  }
  bool number(JsonValue* v) {
    const char* s = p;
    bool integer = true;
    if (p < end && *p == '-') ++p;
    if (p >= end || !(*p >= '0' && *p <= '9')) return fail("bad number");
    if (*p == '0') {
      ++p;
    } else {
      while (p < end && *p >= '0' && *p <= '9') ++p;
    }
    if (p < end && *p == '.') {
      integer = false;
      ++p;
      if (p >= end || !(*p >= '0' && *p <= '9')) return fail("bad fraction");
      while (p < end && *p >= '0' && *p <= '9') ++p;
    }
    if (p < end && (*p == 'e' || *p == 'E')) {
      integer = false;
      ++p;
      if (p < end && (*p == '+' || *p == '-')) ++p;
      if (p >= end || !(*p >= '0' && *p <= '9')) return fail("bad exponent");
      while (p < end && *p >= '0' && *p <= '9') ++p;
    }
    std::string tok(s, p - s);
    v->kind = JsonValue::Number;
    v->num = std::strtod(tok.c_str(), nullptr);
    v->is_integer = false;
    if (integer) {
      errno = 0;
      long long x = std::strtoll(tok.c_str(), nullptr, 10);
      if (errno == 0) {
        v->is_integer = true;
        v->inum = x;
      }
    }
    return true;
  }
  bool value(JsonValue* v) {
    if (++depth > 64) return fail("nesting too deep");
    ws();
    if (p >= end) return fail("unexpected end");
    bool ok = true;
    char c = *p;
    if (c == '{') {
      ++p;
      v->kind = JsonValue::Object;
      ws();
      if (p < end && *p == '}') {
        ++p;
      } else {
        for (;;) {
          ws();
          std::string key;
          if (!string(&key)) { ok = false; break; }
          ws();
          if (p >= end || *p != ':') { ok = fail("expected ':'"); break; }
          ++p;
          JsonValue child;
          if (!value(&child)) { ok = false; break; }
          v->obj.emplace_back(std::move(key), std::move(child));
          ws();
          if (p < end && *p == ',') { ++p; continue; }
          if (p < end && *p == '}') { ++p; break; }
          ok = fail("expected ',' or '}'");
          break;
        }
      }
    } else if (c == '[') {
      ++p;
      v->kind = JsonValue::Array;
      ws();
      if (p < end && *p == ']') {
        ++p;
      } else {
        for (;;) {
          JsonValue child;
          if (!value(&child)) { ok = false; break; }
          v->arr.push_back(std::move(child));
          ws();
          if (p < end && *p == ',') { ++p; continue; }
          if (p < end && *p == ']') { ++p; break; }
          ok = fail("expected ',' or ']'");
          break;
        }
      }
    } else if (c == '"') {
      v->kind = JsonValue::String;
      ok = string(&v->str);
    } else if (c == 't') {
      ok = lit("true") ? (v->kind = JsonValue::Bool, v->b = true, true) : fail("bad literal");
    } else if (c == 'f') {
      ok = lit("false") ? (v->kind = JsonValue::Bool, v->b = false, true) : fail("bad literal");
    } else if (c == 'n') {
      ok = lit("null") ? (v->kind = JsonValue::Null, true) : fail("bad literal");
    } else {
      ok = number(v);
    }
    --depth;
    return ok;
  }
};

}  // namespace

bool json_parse(const char* text, size_t len, JsonValue* out, std::string* err) {
  Reader r{text, text + len, text, std::string()};
  JsonValue v;
  if (!r.value(&v)) {
    *err = r.err;
    return false;
  }
  r.ws();
  if (r.p != r.end) {
    r.fail("trailing characters");
    *err = r.err;
    return false;
  }
  *out = std::move(v);
  return true;
}

}  // namespace byoc
