// Host-side driver for the sanitizer test: feeds serialized subgraphs to
// byoc_subgraph_validate (parser and schema checks) and byoc_subgraph_create
// (which plans the launch sequence on the host before it touches a device;
// on a host without a GPU it then returns BYOC_ERR_DEVICE).
//
// Usage: byoc_plan_driver LIST
// LIST holds one case per line: "<json path> <constants path>".  The
// constants file holds one constant per line, "<dtype 0|1> <ndim> <d0> ...",
// in the order of their JSON "index"; the driver fills them with
// deterministic pseudo-random values in [-1, 1).  For every case it prints
// "<json path> validate=<status> create=<status>".
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

#include "byoc.h"

namespace {

struct ConstBuf {
  int32_t dtype = 0;
  std::vector<int64_t> shape;
  std::vector<float> f32;
  std::vector<uint16_t> bf16;
};

bool read_file(const std::string& path, std::string* out) {
  std::ifstream f(path, std::ios::binary);
  if (!f) return false;
  std::ostringstream ss;
  ss << f.rdbuf();
  *out = ss.str();
  return true;
}

// xorshift32 -> [-1, 1)
float next_value(uint32_t* s) {
  uint32_t x = *s;
  x ^= x << 13;
  x ^= x >> 17;
  x ^= x << 5;
  *s = x;
  return (float)((double)x / 2147483648.0 - 1.0);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s LIST\n", argv[0]);
    return 2;
  }
  std::ifstream list(argv[1]);
  if (!list) {
    std::fprintf(stderr, "cannot open %s\n", argv[1]);
    return 2;
  }
  std::string line;
  int cases = 0;
  while (std::getline(list, line)) {
    std::istringstream ls(line);
    std::string jpath, cpath;
    if (!(ls >> jpath >> cpath)) continue;
    std::string json, cdesc;
    if (!read_file(jpath, &json) || !read_file(cpath, &cdesc)) {
      std::fprintf(stderr, "cannot read case %s\n", line.c_str());
      return 2;
    }
    std::vector<ConstBuf> bufs;
    std::istringstream cs(cdesc);
    std::string cl;
    uint32_t seed = 0x9e3779b9u;
    while (std::getline(cs, cl)) {
      std::istringstream ws(cl);
      ConstBuf b;
      int ndim = 0;
      if (!(ws >> b.dtype >> ndim)) continue;
      int64_t n = 1;
      for (int i = 0; i < ndim; ++i) {
        int64_t d = 0;
        ws >> d;
        b.shape.push_back(d);
        n *= d > 0 ? d : 0;
      }
      if (b.dtype == 1) {
        b.bf16.resize((size_t)n);
        for (auto& v : b.bf16) {
          const float f = next_value(&seed);
          uint32_t u;
          std::memcpy(&u, &f, 4);
          v = (uint16_t)(u >> 16);
        }
      } else {
        b.f32.resize((size_t)n);
        for (auto& v : b.f32) v = next_value(&seed);
      }
      bufs.push_back(std::move(b));
    }
    std::vector<byoc_const> consts(bufs.size());
    for (size_t i = 0; i < bufs.size(); ++i) {
      consts[i].data = bufs[i].dtype == 1 ? (const void*)bufs[i].bf16.data() : (const void*)bufs[i].f32.data();
      consts[i].dtype = bufs[i].dtype;
      consts[i].ndim = (int32_t)bufs[i].shape.size();
      consts[i].shape = bufs[i].shape.data();
    }
    const byoc_const* cp = consts.empty() ? nullptr : consts.data();
    const byoc_status v = byoc_subgraph_validate(json.data(), json.size(), cp, (int32_t)consts.size());
    std::string verr = byoc_last_error();
    byoc_subgraph* g = nullptr;
    const byoc_status c = byoc_subgraph_create(json.data(), json.size(), cp, (int32_t)consts.size(), 0, &g);
    std::string cerr = byoc_last_error();
    if (c == BYOC_OK) byoc_subgraph_destroy(g);
    if (c != BYOC_OK && g != nullptr) {
      std::fprintf(stderr, "%s: create failed but returned a handle\n", jpath.c_str());
      return 3;
    }
    std::printf("%s validate=%d create=%d | %s | %s\n", jpath.c_str(), (int)v, (int)c, verr.c_str(), cerr.c_str());
    ++cases;
  }
  std::printf("cases %d\n", cases);
  return 0;
}
