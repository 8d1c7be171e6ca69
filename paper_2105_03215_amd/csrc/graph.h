// Subgraph IR: the parsed and validated form of a serialized composite-op
// list (the JSON graph representation of Sec. 3.3, Option 1).  Host only;
// nothing here touches the device.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/byoc.h"

namespace byoc {

struct Status {
  byoc_status code = BYOC_OK;
  std::string msg;
  bool ok() const { return code == BYOC_OK; }
  static Status Ok() { return Status(); }
  static Status Err(byoc_status c, std::string m) {
    Status s;
    s.code = c;
    s.msg = std::move(m);
    return s;
  }
};

// I8: the compute type of a partially quantized graph (int8 codes with an
// affine scale and zero point per tensor); never an external dtype.
enum class DType { F32 = BYOC_F32, BF16 = BYOC_BF16, I8 = 2 };
enum class Act { None = 0, Relu = 1, Relu6 = 2, Gelu = 3, Leaky = 4 };
// AvgPool: global average pool; AvgPoolWin: windowed average pool.
enum class OpKind { Conv, Dense, MaxPool, AvgPool, Add, AvgPoolWin, Concat };

// A named tensor of the graph: a subgraph input, a constant or a node output.
struct Value {
  std::string name;
  std::vector<int64_t> shape;  // external layout: NCHW or [M, K]
  DType dtype = DType::F32;
  enum Source { Input, Const, Node } source = Input;
  int index = -1;  // input number, constant index or node number
  // int8 graphs: affine codes of this tensor, value = qscale * (code - qzero)
  bool has_q = false;
  double qscale = 0.0;
  int qzero = 0;
};

struct Node {
  std::string name;
  std::string composite;
  OpKind op = OpKind::Conv;
  bool has_bias = false;
  bool has_add = false;
  Act act = Act::None;
  float alpha = 0.1f;  // leaky ReLU slope (attrs.alpha)
  int data = -1, weight = -1, bias = -1, residual = -1, other = -1;  // value ids
  int out = -1;                                                      // value id
  int stride[2] = {1, 1};
  int pad[4] = {0, 0, 0, 0};  // top, left, bottom, right
  int pool[2] = {1, 1};
  int groups = 1;
  bool depthwise = false;
  bool count_include_pad = false;  // AvgPoolWin
  std::vector<int> cat;            // Concat: the joined values, in channel order
  int64_t macs = 0;
};

struct IoDesc {
  int value = -1;
  DType dtype = DType::F32;
  byoc_layout layout = BYOC_NCHW;
};

struct Graph {
  std::vector<Value> values;
  std::vector<Node> nodes;
  std::vector<IoDesc> inputs;
  std::vector<IoDesc> outputs;
  std::vector<int> const_values;  // value id of constant index i
  DType compute = DType::BF16;
  int64_t macs = 0;
};

// Parses and validates text against the constants.  consts may be NULL when
// n_consts is 0.  Pure host code.
Status parse_graph(const char* json, size_t len, const byoc_const* consts, int32_t n_consts,
                   Graph* out);

const char* act_name(Act a);

}  // namespace byoc
