// Parsing and validation of the serialized subgraph.  Every error names the
// node (or input / constant) and the field at fault.
#include "graph.h"

#include <cmath>
#include <map>
#include <sstream>

#include "json.h"

namespace byoc {
namespace {

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

std::string shape_str(const std::vector<int64_t>& s) {
  std::ostringstream o;
  o << "[";
  for (size_t i = 0; i < s.size(); ++i) o << (i ? "," : "") << s[i];
  o << "]";
  return o.str();
}

int64_t numel(const std::vector<int64_t>& s) {
  int64_t n = 1;
  for (int64_t d : s) n *= d;
  return n;
}

Status perr(const std::string& m) { return Status::Err(BYOC_ERR_PARSE, m); }
Status serr(const std::string& m) { return Status::Err(BYOC_ERR_SHAPE, m); }
Status uerr(const std::string& m) { return Status::Err(BYOC_ERR_UNSUPPORTED, m); }

bool get_string(const JsonValue& o, const char* key, std::string* out) {
  const JsonValue* v = o.get(key);
  if (!v || v->kind != JsonValue::String) return false;
  *out = v->str;
  return true;
}

// Reads an array of integers; false if missing or malformed.
bool get_ints(const JsonValue* v, std::vector<int64_t>* out) {
  if (!v || v->kind != JsonValue::Array) return false;
  out->clear();
  for (const auto& e : v->arr) {
    if (e.kind != JsonValue::Number || !e.is_integer) return false;
    out->push_back(e.inum);
  }
  return true;
}

bool parse_dtype(const std::string& s, DType* d) {
  if (s == "f32" || s == "float32") {
    *d = DType::F32;
    return true;
  }
  if (s == "bf16" || s == "bfloat16") {
    *d = DType::BF16;
    return true;
  }
  return false;
}

// Optional "quant": {"scale": S > 0, "zero_point": Z in [-128, 127]}.
Status parse_quant(const JsonValue& d, const std::string& where, Value* v) {
  const JsonValue* q = d.get("quant");
  if (!q) return Status::Ok();
  if (q->kind != JsonValue::Object) return perr(where + ": quant must be an object");
  const JsonValue* sc = q->get("scale");
  const JsonValue* zp = q->get("zero_point");
  if (!sc || sc->kind != JsonValue::Number || !(sc->num > 0.0) || !std::isfinite(sc->num))
    return perr(where + ": quant.scale must be a positive finite number");
  if (!zp || zp->kind != JsonValue::Number || !zp->is_integer || zp->inum < -128 || zp->inum > 127)
    return perr(where + ": quant.zero_point must be an integer in [-128, 127]");
  v->has_q = true;
  v->qscale = sc->num;
  v->qzero = (int)zp->inum;
  return Status::Ok();
}

// Optional integer-pair attribute (e.g. strides) with a default.
Status attr_pair(const JsonValue* attrs, const char* key, const std::string& where, int lo,
                 int def0, int def1, int out[2]) {
  out[0] = def0;
  out[1] = def1;
  if (!attrs) return Status::Ok();
  const JsonValue* v = attrs->get(key);
  if (!v) return Status::Ok();
  std::vector<int64_t> xs;
  if (!get_ints(v, &xs) || xs.size() != 2)
    return perr(where + ": attrs." + key + " must be a list of 2 integers");
  for (int i = 0; i < 2; ++i) {
    if (xs[i] < lo || xs[i] > 4096)
      return perr(where + ": attrs." + key + " value " + std::to_string(xs[i]) + " out of range");
    out[i] = (int)xs[i];
  }
  return Status::Ok();
}

Status attr_padding(const JsonValue* attrs, const std::string& where, int out[4]) {
  for (int i = 0; i < 4; ++i) out[i] = 0;
  if (!attrs) return Status::Ok();
  const JsonValue* v = attrs->get("padding");
  if (!v) return Status::Ok();
  std::vector<int64_t> xs;
  if (!get_ints(v, &xs) || (xs.size() != 2 && xs.size() != 4))
    return perr(where + ": attrs.padding must be a list of 2 or 4 integers");
  if (xs.size() == 2) xs = {xs[0], xs[1], xs[0], xs[1]};
  for (int i = 0; i < 4; ++i) {
    if (xs[i] < 0 || xs[i] > 4096) return perr(where + ": attrs.padding value out of range");
    out[i] = (int)xs[i];
  }
  return Status::Ok();
}

struct CompositeName {
  OpKind op;
  bool bias = false, add = false;
  Act act = Act::None;
};

bool split_composite(const std::string& name, CompositeName* c) {
  if (name == "max_pool2d") {
    c->op = OpKind::MaxPool;
    return true;
  }
  if (name == "global_avg_pool2d") {
    c->op = OpKind::AvgPool;
    return true;
  }
  if (name == "avg_pool2d") {
    c->op = OpKind::AvgPoolWin;
    return true;
  }
  if (name == "concatenate") {
    c->op = OpKind::Concat;
    return true;
  }
  std::vector<std::string> parts;
  std::string cur;
  for (char ch : name) {
    if (ch == '_') {
      parts.push_back(cur);
      cur.clear();
    } else {
      cur += ch;
    }
  }
  parts.push_back(cur);
  size_t i = 0;
  if (parts[0] == "conv2d") c->op = OpKind::Conv;
  else if (parts[0] == "dense") c->op = OpKind::Dense;
  else if (parts[0] == "add") c->op = OpKind::Add;
  else return false;
  ++i;
  if (c->op == OpKind::Add) {
    c->add = true;
  } else {
    if (i < parts.size() && parts[i] == "bias") c->bias = true, ++i;
    if (i < parts.size() && parts[i] == "add") c->add = true, ++i;
  }
  if (i < parts.size()) {
    if (parts[i] == "relu") c->act = Act::Relu;
    else if (parts[i] == "relu6") c->act = Act::Relu6;
    else if (parts[i] == "gelu") c->act = Act::Gelu;
    else if (parts[i] == "leaky") c->act = Act::Leaky;
    else return false;
    ++i;
  }
  return i == parts.size();
}

}  // namespace

const char* act_name(Act a) {
  switch (a) {
    case Act::Relu: return "relu";
    case Act::Relu6: return "relu6";
    case Act::Gelu: return "gelu";
    case Act::Leaky: return "leaky";
    default: return "none";
  }
}

Status parse_graph(const char* text, size_t len, const byoc_const* consts, int32_t n_consts,
                   Graph* out) {
  if (!text) return Status::Err(BYOC_ERR_INVALID_ARG, "json is NULL");
  if (n_consts < 0 || (n_consts > 0 && !consts))
    return Status::Err(BYOC_ERR_INVALID_ARG, "constant array is NULL or n_consts < 0");
  JsonValue root;
  std::string jerr;
  if (!json_parse(text, len, &root, &jerr)) return perr(jerr);
  if (root.kind != JsonValue::Object) return perr("top level must be an object");
  std::string fmt;
  if (!get_string(root, "format", &fmt) || fmt != "byoc-subgraph")
    return perr("format must be \"byoc-subgraph\"");
  const JsonValue* ver = root.get("version");
  if (!ver || ver->kind != JsonValue::Number || !ver->is_integer || ver->inum != 1)
    return uerr("version must be 1");

  Graph g;
  std::map<std::string, int> by_name;
  auto add_value = [&](Value v) -> int {
    by_name[v.name] = (int)g.values.size();
    g.values.push_back(std::move(v));
    return (int)g.values.size() - 1;
  };

  // ---- inputs --------------------------------------------------------------
  const JsonValue* ins = root.get("inputs");
  if (!ins || ins->kind != JsonValue::Array || ins->arr.empty())
    return perr("inputs must be a non-empty list");
  for (size_t i = 0; i < ins->arr.size(); ++i) {
    const JsonValue& d = ins->arr[i];
    std::string where = "input " + std::to_string(i);
    if (d.kind != JsonValue::Object) return perr(where + ": must be an object");
    Value v;
    if (!get_string(d, "name", &v.name) || v.name.empty()) return perr(where + ": missing name");
    where += " (" + v.name + ")";
    if (by_name.count(v.name)) return perr(where + ": duplicate name");
    if (!get_ints(d.get("shape"), &v.shape)) return perr(where + ": shape must be integers");
    if (v.shape.size() != 2 && v.shape.size() != 4)
      return uerr(where + ": rank must be 2 or 4, got " + shape_str(v.shape));
    for (int64_t s : v.shape)
      if (s < 1) return serr(where + ": non-positive extent in " + shape_str(v.shape));
    if (numel(v.shape) > kMaxElems) return uerr(where + ": more than 2^31-1 elements");
    std::string dt;
    if (!get_string(d, "dtype", &dt) || !parse_dtype(dt, &v.dtype))
      return perr(where + ": dtype must be \"f32\" or \"bf16\"");
    IoDesc io;
    io.dtype = v.dtype;
    std::string lay;
    io.layout = v.shape.size() == 4 ? BYOC_NCHW : BYOC_ROWMAJOR;
    if (get_string(d, "layout", &lay)) {
      if ((v.shape.size() == 4 && lay != "NCHW") || (v.shape.size() == 2 && lay != "ROWMAJOR"))
        return uerr(where + ": layout " + lay + " not supported for rank " +
                    std::to_string(v.shape.size()));
    }
    Status qs = parse_quant(d, where, &v);
    if (!qs.ok()) return qs;
    v.source = Value::Input;
    v.index = (int)i;
    io.value = add_value(v);
    g.inputs.push_back(io);
  }

  // ---- constants -----------------------------------------------------------
  g.const_values.assign(n_consts, -1);
  const JsonValue* cs = root.get("constants");
  if (cs && cs->kind != JsonValue::Array) return perr("constants must be a list");
  if (cs) {
    for (size_t i = 0; i < cs->arr.size(); ++i) {
      const JsonValue& d = cs->arr[i];
      std::string where = "constant " + std::to_string(i);
      if (d.kind != JsonValue::Object) return perr(where + ": must be an object");
      Value v;
      if (!get_string(d, "name", &v.name) || v.name.empty()) return perr(where + ": missing name");
      where += " (" + v.name + ")";
      if (by_name.count(v.name)) return perr(where + ": duplicate name");
      const JsonValue* ix = d.get("index");
      if (!ix || ix->kind != JsonValue::Number || !ix->is_integer)
        return perr(where + ": index must be an integer");
      if (ix->inum < 0 || ix->inum >= n_consts)
        return Status::Err(BYOC_ERR_INVALID_ARG, where + ": index " + std::to_string(ix->inum) +
                                                     " outside the " + std::to_string(n_consts) +
                                                     " constants passed");
      int ci = (int)ix->inum;
      if (g.const_values[ci] >= 0) return perr(where + ": index used twice");
      if (!get_ints(d.get("shape"), &v.shape) || v.shape.empty() || v.shape.size() > 8)
        return perr(where + ": shape must be 1 to 8 integers");
      for (int64_t s : v.shape)
        if (s < 1) return serr(where + ": non-positive extent in " + shape_str(v.shape));
      if (numel(v.shape) > kMaxElems) return uerr(where + ": more than 2^31-1 elements");
      std::string dt;
      if (!get_string(d, "dtype", &dt) || !parse_dtype(dt, &v.dtype))
        return perr(where + ": dtype must be \"f32\" or \"bf16\"");
      const byoc_const& c = consts[ci];
      if (!c.data) return Status::Err(BYOC_ERR_INVALID_ARG, where + ": data pointer is NULL");
      if (c.dtype != (int32_t)v.dtype)
        return serr(where + ": passed dtype differs from the declared " + dt);
      std::vector<int64_t> given;
      if (c.ndim < 1 || c.ndim > 8 || !c.shape)
        return Status::Err(BYOC_ERR_INVALID_ARG, where + ": passed ndim/shape invalid");
      for (int k = 0; k < c.ndim; ++k) given.push_back(c.shape[k]);
      if (given != v.shape)
        return serr(where + ": passed shape " + shape_str(given) + " != declared " +
                    shape_str(v.shape));
      v.source = Value::Const;
      v.index = ci;
      g.const_values[ci] = add_value(v);
    }
  }

  // ---- nodes ---------------------------------------------------------------
  const JsonValue* ns = root.get("nodes");
  if (!ns || ns->kind != JsonValue::Array || ns->arr.empty())
    return perr("nodes must be a non-empty list");
  for (size_t ni = 0; ni < ns->arr.size(); ++ni) {
    const JsonValue& d = ns->arr[ni];
    std::string where = "node " + std::to_string(ni);
    if (d.kind != JsonValue::Object) return perr(where + ": must be an object");
    Node n;
    if (!get_string(d, "name", &n.name) || n.name.empty()) return perr(where + ": missing name");
    if (!get_string(d, "composite", &n.composite)) return perr(where + ": missing composite");
    where += " (" + n.composite + ")";
    if (by_name.count(n.name)) return perr(where + ": duplicate name " + n.name);
    CompositeName cn;
    if (!split_composite(n.composite, &cn)) return uerr(where + ": unknown composite");
    n.op = cn.op;
    n.has_bias = cn.bias;
    n.has_add = cn.add;
    n.act = cn.act;
    std::string odt;
    DType out_dtype;
    if (get_string(d, "out_dtype", &odt) && (odt == "int8" || odt == "i8")) out_dtype = DType::I8;
    else if (odt.empty() || !parse_dtype(odt, &out_dtype))
      return perr(where + ": out_dtype must be \"f32\", \"bf16\" or \"int8\"");
    if (ni == 0) g.compute = out_dtype;
    else if (out_dtype != g.compute)
      return uerr(where + ": mixed out_dtype in one graph (graph computes in " +
                  std::string(g.compute == DType::BF16 ? "bf16" : (g.compute == DType::I8 ? "int8" : "f32")) + ")");
    const JsonValue* refs = d.get("inputs");
    if (!refs || refs->kind != JsonValue::Array) return perr(where + ": inputs must be a list");
    std::vector<int> args;
    for (size_t k = 0; k < refs->arr.size(); ++k) {
      if (refs->arr[k].kind != JsonValue::String) return perr(where + ": input refs must be strings");
      auto it = by_name.find(refs->arr[k].str);
      if (it == by_name.end())
        return perr(where + ": input " + std::to_string(k) + " refers to unknown or later value '" +
                    refs->arr[k].str + "'");
      args.push_back(it->second);
    }
    const JsonValue* attrs = d.get("attrs");
    if (attrs && attrs->kind != JsonValue::Object) return perr(where + ": attrs must be an object");
    auto is_const = [&](int v) { return g.values[v].source == Value::Const; };
    auto shp = [&](int v) -> const std::vector<int64_t>& { return g.values[v].shape; };
    std::vector<int64_t> oshape;

    size_t want = 0;
    switch (n.op) {
      case OpKind::Conv:
      case OpKind::Dense: want = 2 + (n.has_bias ? 1 : 0) + (n.has_add ? 1 : 0); break;
      case OpKind::MaxPool:
      case OpKind::AvgPool:
      case OpKind::AvgPoolWin: want = 1; break;
      case OpKind::Add: want = 2; break;
      case OpKind::Concat: want = args.empty() ? 1 : args.size(); break;  // one or more
    }
    if (args.size() != want)
      return perr(where + ": expects " + std::to_string(want) + " inputs, got " +
                  std::to_string(args.size()));
    for (size_t k = 0; k < args.size(); ++k) {
      bool weight_slot = (n.op == OpKind::Conv || n.op == OpKind::Dense) &&
                         (k == 1 || (k == 2 && n.has_bias));
      if (weight_slot && !is_const(args[k]))
        return uerr(where + ": input " + std::to_string(k) + " must be a constant");
      if (!weight_slot && is_const(args[k]))
        return uerr(where + ": input " + std::to_string(k) + " must be an activation, got constant '" +
                    g.values[args[k]].name + "'");
    }
    n.data = args[0];
    if (n.op == OpKind::Conv || n.op == OpKind::Dense) {
      n.weight = args[1];
      size_t k = 2;
      if (n.has_bias) n.bias = args[k++];
      if (n.has_add) n.residual = args[k++];
    } else if (n.op == OpKind::Add) {
      n.other = args[1];
    } else if (n.op == OpKind::Concat) {
      n.cat = args;
    }
    const auto& xs = shp(n.data);
    if (n.act == Act::Leaky && attrs && attrs->get("alpha")) {
      const JsonValue* av = attrs->get("alpha");
      if (av->kind != JsonValue::Number || !(av->num >= 0.0 && av->num < 1.0))
        return perr(where + ": attrs.alpha must be a number in [0, 1)");
      n.alpha = (float)av->num;
    }

    if (n.op == OpKind::Conv) {
      if (xs.size() != 4) return serr(where + ": data must be 4-D NCHW, got " + shape_str(xs));
      const auto& ws = shp(n.weight);
      if (ws.size() != 4) return serr(where + ": weight must be 4-D OIHW, got " + shape_str(ws));
      Status st = attr_pair(attrs, "strides", where, 1, 1, 1, n.stride);
      if (!st.ok()) return st;
      st = attr_padding(attrs, where, n.pad);
      if (!st.ok()) return st;
      int dil[2];
      st = attr_pair(attrs, "dilation", where, 1, 1, 1, dil);
      if (!st.ok()) return st;
      if (dil[0] != 1 || dil[1] != 1) return uerr(where + ": dilation other than 1");
      n.groups = 1;
      if (attrs && attrs->get("groups")) {
        const JsonValue* gv = attrs->get("groups");
        if (gv->kind != JsonValue::Number || !gv->is_integer || gv->inum < 1)
          return perr(where + ": attrs.groups must be a positive integer");
        n.groups = (int)gv->inum;
      }
      int64_t C = xs[1], K = ws[0];
      if (C % n.groups || K % n.groups || ws[1] != C / n.groups)
        return serr(where + ": weight " + shape_str(ws) + " does not match data channels " +
                    std::to_string(C) + " with groups " + std::to_string(n.groups));
      if (n.groups != 1) {
        if (n.groups == C && K == C) n.depthwise = true;
        else return uerr(where + ": grouped conv other than depthwise (groups == C == K)");
      }
      if (ws[2] > 15 || ws[3] > 15) return uerr(where + ": kernel larger than 15x15");
      int64_t H = xs[2], W = xs[3], R = ws[2], S = ws[3];
      if (H + n.pad[0] + n.pad[2] < R || W + n.pad[1] + n.pad[3] < S)
        return serr(where + ": kernel larger than the padded input");
      int64_t P = (H + n.pad[0] + n.pad[2] - R) / n.stride[0] + 1;
      int64_t Q = (W + n.pad[1] + n.pad[3] - S) / n.stride[1] + 1;
      oshape = {xs[0], K, P, Q};
      if (n.has_bias && shp(n.bias) != std::vector<int64_t>{K})
        return serr(where + ": bias shape " + shape_str(shp(n.bias)) + " != [" + std::to_string(K) + "]");
      n.macs = xs[0] * K * P * Q * (C / n.groups) * R * S;
    } else if (n.op == OpKind::Dense) {
      if (xs.size() != 2) return serr(where + ": data must be 2-D [M,K], got " + shape_str(xs));
      const auto& ws = shp(n.weight);
      if (ws.size() != 2 || ws[1] != xs[1])
        return serr(where + ": weight " + shape_str(ws) + " does not match data " + shape_str(xs));
      oshape = {xs[0], ws[0]};
      if (n.has_bias && shp(n.bias) != std::vector<int64_t>{ws[0]})
        return serr(where + ": bias shape " + shape_str(shp(n.bias)) + " != [" +
                    std::to_string(ws[0]) + "]");
      n.macs = xs[0] * ws[0] * xs[1];
    } else if (n.op == OpKind::MaxPool) {
      if (xs.size() != 4) return serr(where + ": data must be 4-D NCHW, got " + shape_str(xs));
      if (!attrs || !attrs->get("pool_size")) return perr(where + ": attrs.pool_size missing");
      Status st = attr_pair(attrs, "pool_size", where, 1, 1, 1, n.pool);
      if (!st.ok()) return st;
      st = attr_pair(attrs, "strides", where, 1, n.pool[0], n.pool[1], n.stride);
      if (!st.ok()) return st;
      st = attr_padding(attrs, where, n.pad);
      if (!st.ok()) return st;
      if (n.pad[0] >= n.pool[0] || n.pad[2] >= n.pool[0] || n.pad[1] >= n.pool[1] ||
          n.pad[3] >= n.pool[1])
        return uerr(where + ": padding must be smaller than the pool window");
      int64_t H = xs[2], W = xs[3];
      if (H + n.pad[0] + n.pad[2] < n.pool[0] || W + n.pad[1] + n.pad[3] < n.pool[1])
        return serr(where + ": window larger than the padded input");
      int64_t P = (H + n.pad[0] + n.pad[2] - n.pool[0]) / n.stride[0] + 1;
      int64_t Q = (W + n.pad[1] + n.pad[3] - n.pool[1]) / n.stride[1] + 1;
      oshape = {xs[0], xs[1], P, Q};
    } else if (n.op == OpKind::AvgPool) {
      if (xs.size() != 4) return serr(where + ": data must be 4-D NCHW, got " + shape_str(xs));
      oshape = {xs[0], xs[1]};
    } else if (n.op == OpKind::AvgPoolWin) {
      if (xs.size() != 4) return serr(where + ": data must be 4-D NCHW, got " + shape_str(xs));
      if (!attrs || !attrs->get("pool_size")) return perr(where + ": attrs.pool_size missing");
      Status st = attr_pair(attrs, "pool_size", where, 1, 1, 1, n.pool);
      if (!st.ok()) return st;
      st = attr_pair(attrs, "strides", where, 1, 1, 1, n.stride);
      if (!st.ok()) return st;
      st = attr_padding(attrs, where, n.pad);
      if (!st.ok()) return st;
      if (n.pad[0] >= n.pool[0] || n.pad[2] >= n.pool[0] || n.pad[1] >= n.pool[1] || n.pad[3] >= n.pool[1])
        return uerr(where + ": padding must be smaller than the pool window");
      if (const JsonValue* ci = attrs->get("count_include_pad")) {
        if (ci->kind != JsonValue::Bool) return perr(where + ": attrs.count_include_pad must be a boolean");
        n.count_include_pad = ci->b;
      }
      int64_t H = xs[2], W = xs[3];
      if (H + n.pad[0] + n.pad[2] < n.pool[0] || W + n.pad[1] + n.pad[3] < n.pool[1])
        return serr(where + ": window larger than the padded input");
      oshape = {xs[0], xs[1], (H + n.pad[0] + n.pad[2] - n.pool[0]) / n.stride[0] + 1,
                (W + n.pad[1] + n.pad[3] - n.pool[1]) / n.stride[1] + 1};
    } else if (n.op == OpKind::Concat) {
      if (attrs && attrs->get("axis")) {
        const JsonValue* ax = attrs->get("axis");
        if (ax->kind != JsonValue::Number || !ax->is_integer || ax->inum != 1)
          return uerr(where + ": concatenation along an axis other than 1 (channels)");
      }
      int64_t ctot = 0;
      for (int a : n.cat) {
        const auto& s = shp(a);
        if (s.size() != 4 || s[0] != xs[0] || s[2] != xs[2] || s[3] != xs[3])
          return serr(where + ": input '" + g.values[a].name + "' " + shape_str(s) +
                      " does not match the batch and image of " + shape_str(xs));
        ctot += s[1];
      }
      oshape = {xs[0], ctot, xs[2], xs[3]};
    } else {
      if (shp(n.other) != xs)
        return serr(where + ": operand shapes " + shape_str(xs) + " and " + shape_str(shp(n.other)) +
                    " differ");
      oshape = xs;
    }
    if ((n.op == OpKind::MaxPool || n.op == OpKind::AvgPool || n.op == OpKind::AvgPoolWin ||
         n.op == OpKind::Concat) && n.act != Act::None)
      return uerr(where + ": activation on a pool or a concatenation");
    if ((n.op == OpKind::AvgPoolWin || n.op == OpKind::Concat) && out_dtype != DType::BF16)
      return uerr(where + ": " + n.composite + " only in bf16 graphs");
    if (n.op == OpKind::Concat)
      for (int a : n.cat)
        if (shp(a)[1] % 8 != 0)
          return uerr(where + ": input '" + g.values[a].name + "' has " + std::to_string(shp(a)[1]) +
                      " channels (concatenated inputs need a multiple of 8)");
    if (n.residual >= 0 && shp(n.residual) != oshape)
      return serr(where + ": residual shape " + shape_str(shp(n.residual)) + " != output shape " +
                  shape_str(oshape));
    if (numel(oshape) > kMaxElems) return uerr(where + ": output has more than 2^31-1 elements");
    Value ov;
    ov.name = n.name;
    ov.shape = oshape;
    ov.dtype = out_dtype;
    ov.source = Value::Node;
    ov.index = (int)ni;
    Status qs = parse_quant(d, where, &ov);
    if (!qs.ok()) return qs;
    if (out_dtype == DType::I8) {
      // the int8 forms: every tensor quantized, no GELU; a max
      // pool keeps its input's codes (and inherits them when none are given)
      for (int a : {n.data, n.residual, n.other}) {
        if (a < 0 || g.values[a].has_q) continue;
        return serr(where + ": int8 operand '" + g.values[a].name + "' has no quant parameters");
      }
      if (n.act == Act::Gelu)
        return uerr(where + ": " + act_name(n.act) + " has no int8 form");
      if (n.op == OpKind::MaxPool) {
        const Value& xv = g.values[n.data];
        if (ov.has_q && (ov.qscale != xv.qscale || ov.qzero != xv.qzero))
          return serr(where + ": an int8 max pool keeps its input's scale and zero point");
        ov.has_q = true;
        ov.qscale = xv.qscale;
        ov.qzero = xv.qzero;
      }
      if (!ov.has_q) return perr(where + ": int8 node needs quant {scale, zero_point}");
    } else if (ov.has_q) {
      return uerr(where + ": quant parameters only in int8 graphs");
    }
    n.out = add_value(ov);
    g.macs += n.macs;
    g.nodes.push_back(n);
  }

  for (const IoDesc& in : g.inputs) {
    const Value& v = g.values[in.value];
    if (g.compute != DType::I8 && v.has_q)
      return uerr("input " + v.name + ": quant parameters only in int8 graphs");
  }

  // ---- outputs -------------------------------------------------------------
  const JsonValue* os = root.get("outputs");
  if (!os || os->kind != JsonValue::Array || os->arr.empty())
    return perr("outputs must be a non-empty list");
  for (size_t i = 0; i < os->arr.size(); ++i) {
    const JsonValue& d = os->arr[i];
    std::string where = "output " + std::to_string(i);
    if (d.kind != JsonValue::Object) return perr(where + ": must be an object");
    std::string name;
    if (!get_string(d, "name", &name)) return perr(where + ": missing name");
    auto it = by_name.find(name);
    if (it == by_name.end()) return perr(where + ": unknown value '" + name + "'");
    if (g.values[it->second].source == Value::Const)
      return uerr(where + ": a constant cannot be a subgraph output");
    IoDesc io;
    io.value = it->second;
    const auto& s = g.values[io.value].shape;
    std::string dt;
    io.dtype = g.values[io.value].dtype == DType::I8 ? DType::F32 : g.values[io.value].dtype;
    if (get_string(d, "dtype", &dt) && !parse_dtype(dt, &io.dtype))
      return perr(where + ": dtype must be \"f32\" or \"bf16\"");
    io.layout = s.size() == 4 ? BYOC_NCHW : BYOC_ROWMAJOR;
    std::string lay;
    if (get_string(d, "layout", &lay)) {
      if ((s.size() == 4 && lay != "NCHW") || (s.size() == 2 && lay != "ROWMAJOR"))
        return uerr(where + ": layout " + lay + " not supported for rank " + std::to_string(s.size()));
    }
    g.outputs.push_back(io);
  }
  *out = std::move(g);
  return Status::Ok();
}

}  // namespace byoc
