// Cost table <-> JSON (the profiling data T(r) and adapt times of Sec. IV-A).
// Persisting the table lets a net be re-selected without profiling again.
#include <cctype>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <sstream>

#include "core.hpp"

namespace sn {

std::string costs_to_json(const Graph& g) {
  std::ostringstream o;
  o << "{\"dtype\":" << g.dtype << ",\"layers\":[";
  for (int i = 0; i < g.n_layers(); ++i) {
    const Layer& L = g.layers[i];
    if (i) o << ",";
    o << "{\"id\":" << i << ",\"type\":" << L.type << ",\"routines\":[";
    for (size_t r = 0; r < L.routines.size(); ++r) {
      const Routine& R = L.routines[r];
      if (r) o << ",";
      o << "{\"rid\":" << R.id << ",\"layout\":" << R.layout << ",\"algo\":" << R.algo
        << ",\"param\":" << R.param << ",\"dtype\":" << R.dtype << ",\"schema\":" << R.schema()
        << ",\"ns\":" << L.cost[r] << ",\"name\":\"" << R.name << "\"";
      const ChildNet& c = L.child[r];
      if (!c.empty()) {  // a childnet: its sub-layers, sub-routines, their times and its path
        o << ",\"child\":{\"layers\":[";
        for (size_t s = 0; s < c.layer.size(); ++s) o << (s ? "," : "") << "\"" << c.layer[s] << "\"";
        o << "],\"routines\":[";
        for (size_t s = 0; s < c.routine.size(); ++s) {
          o << (s ? "," : "") << "[";
          for (size_t q = 0; q < c.routine[s].size(); ++q) o << (q ? "," : "") << "\"" << c.routine[s][q] << "\"";
          o << "]";
        }
        o << "],\"ns\":[";
        for (size_t s = 0; s < c.cost.size(); ++s) {
          o << (s ? "," : "") << "[";
          for (size_t q = 0; q < c.cost[s].size(); ++q) o << (q ? "," : "") << c.cost[s][q];
          o << "]";
        }
        o << "],\"path\":[";
        for (size_t s = 0; s < c.path.size(); ++s) o << (s ? "," : "") << c.path[s];
        o << "]}";
      }
      o << "}";
    }
    o << "]}";
  }
  o << ",{\"id\":" << g.n_layers() << ",\"type\":" << SN_LAYER_OUTPUT
    << ",\"routines\":[{\"rid\":0,\"layout\":0,\"algo\":0,\"param\":0,\"dtype\":" << g.dtype
    << ",\"schema\":" << schema_of(g.dtype, SN_NCHW) << ",\"ns\":0,\"name\":\"output/nchw\"}]}";
  o << "],\"edges\":[";
  auto E = all_edges(g);
  for (size_t k = 0; k < E.size(); ++k) {
    if (k) o << ",";
    // one dtype: the 3 x 3 layout matrix of the run dtype; else 9 x 9 by schema
    o << "{\"from\":" << E[k].from << ",\"to\":" << E[k].to << ",\"ns\":[";
    const int S = g.multi_dtype() ? kNumSchemas : SN_NUM_LAYOUTS;
    const int base = g.multi_dtype() ? 0 : schema_of(g.dtype, 0);
    for (int a = 0; a < S; ++a) {
      if (a) o << ",";
      o << "[";
      for (int b = 0; b < S; ++b) {
        if (b) o << ",";
        o << (a == b ? 0 : E[k].adapt[base + a][base + b]);
      }
      o << "]";
    }
    o << "]}";
  }
  o << "]}";
  return o.str();
}

namespace {

// Minimal JSON reader: objects, arrays, integers/numbers, strings, literals.
struct JVal {
  enum Kind { NUL, NUM, STR, ARR, OBJ, BOOL } kind = NUL;
  double num = 0;
  long long inum = 0;
  bool is_int = false;
  std::string str;
  std::vector<JVal> arr;
  std::map<std::string, JVal> obj;
  const JVal& at(const std::string& k) const {
    auto it = obj.find(k);
    if (kind != OBJ || it == obj.end()) fail(SN_E_INVALID, "JSON: missing key '" + k + "'");
    return it->second;
  }
  long long as_int() const {
    if (kind != NUM || !is_int) fail(SN_E_INVALID, "JSON: integer expected");
    return inum;
  }
  const std::vector<JVal>& as_arr() const {
    if (kind != ARR) fail(SN_E_INVALID, "JSON: array expected");
    return arr;
  }
};

struct Parser {
  const char* p;
  int depth = 0;
  void ws() {
    while (*p && std::isspace((unsigned char)*p)) ++p;
  }
  [[noreturn]] void bad(const char* what) { fail(SN_E_INVALID, std::string("JSON: ") + what); }
  JVal value() {
    if (++depth > 64) bad("nesting too deep");
    ws();
    JVal v;
    if (*p == '{') {
      v.kind = JVal::OBJ;
      ++p;
      ws();
      if (*p == '}') {
        ++p;
      } else {
        for (;;) {
          ws();
          if (*p != '"') bad("key expected");
          std::string k = string();
          ws();
          if (*p != ':') bad("':' expected");
          ++p;
          v.obj[k] = value();
          ws();
          if (*p == ',') {
            ++p;
            continue;
          }
          if (*p == '}') {
            ++p;
            break;
          }
          bad("',' or '}' expected");
        }
      }
    } else if (*p == '[') {
      v.kind = JVal::ARR;
      ++p;
      ws();
      if (*p == ']') {
        ++p;
      } else {
        for (;;) {
          v.arr.push_back(value());
          ws();
          if (*p == ',') {
            ++p;
            continue;
          }
          if (*p == ']') {
            ++p;
            break;
          }
          bad("',' or ']' expected");
        }
      }
    } else if (*p == '"') {
      v.kind = JVal::STR;
      v.str = string();
    } else if (*p == '-' || std::isdigit((unsigned char)*p)) {
      v.kind = JVal::NUM;
      const char* s = p;
      char* e = nullptr;
      v.inum = std::strtoll(s, &e, 10);
      v.is_int = true;
      if (*e == '.' || *e == 'e' || *e == 'E') {
        v.num = std::strtod(s, &e);
        v.is_int = false;
      } else {
        v.num = (double)v.inum;
      }
      if (e == s) bad("bad number");
      p = e;
    } else if (!std::strncmp(p, "true", 4) || !std::strncmp(p, "false", 5)) {
      v.kind = JVal::BOOL;
      v.num = *p == 't';
      p += *p == 't' ? 4 : 5;
    } else if (!std::strncmp(p, "null", 4)) {
      p += 4;
    } else {
      bad("unexpected character");
    }
    --depth;
    return v;
  }
  std::string string() {
    std::string s;
    ++p;  // opening quote
    while (*p && *p != '"') {
      if (*p == '\\') {
        ++p;
        if (!*p) bad("bad escape");
      }
      s += *p++;
    }
    if (*p != '"') bad("unterminated string");
    ++p;
    return s;
  }
};

}  // namespace

void costs_from_json(Graph& g, const char* json) {
  if (!json) fail(SN_E_INVALID, "null JSON");
  Parser ps{json};
  JVal root = ps.value();
  ps.ws();
  if (*ps.p) fail(SN_E_INVALID, "JSON: trailing characters");
  const auto& layers = root.at("layers").as_arr();
  if ((int)layers.size() != g.n_layers() + 1)
    fail(SN_E_INVALID, "cost table lists a different number of layers");
  std::vector<std::vector<int64_t>> cost(g.n_layers());
  std::vector<std::vector<ChildNet>> child(g.n_layers());
  for (int i = 0; i < g.n_layers(); ++i) {
    const JVal& jl = layers[i];
    if (jl.at("id").as_int() != i) fail(SN_E_INVALID, "layers must be listed in id order");
    const auto& rts = jl.at("routines").as_arr();
    const Layer& L = g.layers[i];
    if (rts.size() != L.routines.size())
      fail(SN_E_INVALID, "layer " + std::to_string(i) + ": routine count differs");
    for (size_t r = 0; r < rts.size(); ++r) {
      const Routine& R = L.routines[r];
      if (rts[r].at("rid").as_int() != R.id || rts[r].at("layout").as_int() != R.layout ||
          rts[r].at("algo").as_int() != R.algo || rts[r].at("param").as_int() != R.param ||
          (rts[r].obj.count("dtype") && rts[r].at("dtype").as_int() != R.dtype))
        fail(SN_E_INVALID, "layer " + std::to_string(i) + ": routine list differs");
      long long ns = rts[r].at("ns").as_int();
      if (ns < -1) fail(SN_E_INVALID, "negative time");
      ChildNet c = L.child[r];
      if (rts[r].obj.count("child")) {
        // a childnet's sub-routine times: when any is known, the routine's
        // time is the DPRS optimum over them (the listed "ns" is not used);
        // a childnet never profiled keeps the routine's own time
        if (c.empty()) fail(SN_E_INVALID, "layer " + std::to_string(i) + ": child times for a plain routine");
        const auto& rows = rts[r].at("child").at("ns").as_arr();
        if (rows.size() != c.cost.size()) fail(SN_E_INVALID, "childnet sub-layer count differs");
        for (size_t s = 0; s < rows.size(); ++s) {
          const auto& row = rows[s].as_arr();
          if (row.size() != c.cost[s].size()) fail(SN_E_INVALID, "childnet sub-routine count differs");
          for (size_t q = 0; q < row.size(); ++q) {
            const long long v = row[q].as_int();
            if (v < -1) fail(SN_E_INVALID, "negative time");
            c.cost[s][q] = v;
          }
        }
        if (c.profiled()) ns = childnet_select(c);
      }
      cost[i].push_back(ns);
      child[i].push_back(c);
    }
  }
  for (int i = 0; i < g.n_layers(); ++i)
    if (g.layers[i].type == SN_LAYER_INPUT && (cost[i].empty() || cost[i][0] != 0))
      fail(SN_E_INVALID, "input layer time must be 0");
  const auto& edges = root.at("edges").as_arr();
  auto E = all_edges(g);
  if (edges.size() != E.size()) fail(SN_E_INVALID, "cost table lists a different number of edges");
  std::vector<Edge> parsed = E;
  for (size_t k = 0; k < E.size(); ++k) {
    if (edges[k].at("from").as_int() != E[k].from || edges[k].at("to").as_int() != E[k].to)
      fail(SN_E_INVALID, "edge list differs");
    // 3 x 3 by layout (a graph with one dtype) or 9 x 9 by schema
    const auto& rows = edges[k].at("ns").as_arr();
    const int S = (int)rows.size();
    if (S != kNumSchemas && !(S == SN_NUM_LAYOUTS && !g.multi_dtype()))
      fail(SN_E_INVALID, g.multi_dtype() ? "adapt matrix must be 9 x 9" : "adapt matrix must be 3 x 3 or 9 x 9");
    const int base = S == kNumSchemas ? 0 : schema_of(g.dtype, 0);
    for (auto& row : parsed[k].adapt)
      for (auto& v : row) v = -1;
    for (int a = 0; a < S; ++a) {
      const auto& row = rows[a].as_arr();
      if ((int)row.size() != S) fail(SN_E_INVALID, "adapt matrix must be square");
      for (int b = 0; b < S; ++b) {
        long long v = row[b].as_int();
        if (v < -1) fail(SN_E_INVALID, "negative time");
        parsed[k].adapt[base + a][base + b] = a == b ? 0 : v;
      }
    }
  }
  for (int i = 0; i < g.n_layers(); ++i) {
    g.layers[i].cost = cost[i];
    g.layers[i].child = child[i];
  }
  for (size_t k = 0; k < g.edges.size(); ++k)
    std::memcpy(g.edges[k].adapt, parsed[k].adapt, sizeof(parsed[k].adapt));
  g.out_edges.assign(parsed.begin() + g.edges.size(), parsed.end());
  g.have_costs = true;
}

}  // namespace sn
