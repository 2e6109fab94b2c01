// Net construction (Sec. III-B of the paper: a net is a DAG of layers that
// exchange blobs; every layer has a type, layer parameters and weights) and
// routine enumeration (Sec. III-C: routines are interchangeable
// implementations of a layer, identified by schema/algorithm and carrying
// routine parameters).
#include <algorithm>
#include <sstream>

#include "core.hpp"
#include "kernels/launch.hpp"
#include "kernels/wino.hpp"

namespace sn {

static const char* kLayoutName[SN_NUM_LAYOUTS] = {"nchw", "nhwc", "nc8hw8"};
static const char* kDtypeName[3] = {"f32", "f16", "bf16"};
static const char* kAlgoName[SN_NUM_ALGOS] = {"direct", "igemm", "winograd"};

static Edge blank_edge(int from, int to) {
  Edge e;
  e.from = from;
  e.to = to;
  for (auto& row : e.adapt)
    for (auto& v : row) v = -1;
  return e;
}

std::vector<int> net_outputs(const Graph& g) {
  if (!g.marked_outputs.empty()) return g.marked_outputs;
  return {g.n_layers() - 1};
}

// The layer edges, then one edge from every net output to the auxiliary
// output layer (id n_layers()), which merges them (Sec. IV-E).
std::vector<Edge> all_edges(const Graph& g) {
  std::vector<Edge> e = g.edges;
  const std::vector<int> outs = net_outputs(g);
  for (size_t k = 0; k < outs.size(); ++k) {
    Edge o = k < g.out_edges.size() ? g.out_edges[k] : blank_edge(0, 0);
    o.from = outs[k];
    o.to = g.n_layers();
    e.push_back(o);
  }
  return e;
}

static Layer input_layer(int id, int dtype, Shape s) {
  Layer L;
  L.id = id;
  L.type = SN_LAYER_INPUT;
  L.out = s;
  Routine r;
  r.id = 0;
  r.layout = SN_NCHW;
  r.algo = SN_ALGO_DIRECT;
  r.dtype = dtype;
  r.name = "input/nchw";
  L.routines.push_back(r);
  L.cost.push_back(0);
  L.child.emplace_back();
  L.signature = "input";
  return L;
}

void graph_init(Graph& g, int dtype, Shape in, int device) {
  g.dtype = dtype;
  g.opt_dtypes = int64_t(1) << dtype;
  g.in = in;
  g.device = device;
  g.layers.push_back(input_layer(0, dtype, in));
}

// The paper joins the inputs of a multi-input net with an auxiliary input
// layer of zero cost (Sec. IV-E).  Layer 0 carries the first input and plays
// that role: every further input layer gets an edge from it that carries no
// data and costs nothing (both ends have the one run-dtype NCHW schema), so
// the layer graph keeps a single source.
int graph_add_input(Graph& g, int c, int h, int w) {
  if (!g.path.empty()) fail(SN_E_STATE, "cannot add inputs after a path was selected");
  if (c <= 0 || h <= 0 || w <= 0) fail(SN_E_INVALID, "input dims must be positive");
  const Shape s{g.in.n, c, h, w};
  check_tensor_size_any(s, g.opt_dtypes | (int64_t(1) << g.dtype), "input tensor");
  const int id = g.n_layers();
  Layer L = input_layer(id, g.dtype, s);
  L.inputs.push_back(0);
  g.layers.push_back(std::move(L));
  Edge e = blank_edge(0, id);
  e.adapt[schema_of(g.dtype, SN_NCHW)][schema_of(g.dtype, SN_NCHW)] = 0;
  g.edges.push_back(e);
  g.net_inputs.push_back(id);
  g.have_costs = false;
  if (!g.host_only()) dev_upload_layer(g, id);
  return id;
}

// Net outputs, in the order of the caller's output tensors; the implicit
// auxiliary output layer merges them (Sec. IV-E).
void graph_mark_output(Graph& g, int layer) {
  if (!g.path.empty()) fail(SN_E_STATE, "cannot mark outputs after a path was selected");
  if (layer < 1 || layer >= g.n_layers()) fail(SN_E_INVALID, "unknown layer");
  if (g.layers[layer].type == SN_LAYER_INPUT) fail(SN_E_INVALID, "an input layer cannot be a net output");
  if (std::find(g.marked_outputs.begin(), g.marked_outputs.end(), layer) != g.marked_outputs.end())
    fail(SN_E_INVALID, "layer is already a net output");
  g.marked_outputs.push_back(layer);
  g.out_edges.clear();
  g.have_costs = false;
}

bool winograd_applicable(const Layer& L, const Shape& in) {
  const auto& d = L.d;
  return L.type == SN_LAYER_CONV2D && d.groups == 1 && d.r == 3 && d.s == 3 && d.stride == 1 &&
         d.pad == 1 && in.c >= 1;
}

static bool is_depthwise(const Layer& L, const Shape& in) {
  return L.type == SN_LAYER_CONV2D && L.d.groups > 1 && L.d.groups == in.c && L.d.k == in.c;
}

std::string routine_name(const Graph& g, const Layer& L, const Routine& r) {
  std::ostringstream o;
  if (g.multi_dtype()) o << kDtypeName[r.dtype] << ":";
  o << kLayoutName[r.layout] << "/" << kAlgoName[r.algo];
  if (L.type == SN_LAYER_CONV2D && r.algo == SN_ALGO_IGEMM) o << ":p" << r.param;
  if (L.type == SN_LAYER_CONV2D && r.algo == SN_ALGO_WINOGRAD && r.param == k::winograd_f4_param()) o << ":f4x4";
  else if (L.type == SN_LAYER_CONV2D && r.algo == SN_ALGO_WINOGRAD && r.param > 0) o << ":fused:p" << r.param - 1;
  if (L.type == SN_LAYER_CONV2D && r.algo == SN_ALGO_DIRECT && r.param > 0) o << ":strip" << k::dw_strip_len(r.param);
  if (L.type == SN_LAYER_FC && r.algo == SN_ALGO_IGEMM) o << ":1x1conv:p" << r.param;
  return o.str();
}

std::vector<Routine> enumerate_routines(const Graph& g, const Layer& L) {
  std::vector<Routine> out;
  if (L.type == SN_LAYER_INPUT) return out;
  const Shape& in = g.layers[L.inputs[0]].out;
  const int residual = L.type == SN_LAYER_CONV2D && L.inputs.size() == 2;
  // the run dtype first (so a single-dtype graph numbers its routines as
  // before), then the other allowed dtypes in sn_dtype order
  std::vector<int> dts;
  if (g.opt_dtypes >> g.dtype & 1) dts.push_back(g.dtype);
  for (int d = 0; d < 3; ++d)
    if (d != g.dtype && (g.opt_dtypes >> d & 1)) dts.push_back(d);
  int dt = g.dtype;
  auto add = [&](int layout, int algo, int param) {
    Routine r;
    r.id = (int)out.size();
    r.layout = layout;
    r.algo = algo;
    r.param = param;
    r.dtype = dt;
    r.name = routine_name(g, L, r);
    out.push_back(r);
  };
  for (int d : dts) {
    dt = d;
    for (int lay = 0; lay < SN_NUM_LAYOUTS; ++lay) {
      if (!(g.opt_layouts >> lay & 1)) continue;
      switch (L.type) {
        case SN_LAYER_CONV2D:
          if (L.proj_stride > 0) {
            // projection, then the convolution with it as residual (two
            // launches, any layout and dtype); both products in one
            // reduction on the LDS-DMA tiles
            add(lay, SN_ALGO_DIRECT, 0);
            if (g.opt_algos >> SN_ALGO_IGEMM & 1) {
              const Shape& sc = g.layers[L.inputs[1]].out;
              for (int p = 0; p < k::igemm_num_params(dt); ++p)
                if (k::igemm_param_takes_projection(dt, p, lay, in.n, in.c, in.h, in.w, L.d.r, L.d.s,
                                                    L.d.stride, L.d.pad, L.d.k, sc.c)) {
                  add(lay, SN_ALGO_IGEMM, p);
                  if (!g.opt_params) break;
                }
            }
            break;
          }
          if (is_depthwise(L, in)) {
            add(lay, SN_ALGO_DIRECT, 0);  // depthwise has its own direct routine
            if (g.opt_params)             // ... and strip lengths as routine parameters
              for (int p = 1; p <= k::dw_num_strip_params(dt, lay, in.c, L.d.r, L.d.s, L.d.stride); ++p)
                add(lay, SN_ALGO_DIRECT, p);
            break;
          }
          if (g.opt_algos >> SN_ALGO_DIRECT & 1) add(lay, SN_ALGO_DIRECT, 0);
          if (g.opt_algos >> SN_ALGO_IGEMM & 1) {
            int np = g.opt_params ? k::igemm_num_params(dt) : 1;
            for (int p = 0; p < np; ++p)
              if (k::igemm_param_valid(dt, p, lay, in.n, in.c, in.h, in.w, L.d.r, L.d.s, L.d.stride,
                                       L.d.pad, L.d.k) &&
                  (residual == 0 || k::igemm_param_takes_residual(dt, p, lay, L.d.k)))
                add(lay, SN_ALGO_IGEMM, p);
          }
          if ((g.opt_algos >> SN_ALGO_WINOGRAD & 1) && !residual && winograd_applicable(L, in)) {
            add(lay, SN_ALGO_WINOGRAD, 0);  // transforms and tile GEMMs as three kernels
            if (g.opt_params && k::wino_fused_applicable(dt, lay, in.c))
              for (int p = 0; p < k::wino_fused_num_configs(); ++p) add(lay, SN_ALGO_WINOGRAD, p + 1);
            // F(4x4,3x3) in fp32 only: its input transform scales values by up
            // to 100 (coefficients up to 5 in each direction), past fp16's range
            // on deep layers, and bf16's 8-bit mantissa loses the tolerance
            if (g.opt_params && dt == SN_F32) add(lay, SN_ALGO_WINOGRAD, k::winograd_f4_param());
          }
          break;
        case SN_LAYER_FC:
          add(lay, SN_ALGO_DIRECT, 0);
          if (g.opt_algos >> SN_ALGO_IGEMM & 1) {  // the dense childnet: a 1x1 convolution
            int np = g.opt_params ? k::igemm_num_params(dt) : 1;
            for (int p = 0; p < np; ++p)
              if (k::igemm_param_valid(dt, p, lay, in.n, in.c, 1, 1, 1, 1, 1, 0, L.d.k))
                add(lay, SN_ALGO_IGEMM, p);
          }
          break;
        default:
          add(lay, SN_ALGO_DIRECT, 0);
      }
    }
  }
  if (g.opt_ws_limit >= 0) {
    // memory-restricted selection: only routines within the workspace limit
    std::vector<Routine> kept;
    for (const Routine& r : out)
      if ((int64_t)routine_ws_bytes(g, L, r) <= g.opt_ws_limit) {
        kept.push_back(r);
        kept.back().id = (int)kept.size() - 1;
      }
    if (kept.empty()) fail(SN_E_UNSUPPORTED, "no routine of this layer fits the workspace limit");
    out.swap(kept);
  }
  return out;
}

ChildNet make_childnet(const Graph& g, const Layer& L, const Routine& r) {
  ChildNet c;
  if (L.type != SN_LAYER_CONV2D || r.algo != SN_ALGO_WINOGRAD ||
      (r.param != 0 && r.param != k::winograd_f4_param()))
    return c;
  // one GEMM tile only when routine parameters are restricted
  const int ng = g.opt_params ? k::winograd_gemm_num_configs(r.dtype) : 1;
  c.layer = {"wgenc", "wgconv", "wgdec"};
  c.routine = {{"wgenc"}, {}, {"wgdec"}};
  for (int q = 0; q < ng; ++q) c.routine[1].push_back("wgconv:p" + std::to_string(q));
  for (const auto& v : c.routine) c.cost.emplace_back(v.size(), -1);
  c.path.assign(c.layer.size(), 0);
  return c;
}

static std::string signature(const Graph& g, const Layer& L) {
  std::ostringstream o;
  o << "t" << L.type << " k" << L.d.k << " r" << L.d.r << " s" << L.d.s << " st" << L.d.stride
    << " p" << L.d.pad << " g" << L.d.groups << " a" << L.d.act << " dt" << g.dtype << " pj" << L.proj_stride;
  for (int j : L.inputs) {
    const Shape& s = g.layers[j].out;
    o << " [" << s.n << "," << s.c << "," << s.h << "," << s.w << "]";
  }
  return o.str();
}

// proj_stride > 0: a CONV2D whose second input is a shortcut projected by a
// 1 x 1 convolution (sc_weight, sc_bias) and added before the activation
static int add_layer_impl(Graph& g, const sn_layer_desc& d, const int32_t* inputs, int n_inputs,
                          const void* weight, const float* bias, int proj_stride, const void* sc_weight,
                          const float* sc_bias) {
  if (!g.path.empty()) fail(SN_E_STATE, "cannot add layers after a path was selected");
  Layer L;
  L.id = g.n_layers();
  L.type = d.type;
  L.d = d;
  int want = d.type == SN_LAYER_ADD ? 2 : 1;
  if (d.type == SN_LAYER_CONV2D && n_inputs == 2) want = 2;  // convolution with a residual
  if (d.type < SN_LAYER_CONV2D || d.type > SN_LAYER_FC)
    fail(SN_E_INVALID, "unknown layer type " + std::to_string(d.type));
  if (n_inputs != want || !inputs)
    fail(SN_E_INVALID, "layer type " + std::to_string(d.type) + " takes " + std::to_string(want) +
                           " input(s)");
  for (int i = 0; i < n_inputs; ++i) {
    if (inputs[i] < 0 || inputs[i] >= L.id)
      fail(SN_E_INVALID, "input id " + std::to_string(inputs[i]) + " is not an existing layer");
    L.inputs.push_back(inputs[i]);
  }
  if (d.act < SN_ACT_NONE || d.act > SN_ACT_RELU6) fail(SN_E_INVALID, "unknown activation");
  const Shape in = g.layers[L.inputs[0]].out;
  Shape out = in;
  auto outdim = [](int x, int k, int st, int p) { return (x + 2 * p - k) / st + 1; };
  int64_t wbytes = 0;
  int ds = dtype_size(g.dtype);
  switch (d.type) {
    case SN_LAYER_CONV2D: {
      if (d.k <= 0 || d.r <= 0 || d.s <= 0 || d.stride <= 0 || d.pad < 0 || d.groups <= 0)
        fail(SN_E_INVALID, "bad convolution parameters");
      if (d.groups != 1 && !(d.groups == in.c && d.k == in.c))
        fail(SN_E_UNSUPPORTED, "only dense (groups=1) and depthwise (groups=C=K) convolutions");
      if (in.h + 2 * d.pad < d.r || in.w + 2 * d.pad < d.s)
        fail(SN_E_SHAPE, "kernel larger than the padded input");
      out = {in.n, d.k, outdim(in.h, d.r, d.stride, d.pad), outdim(in.w, d.s, d.stride, d.pad)};
      wbytes = (int64_t)d.k * (in.c / d.groups) * d.r * d.s * ds;
      if (L.inputs.size() == 2 && proj_stride > 0) {
        const Shape& sc = g.layers[L.inputs[1]].out;
        if (d.groups != 1) fail(SN_E_INVALID, "a projected shortcut needs a dense convolution");
        if (sc.n != out.n || (sc.h - 1) / proj_stride + 1 != out.h || (sc.w - 1) / proj_stride + 1 != out.w)
          fail(SN_E_SHAPE, "the projected shortcut does not give the output's size");
        if (!sc_weight) fail(SN_E_INVALID, "a projected shortcut needs weights");
      } else if (L.inputs.size() == 2) {
        if (d.groups != 1) fail(SN_E_UNSUPPORTED, "a residual input needs a dense convolution");
        if (!(g.layers[L.inputs[1]].out == out)) fail(SN_E_SHAPE, "residual differs from the output shape");
      }
      if (!weight) fail(SN_E_INVALID, "convolution needs weights");
      break;
    }
    case SN_LAYER_MAXPOOL:
      if (d.r <= 0 || d.stride <= 0 || d.pad < 0 || d.pad >= d.r)
        fail(SN_E_INVALID, "bad pooling parameters");
      if (in.h + 2 * d.pad < d.r || in.w + 2 * d.pad < d.r)
        fail(SN_E_SHAPE, "window larger than the padded input");
      out = {in.n, in.c, outdim(in.h, d.r, d.stride, d.pad), outdim(in.w, d.r, d.stride, d.pad)};
      break;
    case SN_LAYER_GAP:
      out = {in.n, in.c, 1, 1};
      break;
    case SN_LAYER_ADD: {
      const Shape& b = g.layers[L.inputs[1]].out;
      if (!(b == in)) fail(SN_E_SHAPE, "ADD inputs differ in shape");
      break;
    }
    case SN_LAYER_FC:
      if (d.k <= 0) fail(SN_E_INVALID, "FC needs k > 0");
      if (in.h != 1 || in.w != 1) fail(SN_E_SHAPE, "FC input must be N x C x 1 x 1");
      out = {in.n, d.k, 1, 1};
      wbytes = (int64_t)d.k * in.c * ds;
      if (!weight) fail(SN_E_INVALID, "FC needs weights");
      break;
  }
  if (out.h <= 0 || out.w <= 0) fail(SN_E_SHAPE, "empty output");
  check_tensor_size_any(out, g.opt_dtypes, "layer output");
  L.out = out;
  if (wbytes) {
    L.weight.resize(wbytes);
    std::memcpy(L.weight.data(), weight, wbytes);
    L.bias.assign(out.c, 0.f);
    if (bias) std::memcpy(L.bias.data(), bias, sizeof(float) * out.c);
  }
  if (proj_stride > 0) {
    const int64_t pbytes = (int64_t)out.c * g.layers[L.inputs[1]].out.c * ds;
    L.proj_stride = proj_stride;
    L.wproj.resize(pbytes);
    std::memcpy(L.wproj.data(), sc_weight, pbytes);
    L.bproj.assign(out.c, 0.f);
    if (sc_bias) std::memcpy(L.bproj.data(), sc_bias, sizeof(float) * out.c);
  }
  L.signature = signature(g, L);
  L.routines = enumerate_routines(g, L);  // (may refuse the layer: the workspace limit)
  g.layers.push_back(std::move(L));
  Layer& ref = g.layers.back();
  ref.cost.assign(ref.routines.size(), -1);
  for (const Routine& r : ref.routines) ref.child.push_back(make_childnet(g, ref, r));
  for (int j : ref.inputs) g.edges.push_back(blank_edge(j, ref.id));
  g.have_costs = false;
  if (!g.host_only()) dev_upload_layer(g, ref.id);
  return ref.id;
}

int graph_add_layer(Graph& g, const sn_layer_desc& d, const int32_t* inputs, int n_inputs,
                    const void* weight, const float* bias) {
  return add_layer_impl(g, d, inputs, n_inputs, weight, bias, 0, nullptr, nullptr);
}

int graph_add_projected(Graph& g, const sn_layer_desc& d, int input, int shortcut, int stride,
                        const void* weight, const float* bias, const void* sc_weight, const float* sc_bias) {
  if (d.type != SN_LAYER_CONV2D) fail(SN_E_INVALID, "a projected shortcut belongs to a convolution");
  if (stride < 1) fail(SN_E_INVALID, "shortcut stride must be >= 1");
  const int32_t ins[2] = {input, shortcut};
  return add_layer_impl(g, d, ins, 2, weight, bias, stride, sc_weight, sc_bias);
}

}  // namespace sn
