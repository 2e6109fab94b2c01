// Net construction (Sec. III-B of the paper: a net is a DAG of layers that
// exchange blobs; every layer has a type, layer parameters and weights) and
// routine enumeration (Sec. III-C: routines are interchangeable
// implementations of a layer, identified by schema/algorithm and carrying
// routine parameters).
#include <algorithm>
#include <sstream>

#include "core.hpp"
#include "kernels/launch.hpp"

namespace sn {

static const char* kLayoutName[SN_NUM_LAYOUTS] = {"nchw", "nhwc", "nc8hw8"};
static const char* kAlgoName[SN_NUM_ALGOS] = {"direct", "igemm", "winograd"};

std::vector<Edge> all_edges(const Graph& g) {
  std::vector<Edge> e = g.edges;
  Edge o = g.out_edge;
  o.from = g.n_layers() - 1;
  o.to = g.n_layers();
  e.push_back(o);
  return e;
}

void graph_init(Graph& g, int dtype, Shape in, int device) {
  for (auto& row : g.out_edge.adapt)
    for (auto& v : row) v = -1;
  g.dtype = dtype;
  g.in = in;
  g.device = device;
  Layer L;
  L.id = 0;
  L.type = SN_LAYER_INPUT;
  L.out = in;
  Routine r;
  r.id = 0;
  r.layout = SN_NCHW;
  r.algo = SN_ALGO_DIRECT;
  r.name = "input/nchw";
  L.routines.push_back(r);
  L.cost.push_back(0);
  L.signature = "input";
  g.layers.push_back(std::move(L));
}

bool winograd_applicable(const Layer& L, const Shape& in) {
  const auto& d = L.d;
  return L.type == SN_LAYER_CONV2D && d.groups == 1 && d.r == 3 && d.s == 3 && d.stride == 1 &&
         d.pad == 1 && in.c >= 1;
}

static bool is_depthwise(const Layer& L, const Shape& in) {
  return L.type == SN_LAYER_CONV2D && L.d.groups > 1 && L.d.groups == in.c && L.d.k == in.c;
}

std::string routine_name(const Layer& L, const Routine& r) {
  std::ostringstream o;
  o << kLayoutName[r.layout] << "/" << kAlgoName[r.algo];
  if (L.type == SN_LAYER_CONV2D && r.algo == SN_ALGO_IGEMM) o << ":p" << r.param;
  if (L.type == SN_LAYER_FC && r.algo == SN_ALGO_IGEMM) o << ":1x1conv:p" << r.param;
  return o.str();
}

std::vector<Routine> enumerate_routines(const Graph& g, const Layer& L) {
  std::vector<Routine> out;
  if (L.type == SN_LAYER_INPUT) return out;
  const Shape& in = g.layers[L.inputs[0]].out;
  const int residual = L.type == SN_LAYER_CONV2D && L.inputs.size() == 2;
  auto add = [&](int layout, int algo, int param) {
    Routine r;
    r.id = (int)out.size();
    r.layout = layout;
    r.algo = algo;
    r.param = param;
    r.name = routine_name(L, r);
    out.push_back(r);
  };
  for (int lay = 0; lay < SN_NUM_LAYOUTS; ++lay) {
    if (!(g.opt_layouts >> lay & 1)) continue;
    switch (L.type) {
      case SN_LAYER_CONV2D:
        if (is_depthwise(L, in)) {
          add(lay, SN_ALGO_DIRECT, 0);  // depthwise has its own direct routine
          break;
        }
        if (g.opt_algos >> SN_ALGO_DIRECT & 1) add(lay, SN_ALGO_DIRECT, 0);
        if (g.opt_algos >> SN_ALGO_IGEMM & 1) {
          int np = g.opt_params ? k::igemm_num_params(g.dtype) : 1;
          for (int p = 0; p < np; ++p)
            if (k::igemm_param_valid(g.dtype, p, lay, in.n, in.c, in.h, in.w, L.d.r, L.d.s, L.d.stride,
                                     L.d.pad, L.d.k) &&
                (residual == 0 || k::igemm_param_takes_residual(g.dtype, p, lay, L.d.k)))
              add(lay, SN_ALGO_IGEMM, p);
        }
        if ((g.opt_algos >> SN_ALGO_WINOGRAD & 1) && !residual && winograd_applicable(L, in))
          add(lay, SN_ALGO_WINOGRAD, 0);
        break;
      case SN_LAYER_FC:
        add(lay, SN_ALGO_DIRECT, 0);
        if (g.opt_algos >> SN_ALGO_IGEMM & 1) {  // the dense childnet: a 1x1 convolution
          int np = g.opt_params ? k::igemm_num_params(g.dtype) : 1;
          for (int p = 0; p < np; ++p)
            if (k::igemm_param_valid(g.dtype, p, lay, in.n, in.c, 1, 1, 1, 1, 1, 0, L.d.k))
              add(lay, SN_ALGO_IGEMM, p);
        }
        break;
      default:
        add(lay, SN_ALGO_DIRECT, 0);
    }
  }
  return out;
}

static std::string signature(const Graph& g, const Layer& L) {
  std::ostringstream o;
  o << "t" << L.type << " k" << L.d.k << " r" << L.d.r << " s" << L.d.s << " st" << L.d.stride
    << " p" << L.d.pad << " g" << L.d.groups << " a" << L.d.act << " dt" << g.dtype;
  for (int j : L.inputs) {
    const Shape& s = g.layers[j].out;
    o << " [" << s.n << "," << s.c << "," << s.h << "," << s.w << "]";
  }
  return o.str();
}

int graph_add_layer(Graph& g, const sn_layer_desc& d, const int32_t* inputs, int n_inputs,
                    const void* weight, const float* bias) {
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
      if (L.inputs.size() == 2) {
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
  check_tensor_size(out, g.dtype, "layer output");
  L.out = out;
  if (wbytes) {
    L.weight.resize(wbytes);
    std::memcpy(L.weight.data(), weight, wbytes);
    L.bias.assign(out.c, 0.f);
    if (bias) std::memcpy(L.bias.data(), bias, sizeof(float) * out.c);
  }
  L.signature = signature(g, L);
  g.layers.push_back(std::move(L));
  Layer& ref = g.layers.back();
  ref.routines = enumerate_routines(g, ref);
  ref.cost.assign(ref.routines.size(), -1);
  for (int j : ref.inputs) {
    Edge e;
    e.from = j;
    e.to = ref.id;
    for (auto& row : e.adapt)
      for (auto& v : row) v = -1;
    g.edges.push_back(e);
  }
  g.have_costs = false;
  if (!g.host_only()) dev_upload_layer(g, ref.id);
  return ref.id;
}

}  // namespace sn
