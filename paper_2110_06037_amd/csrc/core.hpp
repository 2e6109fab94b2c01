// Internal types of the routine-selection library (host side).
#pragma once

#include <cstdint>
#include <cstring>
#include <memory>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/softneuro.h"

namespace sn {

constexpr int64_t kInf = INT64_MAX / 4;

// Error carried to the C boundary as a status code plus message.
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};
[[noreturn]] inline void fail(int code, const std::string& msg) { throw Error(code, msg); }

struct Shape {
  int n = 0, c = 0, h = 0, w = 0;
  int64_t numel() const { return (int64_t)n * c * h * w; }
  bool operator==(const Shape& o) const { return n == o.n && c == o.c && h == o.h && w == o.w; }
};

inline int round8(int c) { return (c + 7) / 8 * 8; }
inline int dtype_size(int dt) { return dt == SN_F32 ? 4 : 2; }

// A schema is a (dtype, layout) pair (Sec. III-C: a routine's schema names
// the data representation it works in; converting between schemas is an
// adapt job).  Index = dtype * SN_NUM_LAYOUTS + layout.
constexpr int kNumSchemas = SN_NUM_SCHEMAS;
inline int schema_of(int dtype, int layout) { return dtype * SN_NUM_LAYOUTS + layout; }
inline int schema_dtype(int schema) { return schema / SN_NUM_LAYOUTS; }
inline int schema_layout(int schema) { return schema % SN_NUM_LAYOUTS; }

// Channels as stored by a layout (NC8HW8 pads to a multiple of 8).
inline int stored_c(const Shape& s, int layout) { return layout == SN_NC8HW8 ? round8(s.c) : s.c; }
inline int64_t stored_numel(const Shape& s, int layout) {
  return (int64_t)s.n * stored_c(s, layout) * s.h * s.w;
}

// Every kernel addresses a tensor with 32-bit byte offsets (buffer resources),
// so a tensor's stored size (channels padded to 8, the largest of the three
// layouts) must stay below 2 GiB.
inline void check_tensor_size(const Shape& s, int dtype, const char* what) {
  const int64_t bytes = (int64_t)s.n * round8(s.c) * s.h * s.w * dtype_size(dtype);
  if (bytes >= (int64_t(1) << 31))
    fail(SN_E_UNSUPPORTED, std::string(what) + " of " + std::to_string(bytes) +
                               " bytes exceeds the 2 GiB a kernel addresses");
}
inline void check_tensor_size_any(const Shape& s, int64_t dtype_mask, const char* what) {
  for (int d = 0; d < 3; ++d)
    if (dtype_mask >> d & 1) check_tensor_size(s, d, what);
}

// Two layouts hold identical bytes for this shape (the adapt is void); for
// schemas the dtypes must agree too (see schemas_equivalent).
inline bool layouts_equivalent(const Shape& s, int a, int b) {
  if (a == b) return true;
  auto canon = [&](int l) { return l == SN_NC8HW8 && s.c % 8 != 0 ? -1 : l; };
  if (canon(a) < 0 || canon(b) < 0) return false;  // padded NC8HW8 differs from the others
  bool spatial1 = (int64_t)s.h * s.w == 1;
  if (spatial1) return true;                        // N x C x 1 x 1 in all three
  // NCHW == NHWC when C == 1; NC8HW8 == NHWC when C == 8
  auto pair = [&](int x, int y) { return (a == x && b == y) || (a == y && b == x); };
  if (pair(SN_NCHW, SN_NHWC)) return s.c == 1;
  if (pair(SN_NHWC, SN_NC8HW8)) return s.c == 8;
  return false;
}

// Two schemas hold identical bytes for this shape.
inline bool schemas_equivalent(const Shape& s, int a, int b) {
  return schema_dtype(a) == schema_dtype(b) && layouts_equivalent(s, schema_layout(a), schema_layout(b));
}

struct Routine {
  int id = 0;
  int layout = 0;
  int algo = 0;
  int param = 0;
  int dtype = 0;  // element type it reads and writes
  std::string name;
  int schema() const { return schema_of(dtype, layout); }
};

// A routine built from sub-layers, each with routines of its own (a
// childnet, Sec. III-D).  Its sub-routines are profiled one by one and its
// time is the DPRS optimum over the sub-layers, found before the net's own
// DPRS runs (the algorithm applied from the innermost childnet outward).
// The sub-layers pass internal tensors of one fixed format, so the
// childnet has one schema and no adapts.
struct ChildNet {
  std::vector<std::string> layer;                 // sub-layer names
  std::vector<std::vector<std::string>> routine;  // [sub-layer][sub-routine] names
  std::vector<std::vector<int64_t>> cost;         // [sub-layer][sub-routine] ns, -1 = unknown
  std::vector<int> path;                          // selected sub-routine per sub-layer
  bool empty() const { return layer.empty(); }
  bool profiled() const {
    for (const auto& v : cost)
      for (int64_t c : v)
        if (c >= 0) return true;
    return false;
  }
};

struct Layer {
  int id = 0;
  int type = SN_LAYER_INPUT;
  sn_layer_desc d{};
  std::vector<int> inputs;
  Shape out;
  // host copies of the user's weights (run dtype bytes, OIHW / [K][C]) and bias
  std::vector<uint8_t> weight;
  std::vector<float> bias;
  // CONV2D with a projected shortcut (second input read by a 1 x 1
  // convolution at proj_stride): its weights [K][C2] and bias
  int proj_stride = 0;
  std::vector<uint8_t> wproj;
  std::vector<float> bproj;
  std::vector<Routine> routines;
  std::vector<int64_t> cost;  // per routine, ns; -1 = not profiled
  std::vector<ChildNet> child;  // per routine; empty for routines that are not childnets
  std::string signature;      // identical signatures share profiling results
};

struct Edge {
  int from = 0, to = 0;
  int64_t adapt[kNumSchemas][kNumSchemas];  // ns by schema index, -1 = unavailable
};

struct Plan;      // execution plan (plan.cpp)
struct DevState;  // device-side weights and profiling caches (device.cpp)

struct DPLayerStats {
  int64_t states = 0;      // (schema, constraint) states evaluated at the layer
  int64_t candidates = 0;  // candidate unions per state (|Lambda|^|H|)
};

// One routine path timed end to end by integrated profiling.
struct Candidate {
  std::vector<int> path;
  int64_t model_ns = -1;     // T(S) under the unit-profiled table
  int64_t measured_ns = -1;  // end-to-end time per run, -1 = not measured
  int kind = 0;              // 0: DPRS over the layouts in mask a; 1: fixed (layout a, algo b)
  int a = 0, b = 0;
};

struct Graph {
  int dtype = SN_F32;
  int device = -1;
  Shape in;
  int64_t opt_layouts = 7, opt_algos = 7, opt_params = 1, opt_hipgraph = 0, opt_seed = 1;
  int64_t opt_dtypes = 0;  // compute dtypes allowed (bit = sn_dtype); set to the run dtype at init
  int64_t opt_flush = 0;  // bytes written before each layer of a timed run (0 = none)
  int64_t opt_keep = 0;   // 1: the plan gives every buffer its own bytes
  int64_t opt_ws_limit = -1;  // largest routine workspace admitted (bytes), -1: no limit
  std::vector<Layer> layers;  // layers[0] = auxiliary input
  std::vector<Edge> edges;    // every (input -> layer) edge, in insertion order
  std::vector<int> net_inputs{0};  // layers carrying the caller's input tensors, in order
  std::vector<int> marked_outputs; // net outputs in order; empty = the last layer
  std::vector<Edge> out_edges;     // (net output k -> auxiliary output); from/to set on use
  bool have_costs = false;
  std::vector<int> path;      // routine index per layer; empty = none
  int64_t path_cost = -1;
  std::vector<DPLayerStats> dp_stats;
  std::vector<Candidate> candidates;  // last integrated profiling
  std::unique_ptr<Plan> plan;
  std::unique_ptr<DevState> dev;
  bool host_only() const { return device < 0; }
  bool multi_dtype() const { return opt_dtypes != (int64_t(1) << dtype); }
  // schemas the DP may use: allowed layouts x allowed dtypes, plus the
  // run-dtype NCHW schema of the auxiliary input and output layers
  bool schema_allowed(int sc) const {
    return sc == schema_of(dtype, SN_NCHW) ||
           ((opt_layouts >> schema_layout(sc) & 1) && (opt_dtypes >> schema_dtype(sc) & 1));
  }
  int n_layers() const { return (int)layers.size(); }
  Graph();
  ~Graph();
};

// graph.cpp
void graph_init(Graph& g, int dtype, Shape in, int device);
// a further net input (N x c x h x w, run dtype, NCHW): a zero-cost input
// layer joined to the auxiliary input layer 0 by a structural edge
int graph_add_input(Graph& g, int c, int h, int w);
void graph_mark_output(Graph& g, int layer);
std::vector<int> net_outputs(const Graph& g);
int graph_add_projected(Graph& g, const sn_layer_desc& d, int input, int shortcut, int stride,
                        const void* weight, const float* bias, const void* sc_weight, const float* sc_bias);
int graph_add_layer(Graph& g, const sn_layer_desc& d, const int32_t* inputs, int n_inputs,
                    const void* weight, const float* bias);
// all edges including the one into the auxiliary output layer (id = n_layers())
std::vector<Edge> all_edges(const Graph& g);
std::vector<Routine> enumerate_routines(const Graph& g, const Layer& L);
bool winograd_applicable(const Layer& L, const Shape& in);
std::string routine_name(const Graph& g, const Layer& L, const Routine& r);
// the childnet of a routine (empty when the routine is a single kernel
// sequence of its own): the split Winograd F(2x2,3x3) routine is wgenc ->
// wgconv (one sub-routine per GEMM tile) -> wgdec
ChildNet make_childnet(const Graph& g, const Layer& L, const Routine& r);

// select.cpp
void select_dprs(Graph& g, int layout_mask = -1, int dtype_mask = -1);
// DPRS over a childnet (a chain of sub-layers, one schema): sets c.path and
// returns its time, -1 when some sub-layer has no timed sub-routine
int64_t childnet_select(ChildNet& c);
// integrated profiling's candidate paths (Sec. III-C): DPRS over every
// non-empty subset of the allowed layouts, then every fixed path; identical
// paths kept once; g.path is left unchanged
std::vector<Candidate> integrated_candidates(Graph& g);
// dtype -1: the run dtype if allowed, else the lowest allowed one
void select_fixed(Graph& g, int layout, int algo, int dtype = -1);
void set_path(Graph& g, const int32_t* ids, int n);
int64_t path_total(const Graph& g, const std::vector<int>& path);

// json.cpp
std::string costs_to_json(const Graph& g);
void costs_from_json(Graph& g, const char* json);

// device.cpp (HIP)
void dev_create(Graph& g);
void dev_destroy(Graph& g);
void dev_upload_layer(Graph& g, int layer);
// Device workspace a routine of layer L needs beyond its input and output
// tensors (host arithmetic only; also for host-only graphs).
size_t routine_ws_bytes(const Graph& g, const Layer& L, const Routine& r);
void dev_profile(Graph& g, int warmup, int reps, void* stream);
void plan_compile(Graph& g);
// d_in / d_out: one device pointer per net input / output, in order
void plan_run(Graph& g, const void* const* d_in, void* const* d_out, void* stream, float* layer_ms = nullptr,
              int reps = 1);
void plan_destroy(Graph& g);
// noalloc_scratch.hip: the static per-device region of sn_run_noalloc
size_t noalloc_scratch_bytes();
void* noalloc_scratch_ptr(int device);  // the region's device address (device must be current)
void plan_run_in(const Graph& g, void* base, size_t cap, const void* const* d_in, void* const* d_out,
                 void* stream);
size_t plan_arena_bytes(const Graph& g);
std::vector<int> plan_launch_layers(const Graph& g);
void plan_layer_output(const Graph& g, int layer, void* d_dst, size_t cap, size_t* bytes, int* layout,
                       void* stream);
// times every candidate end to end and selects the fastest (compiles its plan)
void integrated_measure(Graph& g, std::vector<Candidate>& cands, int warmup, int reps,
                        void* stream);
// in-path refinement of g.path (sn_refine_in_path); returns the number of
// layers whose routine changed
int refine_in_path(Graph& g, int tol_permille, int max_alts, int reps, void* stream);

}  // namespace sn
