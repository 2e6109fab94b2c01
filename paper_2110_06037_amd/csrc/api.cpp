// C ABI: status codes in, no exception out (see include/softneuro.h).
#include <algorithm>
#include <cstdio>
#include <string>

#include <hip/hip_runtime.h>

#include "core.hpp"

using namespace sn;

struct sn_graph {
  Graph g;
};

static thread_local std::string t_err;

template <class F>
static int guarded(F&& f) {
  try {
    f();
    return SN_OK;
  } catch (const Error& e) {
    t_err = e.what();
    return e.code;
  } catch (const std::bad_alloc&) {
    t_err = "out of host memory";
    return SN_E_INTERNAL;
  } catch (const std::exception& e) {
    t_err = e.what();
    return SN_E_INTERNAL;
  } catch (...) {
    t_err = "unknown error";
    return SN_E_INTERNAL;
  }
}

#define CHECK_G(gp)                                         \
  do {                                                      \
    if (!(gp)) fail(SN_E_INVALID, "null graph pointer");    \
  } while (0)

extern "C" {

const char* sn_last_error(void) { return t_err.c_str(); }

int sn_graph_create(int32_t dtype, int32_t n, int32_t c, int32_t h, int32_t w, int32_t device,
                    sn_graph** out) {
  return guarded([&] {
    if (!out) fail(SN_E_INVALID, "null output pointer");
    *out = nullptr;
    if (dtype < SN_F32 || dtype > SN_BF16) fail(SN_E_INVALID, "unknown dtype");
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0) fail(SN_E_INVALID, "input dims must be positive");
    if (device < -1) fail(SN_E_INVALID, "device must be >= -1");
    check_tensor_size(Shape{n, c, h, w}, dtype, "input tensor");
    auto* gp = new sn_graph;
    try {
      graph_init(gp->g, dtype, Shape{n, c, h, w}, device);
      if (device >= 0) dev_create(gp->g);
    } catch (...) {
      delete gp;
      throw;
    }
    *out = gp;
  });
}

void sn_graph_destroy(sn_graph* gp) {
  if (!gp) return;
  try {
    if (!gp->g.host_only()) {
      plan_destroy(gp->g);
      dev_destroy(gp->g);
    }
  } catch (...) {
  }
  delete gp;
}

int sn_set_option(sn_graph* gp, int32_t option, int64_t value) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    bool routine_set = option == SN_OPT_LAYOUTS || option == SN_OPT_ALGOS || option == SN_OPT_PARAMS ||
                       option == SN_OPT_DTYPES || option == SN_OPT_WS_LIMIT;
    if (routine_set && g.n_layers() > 1)
      fail(SN_E_STATE, "routine-set options must be set before adding layers");
    switch (option) {
      case SN_OPT_LAYOUTS:
        if (value <= 0 || value > 7) fail(SN_E_INVALID, "layout mask must be in 1..7");
        g.opt_layouts = value;
        break;
      case SN_OPT_ALGOS:
        if (value <= 0 || value > 7) fail(SN_E_INVALID, "algorithm mask must be in 1..7");
        g.opt_algos = value;
        break;
      case SN_OPT_PARAMS:
        if (value != 0 && value != 1) fail(SN_E_INVALID, "PARAMS is 0 or 1");
        g.opt_params = value;
        break;
      case SN_OPT_HIPGRAPH:
        if (value != 0 && value != 1) fail(SN_E_INVALID, "HIPGRAPH is 0 or 1");
        g.opt_hipgraph = value;
        break;
      case SN_OPT_SEED:
        g.opt_seed = value;
        break;
      case SN_OPT_DTYPES:
        if (value <= 0 || value > 7) fail(SN_E_INVALID, "dtype mask must be in 1..7");
        g.opt_dtypes = value;
        break;
      case SN_OPT_KEEP:
        if (value != 0 && value != 1) fail(SN_E_INVALID, "KEEP is 0 or 1");
        if (g.opt_keep != value && g.plan) {
          g.opt_keep = value;
          plan_compile(g);  // re-place the buffers
        }
        g.opt_keep = value;
        break;
      case SN_OPT_FLUSH:
        if (value < 0 || value > (int64_t(1) << 34)) fail(SN_E_INVALID, "FLUSH is 0..16 GiB");
        g.opt_flush = value;
        break;
      case SN_OPT_WS_LIMIT:
        if (value < -1) fail(SN_E_INVALID, "WS_LIMIT is -1 (no limit) or a byte count");
        g.opt_ws_limit = value;
        break;
      default:
        fail(SN_E_INVALID, "unknown option");
    }
  });
}

int sn_add_layer(sn_graph* gp, const sn_layer_desc* d, const int32_t* inputs, int32_t n_inputs,
                 const void* weight, const float* bias, int32_t* out_id) {
  return guarded([&] {
    CHECK_G(gp);
    if (!d) fail(SN_E_INVALID, "null layer description");
    int id = graph_add_layer(gp->g, *d, inputs, n_inputs, weight, bias);
    if (out_id) *out_id = id;
  });
}

int sn_add_projected_conv(sn_graph* gp, const sn_layer_desc* d, int32_t input, int32_t shortcut,
                          int32_t shortcut_stride, const void* weight, const float* bias,
                          const void* shortcut_weight, const float* shortcut_bias, int32_t* out_id) {
  return guarded([&] {
    CHECK_G(gp);
    if (!d) fail(SN_E_INVALID, "null layer description");
    int id = graph_add_projected(gp->g, *d, input, shortcut, shortcut_stride, weight, bias, shortcut_weight,
                                 shortcut_bias);
    if (out_id) *out_id = id;
  });
}

int sn_add_input(sn_graph* gp, int32_t c, int32_t h, int32_t w, int32_t* out_id) {
  return guarded([&] {
    CHECK_G(gp);
    int id = graph_add_input(gp->g, c, h, w);
    if (out_id) *out_id = id;
  });
}

int sn_mark_output(sn_graph* gp, int32_t layer) {
  return guarded([&] {
    CHECK_G(gp);
    graph_mark_output(gp->g, layer);
  });
}

int sn_num_io(const sn_graph* gp, int32_t* n_inputs, int32_t* n_outputs) {
  return guarded([&] {
    CHECK_G(gp);
    if (n_inputs) *n_inputs = (int32_t)gp->g.net_inputs.size();
    if (n_outputs) *n_outputs = (int32_t)net_outputs(gp->g).size();
  });
}

int sn_profile(sn_graph* gp, int32_t warmup, int32_t reps, void* stream) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot profile");
    if (g.n_layers() < 2) fail(SN_E_STATE, "graph has no layers");
    if (warmup < 0 || reps < 1) fail(SN_E_INVALID, "warmup >= 0 and reps >= 1 required");
    dev_profile(g, warmup, reps, stream);
    g.have_costs = true;
  });
}

static void compile_if_device(Graph& g) {
  if (!g.host_only()) plan_compile(g);
}

int sn_select_path(sn_graph* gp, int32_t mode, int32_t layout, int32_t algo) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.n_layers() < 2) fail(SN_E_STATE, "graph has no layers");
    std::vector<int> old = g.path;
    if (mode == SN_SELECT_DPRS) {
      select_dprs(g);
    } else if (mode == SN_SELECT_FIXED) {
      select_fixed(g, layout, algo);
    } else {
      fail(SN_E_INVALID, "unknown selection mode");
    }
    try {
      compile_if_device(g);
    } catch (...) {
      g.path = old;
      throw;
    }
  });
}

int sn_set_path(sn_graph* gp, const int32_t* ids, int32_t n) {
  return guarded([&] {
    CHECK_G(gp);
    if (!ids) fail(SN_E_INVALID, "null routine ids");
    Graph& g = gp->g;
    if (g.n_layers() < 2) fail(SN_E_STATE, "graph has no layers");
    std::vector<int> old = g.path;
    set_path(g, ids, n);
    try {
      compile_if_device(g);
    } catch (...) {
      g.path = old;
      throw;
    }
  });
}

static void require_single_io(const Graph& g) {
  if (g.net_inputs.size() != 1 || net_outputs(g).size() != 1)
    fail(SN_E_INVALID, "the net has several inputs or outputs: use sn_run_mimo");
}

int sn_run(sn_graph* gp, const void* d_in, void* d_out, void* stream) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run");
    if (g.path.empty()) fail(SN_E_STATE, "no routine path selected");
    if (!d_in || !d_out) fail(SN_E_INVALID, "null device pointer");
    require_single_io(g);
    plan_run(g, &d_in, &d_out, stream, nullptr);
  });
}

int sn_run_mimo(sn_graph* gp, const void* const* d_ins, int32_t n_in, void* const* d_outs, int32_t n_out,
                void* stream) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run");
    if (g.path.empty()) fail(SN_E_STATE, "no routine path selected");
    if (!d_ins || !d_outs || n_in != (int32_t)g.net_inputs.size() || n_out != (int32_t)net_outputs(g).size())
      fail(SN_E_INVALID, "one device pointer per net input and per net output required");
    for (int i = 0; i < n_in; ++i)
      if (!d_ins[i]) fail(SN_E_INVALID, "null device pointer");
    for (int i = 0; i < n_out; ++i)
      if (!d_outs[i]) fail(SN_E_INVALID, "null device pointer");
    plan_run(g, d_ins, d_outs, stream, nullptr);
  });
}

int sn_run_noalloc(sn_graph* gp, const void* d_in, void* d_out, void* stream) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run");
    if (g.path.empty() || !g.plan) fail(SN_E_STATE, "no routine path selected");
    if (!d_in || !d_out) fail(SN_E_INVALID, "null device pointer");
    if (plan_arena_bytes(g) > noalloc_scratch_bytes())
      fail(SN_E_UNSUPPORTED, "the plan needs " + std::to_string(plan_arena_bytes(g)) +
                                 " bytes of intermediate memory; the static region holds " +
                                 std::to_string(noalloc_scratch_bytes()));
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) fail(SN_E_DEVICE, "hipGetDevice failed");
    if (cur != g.device && hipSetDevice(g.device) != hipSuccess) fail(SN_E_DEVICE, "hipSetDevice failed");
    require_single_io(g);
    void* base = noalloc_scratch_ptr(g.device);
    plan_run_in(g, base, noalloc_scratch_bytes(), &d_in, &d_out, stream);
  });
}

int sn_run_timed(sn_graph* gp, const void* d_in, void* d_out, void* stream, int32_t reps,
                 float* layer_ms, int32_t n) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run");
    if (g.path.empty()) fail(SN_E_STATE, "no routine path selected");
    if (!d_in || !d_out || !layer_ms) fail(SN_E_INVALID, "null pointer");
    if (n != g.n_layers()) fail(SN_E_INVALID, "layer_ms must have one entry per layer");
    if (reps < 1 || reps > 10000) fail(SN_E_INVALID, "reps must be in 1..10000");
    require_single_io(g);
    plan_run(g, &d_in, &d_out, stream, layer_ms, reps);
  });
}

int sn_layer_output(const sn_graph* gp, int32_t layer, void* d_dst, size_t cap, size_t* bytes,
                    int32_t* layout, void* stream) {
  return guarded([&] {
    CHECK_G(gp);
    const Graph& g = gp->g;
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph has no device tensors");
    int lay = 0;
    plan_layer_output(g, layer, d_dst, cap, bytes, &lay, stream);
    if (layout) *layout = lay;
  });
}

int sn_plan_launches(const sn_graph* gp, int32_t* layer_of_launch, int32_t cap, int32_t* n) {
  return guarded([&] {
    CHECK_G(gp);
    if (gp->g.host_only()) fail(SN_E_DEVICE, "host-only graph has no plan");
    const std::vector<int> v = plan_launch_layers(gp->g);
    if (n) *n = (int32_t)v.size();
    if (!layer_of_launch) return;
    if (cap < (int32_t)v.size()) fail(SN_E_NOMEM, "buffer smaller than the launch count");
    for (size_t i = 0; i < v.size(); ++i) layer_of_launch[i] = v[i];
  });
}

int sn_profile_integrated(sn_graph* gp, int32_t warmup, int32_t reps, void* stream,
                          int32_t* n_candidates) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (g.n_layers() < 2) fail(SN_E_STATE, "graph has no layers");
    if (warmup < 0 || reps < 0 || reps > 10000)
      fail(SN_E_INVALID, "warmup >= 0 and reps in 0..10000 required");
    if (reps > 0 && g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run candidates");
    std::vector<Candidate> c = integrated_candidates(g);
    if (reps > 0) integrated_measure(g, c, warmup, reps, stream);
    g.candidates = std::move(c);
    if (n_candidates) *n_candidates = (int32_t)g.candidates.size();
  });
}

int sn_refine_in_path(sn_graph* gp, int32_t tol_permille, int32_t max_alts, int32_t reps, void* stream,
                      int32_t* n_changed) {
  return guarded([&] {
    CHECK_G(gp);
    Graph& g = gp->g;
    if (tol_permille < 0 || tol_permille > 1000 || max_alts < 1 || max_alts > 16 || reps < 1 || reps > 1000)
      fail(SN_E_INVALID, "tol_permille in 0..1000, max_alts in 1..16 and reps in 1..1000 required");
    if (!g.have_costs) fail(SN_E_STATE, "no costs: profile or load a cost table first");
    if (g.path.empty()) fail(SN_E_STATE, "no selected path");
    if (g.host_only()) fail(SN_E_DEVICE, "host-only graph cannot run paths");
    const int c = refine_in_path(g, tol_permille, max_alts, reps, stream);
    if (n_changed) *n_changed = c;
  });
}

int sn_integrated_candidate(const sn_graph* gp, int32_t idx, int32_t* routine_ids, int32_t n,
                            int64_t* model_ns, int64_t* measured_ns, int32_t* kind_ab) {
  return guarded([&] {
    CHECK_G(gp);
    const Graph& g = gp->g;
    if (idx < 0 || idx >= (int32_t)g.candidates.size()) fail(SN_E_INVALID, "candidate index out of range");
    const Candidate& c = g.candidates[idx];
    if (routine_ids) {
      if (n != g.n_layers()) fail(SN_E_INVALID, "routine_ids must have one entry per layer");
      for (int i = 0; i < n; ++i) routine_ids[i] = c.path[i];
    }
    if (model_ns) *model_ns = c.model_ns;
    if (measured_ns) *measured_ns = c.measured_ns;
    if (kind_ab) {
      kind_ab[0] = c.kind;
      kind_ab[1] = c.a;
      kind_ab[2] = c.b;
    }
  });
}

int sn_get_costs(const sn_graph* gp, char* json, size_t cap, size_t* len) {
  return guarded([&] {
    CHECK_G(gp);
    std::string s = costs_to_json(gp->g);
    if (len) *len = s.size() + 1;
    if (!json || cap < s.size() + 1) fail(SN_E_NOMEM, "buffer too small for the cost table");
    std::memcpy(json, s.c_str(), s.size() + 1);
  });
}

int sn_set_costs(sn_graph* gp, const char* json) {
  return guarded([&] {
    CHECK_G(gp);
    costs_from_json(gp->g, json);
  });
}

int sn_get_path(const sn_graph* gp, int32_t* ids, int32_t n, int64_t* total_ns) {
  return guarded([&] {
    CHECK_G(gp);
    const Graph& g = gp->g;
    if (g.path.empty()) fail(SN_E_STATE, "no routine path selected");
    if (n != g.n_layers()) fail(SN_E_INVALID, "n must equal the number of layers");
    if (ids)
      for (int i = 0; i < n; ++i) ids[i] = g.path[i];
    if (total_ns) *total_ns = g.path_cost;
  });
}

int sn_num_layers(const sn_graph* gp, int32_t* n) {
  return guarded([&] {
    CHECK_G(gp);
    if (!n) fail(SN_E_INVALID, "null pointer");
    *n = gp->g.n_layers();
  });
}

int sn_num_routines(const sn_graph* gp, int32_t layer, int32_t* count) {
  return guarded([&] {
    CHECK_G(gp);
    if (!count) fail(SN_E_INVALID, "null pointer");
    if (layer < 0 || layer >= gp->g.n_layers()) fail(SN_E_INVALID, "unknown layer");
    *count = (int32_t)gp->g.layers[layer].routines.size();
  });
}

int sn_routine_info(const sn_graph* gp, int32_t layer, int32_t idx, sn_routine_desc* out) {
  return guarded([&] {
    CHECK_G(gp);
    if (!out) fail(SN_E_INVALID, "null pointer");
    const Graph& g = gp->g;
    if (layer < 0 || layer >= g.n_layers()) fail(SN_E_INVALID, "unknown layer");
    const Layer& L = g.layers[layer];
    if (idx < 0 || idx >= (int)L.routines.size()) fail(SN_E_INVALID, "unknown routine");
    const Routine& r = L.routines[idx];
    out->id = r.id;
    out->layout = r.layout;
    out->algo = r.algo;
    out->param = r.param;
    out->dtype = r.dtype;
    out->schema = r.schema();
    out->cost_ns = L.cost[idx];
    out->ws_bytes = (int64_t)routine_ws_bytes(g, L, r);
    std::snprintf(out->name, sizeof(out->name), "%s", r.name.c_str());
  });
}

int sn_layer_shape(const sn_graph* gp, int32_t layer, int32_t* nchw) {
  return guarded([&] {
    CHECK_G(gp);
    if (!nchw) fail(SN_E_INVALID, "null pointer");
    if (layer < 0 || layer >= gp->g.n_layers()) fail(SN_E_INVALID, "unknown layer");
    const Shape& s = gp->g.layers[layer].out;
    nchw[0] = s.n;
    nchw[1] = s.c;
    nchw[2] = s.h;
    nchw[3] = s.w;
  });
}

int sn_dp_stats(const sn_graph* gp, int32_t layer, int64_t* n_states, int64_t* n_candidates) {
  return guarded([&] {
    CHECK_G(gp);
    const Graph& g = gp->g;
    if (layer < 0 || layer >= (int)g.dp_stats.size()) fail(SN_E_INVALID, "no DPRS statistics");
    if (n_states) *n_states = g.dp_stats[layer].states;
    if (n_candidates) *n_candidates = g.dp_stats[layer].candidates;
  });
}

}  // extern "C"
