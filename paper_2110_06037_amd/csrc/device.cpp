// Device side of the library: weight preparation per routine format, unit
// profiling (Sec. III-C), plan compilation with adapt (layout converter)
// insertion on edges whose routines use different schemas (Sec. III-C,
// Definition 1), liveness-based activation memory, and execution (optionally
// replayed from a captured HIP graph).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <map>

#include "core.hpp"
#include "kernels/launch.hpp"
#include "kernels/wino.hpp"

namespace sn {

#define HIPCHK(expr)                                                                        \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) fail(SN_E_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

static size_t align256(size_t b) { return (b + 255) / 256 * 256; }

struct DevLayer {
  void* w[3] = {};      // per dtype: dense [Kp][R][S][C8] | depthwise [R][S][C8] | fc [Kp][C8]
  void* wu[3] = {};     // per dtype: Winograd U [16][Kp][C8]
  void* wu4[3] = {};    // per dtype: Winograd F(4x4,3x3) U [36][Kp][C8]
  void* wp[3] = {};     // per dtype: projected-shortcut weights [Kp][C2_8]
  void* wcat[3] = {};   // per dtype: 1x1 layer with a projected shortcut, both weights [Kp][C + C2]
  float* bias = nullptr;  // [Kp] (with a projected shortcut: the two biases summed)
  float* zbias = nullptr;  // [Kp] zeros (the shortcut's own launch in the two-launch routine)
};

struct DevState {
  int device = 0;
  unsigned* fixup_cnt = nullptr;  // kFixupMaxTiles zeroed tile counters (split reductions)
  std::vector<DevLayer> L;
  std::map<std::string, int64_t> cost_cache;  // "signature|routine" or "cvt|shape|a|b" -> ns
};

struct BufRef {
  int kind = 0;  // 0 arena, 1 user input, 2 user output
  size_t off = 0;
  int idx = 0;   // which user input / output
};

struct Step {
  int type = 0;   // 0 convert, 1 layer
  int layer = 0;  // layer the step is accounted to
  BufRef src, dst;
  k::TDesc sd{}, dd{};
  int sdt = 0, ddt = 0;  // converter: source and destination element types
  int n_in = 0;
  BufRef in[2];
  k::TDesc ind[2]{};
  BufRef out;
  k::TDesc outd{};
  BufRef ws;
  size_t ws_bytes = 0;
};

struct Plan {
  std::vector<Step> steps;
  void* arena = nullptr;
  size_t arena_bytes = 0;
  std::vector<int> first_step, last_step;  // per layer (steps of a layer are contiguous)
  std::vector<BufRef> layer_out;           // per layer: where its routine stores its output
  std::vector<hipEvent_t> ev;              // timed runs: 2 per layer
  hipStream_t gstream = nullptr;           // stream the captured graph replays on
  hipGraphExec_t gexec = nullptr;
  hipGraph_t graph = nullptr;
  std::vector<const void*> g_in;           // the user tensors the captured graph was made for
  std::vector<void*> g_out;
  hipEvent_t gev[2] = {nullptr, nullptr};
};

Graph::Graph() = default;
Graph::~Graph() = default;

// ------------------------------------------------------------------ helpers
static k::TDesc tdesc(const Shape& s, int layout) {
  return k::TDesc{s.n, s.c, s.h, s.w, stored_c(s, layout), layout};
}

static double decode(const uint8_t* p, int dtype) {
  if (dtype == SN_F32) {
    float f;
    std::memcpy(&f, p, 4);
    return f;
  }
  uint16_t b;
  std::memcpy(&b, p, 2);
  if (dtype == SN_F16) {
    _Float16 h;
    std::memcpy(&h, &b, 2);
    return (double)h;
  }
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

static void encode(double v, int dtype, uint8_t* p) {
  if (dtype == SN_F32) {
    float f = (float)v;
    std::memcpy(p, &f, 4);
  } else if (dtype == SN_F16) {
    _Float16 h = (_Float16)v;  // one rounding, nearest-even
    std::memcpy(p, &h, 2);
  } else {
    __bf16 b = (__bf16)v;      // one rounding, nearest-even
    std::memcpy(p, &b, 2);
  }
}

static void* dev_upload(const void* host, size_t bytes) {
  void* d = nullptr;
  HIPCHK(hipMalloc(&d, std::max<size_t>(bytes, 256)));
  HIPCHK(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

static bool is_depthwise(const Graph& g, const Layer& L) {
  return L.type == SN_LAYER_CONV2D && L.d.groups > 1;
}

// ------------------------------------------------------------------ lifetime
void dev_create(Graph& g) {
  int n = 0;
  HIPCHK(hipGetDeviceCount(&n));
  if (g.device >= n) fail(SN_E_DEVICE, "no such HIP device");
  HIPCHK(hipSetDevice(g.device));
  g.dev.reset(new DevState);
  g.dev->device = g.device;
  g.dev->L.resize(1);
  // the tile counters of split-reduction launches: zero here, and every such
  // launch leaves them at zero
  HIPCHK(hipMalloc(&g.dev->fixup_cnt, k::kFixupMaxTiles * sizeof(unsigned)));
  HIPCHK(hipMemset(g.dev->fixup_cnt, 0, k::kFixupMaxTiles * sizeof(unsigned)));
  HIPCHK(hipDeviceSynchronize());
}

void plan_destroy(Graph& g) {
  if (!g.plan) return;
  Plan& p = *g.plan;
  if (p.gexec) (void)hipGraphExecDestroy(p.gexec);
  if (p.graph) (void)hipGraphDestroy(p.graph);
  for (auto e : p.ev) (void)hipEventDestroy(e);
  for (auto e : p.gev)
    if (e) (void)hipEventDestroy(e);
  if (p.gstream) (void)hipStreamDestroy(p.gstream);
  if (p.arena) (void)hipFree(p.arena);
  g.plan.reset();
}

void dev_destroy(Graph& g) {
  if (!g.dev) return;
  (void)hipSetDevice(g.dev->device);
  for (auto& d : g.dev->L) {
    for (void* p : d.w)
      if (p) (void)hipFree(p);
    for (void* p : d.wu)
      if (p) (void)hipFree(p);
    for (void* p : d.wu4)
      if (p) (void)hipFree(p);
    for (void* p : d.wp)
      if (p) (void)hipFree(p);
    for (void* p : d.wcat)
      if (p) (void)hipFree(p);
    if (d.bias) (void)hipFree(d.bias);
    if (d.zbias) (void)hipFree(d.zbias);
  }
  if (g.dev->fixup_cnt) (void)hipFree(g.dev->fixup_cnt);
  g.dev.reset();
}

// Prepared weight formats (see kernels/launch.hpp), one copy per allowed
// dtype: the caller's weights (run dtype) are decoded exactly and rounded
// once to each dtype.
void dev_upload_layer(Graph& g, int id) {
  HIPCHK(hipSetDevice(g.device));
  DevState& D = *g.dev;
  D.L.resize(g.n_layers());
  Layer& L = g.layers[id];
  DevLayer& dl = D.L[id];
  if (L.weight.empty()) return;
  const int ies = dtype_size(g.dtype);
  const Shape& in = g.layers[L.inputs[0]].out;
  const int K = L.out.c, Kp = round8(K), C = in.c, C8 = round8(C);
  std::vector<float> bias(Kp, 0.f);
  std::copy(L.bias.begin(), L.bias.end(), bias.begin());
  if (L.proj_stride > 0) {  // the two biases, summed in float64 and rounded once
    for (int kk = 0; kk < K; ++kk) bias[kk] = (float)((double)L.bias[kk] + (double)L.bproj[kk]);
    std::vector<float> z(Kp, 0.f);
    dl.zbias = static_cast<float*>(dev_upload(z.data(), z.size() * 4));
  }
  dl.bias = static_cast<float*>(dev_upload(bias.data(), bias.size() * 4));
  const uint8_t* src = L.weight.data();
  const int R = L.d.r, S = L.d.s;
  for (int dt = 0; dt < 3; ++dt) {
    if (!(g.opt_dtypes >> dt & 1)) continue;
    const int es = dtype_size(dt);
    // element e of the caller's weights, in dtype dt
    auto put = [&](uint8_t* dst, size_t e) {
      if (dt == g.dtype) std::memcpy(dst, src + e * ies, ies);
      else encode(decode(src + e * ies, g.dtype), dt, dst);
    };
    if (L.type == SN_LAYER_FC) {
      std::vector<uint8_t> w((size_t)Kp * C8 * es, 0);
      for (int kk = 0; kk < K; ++kk)
        for (int c = 0; c < C; ++c) put(&w[((size_t)kk * C8 + c) * es], (size_t)kk * C + c);
      dl.w[dt] = dev_upload(w.data(), w.size());
      continue;
    }
    if (is_depthwise(g, L)) {  // OIHW [C][1][R][S] -> [R][S][C8]
      std::vector<uint8_t> w((size_t)R * S * C8 * es, 0);
      for (int c = 0; c < C; ++c)
        for (int r = 0; r < R; ++r)
          for (int s2 = 0; s2 < S; ++s2)
            put(&w[(((size_t)r * S + s2) * C8 + c) * es], ((size_t)c * R + r) * S + s2);
      dl.w[dt] = dev_upload(w.data(), w.size());
      continue;
    }
    // dense OIHW [K][C][R][S] -> [Kp][R][S][C8]
    std::vector<uint8_t> w((size_t)Kp * R * S * C8 * es, 0);
    for (int kk = 0; kk < K; ++kk)
      for (int c = 0; c < C; ++c)
        for (int r = 0; r < R; ++r)
          for (int s2 = 0; s2 < S; ++s2)
            put(&w[((((size_t)kk * R + r) * S + s2) * C8 + c) * es], (((size_t)kk * C + c) * R + r) * S + s2);
    dl.w[dt] = dev_upload(w.data(), w.size());
    if (L.proj_stride > 0) {  // shortcut [K][C2] -> [Kp][C2_8]
      const int C2 = g.layers[L.inputs[1]].out.c, C28 = round8(C2);
      std::vector<uint8_t> w2((size_t)Kp * C28 * es, 0);
      for (int kk = 0; kk < K; ++kk)
        for (int c = 0; c < C2; ++c) {
          const size_t e = (size_t)kk * C2 + c;
          if (dt == g.dtype) std::memcpy(&w2[((size_t)kk * C28 + c) * es], L.wproj.data() + e * ies, ies);
          else encode(decode(L.wproj.data() + e * ies, g.dtype), dt, &w2[((size_t)kk * C28 + c) * es]);
        }
      dl.wp[dt] = dev_upload(w2.data(), w2.size());
      if (R == 1 && S == 1 && C % 64 == 0 && C2 % 64 == 0) {  // the streaming kernel's filter rows
        std::vector<uint8_t> wc((size_t)Kp * (C + C2) * es);
        for (int kk = 0; kk < Kp; ++kk) {
          std::memcpy(&wc[(size_t)kk * (C + C2) * es], &w[(size_t)kk * C * es], (size_t)C * es);
          std::memcpy(&wc[((size_t)kk * (C + C2) + C) * es], &w2[(size_t)kk * C2 * es], (size_t)C2 * es);
        }
        dl.wcat[dt] = dev_upload(wc.data(), wc.size());
      }
    }
    if (winograd_applicable(L, in)) {
      // U = G g G^T per (k, c), in float64 from the caller's weights, rounded
      // once to the dtype
      static const double G[4][3] = {{1, 0, 0}, {0.5, 0.5, 0.5}, {0.5, -0.5, 0.5}, {0, 0, 1}};
      std::vector<uint8_t> u((size_t)16 * Kp * C8 * es, 0);
      for (int kk = 0; kk < K; ++kk)
        for (int c = 0; c < C; ++c) {
          double gg[3][3], t[4][3];
          for (int r = 0; r < 3; ++r)
            for (int s2 = 0; s2 < 3; ++s2)
              gg[r][s2] = decode(src + ((((size_t)kk * C + c) * 3 + r) * 3 + s2) * ies, g.dtype);
          for (int i = 0; i < 4; ++i)
            for (int s2 = 0; s2 < 3; ++s2) t[i][s2] = G[i][0] * gg[0][s2] + G[i][1] * gg[1][s2] + G[i][2] * gg[2][s2];
          for (int i = 0; i < 4; ++i)
            for (int j = 0; j < 4; ++j) {
              double v = t[i][0] * G[j][0] + t[i][1] * G[j][1] + t[i][2] * G[j][2];
              encode(v, dt, &u[(((size_t)(i * 4 + j) * Kp + kk) * C8 + c) * es]);
            }
        }
      dl.wu[dt] = dev_upload(u.data(), u.size());
      // F(4x4,3x3): G of the Toom-Cook construction on 0, 1, -1, 2, -2, infinity
      static const double G4[6][3] = {{1.0 / 4, 0, 0},
                                      {-1.0 / 6, -1.0 / 6, -1.0 / 6},
                                      {-1.0 / 6, 1.0 / 6, -1.0 / 6},
                                      {1.0 / 24, 1.0 / 12, 1.0 / 6},
                                      {1.0 / 24, -1.0 / 12, 1.0 / 6},
                                      {0, 0, 1}};
      std::vector<uint8_t> u4((size_t)36 * Kp * C8 * es, 0);
      for (int kk = 0; kk < K; ++kk)
        for (int c = 0; c < C; ++c) {
          double gg[3][3], t[6][3];
          for (int r = 0; r < 3; ++r)
            for (int s2 = 0; s2 < 3; ++s2)
              gg[r][s2] = decode(src + ((((size_t)kk * C + c) * 3 + r) * 3 + s2) * ies, g.dtype);
          for (int i = 0; i < 6; ++i)
            for (int s2 = 0; s2 < 3; ++s2)
              t[i][s2] = G4[i][0] * gg[0][s2] + G4[i][1] * gg[1][s2] + G4[i][2] * gg[2][s2];
          for (int i = 0; i < 6; ++i)
            for (int j = 0; j < 6; ++j) {
              double v = t[i][0] * G4[j][0] + t[i][1] * G4[j][1] + t[i][2] * G4[j][2];
              encode(v, dt, &u4[(((size_t)(i * 6 + j) * Kp + kk) * C8 + c) * es]);
            }
        }
      dl.wu4[dt] = dev_upload(u4.data(), u4.size());
    }
  }
}

// ------------------------------------------------------------------ launching
size_t routine_ws_bytes(const Graph& g, const Layer& L, const Routine& r) {
  if (L.inputs.empty()) return 0;  // the input layer
  const Shape& in = g.layers[L.inputs[0]].out;
  if (L.type == SN_LAYER_FC && r.algo == SN_ALGO_IGEMM)
    return k::igemm_ws_bytes(r.dtype, r.param, tdesc(in, r.layout), tdesc(L.out, r.layout), 1, 1);
  if (L.type != SN_LAYER_CONV2D || L.d.groups > 1) return 0;
  if (L.proj_stride > 0) {
    if (r.algo == SN_ALGO_DIRECT)  // the shortcut's projection, stored in the output's schema
      return align256((size_t)stored_numel(L.out, r.layout) * dtype_size(r.dtype));
    return k::igemm_ws_bytes(r.dtype, r.param, tdesc(in, r.layout), tdesc(L.out, r.layout), L.d.r, L.d.s,
                             g.layers[L.inputs[1]].out.c);
  }
  if (r.algo == SN_ALGO_WINOGRAD) {  // the fused routines keep their transforms on chip
    if (r.param == 0) return k::winograd_ws_bytes(r.dtype, tdesc(in, r.layout), L.out.c, 2);
    if (r.param == k::winograd_f4_param()) return k::winograd_ws_bytes(r.dtype, tdesc(in, r.layout), L.out.c, 4);
    return 0;
  }
  if (r.algo == SN_ALGO_IGEMM)
    return k::igemm_ws_bytes(r.dtype, r.param, tdesc(in, r.layout), tdesc(L.out, r.layout), L.d.r, L.d.s);
  return 0;
}

// sub >= 0 launches only that sub-layer of a childnet routine, with
// sub-routine sub_routine (unit profiling of the childnet's sub-routines)
static void launch_layer(const Graph& g, int id, const Routine& r, const void* const* in,
                         const k::TDesc* ind, void* out, const k::TDesc& outd, void* ws,
                         size_t ws_bytes, hipStream_t st, int sub = -1, int sub_routine = 0) {
  const Layer& L = g.layers[id];
  const DevLayer& dl = g.dev->L[id];
  const int dt = r.dtype;
  switch (L.type) {
    case SN_LAYER_CONV2D: {
      k::ConvArgs a{};
      a.x = in[0];
      a.xd = ind[0];
      a.w = r.algo != SN_ALGO_WINOGRAD ? dl.w[dt] : r.param == k::winograd_f4_param() ? dl.wu4[dt] : dl.wu[dt];
      a.bias = dl.bias;
      a.y = out;
      a.yd = outd;
      a.r = L.d.r;
      a.s = L.d.s;
      a.stride = L.d.stride;
      a.pad = L.d.pad;
      a.act = L.d.act;
      a.ws = ws;
      a.ws_bytes = ws_bytes;
      a.cnt = g.dev->fixup_cnt;
      a.res = L.inputs.size() > 1 ? in[1] : nullptr;
      if (L.proj_stride > 0) {
        a.res = nullptr;
        if (r.algo == SN_ALGO_DIRECT) {
          // two launches: the shortcut's 1 x 1 projection (bias zero, no
          // activation) into the workspace, then the convolution adding it
          k::ConvArgs p = a;
          p.x = in[1];
          p.xd = ind[1];
          p.w = dl.wp[dt];
          p.bias = dl.zbias;
          p.y = ws;
          p.r = p.s = 1;
          p.stride = L.proj_stride;
          p.pad = 0;
          p.act = SN_ACT_NONE;
          p.ws = nullptr;
          p.ws_bytes = 0;
          k::conv_direct(dt, p, st);
          a.res = ws;
          a.ws = nullptr;
          a.ws_bytes = 0;
          k::conv_direct(dt, a, st);
        } else {
          a.x2 = in[1];
          a.x2d = ind[1];
          a.w2 = dl.wp[dt];
          a.wcat = dl.wcat[dt];
          a.stride2 = L.proj_stride;
          k::conv_igemm(dt, r.param, a, st);
        }
        break;
      }
      if (L.d.groups > 1) {
        k::dwconv(dt, a, r.param, st);
      } else if (r.algo == SN_ALGO_DIRECT) {
        k::conv_direct(dt, a, st);
      } else if (r.algo == SN_ALGO_IGEMM) {
        k::conv_igemm(dt, r.param, a, st);
      } else if (r.param == 0 || r.param == k::winograd_f4_param()) {  // childnet wgenc -> wgconv -> wgdec
        const int tile = r.param == 0 ? 2 : 4;
        if (sub >= 0) {
          k::winograd_sub(dt, tile, sub, sub_routine, a, st);
        } else {
          const ChildNet& cn = L.child[r.id];
          k::conv_winograd(dt, tile, a, cn.path.size() > 1 ? cn.path[1] : 0, st);
        }
      } else {
        k::conv_wino_fused(dt, r.param - 1, a, st);
      }
      break;
    }
    case SN_LAYER_MAXPOOL:
      k::maxpool(dt, in[0], ind[0], out, outd, L.d.r, L.d.stride, L.d.pad, st);
      break;
    case SN_LAYER_GAP:
      k::gap(dt, in[0], ind[0], out, outd, st);
      break;
    case SN_LAYER_ADD: {
      const Shape& s = L.out;
      k::add_act(dt, in[0], in[1], out, stored_numel(s, r.layout), L.d.act, st);
      break;
    }
    case SN_LAYER_FC: {
      const Shape& xs = g.layers[L.inputs[0]].out;
      if (r.algo == SN_ALGO_IGEMM) {  // dense childnet: 1x1 convolution
        k::ConvArgs a{};
        a.x = in[0];
        a.xd = ind[0];
        a.w = dl.w[dt];
        a.bias = dl.bias;
        a.y = out;
        a.yd = outd;
        a.r = a.s = 1;
        a.stride = 1;
        a.pad = 0;
        a.act = L.d.act;
        a.ws = ws;
        a.ws_bytes = ws_bytes;
        a.cnt = g.dev->fixup_cnt;
        k::conv_igemm(dt, r.param, a, st);
      } else {
        k::fc_direct(dt, in[0], xs.n, xs.c, stored_c(xs, r.layout), dl.w[dt], round8(xs.c), dl.bias, out,
                     L.out.c, stored_c(L.out, r.layout), L.d.act, st);
      }
      break;
    }
    default:
      fail(SN_E_INTERNAL, "no launcher for layer type");
  }
}

// ------------------------------------------------------------------ profiling
void dev_profile(Graph& g, int warmup, int reps, void* stream) {
  HIPCHK(hipSetDevice(g.device));
  hipStream_t st = static_cast<hipStream_t>(stream);
  DevState& D = *g.dev;
  // scratch sized for the largest tensor of any schema and the largest workspace
  int es_max = 2;
  for (int d = 0; d < 3; ++d)
    if (g.opt_dtypes >> d & 1 || d == g.dtype) es_max = std::max(es_max, dtype_size(d));
  size_t tmax = 0, wsmax = 0;
  for (const Layer& L : g.layers) {
    for (int l = 0; l < SN_NUM_LAYOUTS; ++l) tmax = std::max(tmax, (size_t)stored_numel(L.out, l) * es_max);
    for (const Routine& r : L.routines) wsmax = std::max(wsmax, routine_ws_bytes(g, L, r));
  }
  tmax = align256(tmax);
  void *in0 = nullptr, *in1 = nullptr, *outb = nullptr, *ws = nullptr, *flush = nullptr;
  std::vector<hipEvent_t> ev(2, nullptr);
  auto cleanup = [&]() {
    for (auto e : ev)
      if (e) (void)hipEventDestroy(e);
    for (void* p : {in0, in1, outb, ws, flush})
      if (p) (void)hipFree(p);
  };
  // cache-cold mode: costs are keyed apart from the warm ones
  const std::string mode_key = g.opt_flush > 0 ? "|cold" + std::to_string(g.opt_flush) : std::string();
  try {
    HIPCHK(hipMalloc(&in0, tmax));
    HIPCHK(hipMalloc(&in1, tmax));
    HIPCHK(hipMalloc(&outb, tmax));
    if (wsmax) HIPCHK(hipMalloc(&ws, wsmax));
    if (g.opt_flush > 0) HIPCHK(hipMalloc(&flush, (size_t)g.opt_flush));
    for (auto& e : ev) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
    // operands hold values of the dtype being timed (refilled when it changes)
    int filled = -1;
    auto fill = [&](int dt) {
      if (dt == filled) return;
      k::fill_random(dt, in0, tmax / dtype_size(dt), (uint64_t)g.opt_seed, st);
      k::fill_random(dt, in1, tmax / dtype_size(dt), (uint64_t)g.opt_seed + 7, st);
      HIPCHK(hipGetLastError());
      filled = dt;
    };
    struct Clear {
      ~Clear() { k::g_timing = k::LaunchTiming{}; }
    } clear_on_exit;
    // a routine's cost is the mean time of reps back-to-back runs: events
    // are tied to the start of the first run's first kernel and to the end
    // of the last run's last kernel, so host launch latency and the events'
    // own dispatch gaps are amortised over the block
    //
    // cache-cold mode (SN_OPT_FLUSH > 0): before each run an untimed kernel
    // writes the flush buffer, evicting the operands and weights from the
    // caches; each run is timed on its own and the cost is the median
    auto time_cold = [&](auto&& launch) -> int64_t {
      for (int i = 0; i < warmup; ++i) launch();
      std::vector<float> t(reps);
      for (int i = 0; i < reps; ++i) {
        k::fill_random(SN_F32, flush, g.opt_flush / 4, (uint64_t)i, st);
        k::g_timing = k::LaunchTiming{ev[0], ev[1]};
        launch();
        k::g_timing = k::LaunchTiming{};
        HIPCHK(hipGetLastError());
        HIPCHK(hipEventSynchronize(ev[1]));
        HIPCHK(hipEventElapsedTime(&t[i], ev[0], ev[1]));
      }
      std::nth_element(t.begin(), t.begin() + reps / 2, t.end());
      return std::max<int64_t>(1, (int64_t)std::llround((double)t[reps / 2] * 1e6));
    };
    auto time_it = [&](auto&& launch) -> int64_t {
      if (flush) return time_cold(launch);
      for (int i = 0; i < warmup; ++i) launch();
      for (int i = 0; i < reps; ++i) {
        k::g_timing = k::LaunchTiming{i == 0 ? ev[0] : nullptr, i == reps - 1 ? ev[1] : nullptr};
        launch();
        k::g_timing = k::LaunchTiming{};
      }
      HIPCHK(hipGetLastError());
      HIPCHK(hipEventSynchronize(ev[1]));
      float ms = 0.f;
      HIPCHK(hipEventElapsedTime(&ms, ev[0], ev[1]));
      return (int64_t)std::llround((double)ms * 1e6 / reps);
    };
    for (int i = 1; i < g.n_layers(); ++i) {
      Layer& L = g.layers[i];
      if (L.type == SN_LAYER_INPUT) continue;  // a net input: its one routine costs 0
      for (size_t ri = 0; ri < L.routines.size(); ++ri) {
        const Routine& r = L.routines[ri];
        ChildNet& cn = L.child[ri];
        if (!cn.empty()) {
          // a childnet: every sub-routine is profiled on its own, and the
          // routine's time is the DPRS optimum over the sub-layers
          fill(r.dtype);
          const void* ins[2] = {in0, in1};
          k::TDesc ind[2];
          for (size_t q = 0; q < L.inputs.size(); ++q) ind[q] = tdesc(g.layers[L.inputs[q]].out, r.layout);
          const k::TDesc od = tdesc(L.out, r.layout);
          const size_t wsb = routine_ws_bytes(g, L, r);
          for (size_t sl = 0; sl < cn.layer.size(); ++sl)
            for (size_t q = 0; q < cn.routine[sl].size(); ++q) {
              const std::string skey = L.signature + "|" + r.name + "|" + cn.layer[sl] + "/" + cn.routine[sl][q] + mode_key;
              auto it = D.cost_cache.find(skey);
              if (it == D.cost_cache.end()) {
                const int64_t ns =
                    time_it([&] { launch_layer(g, i, r, ins, ind, outb, od, ws, wsb, st, (int)sl, (int)q); });
                it = D.cost_cache.emplace(skey, ns).first;
              }
              cn.cost[sl][q] = it->second;
            }
          L.cost[ri] = childnet_select(cn);
          continue;
        }
        std::string key = L.signature + "|" + r.name + mode_key;
        auto it = D.cost_cache.find(key);
        if (it != D.cost_cache.end()) {
          L.cost[ri] = it->second;
          continue;
        }
        fill(r.dtype);
        const void* ins[2] = {in0, in1};
        k::TDesc ind[2];
        for (size_t q = 0; q < L.inputs.size(); ++q) ind[q] = tdesc(g.layers[L.inputs[q]].out, r.layout);
        k::TDesc od = tdesc(L.out, r.layout);
        size_t wsb = routine_ws_bytes(g, L, r);
        int64_t ns = time_it([&] { launch_layer(g, i, r, ins, ind, outb, od, ws, wsb, st); });
        D.cost_cache[key] = ns;
        L.cost[ri] = ns;
      }
    }
    // adapt costs: every ordered pair of allowed schemas on every edge
    auto edge_costs = [&](Edge& e, const Shape& s) {
      for (int a = 0; a < kNumSchemas; ++a)
        for (int b = 0; b < kNumSchemas; ++b) {
          if (a == b) {
            e.adapt[a][b] = 0;
            continue;
          }
          if (!g.schema_allowed(a) || !g.schema_allowed(b)) {
            e.adapt[a][b] = -1;
            continue;
          }
          if (schemas_equivalent(s, a, b)) {
            e.adapt[a][b] = 0;  // identical bytes: void adapt
            continue;
          }
          std::string key = "cvt|" + std::to_string(s.n) + "," + std::to_string(s.c) + "," +
                            std::to_string(s.h) + "," + std::to_string(s.w) + "|" +
                            std::to_string(a) + ">" + std::to_string(b) + mode_key;
          auto it = D.cost_cache.find(key);
          if (it == D.cost_cache.end()) {
            fill(schema_dtype(a));
            k::TDesc sd = tdesc(s, schema_layout(a)), dd = tdesc(s, schema_layout(b));
            int64_t ns = time_it([&] { k::convert_cast(schema_dtype(a), in0, sd, schema_dtype(b), outb, dd, st); });
            it = D.cost_cache.emplace(key, ns).first;
          }
          e.adapt[a][b] = it->second;
        }
    };
    for (Edge& e : g.edges)
      if (g.layers[e.to].type != SN_LAYER_INPUT) edge_costs(e, g.layers[e.from].out);
    const std::vector<int> outs = net_outputs(g);
    g.out_edges.resize(outs.size());
    for (size_t k2 = 0; k2 < outs.size(); ++k2) edge_costs(g.out_edges[k2], g.layers[outs[k2]].out);
    HIPCHK(hipStreamSynchronize(st));
  } catch (...) {
    cleanup();
    throw;
  }
  cleanup();
}

// ------------------------------------------------------------------ plan
void plan_compile(Graph& g) {
  HIPCHK(hipSetDevice(g.device));
  plan_destroy(g);
  std::unique_ptr<Plan> P(new Plan);
  const int n = g.n_layers();
  const std::vector<int> outs = net_outputs(g);
  const int io_schema = schema_of(g.dtype, SN_NCHW);
  struct Buf {
    size_t bytes;
    int def, last;
    size_t off;
  };
  std::vector<Buf> bufs;
  // with opt_keep every buffer lives to the end of the plan (nothing shares
  // bytes), so every layer's stored output can be read after a run
  const int never = g.opt_keep ? INT32_MAX : -1;
  auto new_buf = [&](size_t bytes, int def) {
    bufs.push_back(Buf{align256(bytes), def, std::max(def, never), 0});
    return (int)bufs.size() - 1;
  };
  auto schema_bytes = [&](const Shape& sh, int sc) {
    return (size_t)stored_numel(sh, schema_layout(sc)) * dtype_size(schema_dtype(sc));
  };
  // output tensor of each layer: kind/buffer index
  std::vector<int> out_buf(n, -1);  // -1 = a user tensor
  std::vector<BufRef> out_ref(n);
  std::vector<std::vector<int>> step_bufs;
  out_ref[0].kind = 1;
  P->first_step.assign(n, -1);
  P->last_step.assign(n, -1);
  auto push = [&](Step s, std::vector<int> uses) {
    int idx = (int)P->steps.size();
    if (P->first_step[s.layer] < 0) P->first_step[s.layer] = idx;
    P->last_step[s.layer] = idx;
    for (int b : uses) bufs[b].last = std::max(bufs[b].last, idx);
    P->steps.push_back(s);
    step_bufs.push_back(uses);
  };
  for (int i = 1; i < n; ++i) {
    const Layer& L = g.layers[i];
    if (L.type == SN_LAYER_INPUT) {  // a further net input: the caller's tensor
      out_ref[i].kind = 1;
      out_ref[i].idx = (int)(std::find(g.net_inputs.begin(), g.net_inputs.end(), i) - g.net_inputs.begin());
      continue;
    }
    const Routine& r = L.routines[g.path[i]];
    const int rs = r.schema();
    Step s;
    s.type = 1;
    s.layer = i;
    s.n_in = (int)L.inputs.size();
    std::vector<int> uses;
    for (int q = 0; q < s.n_in; ++q) {
      const int j = L.inputs[q];
      const Shape& js = g.layers[j].out;
      const int sj = g.layers[j].routines[g.path[j]].schema();
      s.ind[q] = tdesc(js, r.layout);
      if (schemas_equivalent(js, sj, rs)) {
        s.in[q] = out_ref[j];
        if (out_buf[j] >= 0) uses.push_back(out_buf[j]);
      } else {
        Step c;
        c.type = 0;
        c.layer = i;
        c.src = out_ref[j];
        c.sd = tdesc(js, schema_layout(sj));
        c.dd = tdesc(js, r.layout);
        c.sdt = schema_dtype(sj);
        c.ddt = r.dtype;
        const int step_idx = (int)P->steps.size();
        int b = new_buf(schema_bytes(js, rs), step_idx);
        c.dst.kind = 0;
        c.dst.off = (size_t)b;  // buffer id; resolved to an offset below
        std::vector<int> cu{b};
        if (out_buf[j] >= 0) cu.push_back(out_buf[j]);
        push(c, cu);
        s.in[q] = c.dst;
        uses.push_back(b);
        // a timed run repeats the converter after the layer's routine: its
        // source must outlive the routine, so the routine's output never
        // takes the source's bytes
        if (out_buf[j] >= 0) uses.push_back(out_buf[j]);
      }
    }
    s.outd = tdesc(L.out, r.layout);
    const int out_k = (int)(std::find(outs.begin(), outs.end(), i) - outs.begin());
    const bool is_out = out_k < (int)outs.size();
    const int step_idx = (int)P->steps.size();
    if (is_out && schemas_equivalent(L.out, rs, io_schema)) {
      s.out.kind = 2;  // straight into the caller's output tensor
      s.out.idx = out_k;
    } else {
      int b = new_buf(schema_bytes(L.out, rs), step_idx);
      out_buf[i] = b;
      s.out.kind = 0;
      s.out.off = (size_t)b;
      uses.push_back(b);
    }
    s.ws_bytes = routine_ws_bytes(g, L, r);
    if (s.ws_bytes) {
      int b = new_buf(s.ws_bytes, step_idx);
      s.ws.kind = 0;
      s.ws.off = (size_t)b;
      uses.push_back(b);
    }
    out_ref[i] = s.out;
    push(s, uses);
    if (is_out && s.out.kind != 2) {  // adapt into the caller's NCHW output (run dtype)
      Step c;
      c.type = 0;
      c.layer = i;
      c.src = s.out;
      c.sd = s.outd;
      c.dd = tdesc(L.out, SN_NCHW);
      c.sdt = r.dtype;
      c.ddt = g.dtype;
      c.dst.kind = 2;
      c.dst.idx = out_k;
      push(c, {out_buf[i]});
    }
  }
  // first-fit offsets, largest buffers first; buffers whose step ranges
  // overlap never share bytes
  std::vector<int> order(bufs.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
  std::sort(order.begin(), order.end(), [&](int a, int b) {
    return bufs[a].bytes != bufs[b].bytes ? bufs[a].bytes > bufs[b].bytes : a < b;
  });
  std::vector<int> placed;
  size_t total = 0;
  for (int b : order) {
    std::vector<std::pair<size_t, size_t>> busy;
    for (int o : placed)
      if (!(bufs[o].last < bufs[b].def || bufs[b].last < bufs[o].def))
        busy.push_back({bufs[o].off, bufs[o].off + bufs[o].bytes});
    std::sort(busy.begin(), busy.end());
    size_t off = 0;
    for (auto& iv : busy) {
      if (off + bufs[b].bytes <= iv.first) break;
      off = std::max(off, iv.second);
    }
    bufs[b].off = off;
    total = std::max(total, off + bufs[b].bytes);
    placed.push_back(b);
  }
  auto resolve = [&](BufRef& r) {
    if (r.kind == 0) r.off = bufs[r.off].off;
  };
  for (Step& s : P->steps) {
    if (s.type == 0) {
      resolve(s.src);
      resolve(s.dst);
    } else {
      for (int q = 0; q < s.n_in; ++q) resolve(s.in[q]);
      resolve(s.out);
      if (s.ws_bytes) resolve(s.ws);
    }
  }
  P->layer_out = out_ref;
  for (BufRef& r : P->layer_out) resolve(r);
  P->arena_bytes = std::max<size_t>(total, 256);
  HIPCHK(hipMalloc(&P->arena, P->arena_bytes));
  P->ev.resize(2 * n, nullptr);
  for (auto& e : P->ev) HIPCHK(hipEventCreateWithFlags(&e, hipEventDisableSystemFence));
  g.plan = std::move(P);
}

static void enqueue_step(const Graph& g, const Plan& P, char* base, const Step& s, const void* const* d_in,
                         void* const* d_out, hipStream_t st) {
  auto ptr = [&](const BufRef& r) -> void* {
    if (r.kind == 1) return const_cast<void*>(d_in[r.idx]);
    if (r.kind == 2) return d_out[r.idx];
    return base + r.off;
  };
  if (s.type == 0) {
    k::convert_cast(s.sdt, ptr(s.src), s.sd, s.ddt, ptr(s.dst), s.dd, st);
  } else {
    const Routine& r = g.layers[s.layer].routines[g.path[s.layer]];
    const void* ins[2] = {ptr(s.in[0]), s.n_in > 1 ? ptr(s.in[1]) : nullptr};
    launch_layer(g, s.layer, r, ins, s.ind, ptr(s.out), s.outd, s.ws_bytes ? ptr(s.ws) : nullptr,
                 s.ws_bytes, st);
  }
}

static void enqueue_steps(const Graph& g, const Plan& P, char* base, const void* const* d_in,
                          void* const* d_out, hipStream_t st) {
  for (const Step& s : P.steps) enqueue_step(g, P, base, s, d_in, d_out, st);
  HIPCHK(hipGetLastError());
}

// Timed run: each layer's steps (converters feeding it, then its routine) are
// enqueued reps times back to back, with events tied to the start of the
// first repetition's first kernel and the end of the last repetition's last
// kernel.  Every step writes buffers distinct from the ones it reads, so a
// repetition recomputes the same values and the run's result is unchanged.
static void enqueue_timed(const Graph& g, const Plan& P, const void* const* d_in, void* const* d_out,
                          hipStream_t st, int reps, void* flush, int64_t flush_bytes) {
  struct Clear {
    ~Clear() { k::g_timing = k::LaunchTiming{}; }
  } clear_on_exit;
  for (int i = 1; i < g.n_layers(); ++i) {
    const int a = P.first_step[i], b = P.last_step[i];
    if (a < 0) continue;  // a net input: nothing runs
    if (flush) {  // untimed: evict the caches before the layer
      k::g_timing = k::LaunchTiming{};
      k::fill_random(SN_F32, flush, flush_bytes / 4, (uint64_t)i, st);
    }
    for (int rep = 0; rep < reps; ++rep)
      for (int si = a; si <= b; ++si) {
        k::g_timing = k::LaunchTiming{rep == 0 && si == a ? P.ev[2 * i] : nullptr,
                                      rep == reps - 1 && si == b ? P.ev[2 * i + 1] : nullptr};
        enqueue_step(g, P, static_cast<char*>(P.arena), P.steps[si], d_in, d_out, st);
      }
  }
  k::g_timing = k::LaunchTiming{};
  HIPCHK(hipGetLastError());
}

void plan_run(Graph& g, const void* const* d_in, void* const* d_out, void* stream, float* layer_ms, int reps) {
  if (!g.plan) fail(SN_E_STATE, "no execution plan");
  HIPCHK(hipSetDevice(g.device));
  Plan& P = *g.plan;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (layer_ms) {
    void* flush = nullptr;
    if (g.opt_flush > 0) HIPCHK(hipMalloc(&flush, (size_t)g.opt_flush));
    try {
      enqueue_timed(g, P, d_in, d_out, st, reps, flush, g.opt_flush);
      HIPCHK(hipStreamSynchronize(st));
    } catch (...) {
      if (flush) (void)hipFree(flush);
      throw;
    }
    if (flush) HIPCHK(hipFree(flush));
    layer_ms[0] = 0.f;
    for (int i = 1; i < g.n_layers(); ++i) {
      layer_ms[i] = 0.f;
      if (P.first_step[i] < 0) continue;
      HIPCHK(hipEventElapsedTime(&layer_ms[i], P.ev[2 * i], P.ev[2 * i + 1]));
      layer_ms[i] /= (float)reps;
    }
    return;
  }
  if (!g.opt_hipgraph) {
    enqueue_steps(g, P, static_cast<char*>(P.arena), d_in, d_out, st);
    return;
  }
  // replay a captured graph on the plan's stream, ordered after/before the caller's stream
  if (!P.gstream) {
    HIPCHK(hipStreamCreateWithFlags(&P.gstream, hipStreamNonBlocking));
    HIPCHK(hipEventCreateWithFlags(&P.gev[0], hipEventDisableTiming));
    HIPCHK(hipEventCreateWithFlags(&P.gev[1], hipEventDisableTiming));
  }
  const std::vector<const void*> ins(d_in, d_in + g.net_inputs.size());
  const std::vector<void*> outs(d_out, d_out + net_outputs(g).size());
  if (!P.gexec || P.g_in != ins || P.g_out != outs) {
    if (P.gexec) HIPCHK(hipGraphExecDestroy(P.gexec));
    if (P.graph) HIPCHK(hipGraphDestroy(P.graph));
    P.gexec = nullptr;
    P.graph = nullptr;
    HIPCHK(hipStreamBeginCapture(P.gstream, hipStreamCaptureModeThreadLocal));
    try {
      enqueue_steps(g, P, static_cast<char*>(P.arena), d_in, d_out, P.gstream);
    } catch (...) {
      hipGraph_t tmp = nullptr;
      (void)hipStreamEndCapture(P.gstream, &tmp);
      if (tmp) (void)hipGraphDestroy(tmp);
      throw;
    }
    HIPCHK(hipStreamEndCapture(P.gstream, &P.graph));
    HIPCHK(hipGraphInstantiate(&P.gexec, P.graph, nullptr, nullptr, 0));
    P.g_in = ins;
    P.g_out = outs;
  }
  HIPCHK(hipEventRecord(P.gev[0], st));
  HIPCHK(hipStreamWaitEvent(P.gstream, P.gev[0], 0));
  HIPCHK(hipGraphLaunch(P.gexec, P.gstream));
  HIPCHK(hipEventRecord(P.gev[1], P.gstream));
  HIPCHK(hipStreamWaitEvent(st, P.gev[1], 0));
}

// sn_run with the plan's intermediate tensors and workspaces placed in a
// caller-provided device region of cap bytes instead of the plan's own
// memory (same offsets, same launches, hence the same results).  Enqueues
// only kernel launches: no allocation, no memset.
void plan_run_in(const Graph& g, void* base, size_t cap, const void* const* d_in, void* const* d_out,
                 void* stream) {
  if (!g.plan) fail(SN_E_STATE, "no execution plan");
  const Plan& P = *g.plan;
  if (P.arena_bytes > cap)
    fail(SN_E_UNSUPPORTED, "the plan needs " + std::to_string(P.arena_bytes) +
                               " bytes of intermediate memory, more than the " + std::to_string(cap) +
                               " bytes of the static scratch region");
  HIPCHK(hipSetDevice(g.device));
  enqueue_steps(g, P, static_cast<char*>(base), d_in, d_out, static_cast<hipStream_t>(stream));
}

size_t plan_arena_bytes(const Graph& g) { return g.plan ? g.plan->arena_bytes : 0; }

// The layer each kernel launch of one sn_run belongs to, in launch order
// (converters feeding a layer count as the layer's).  The plan's steps are
// enqueued with launches counted, not issued, on placeholder addresses.
std::vector<int> plan_launch_layers(const Graph& g) {
  if (!g.plan) fail(SN_E_STATE, "no execution plan");
  const Plan& P = *g.plan;
  std::vector<const void*> ins(g.net_inputs.size(), reinterpret_cast<const void*>(uintptr_t(1) << 20));
  std::vector<void*> outs(net_outputs(g).size(), reinterpret_cast<void*>(uintptr_t(1) << 21));
  char* base = reinterpret_cast<char*>(uintptr_t(1) << 22);
  std::vector<int> layer_of;
  struct Restore {
    ~Restore() { k::g_count_only = 0; }
  } restore;
  k::g_count_only = 1;
  for (const Step& s : P.steps) {
    const long long before = k::g_launches;
    enqueue_step(g, P, base, s, ins.data(), outs.data(), nullptr);
    for (long long q = before; q < k::g_launches; ++q) layer_of.push_back(s.layer);
  }
  return layer_of;
}

// Copy of a layer's stored output (its routine's layout, channels padded as
// stored) out of the plan's arena; with opt_keep every layer's output
// survives the run.
void plan_layer_output(const Graph& g, int layer, void* d_dst, size_t cap, size_t* bytes,
                       int* layout, void* stream) {
  if (!g.plan) fail(SN_E_STATE, "no execution plan");
  if (layer < 1 || layer >= g.n_layers()) fail(SN_E_INVALID, "unknown layer (the input layer has no stored output)");
  const Plan& P = *g.plan;
  const Layer& L = g.layers[layer];
  if (L.type == SN_LAYER_INPUT) fail(SN_E_INVALID, "a net input layer has no stored output");
  const Routine& R = L.routines[g.path[layer]];
  const int lay = R.layout;
  const size_t b = (size_t)stored_numel(L.out, lay) * dtype_size(R.dtype);
  if (bytes) *bytes = b;
  if (layout) *layout = lay;
  if (!d_dst) return;
  if (cap < b) fail(SN_E_NOMEM, "destination smaller than the stored output");
  const BufRef& r = P.layer_out[layer];
  if (r.kind != 0) fail(SN_E_UNSUPPORTED, "the layer stores straight into the caller's output tensor");
  const std::vector<int> outs = net_outputs(g);
  if (!g.opt_keep && std::find(outs.begin(), outs.end(), layer) == outs.end())
    fail(SN_E_STATE, "intermediate outputs are kept only with SN_OPT_KEEP = 1");
  HIPCHK(hipSetDevice(g.device));
  HIPCHK(hipMemcpyAsync(d_dst, static_cast<char*>(P.arena) + r.off, b, hipMemcpyDeviceToDevice,
                        static_cast<hipStream_t>(stream)));
}

// ------------------------------------------------------------------ integrated profiling
// Every candidate path is compiled and run end to end on scratch tensors
// (zero-filled input): warmup runs, then two rounds (candidate order, then
// reverse order, so slow drift does not favour one end of the list) of reps
// back-to-back runs between HIP events; a candidate's time is the smaller of
// its two block means.  The fastest candidate (earliest on ties) is selected.
// Zero-filled scratch tensors for the net inputs and outputs, and a pair of
// HIP events, for timing whole paths; freed when it goes out of scope.
struct ScratchIO {
  std::vector<void*> din, dout;
  hipEvent_t ev[2] = {nullptr, nullptr};
  ScratchIO(const Graph& g, hipStream_t st) {
    const int es = dtype_size(g.dtype);
    const std::vector<int> outs = net_outputs(g);
    din.assign(g.net_inputs.size(), nullptr);
    dout.assign(outs.size(), nullptr);
    try {
      for (size_t q = 0; q < din.size(); ++q) {
        const size_t b = (size_t)g.layers[g.net_inputs[q]].out.numel() * es;
        HIPCHK(hipMalloc(&din[q], std::max<size_t>(b, 256)));
        HIPCHK(hipMemsetAsync(din[q], 0, b, st));
      }
      for (size_t q = 0; q < dout.size(); ++q)
        HIPCHK(hipMalloc(&dout[q], std::max<size_t>((size_t)g.layers[outs[q]].out.numel() * es, 256)));
      for (auto& e : ev) HIPCHK(hipEventCreate(&e));
    } catch (...) {
      release();
      throw;
    }
  }
  ~ScratchIO() { release(); }
  ScratchIO(const ScratchIO&) = delete;
  ScratchIO& operator=(const ScratchIO&) = delete;
  void release() {
    for (auto& e : ev)
      if (e) (void)hipEventDestroy(e), e = nullptr;
    for (void*& p : din)
      if (p) (void)hipFree(p), p = nullptr;
    for (void*& p : dout)
      if (p) (void)hipFree(p), p = nullptr;
  }
  // mean ns per run of the compiled plan over reps back-to-back runs
  int64_t block_ns(Graph& g, hipStream_t st, int reps) {
    HIPCHK(hipEventRecord(ev[0], st));
    for (int r = 0; r < reps; ++r) plan_run(g, din.data(), dout.data(), st);
    HIPCHK(hipEventRecord(ev[1], st));
    HIPCHK(hipEventSynchronize(ev[1]));
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, ev[0], ev[1]));
    return std::max<int64_t>(1, (int64_t)((double)ms * 1e6 / reps + 0.5));
  }
};

void integrated_measure(Graph& g, std::vector<Candidate>& cands, int warmup, int reps,
                        void* stream) {
  if (cands.empty()) fail(SN_E_INTERNAL, "no candidate paths");
  HIPCHK(hipSetDevice(g.device));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const std::vector<int> saved = g.path;
  const int64_t saved_cost = g.path_cost;
  try {
    ScratchIO io(g, st);
    for (Candidate& c : cands) c.measured_ns = -1;
    const int nc = (int)cands.size();
    for (int round = 0; round < 2; ++round) {
      for (int q = 0; q < nc; ++q) {
        Candidate& c = cands[round == 0 ? q : nc - 1 - q];
        g.path = c.path;
        g.path_cost = c.model_ns;
        plan_compile(g);
        for (int w = 0; w < warmup; ++w) plan_run(g, io.din.data(), io.dout.data(), st);
        const int64_t ns = io.block_ns(g, st, reps);
        if (c.measured_ns < 0 || ns < c.measured_ns) c.measured_ns = ns;
      }
    }
    int best = 0;
    for (int q = 1; q < nc; ++q)
      if (cands[q].measured_ns < cands[best].measured_ns) best = q;
    g.path = cands[best].path;
    g.path_cost = cands[best].model_ns;
    plan_compile(g);
  } catch (...) {
    g.path = saved;
    g.path_cost = saved_cost;
    plan_destroy(g);
    throw;
  }
}

// ------------------------------------------------------------------ in-path refinement
// Layer by layer, the selected routine and its near-tied alternatives of the
// same schema are timed inside the whole path (only that layer swapped; the
// layer's time from the events tied to its first and last launch, median of
// reps timed runs); a clear winner (more than 2 % faster, confirmed by a second
// pair of timings) is kept for the later layers' trials.  The refined path then
// has to beat the selected one end to end (alternating rounds) to be kept.
int refine_in_path(Graph& g, int tol_permille, int max_alts, int reps, void* stream) {
  if (!g.have_costs) fail(SN_E_STATE, "no costs: profile or load a cost table first");
  if (g.path.empty()) fail(SN_E_STATE, "no selected path");
  HIPCHK(hipSetDevice(g.device));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const std::vector<int> saved = g.path;
  const int64_t saved_cost = g.path_cost;
  const int nl = g.n_layers();
  int changed = 0;
  try {
    ScratchIO io(g, st);
    std::vector<float> ms(nl);
    std::vector<float> v(reps);
    auto layer_time = [&](const std::vector<int>& path, int layer) {
      g.path = path;
      plan_compile(g);
      for (int w = 0; w < 2; ++w) plan_run(g, io.din.data(), io.dout.data(), st, ms.data(), 1);
      for (int r = 0; r < reps; ++r) {
        plan_run(g, io.din.data(), io.dout.data(), st, ms.data(), 1);
        v[r] = ms[layer];
      }
      std::nth_element(v.begin(), v.begin() + reps / 2, v.end());
      return v[reps / 2];
    };
    std::vector<int> cur = saved;
    for (int i = 1; i < nl; ++i) {
      const Layer& L = g.layers[i];
      const int r0 = cur[i];
      const int64_t c0 = L.cost[r0];
      if (c0 <= 0) continue;
      std::vector<int> alts;
      for (int r = 0; r < (int)L.routines.size(); ++r)
        if (r != r0 && L.routines[r].schema() == L.routines[r0].schema() && L.cost[r] > 0 &&
            (double)L.cost[r] <= (double)c0 * (1.0 + tol_permille / 1000.0))
          alts.push_back(r);
      if (alts.empty()) continue;
      std::stable_sort(alts.begin(), alts.end(), [&](int a, int b) { return L.cost[a] < L.cost[b]; });
      if ((int)alts.size() > max_alts) alts.resize(max_alts);
      const float t0 = layer_time(cur, i);
      float best_t = t0;
      int best = r0;
      for (int r : alts) {
        std::vector<int> p = cur;
        p[i] = r;
        const float t = layer_time(p, i);
        if (t < best_t) best_t = t, best = r;
      }
      if (best == r0 || best_t >= 0.98f * t0) continue;
      // a second, fresh pair of timings has to confirm the win: with several
      // alternatives the fastest of a noisy set is biased low
      std::vector<int> p = cur;
      p[i] = best;
      const float t0b = layer_time(cur, i);
      const float t1b = layer_time(p, i);
      if (t1b < 0.98f * t0b) cur[i] = best;
    }
    for (int i = 0; i < nl; ++i) changed += cur[i] != saved[i];
    if (changed) {
      // the refined path has to win end to end: four alternating rounds
      std::vector<int64_t> ta, tb;
      for (int round = 0; round < 4; ++round)
        for (int k = 0; k < 2; ++k) {
          const bool refined = (round % 2 == 0) == (k == 1);
          g.path = refined ? cur : saved;
          plan_compile(g);
          for (int w = 0; w < 3; ++w) plan_run(g, io.din.data(), io.dout.data(), st);
          (refined ? tb : ta).push_back(io.block_ns(g, st, 20));
        }
      std::sort(ta.begin(), ta.end());
      std::sort(tb.begin(), tb.end());
      if (tb[1] + tb[2] >= ta[1] + ta[2]) changed = 0;
    }
    g.path = changed ? cur : saved;
    g.path_cost = changed ? path_total(g, cur) : saved_cost;
    plan_compile(g);
  } catch (...) {
    g.path = saved;
    g.path_cost = saved_cost;
    plan_destroy(g);
    throw;
  }
  return changed;
}

}  // namespace sn
