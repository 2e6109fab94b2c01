// Routine-path selection.
//
// select_dprs implements DPRS (Sec. IV, Algorithm 1 of the paper): dynamic
// programming over the layer DAG in topological order, where the state of a
// layer is its own schema plus the schemas of the open branching layers
// upstream (the constraint set C_i, Sec. IV-C), constraints are relaxed at a
// merging layer for the branching layers it post-dominates (Sec. IV-D,
// Proposition 3), and a branching layer adds itself to the constraint set.
//
// Readings where the paper is silent or ambiguous:
//  * Subpath union: a state carries the full routine assignment of the
//    layers it covers (the ancestors of the layer plus the layer), and the
//    time of a union is recomputed from the union itself, so layers and edges
//    shared by several predecessors' subpaths are counted once (T(S) sums
//    over a set, Definition 1).
//  * C_i is the union of the predecessors' constraint sets; each
//    predecessor's subpath is looked up with the restriction of the
//    constraint tuple to its own set.  (The pseudo-code takes one
//    predecessor's set and assumes all are equal.)
//  * A branching layer that is itself an input of a merge must agree with
//    its constraint: its table is +inf when its schema differs from the
//    constrained one.
//  * "fastest" breaks ties by the routine-id vector in layer order, so the
//    returned path is the unique (time, lexicographic) minimum.
//  * The auxiliary input layer has one NCHW routine of time 0 (as has every
//    further net input, joined to it by a zero-cost edge); an implicit
//    auxiliary output layer with one NCHW routine of time 0 takes every net
//    output (Sec. IV-E), so the final constraint set is empty (Sec. IV-F).
//  * A schema is a (dtype, layout) pair; with one dtype the schemas are the
//    layouts.  The DP is the same for any schema set (Sec. IV-F: hybrid
//    tuning only enlarges it).
#include <algorithm>
#include <numeric>

#include "core.hpp"

namespace sn {

namespace {

struct Problem {
  int L = 0;                                  // layers incl. auxiliary output
  int S = 0;                                  // number of schemas in use
  std::vector<int> index_of_schema;           // schema (dtype x layout) -> index or -1
  std::vector<std::vector<int64_t>> cost;     // [i][r], kInf = unavailable
  std::vector<std::vector<int>> schema;       // [i][r], schema index
  std::vector<std::vector<int>> preds, succs; // distinct neighbours
  struct E {
    int a, b;
    std::vector<int64_t> A;                   // S x S by schema index, kInf = unavailable
    int64_t at(int x, int y, int S_) const { return A[(size_t)x * S_ + y]; }
  };
  std::vector<E> edges;
};

// layout_mask / dtype_mask restrict the routines of layers 1..n-1 to those
// layouts / dtypes (the auxiliary layers keep their run-dtype NCHW routine)
Problem make_problem(const Graph& g, int layout_mask = -1, int dtype_mask = -1) {
  Problem P;
  int n = g.n_layers();
  P.L = n + 1;
  P.index_of_schema.assign(kNumSchemas, -1);
  for (int sc = 0; sc < kNumSchemas; ++sc)
    if (g.schema_allowed(sc)) P.index_of_schema[sc] = P.S++;
  P.cost.resize(P.L);
  P.schema.resize(P.L);
  for (int i = 0; i < n; ++i) {
    const Layer& L = g.layers[i];
    for (size_t r = 0; r < L.routines.size(); ++r) {
      const Routine& R = L.routines[r];
      int64_t c = L.cost[r];
      if (L.type != SN_LAYER_INPUT && (!(layout_mask >> R.layout & 1) || !(dtype_mask >> R.dtype & 1))) c = -1;
      const int si = P.index_of_schema[R.schema()];
      if (si < 0) c = -1;
      P.cost[i].push_back(c < 0 ? kInf : c);
      P.schema[i].push_back(si < 0 ? 0 : si);
    }
  }
  P.cost[n] = {0};
  P.schema[n] = {P.index_of_schema[schema_of(g.dtype, SN_NCHW)]};
  P.preds.resize(P.L);
  P.succs.resize(P.L);
  for (const Edge& e : all_edges(g)) {
    Problem::E pe;
    pe.a = e.from;
    pe.b = e.to;
    pe.A.assign((size_t)P.S * P.S, kInf);
    for (int x = 0; x < kNumSchemas; ++x)
      for (int y = 0; y < kNumSchemas; ++y) {
        int sx = P.index_of_schema[x], sy = P.index_of_schema[y];
        if (sx < 0 || sy < 0) continue;
        int64_t v = x == y ? 0 : e.adapt[x][y];
        pe.A[(size_t)sx * P.S + sy] = v < 0 ? kInf : v;
      }
    P.edges.push_back(pe);
    auto& pr = P.preds[e.to];
    if (std::find(pr.begin(), pr.end(), e.from) == pr.end()) pr.push_back(e.from);
    auto& su = P.succs[e.from];
    if (std::find(su.begin(), su.end(), e.to) == su.end()) su.push_back(e.to);
  }
  for (auto& v : P.preds) std::sort(v.begin(), v.end());
  for (int i = 0; i + 1 < P.L; ++i)
    if (P.succs[i].empty())
      fail(SN_E_INVALID, "layer " + std::to_string(i) +
                             " has no consumer: every layer must reach a net output");
  return P;
}

// Time of a (partial) assignment: routines of the assigned layers plus the
// adapts of the edges whose two ends are assigned.
int64_t assignment_time(const Problem& P, const std::vector<int32_t>& U) {
  int64_t t = 0;
  for (int i = 0; i < P.L; ++i)
    if (U[i] >= 0) {
      int64_t c = P.cost[i][U[i]];
      if (c >= kInf) return kInf;
      t += c;
    }
  for (const auto& e : P.edges) {
    if (U[e.a] < 0 || U[e.b] < 0) continue;
    int sa = P.schema[e.a][U[e.a]], sb = P.schema[e.b][U[e.b]];
    if (sa == sb) continue;
    int64_t c = e.at(sa, sb, P.S);
    if (c >= kInf) return kInf;
    t += c;
  }
  return t;
}

struct State {
  int64_t t = kInf;
  std::vector<int32_t> U;
};

bool better(const State& a, const State& b) {  // a strictly before b in (time, lex) order
  if (a.t != b.t) return a.t < b.t;
  return std::lexicographical_compare(a.U.begin(), a.U.end(), b.U.begin(), b.U.end());
}

struct Table {
  std::vector<int> C;         // constrained layers, ascending
  std::vector<State> st;      // index: lambda + S * sum_k lambda_C[k] * S^k
};

int64_t ipow(int64_t b, int e) {
  int64_t r = 1;
  while (e-- > 0) r *= b;
  return r;
}

// DPRS over a problem: the (time, lexicographic) minimum complete state;
// per-layer statistics into *stats when given.
State dprs_solve(const Problem& P, std::vector<DPLayerStats>* stats) {
  const int L = P.L, S = P.S;

  // post-dominator sets on the 1-in-1-out DAG (the output post-dominates all)
  std::vector<std::vector<char>> pdom(L, std::vector<char>(L, 0));
  for (int i = L - 1; i >= 0; --i) {
    if (P.succs[i].empty()) {
      pdom[i][i] = 1;
      continue;
    }
    std::vector<char> acc = pdom[P.succs[i][0]];
    for (size_t k = 1; k < P.succs[i].size(); ++k)
      for (int j = 0; j < L; ++j) acc[j] = acc[j] && pdom[P.succs[i][k]][j];
    acc[i] = 1;
    pdom[i] = acc;
  }

  // F_i(lambda): fastest routine of each schema, lowest id on ties (Eq. 1)
  std::vector<std::vector<int>> F(L, std::vector<int>(S, -1));
  for (int i = 0; i < L; ++i)
    for (size_t r = 0; r < P.cost[i].size(); ++r) {
      int s = P.schema[i][r];
      if (s < 0 || P.cost[i][r] >= kInf) continue;
      int& f = F[i][s];
      if (f < 0 || P.cost[i][r] < P.cost[i][f]) f = (int)r;
    }

  std::vector<Table> T(L);
  if (stats) stats->assign(L, DPLayerStats{});
  int64_t conflicts = 0;
  for (int i = 0; i < L; ++i) {
    const auto& H = P.preds[i];
    Table& ti = T[i];
    for (int h : H)
      for (int c : T[h].C)
        if (std::find(ti.C.begin(), ti.C.end(), c) == ti.C.end()) ti.C.push_back(c);
    std::sort(ti.C.begin(), ti.C.end());
    if (ti.C.size() > 12 || ipow(S, (int)ti.C.size() + 1) > (int64_t(1) << 26))
      fail(SN_E_UNSUPPORTED, "too many open branches for DPRS");
    const int nc = (int)ti.C.size();
    const int64_t nCt = ipow(S, nc);
    ti.st.assign(S * nCt, State{});
    // position of each predecessor's constrained layers inside C_i
    std::vector<std::vector<int>> pos(H.size());
    for (size_t k = 0; k < H.size(); ++k)
      for (int c : T[H[k]].C)
        pos[k].push_back((int)(std::find(ti.C.begin(), ti.C.end(), c) - ti.C.begin()));
    const int64_t nH = ipow(S, (int)H.size());
    if (stats) {
      (*stats)[i].states = S * nCt;
      (*stats)[i].candidates = nH;
    }
    std::vector<int> lc(nc), lh(H.size());
    for (int64_t ci = 0; ci < nCt; ++ci) {
      for (int k = 0, v = (int)ci; k < nc; ++k, v /= S) lc[k] = v % S;
      for (int lam = 0; lam < S; ++lam) {
        State& best = ti.st[lam + S * ci];
        int f = F[i][lam];
        if (f < 0) continue;
        if (H.empty()) {  // the input layer (S_0 of the pseudo-code)
          State s;
          s.U.assign(L, -1);
          s.U[i] = f;
          s.t = assignment_time(P, s.U);
          best = s;
          continue;
        }
        for (int64_t hi = 0; hi < nH; ++hi) {
          for (size_t k = 0, v = (size_t)hi; k < H.size(); ++k, v /= S) lh[k] = (int)(v % S);
          State cand;
          cand.U.assign(L, -1);
          bool ok = true;
          for (size_t k = 0; k < H.size() && ok; ++k) {
            const Table& th = T[H[k]];
            int64_t idx = 0, mul = 1;
            for (size_t q = 0; q < pos[k].size(); ++q, mul *= S) idx += lc[pos[k][q]] * mul;
            const State& sh = th.st[lh[k] + S * idx];
            if (sh.t >= kInf) {
              ok = false;
              break;
            }
            for (int j = 0; j < L; ++j) {
              if (sh.U[j] < 0) continue;
              if (cand.U[j] >= 0 && cand.U[j] != sh.U[j]) {
                ok = false;
                ++conflicts;
                break;
              }
              cand.U[j] = sh.U[j];
            }
          }
          if (!ok) continue;
          cand.U[i] = f;
          cand.t = assignment_time(P, cand.U);
          if (cand.t >= kInf) continue;
          if (best.t >= kInf || better(cand, best)) best = std::move(cand);
        }
      }
    }
    // merging layer: relax the constraints of the branching layers it post-dominates
    if (H.size() >= 2) {
      std::vector<int> keep, relax;
      for (int k = 0; k < nc; ++k) (pdom[ti.C[k]][i] ? relax : keep).push_back(k);
      if (!relax.empty()) {
        Table nt;
        for (int k : keep) nt.C.push_back(ti.C[k]);
        int64_t nKt = ipow(S, (int)keep.size());
        nt.st.assign(S * nKt, State{});
        for (int64_t ci = 0; ci < nCt; ++ci) {
          for (int k = 0, v = (int)ci; k < nc; ++k, v /= S) lc[k] = v % S;
          int64_t ki = 0, mul = 1;
          for (int k : keep) {
            ki += lc[k] * mul;
            mul *= S;
          }
          for (int lam = 0; lam < S; ++lam) {
            const State& s = ti.st[lam + S * ci];
            State& d = nt.st[lam + S * ki];
            if (s.t < kInf && (d.t >= kInf || better(s, d))) d = s;
          }
        }
        ti = std::move(nt);
      }
    }
    // branching layer: constrain its own schema downstream
    if (P.succs[i].size() >= 2) {
      Table nt;
      nt.C = ti.C;
      nt.C.push_back(i);  // i is larger than every id in C_i
      int64_t nOld = ipow(S, (int)ti.C.size());
      nt.st.assign(S * nOld * S, State{});
      for (int64_t ci = 0; ci < nOld; ++ci)
        for (int lam = 0; lam < S; ++lam)
          nt.st[lam + S * (ci + nOld * lam)] = ti.st[lam + S * ci];
      ti = std::move(nt);
    }
    // free tables no successor can read any more
    for (int h : H) {
      bool needed = false;
      for (int s : P.succs[h])
        if (s > i) needed = true;
      if (!needed) T[h].st.clear(), T[h].st.shrink_to_fit();
    }
  }
  if (conflicts) fail(SN_E_INTERNAL, "DPRS: inconsistent subpaths at a merge");
  const Table& last = T[L - 1];
  if (!last.C.empty()) fail(SN_E_INTERNAL, "DPRS: constraint set not empty at the output");
  const State* best = nullptr;
  for (const State& s : last.st)
    if (s.t < kInf && (!best || better(s, *best))) best = &s;
  if (!best) fail(SN_E_UNSUPPORTED, "no routine path of finite time");
  return *best;
}

}  // namespace

void select_dprs(Graph& g, int layout_mask, int dtype_mask) {
  if (!g.have_costs) fail(SN_E_STATE, "no cost table: call sn_profile or sn_set_costs first");
  const Problem P = make_problem(g, layout_mask, dtype_mask);
  const State best = dprs_solve(P, &g.dp_stats);
  g.path.assign(best.U.begin(), best.U.begin() + g.n_layers());
  g.path_cost = best.t;
}

// The childnet as a net of its own: sub-layer 0 takes the role of the
// input layer, the sub-layers form a chain, an auxiliary output closes it,
// and the one schema makes every adapt void.
int64_t childnet_select(ChildNet& c) {
  const int m = (int)c.layer.size();
  Problem P;
  P.L = m + 1;
  P.S = 1;
  P.index_of_schema.assign(kNumSchemas, -1);
  P.cost.resize(P.L);
  P.schema.resize(P.L);
  P.preds.resize(P.L);
  P.succs.resize(P.L);
  for (int i = 0; i < m; ++i) {
    bool any = false;
    for (int64_t v : c.cost[i]) {
      P.cost[i].push_back(v < 0 ? kInf : v);
      P.schema[i].push_back(0);
      any = any || v >= 0;
    }
    if (!any) return -1;
  }
  P.cost[m] = {0};
  P.schema[m] = {0};
  for (int i = 0; i < m; ++i) {
    Problem::E e;
    e.a = i;
    e.b = i + 1;
    e.A = {0};
    P.edges.push_back(e);
    P.preds[i + 1] = {i};
    P.succs[i] = {i + 1};
  }
  const State best = dprs_solve(P, nullptr);
  c.path.assign(best.U.begin(), best.U.begin() + m);
  return best.t;
}

int64_t path_total(const Graph& g, const std::vector<int>& path) {
  Problem P = make_problem(g);
  std::vector<int32_t> U(path.begin(), path.end());
  U.push_back(0);
  int64_t t = assignment_time(P, U);
  return t >= kInf ? -1 : t;
}

void select_fixed(Graph& g, int layout, int algo, int dtype) {
  if (layout < 0 || layout >= SN_NUM_LAYOUTS || algo < 0 || algo >= SN_NUM_ALGOS)
    fail(SN_E_INVALID, "bad layout or algorithm");
  if (dtype < 0) {
    dtype = g.dtype;
    for (int d = 2; d >= 0; --d)
      if (!(g.opt_dtypes >> dtype & 1) && (g.opt_dtypes >> d & 1)) dtype = d;
  }
  if (dtype > 2 || !(g.opt_dtypes >> dtype & 1)) fail(SN_E_INVALID, "dtype not allowed");
  std::vector<int> path(g.n_layers(), 0);
  for (int i = 1; i < g.n_layers(); ++i) {
    const Layer& L = g.layers[i];
    if (L.type == SN_LAYER_INPUT) continue;  // a net input keeps its one routine
    auto pick = [&](int want_algo) {
      int best = -1;
      for (const Routine& r : L.routines) {
        if (r.layout != layout || r.algo != want_algo || r.dtype != dtype) continue;
        if (best < 0) {
          best = r.id;
          continue;
        }
        int64_t cb = L.cost[best], cr = L.cost[r.id];
        if (cr >= 0 && (cb < 0 || cr < cb)) best = r.id;
      }
      return best;
    };
    int r = -1;
    if (L.type == SN_LAYER_CONV2D) {
      r = pick(algo);
      if (r < 0) r = pick(SN_ALGO_IGEMM);
      if (r < 0) r = pick(SN_ALGO_DIRECT);
    } else if (L.type == SN_LAYER_FC) {
      r = pick(algo == SN_ALGO_IGEMM ? SN_ALGO_IGEMM : SN_ALGO_DIRECT);
      if (r < 0) r = pick(SN_ALGO_DIRECT);
    } else {
      r = pick(SN_ALGO_DIRECT);
    }
    if (r < 0)
      fail(SN_E_UNSUPPORTED, "layer " + std::to_string(i) + " has no routine in that layout");
    path[i] = r;
  }
  g.path = path;
  g.path_cost = g.have_costs ? path_total(g, path) : -1;
}

std::vector<Candidate> integrated_candidates(Graph& g) {
  if (!g.have_costs) fail(SN_E_STATE, "no cost table: call sn_profile or sn_set_costs first");
  const std::vector<int> saved = g.path;
  const int64_t saved_cost = g.path_cost;
  std::vector<Candidate> out;
  auto add = [&](int kind, int a, int b) {
    for (const Candidate& c : out)
      if (c.path == g.path) return;
    Candidate c;
    c.path = g.path;
    c.model_ns = g.path_cost;
    c.kind = kind;
    c.a = a;
    c.b = b;
    out.push_back(std::move(c));
  };
  // the schemas the DP may use; subsets in increasing mask order, the full set first
  const int full = (int)(g.opt_layouts & ((1 << SN_NUM_LAYOUTS) - 1));
  std::vector<int> masks{full};
  for (int m = 1; m < full; ++m)
    if ((m & full) == m) masks.push_back(m);
  const int dfull = (int)(g.opt_dtypes & 7);
  try {
    for (int m : masks) {
      try {
        select_dprs(g, m);
      } catch (const Error& e) {
        if (e.code != SN_E_UNSUPPORTED) throw;
        continue;  // some layer has no routine in these layouts
      }
      add(0, m, dfull);
    }
    // with several dtypes: the best path in each dtype alone (the
    // single-schema-family tunings that hybrid tuning is measured against)
    if (g.multi_dtype())
      for (int d = 0; d < 3; ++d) {
        if (!(dfull >> d & 1)) continue;
        try {
          select_dprs(g, full, 1 << d);
        } catch (const Error& e) {
          if (e.code != SN_E_UNSUPPORTED) throw;
          continue;
        }
        add(0, full, 1 << d);
      }
    for (int l = 0; l < SN_NUM_LAYOUTS; ++l) {
      if (!(full >> l & 1)) continue;
      for (int a = 0; a < SN_NUM_ALGOS; ++a) {
        if (!(g.opt_algos >> a & 1)) continue;
        try {
          select_fixed(g, l, a);
        } catch (const Error& e) {
          if (e.code != SN_E_UNSUPPORTED) throw;
          continue;
        }
        add(1, l, a);
      }
    }
  } catch (...) {
    g.path = saved;
    g.path_cost = saved_cost;
    throw;
  }
  g.path = saved;
  g.path_cost = saved_cost;
  return out;
}

void set_path(Graph& g, const int32_t* ids, int n) {
  if (n != g.n_layers()) fail(SN_E_INVALID, "path length differs from the number of layers");
  std::vector<int> path(n);
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= (int)g.layers[i].routines.size())
      fail(SN_E_INVALID, "unknown routine id for layer " + std::to_string(i));
    path[i] = ids[i];
  }
  g.path = path;
  g.path_cost = g.have_costs ? path_total(g, path) : -1;
}

}  // namespace sn
