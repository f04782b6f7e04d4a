// Inter-stage planner (Sec. 5.3, Eq. 1-3): the pipeline partition, gradient-accumulation steps
// and per-stage frontier points that minimise Eq. 2 for one hardware sample, exactly.
//
// Eq. 2 (inner sum read as the time of the stages before i):
//   F = (G - 1) * max_i t_i + sum_i t_i + max_i (d_i - sum_{j<i} t_j)
//     = (G - 1) * max_i t_i + max_i (d_i + sum_{j>=i} t_j).
// In the second form F is non-decreasing in every t_i and d_i, and the last two terms build up
// stage by stage from the last stage to the first: with T = sum_{j>=i} t_j,
// H = max_{j>=i} (d_j + T_j) and M = max_{j>=i} t_j, stage i maps (T, H, M) to
// (t_i + T, max(H, d_i + t_i + T), max(M, t_i)).  A partial plan whose (T, H, M) is no smaller
// in all three than another's with the same stages and layer count can never finish better, so
// a dynamic program over (stage, layers used) keeps only the non-dominated triples and is exact;
// no MILP solver is needed.
//
// Exact also in floating point: every step above (a rounded sum, a maximum) and the final
// (G - 1) * M + H are non-decreasing in T, H and M, so a pruned state's completions never round
// below its dominator's.  Finished plans are therefore ranked by that same suffix-form value,
// fl((G - 1) * M + H), and the winner is its exact minimum over all plans.  The reported F is the
// winner re-evaluated in stage order (sums left to right), the form the paper writes; the two
// forms agree in real arithmetic, so against the minimum of the stage-order form the reported F
// is off by at most the rounding of the two evaluations (a few ulps of the summed stage times per
// stage).

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <map>
#include <new>
#include <string>
#include <tuple>
#include <vector>

#include "mist.h"

namespace mist {
__attribute__((visibility("hidden"))) mist_status lib_fail(mist_status code, const std::string& msg);  // sets the thread's error
}

namespace {

struct Pt {
  double t, d;
  uint64_t id;
};

struct State {
  double T, H, M;
  int prev;     // index of the state of stage i+1 it extends (-1: none, stage S)
  int l;        // this stage's layer count
  int pt;       // index of this stage's point in its candidate list
};

// Keeps the (t, d)-minimal points, lowest id first among equal ones.
std::vector<Pt> pareto_td(std::vector<Pt> v) {
  std::sort(v.begin(), v.end(), [](const Pt& a, const Pt& b) {
    return std::tie(a.t, a.d, a.id) < std::tie(b.t, b.d, b.id);
  });
  std::vector<Pt> out;
  double dmin = std::numeric_limits<double>::infinity();
  for (const Pt& p : v)
    if (p.d < dmin) {
      out.push_back(p);
      dmin = p.d;
    }
  return out;
}

// Appends s unless a kept state is no larger in T, H and M; drops kept states it dominates.
void add_state(std::vector<State>& v, const State& s) {
  for (const State& o : v)
    if (o.T <= s.T && o.H <= s.H && o.M <= s.M) return;
  size_t w = 0;
  for (size_t r = 0; r < v.size(); ++r)
    if (!(s.T <= v[r].T && s.H <= v[r].H && s.M <= v[r].M)) v[w++] = v[r];
  v.resize(w);
  v.push_back(s);
}

double plan_value(int32_t G, const std::vector<double>& t, const std::vector<double>& d) {
  double t_max = t[0], t_sum = 0.0, m = 0.0;
  for (size_t i = 0; i < t.size(); ++i) {
    const double v = d[i] - t_sum;
    m = i == 0 ? v : std::max(m, v);
    t_sum = t_sum + t[i];
    t_max = std::max(t_max, t[i]);
  }
  return ((double)(G - 1) * t_max + t_sum) + m;
}

}  // namespace

extern "C" mist_status mist_plan_points(const mist_stage_point* pts, int64_t n, int32_t n_layers, int32_t pp,
                                        mist_plan* out) {
  using mist::lib_fail;
  if (!out || (!pts && n > 0)) return lib_fail(MIST_E_INVALID, "null argument");
  if (n < 0 || n_layers < 1 || pp < 0 || pp > MIST_MAX_STAGES) return lib_fail(MIST_E_INVALID, "argument out of range");
  try {
    std::memset(out, 0, sizeof(*out));
    out->F = std::numeric_limits<double>::infinity();
    double best_Fs = std::numeric_limits<double>::infinity();  // suffix-form value of *out
    // candidates per (G, PP) -> per k -> per l
    std::map<std::pair<int32_t, int32_t>, std::map<int32_t, std::map<int32_t, std::vector<Pt>>>> cand;
    for (int64_t i = 0; i < n; ++i) {
      const mist_stage_point& p = pts[i];
      if (p.PP < 1 || p.k < 1 || p.k > p.PP || p.l < 1 || p.G < 1 || !std::isfinite(p.t) || !std::isfinite(p.d))
        return lib_fail(MIST_E_INVALID, "invalid stage point");
      if (p.PP > MIST_MAX_STAGES || (pp && p.PP != pp)) continue;
      cand[{p.G, p.PP}][p.k][p.l].push_back(Pt{p.t, p.d, p.id});
    }
    for (auto& gp : cand) {
      const int32_t G = gp.first.first, PP = gp.first.second;
      auto& byk = gp.second;
      // stage i (1-based) runs k = PP - i + 1 microbatches in flight
      std::vector<std::vector<std::pair<int32_t, std::vector<Pt>>>> stage(PP + 1);
      bool ok = true;
      for (int32_t i = 1; i <= PP && ok; ++i) {
        auto it = byk.find(PP - i + 1);
        if (it == byk.end()) { ok = false; break; }
        for (auto& lp : it->second) stage[i].push_back({lp.first, pareto_td(lp.second)});
        ok = !stage[i].empty();
      }
      if (!ok) continue;
      std::vector<int32_t> lmin(PP + 2, 0);  // fewest layers stages i..PP can hold
      for (int32_t i = PP; i >= 1; --i) {
        int32_t m = std::numeric_limits<int32_t>::max();
        for (auto& lp : stage[i]) m = std::min(m, lp.first);
        lmin[i] = lmin[i + 1] + m;
      }
      // states[i][u]: stages i..PP placed, u layers used
      std::vector<std::vector<std::vector<State>>> states(PP + 2, std::vector<std::vector<State>>(n_layers + 1));
      states[PP + 1][0].push_back(State{0.0, -std::numeric_limits<double>::infinity(), 0.0, -1, 0, 0});
      for (int32_t i = PP; i >= 1; --i) {
        for (int32_t u = 0; u <= n_layers; ++u) {
          const auto& from = states[i + 1][u];
          for (int s = 0; s < (int)from.size(); ++s) {
            const State& st = from[s];
            for (auto& lp : stage[i]) {
              const int32_t u2 = u + lp.first;
              if (u2 + lmin[1] - lmin[i] > n_layers) continue;  // stages 1..i-1 still need layers
              if (i == 1 && u2 != n_layers) continue;
              for (int q = 0; q < (int)lp.second.size(); ++q) {
                const Pt& p = lp.second[q];
                const double T = p.t + st.T;
                add_state(states[i][u2], State{T, std::max(st.H, p.d + T), std::max(st.M, p.t), s, lp.first, q});
              }
            }
          }
        }
      }
      // the finished plans: stage 1 placed, all layers used
      const auto& fin = states[1][n_layers];
      for (int s = 0; s < (int)fin.size(); ++s) {
        const double Fs = (double)(G - 1) * fin[s].M + fin[s].H;
        if (!(Fs < best_Fs)) continue;
        best_Fs = Fs;
        std::vector<double> tv, dv;
        mist_plan cand_plan;
        std::memset(&cand_plan, 0, sizeof(cand_plan));
        int cur = s;
        // walk back through the predecessors: stage i's state lives in states[i][u_i]
        int32_t u = n_layers;
        for (int32_t i = 1; i <= PP; ++i) {
          const State& st = states[i][u][cur];
          const Pt* pt = nullptr;
          for (auto& lp : stage[i])
            if (lp.first == st.l) pt = &lp.second[st.pt];
          mist_stage_plan& sp = cand_plan.stage[i - 1];
          sp.l = st.l;
          sp.k = PP - i + 1;
          sp.id = pt->id;
          sp.t = pt->t;
          sp.d = pt->d;
          tv.push_back(pt->t);
          dv.push_back(pt->d);
          cur = st.prev;
          u -= st.l;
        }
        cand_plan.G = G;
        cand_plan.PP = PP;
        cand_plan.found = 1;
        cand_plan.F = plan_value(G, tv, dv);
        *out = cand_plan;
      }
    }
    return MIST_OK;
  } catch (const std::bad_alloc&) {
    return lib_fail(MIST_E_NOMEM, "host allocation failed");
  }
}
