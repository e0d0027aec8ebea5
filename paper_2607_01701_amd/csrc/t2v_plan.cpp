// Cascade planner: the paper's scheduling problem (Section IV-A, Eqs. (1)-(7)) solved as in
// Alg. 1 — a genetic algorithm over per-cascade parallel degrees whose fitness is the
// makespan of a critical-path list scheduler. Host-only C++ (no HIP): the planner feeds the
// cross-GPU orchestration that this library does not run itself; it is exposed so that a
// launcher can plan a batch from the attention cost model (Eq. (9)).
//
// Problem. Cascades c = 0..n-1 with direct predecessors P_c (a DAG); degrees K; latency
// L_{c,k} and memory Mem_{c,k}; N GPUs of W bytes each. Choose one degree per cascade with
// Mem_{c,k} <= W (Eqs. (5), (6)) and launch times s_c >= e_p for every predecessor p
// (Eq. (4)) such that the degrees of the cascades active at any time sum to at most N
// (Eq. (7)), minimising T = max_c (s_c + L_{c,k_c}) (Eqs. (1)-(3)).
//
// List scheduler (the GA's fitness). With the degrees fixed: priority of a cascade = its
// bottom level (its latency plus the longest chain of latencies below it, the critical
// path through it). Repeatedly take the ready cascade (all predecessors placed) of highest
// priority and start it at the earliest time at or after its predecessors' ends at which
// its k GPUs stay free for its whole latency (a serial schedule-generation scheme).
//
// Genetic algorithm. A chromosome is a feasible degree per cascade. The first population
// holds four heuristic assignments (every cascade at its smallest, largest, fastest and
// smallest-area (k * L) feasible degree) and random ones. Each generation keeps the `elite`
// best, and fills the rest with children of two tournament-selected parents (uniform
// crossover), each gene then re-drawn with probability `mutation`. The best schedule seen
// is returned. Deterministic for a seed.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <string>
#include <vector>

#include "../../include/t2vattn.h"
#include "t2v_host.h"

namespace t2v {
namespace {

struct Problem {
  int n = 0;
  std::vector<std::vector<int>> preds, succs;
  std::vector<int> topo;  // a topological order
};

// Builds predecessor / successor lists from CSR input and checks that the graph is acyclic.
int build_problem(int n, const int32_t* pred_ptr, const int32_t* pred_idx, Problem* pr) {
  if (n < 0) return set_error(T2V_ERR_INVALID_ARG, "n_cascades must be >= 0");
  if (n > 0 && pred_ptr == nullptr) return set_error(T2V_ERR_INVALID_ARG, "pred_ptr is NULL");
  pr->n = n;
  pr->preds.assign(n, {});
  pr->succs.assign(n, {});
  if (n == 0) return T2V_OK;
  if (pred_ptr[0] != 0) return set_error(T2V_ERR_INVALID_ARG, "pred_ptr[0] must be 0");
  for (int c = 0; c < n; ++c)
    if (pred_ptr[c + 1] < pred_ptr[c]) return set_error(T2V_ERR_INVALID_ARG, "pred_ptr must be non-decreasing");
  if (pred_ptr[n] > 0 && pred_idx == nullptr) return set_error(T2V_ERR_INVALID_ARG, "pred_idx is NULL");
  for (int c = 0; c < n; ++c) {
    for (int i = pred_ptr[c]; i < pred_ptr[c + 1]; ++i) {
      const int p = pred_idx[i];
      if (p < 0 || p >= n || p == c)
        return set_error(T2V_ERR_INVALID_ARG, "bad predecessor " + std::to_string(p) + " of cascade " +
                                                  std::to_string(c));
      pr->preds[c].push_back(p);
      pr->succs[p].push_back(c);
    }
  }
  std::vector<int> indeg(n);
  for (int c = 0; c < n; ++c) indeg[c] = static_cast<int>(pr->preds[c].size());
  std::vector<int> stack;
  for (int c = n - 1; c >= 0; --c)
    if (indeg[c] == 0) stack.push_back(c);
  while (!stack.empty()) {
    const int c = stack.back();
    stack.pop_back();
    pr->topo.push_back(c);
    for (int s : pr->succs[c])
      if (--indeg[s] == 0) stack.push_back(s);
  }
  if (static_cast<int>(pr->topo.size()) != n)
    return set_error(T2V_ERR_INVALID_ARG, "the cascade graph has a cycle");
  return T2V_OK;
}

struct Placed {
  double s, e;
  int k;
};

// Earliest t >= release at which `need` GPUs are free throughout [t, t + dur), given the
// cascades already placed. Usage changes only at their starts and ends, so the candidates
// are the release time and the ends after it, and a candidate is checked at itself and at
// every start inside its interval.
double earliest_start(double release, double dur, int need, const std::vector<Placed>& placed, int n_gpus) {
  std::vector<double> cand{release};
  for (const auto& p : placed)
    if (p.e > release) cand.push_back(p.e);
  std::sort(cand.begin(), cand.end());
  for (double t : cand) {
    bool ok = true;
    auto used_at = [&](double x) {
      int u = 0;
      for (const auto& p : placed)
        if (p.s <= x && x < p.e) u += p.k;
      return u;
    };
    if (used_at(t) + need > n_gpus) ok = false;
    for (size_t i = 0; ok && i < placed.size(); ++i) {
      const double x = placed[i].s;
      if (x > t && x < t + dur && used_at(x) + need > n_gpus) ok = false;
    }
    if (ok) return t;
  }
  return std::numeric_limits<double>::infinity();  // only when need > n_gpus
}

// Critical-path list schedule for fixed degrees; returns the makespan and fills starts.
double list_schedule(const Problem& pr, const int* deg, const double* lat, int n_gpus, double* start) {
  const int n = pr.n;
  if (n == 0) return 0.0;
  std::vector<double> bottom(n, 0.0);
  for (int i = n - 1; i >= 0; --i) {
    const int c = pr.topo[i];
    double below = 0.0;
    for (int s : pr.succs[c]) below = std::max(below, bottom[s]);
    bottom[c] = lat[c] + below;
  }
  std::vector<int> waiting(n);
  std::vector<char> ready(n, 0);
  for (int c = 0; c < n; ++c) {
    waiting[c] = static_cast<int>(pr.preds[c].size());
    ready[c] = waiting[c] == 0;
  }
  std::vector<double> end(n, 0.0);
  std::vector<Placed> placed;
  placed.reserve(n);
  double makespan = 0.0;
  for (int step = 0; step < n; ++step) {
    int best = -1;
    for (int c = 0; c < n; ++c)
      if (ready[c] == 1 && (best < 0 || bottom[c] > bottom[best])) best = c;
    double release = 0.0;
    for (int p : pr.preds[best]) release = std::max(release, end[p]);
    const double t = earliest_start(release, lat[best], deg[best], placed, n_gpus);
    start[best] = t;
    end[best] = t + lat[best];
    makespan = std::max(makespan, end[best]);
    placed.push_back({t, end[best], deg[best]});
    ready[best] = 2;  // placed
    for (int s : pr.succs[best])
      if (--waiting[s] == 0) ready[s] = 1;
  }
  return makespan;
}

// splitmix64: a small, well-mixed deterministic generator.
struct Rng {
  uint64_t x;
  uint64_t next() {
    uint64_t z = (x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int below(int m) { return static_cast<int>(next() % static_cast<uint64_t>(m)); }
  double unit() { return static_cast<double>(next() >> 11) * (1.0 / 9007199254740992.0); }
};

}  // namespace
}  // namespace t2v

extern "C" {

int t2v_list_schedule(int n_cascades, const int32_t* pred_ptr, const int32_t* pred_idx, const int32_t* degree,
                      const double* latency, int n_gpus, double* start_out, double* makespan_out) {
  using namespace t2v;
  try {
    Problem pr;
    if (int st = build_problem(n_cascades, pred_ptr, pred_idx, &pr)) return st;
    if (makespan_out == nullptr) return set_error(T2V_ERR_INVALID_ARG, "makespan_out is NULL");
    if (n_gpus < 1) return set_error(T2V_ERR_INVALID_ARG, "n_gpus must be >= 1");
    if (n_cascades > 0 && (degree == nullptr || latency == nullptr || start_out == nullptr))
      return set_error(T2V_ERR_INVALID_ARG, "degree, latency or start_out is NULL");
    for (int c = 0; c < n_cascades; ++c) {
      if (degree[c] < 1 || degree[c] > n_gpus)
        return set_error(T2V_ERR_INVALID_ARG, "degree of cascade " + std::to_string(c) + " is outside 1..n_gpus");
      if (!(latency[c] >= 0.0) || !std::isfinite(latency[c]))
        return set_error(T2V_ERR_INVALID_ARG, "latency of cascade " + std::to_string(c) + " is not finite >= 0");
    }
    std::vector<int> deg(degree, degree + n_cascades);
    *makespan_out = list_schedule(pr, deg.data(), latency, n_gpus, start_out);
    return T2V_OK;
  } catch (...) {
    return set_error(T2V_ERR_OOM, "host allocation failed");
  }
}

int t2v_plan_cascades(int n_cascades, const int32_t* pred_ptr, const int32_t* pred_idx, int n_degrees,
                      const int32_t* degrees, const double* latency, const double* mem, double mem_cap, int n_gpus,
                      int population, int generations, double mutation, int elite, uint64_t seed,
                      int32_t* degree_out, double* start_out, double* makespan_out) {
  using namespace t2v;
  try {
    Problem pr;
    if (int st = build_problem(n_cascades, pred_ptr, pred_idx, &pr)) return st;
    if (makespan_out == nullptr) return set_error(T2V_ERR_INVALID_ARG, "makespan_out is NULL");
    if (n_gpus < 1) return set_error(T2V_ERR_INVALID_ARG, "n_gpus must be >= 1");
    if (n_degrees < 1 || degrees == nullptr) return set_error(T2V_ERR_INVALID_ARG, "need at least one degree");
    if (population < 2 || generations < 0 || elite < 0 || elite > population || !(mutation >= 0.0 && mutation <= 1.0))
      return set_error(T2V_ERR_INVALID_ARG, "bad GA hyper-parameters");
    const int n = n_cascades;
    if (n > 0 && (latency == nullptr || mem == nullptr || degree_out == nullptr || start_out == nullptr))
      return set_error(T2V_ERR_INVALID_ARG, "latency, mem, degree_out or start_out is NULL");
    for (int j = 0; j < n_degrees; ++j)
      if (degrees[j] < 1) return set_error(T2V_ERR_INVALID_ARG, "degrees must be >= 1");
    // Feasible degree indices per cascade (Eqs. (5), (6) and k <= N).
    std::vector<std::vector<int>> feas(n);
    for (int c = 0; c < n; ++c) {
      for (int j = 0; j < n_degrees; ++j) {
        const double L = latency[static_cast<size_t>(c) * n_degrees + j];
        const double M = mem[static_cast<size_t>(c) * n_degrees + j];
        if (!std::isfinite(L) || L < 0.0 || std::isnan(M))
          return set_error(T2V_ERR_INVALID_ARG, "latency must be finite >= 0 and mem not NaN");
        if (M <= mem_cap && degrees[j] <= n_gpus) feas[c].push_back(j);
      }
      if (feas[c].empty())
        return set_error(T2V_ERR_INVALID_ARG, "cascade " + std::to_string(c) + " has no feasible degree");
    }
    if (n == 0) {
      *makespan_out = 0.0;
      return T2V_OK;
    }
    Rng rng{seed};
    using Chrom = std::vector<int>;  // degree index per cascade
    auto lat_of = [&](int c, int j) { return latency[static_cast<size_t>(c) * n_degrees + j]; };
    std::vector<int> deg(n);
    std::vector<double> lat(n), start(n);
    auto fitness = [&](const Chrom& ch, double* st_out) {
      for (int c = 0; c < n; ++c) {
        deg[c] = degrees[ch[c]];
        lat[c] = lat_of(c, ch[c]);
      }
      return list_schedule(pr, deg.data(), lat.data(), n_gpus, st_out);
    };
    // Initial population: four heuristic assignments, then random ones.
    std::vector<Chrom> pop;
    auto pick = [&](auto better) {
      Chrom ch(n);
      for (int c = 0; c < n; ++c) {
        int b = feas[c][0];
        for (int j : feas[c])
          if (better(c, j, b)) b = j;
        ch[c] = b;
      }
      return ch;
    };
    pop.push_back(pick([&](int, int j, int b) { return degrees[j] < degrees[b]; }));
    pop.push_back(pick([&](int, int j, int b) { return degrees[j] > degrees[b]; }));
    pop.push_back(pick([&](int c, int j, int b) { return lat_of(c, j) < lat_of(c, b); }));
    pop.push_back(pick([&](int c, int j, int b) { return degrees[j] * lat_of(c, j) < degrees[b] * lat_of(c, b); }));
    while (static_cast<int>(pop.size()) > population) pop.pop_back();
    while (static_cast<int>(pop.size()) < population) {
      Chrom ch(n);
      for (int c = 0; c < n; ++c) ch[c] = feas[c][rng.below(static_cast<int>(feas[c].size()))];
      pop.push_back(ch);
    }
    std::vector<double> fit(pop.size());
    double best_T = std::numeric_limits<double>::infinity();
    Chrom best;
    std::vector<double> best_start(n);
    std::vector<int> order(pop.size());
    for (int g = 0; g <= generations; ++g) {
      for (size_t i = 0; i < pop.size(); ++i) {
        fit[i] = fitness(pop[i], start.data());
        if (fit[i] < best_T) {
          best_T = fit[i];
          best = pop[i];
          best_start = start;
        }
      }
      if (g == generations) break;
      for (size_t i = 0; i < order.size(); ++i) order[i] = static_cast<int>(i);
      std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return fit[a] < fit[b]; });
      std::vector<Chrom> next;
      next.reserve(pop.size());
      for (int i = 0; i < elite; ++i) next.push_back(pop[order[i]]);
      auto tournament = [&]() {
        const int a = rng.below(static_cast<int>(pop.size())), b = rng.below(static_cast<int>(pop.size()));
        return fit[a] <= fit[b] ? a : b;
      };
      while (next.size() < pop.size()) {
        const Chrom& pa = pop[tournament()];
        const Chrom& pb = pop[tournament()];
        Chrom child(n);
        for (int c = 0; c < n; ++c) {
          child[c] = (rng.next() & 1) ? pa[c] : pb[c];
          if (rng.unit() < mutation) child[c] = feas[c][rng.below(static_cast<int>(feas[c].size()))];
        }
        next.push_back(std::move(child));
      }
      pop.swap(next);
    }
    for (int c = 0; c < n; ++c) {
      degree_out[c] = degrees[best[c]];
      start_out[c] = best_start[c];
    }
    *makespan_out = best_T;
    return T2V_OK;
  } catch (...) {
    return set_error(T2V_ERR_OOM, "host allocation failed");
  }
}

}  // extern "C"
