// Adaptive traffic controller (paper Section 4.2.2): the robot-to-GPU
// assignment integer program, eqs (1)-(3), solved exactly by depth-first
// branch and bound on the host.
//
// Variables r[i][j] >= 0 (robots of model i sent to GPU j; zero where the
// placement does not host i on j). eq (1): sum_j r[i][j] = N_i. eq (2):
// sum_i r[i][j] / C_i <= 1, checked exactly in integers as
// sum_i r[i][j] * (L / C_i) <= L with L = lcm(C_i). eq (3): minimise
// sum_j sum_{i<k} r[i][j] r[k][j].
//
// Search: models in order of decreasing population; for each, its robots are
// distributed over its hosting GPUs, GPUs with the fewest robots of earlier
// models first and larger shares first, so good incumbents come early.
// Adding a model adds sum_j r[i][j] * S_j to eq (3), where S_j is the number
// of robots already on GPU j, so a lower bound of the remainder is, for each
// model not yet placed, the least such increment it could have with the
// current S and capacities (fill the GPUs in ascending S): placing more
// models only raises S and lowers capacities. Interchangeable GPUs (same
// hosting column, same robots of every placed model) are taken in
// non-increasing share order (each bounded by its nearest earlier twin).
// The search stops after max_nodes nodes and reports whether the optimum
// was proven.
#include <algorithm>
#include <numeric>
#include <vector>

#include "../../include/vla.h"
#include "../../include/vla_sched.h"
#include "model.h"

namespace {

typedef __int128 i128;

struct TrafficSearch {
  int M = 0, G = 0;
  std::vector<int> host, n, order;   // host [M][G]; order: model visit order
  std::vector<i128> w;               // L / C_i
  i128 L = 1;
  std::vector<i128> load;            // per GPU: sum_i r[i][j] * w_i
  std::vector<long long> robots;     // per GPU: robots already placed (S_j)
  std::vector<int> r, best_r;        // [M][G]
  long long best = -1, nodes = 0, max_nodes = 0;
  bool stopped = false;

  int cap(int i, int j) const {      // most robots of model i GPU j still takes
    if (!host[i * G + j]) return 0;
    const i128 c = (L - load[j]) / w[i];
    return (int)std::min<i128>(c, n[i]);
  }

  // least increment of eq (3) model i could add now; -1 if it cannot fit
  long long least_increment(int i) const {
    std::vector<int> js;
    for (int j = 0; j < G; ++j)
      if (host[i * G + j]) js.push_back(j);
    std::sort(js.begin(), js.end(), [&](int a, int b) { return robots[a] < robots[b]; });
    long long left = n[i], inc = 0;
    for (int j : js) {
      if (left == 0) break;
      const long long t = std::min<long long>(left, cap(i, j));
      inc += t * robots[j];
      left -= t;
    }
    return left > 0 ? -1 : inc;
  }

  bool equivalent(int a, int b, int depth) const {   // GPUs a, b interchangeable so far
    for (int i = 0; i < M; ++i)
      if (host[i * G + a] != host[i * G + b]) return false;
    for (int d = 0; d < depth; ++d) {
      const int i = order[d];
      if (r[i * G + a] != r[i * G + b]) return false;
    }
    return true;
  }

  void model(int depth, long long obj) {
    if (stopped) return;
    if (depth == M) {
      if (best < 0 || obj < best) { best = obj; best_r = r; }
      return;
    }
    long long lb = obj;
    for (int d = depth; d < M; ++d) {
      const long long inc = least_increment(order[d]);
      if (inc < 0) return;                        // cannot fit any more
      lb += inc;
    }
    if (best >= 0 && lb >= best) return;
    const int i = order[depth];
    std::vector<int> js;
    for (int j = 0; j < G; ++j)
      if (host[i * G + j]) js.push_back(j);
    std::stable_sort(js.begin(), js.end(), [&](int a, int b) { return robots[a] < robots[b]; });
    // symmetry: a GPU interchangeable with an earlier one in js takes no more
    std::vector<int> twin(js.size(), -1);
    for (size_t x = 1; x < js.size(); ++x)
      for (size_t y = x; y-- > 0;)
        if (equivalent(js[y], js[x], depth)) { twin[x] = (int)y; break; }
    std::vector<int> share(js.size(), 0);
    distribute(depth, obj, i, js, twin, share, 0, n[i]);
  }

  void distribute(int depth, long long obj, int i, const std::vector<int>& js, const std::vector<int>& twin,
                  std::vector<int>& share, size_t x, int left) {
    if (stopped) return;
    if (++nodes > max_nodes) { stopped = true; return; }
    if (x == js.size()) {
      if (left == 0) model(depth + 1, obj);
      return;
    }
    const int j = js[x];
    // the remaining GPUs must be able to take what this one leaves
    long long rest = 0;
    for (size_t y = x + 1; y < js.size(); ++y) rest += cap(i, js[y]);
    int hi = std::min(left, cap(i, j));
    if (twin[x] >= 0) hi = std::min(hi, share[twin[x]]);
    const int lo = (int)std::max<long long>(0, left - rest);
    for (int t = hi; t >= lo; --t) {
      share[x] = t;
      r[i * G + j] = t;
      load[j] += (i128)t * w[i];
      robots[j] += t;
      distribute(depth, obj + (long long)t * (robots[j] - t), i, js, twin, share, x + 1, left - t);
      robots[j] -= t;
      load[j] -= (i128)t * w[i];
      r[i * G + j] = 0;
      if (stopped) return;
    }
    share[x] = 0;
  }
};

i128 gcd128(i128 a, i128 b) {
  while (b) { const i128 t = a % b; a = b; b = t; }
  return a;
}

}  // namespace

extern "C" {

vla_status vla_traffic_assign(int n_models, int n_gpus, const int* host, const int* n_robots, const int* limits,
                              long long max_nodes, int* r_out, long long* objective, int* optimal) {
  try {
    vla_clear_error();
    VLA_REQUIRE(n_models >= 1 && n_models <= 64 && n_gpus >= 1 && n_gpus <= 64, "n_models, n_gpus must be in [1, 64]");
    VLA_REQUIRE(host && n_robots && limits && r_out, "null argument");
    VLA_REQUIRE(max_nodes >= 1, "max_nodes must be >= 1");
    TrafficSearch s;
    s.M = n_models; s.G = n_gpus; s.max_nodes = max_nodes;
    s.host.assign(host, host + (size_t)n_models * n_gpus);
    s.n.assign(n_robots, n_robots + n_models);
    for (int i = 0; i < n_models; ++i) {
      VLA_REQUIRE(n_robots[i] >= 0 && n_robots[i] <= 1000000, "robot populations must be in [0, 1e6]");
      VLA_REQUIRE(limits[i] >= 1 && limits[i] <= 1000000, "robot limits must be in [1, 1e6]");
      for (int j = 0; j < n_gpus; ++j) VLA_REQUIRE(host[i * n_gpus + j] == 0 || host[i * n_gpus + j] == 1, "host entries must be 0 or 1");
    }
    // L = lcm of the limits (exact capacity test); refuse sets whose lcm overflows
    for (int i = 0; i < n_models; ++i) {
      const i128 c = limits[i], g = gcd128(s.L, c);
      VLA_REQUIRE(s.L / g <= ((i128)1 << 100) / c, "robot limits: least common multiple too large");
      s.L = s.L / g * c;
    }
    for (int i = 0; i < n_models; ++i) s.w.push_back(s.L / limits[i]);
    s.order.resize(n_models);
    std::iota(s.order.begin(), s.order.end(), 0);
    std::stable_sort(s.order.begin(), s.order.end(), [&](int a, int b) { return s.n[a] > s.n[b]; });
    s.load.assign(n_gpus, 0);
    s.robots.assign(n_gpus, 0);
    s.r.assign((size_t)n_models * n_gpus, 0);
    s.model(0, 0);
    if (s.best < 0) {
      if (s.stopped) throw VlaError{VLA_EUNSUPPORTED, "traffic assignment: search limit reached before any feasible assignment"};
      throw VlaError{VLA_EINVAL, "traffic assignment infeasible: change the model placement or add GPUs (eq (1)-(2))"};
    }
    std::copy(s.best_r.begin(), s.best_r.end(), r_out);
    if (objective) *objective = s.best;
    if (optimal) *optimal = s.stopped ? 0 : 1;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

}  // extern "C"
