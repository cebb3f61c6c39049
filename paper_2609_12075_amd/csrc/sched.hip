// Host-side serving scheduler (paper Section 4.1.2 lockstep execution and
// Section 4.1.3 SLO-aware multi-model serving): per-model FIFO queues,
// earliest-SLO-first queue choice, power-of-two fixed batches, a two-slot
// VLM -> action-stage hand-off, and SLO accounting. Runs an arrival trace on
// the GPU (vla_step, wall clock) or against a lockstep-duration table
// (simulated clock).
#include <chrono>
#include <deque>
#include <thread>
#include <vector>

#include "../../include/vla.h"
#include "../../include/vla_sched.h"
#include "model.h"

namespace {

int bucket_of(int b) {
  if (b <= 0) return 0;
  int j = 1;
  while ((1 << (j - 1)) < b) ++j;
  return j;
}

int pow2_floor(int x) {
  int p = 1;
  while (p * 2 <= x) p *= 2;
  return p;
}

}  // namespace

struct vla_sched_s {
  int n_models = 0, max_batch = 1, policy = VLA_SCHED_ESF, n_buckets = 2;
  int mode = VLA_SCHED_LOCKSTEP;
  std::vector<int64_t> slo_ns;
  // executor
  int exec_kind = 0;                       // 0 none, 1 simulated, 2 GPU
  std::vector<int64_t> dur_ns;
  int64_t host_overhead_ns = 0;
  std::vector<vla_sched_model_io> io;
  hipStream_t join = nullptr;
  int default_cu = 256;
  std::vector<int> cu_table;

  size_t combo(int mv, int bv, int ma, int ba) const {
    const int bkv = bucket_of(bv), bka = bucket_of(ba);
    const int iv = mv < 0 ? 0 : mv, ia = ma < 0 ? 0 : ma;
    return (((size_t)iv * n_buckets + bkv) * n_models + ia) * n_buckets + bka;
  }
};

extern "C" {

vla_status vla_sched_create(const vla_sched_config* cfg, vla_sched* out) {
  try {
    vla_clear_error();
    VLA_REQUIRE(cfg && out, "null config or out");
    *out = nullptr;
    VLA_REQUIRE(cfg->n_models >= 1 && cfg->n_models <= 16, "n_models must be in [1, 16]");
    VLA_REQUIRE(cfg->slo_ms, "null slo_ms");
    VLA_REQUIRE(cfg->max_batch >= 1 && cfg->max_batch <= 64 && (cfg->max_batch & (cfg->max_batch - 1)) == 0,
                "max_batch must be a power of two in [1, 64]");
    VLA_REQUIRE(cfg->policy >= VLA_SCHED_ESF && cfg->policy <= VLA_SCHED_LQF, "unknown policy");
    auto* s = new vla_sched_s();
    s->n_models = cfg->n_models;
    s->max_batch = cfg->max_batch;
    s->policy = cfg->policy;
    s->n_buckets = bucket_of(cfg->max_batch) + 1;
    for (int m = 0; m < cfg->n_models; ++m) {
      if (!(cfg->slo_ms[m] > 0)) { delete s; throw VlaError{1, "slo_ms must be > 0"}; }
      s->slo_ns.push_back((int64_t)(cfg->slo_ms[m] * 1e6 + 0.5));
    }
    *out = s;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

void vla_sched_destroy(vla_sched s) { delete s; }

vla_status vla_sched_set_sim_executor(vla_sched s, const int64_t* dur_ns, int64_t host_overhead_ns) {
  try {
    vla_clear_error();
    VLA_REQUIRE(s && dur_ns, "null scheduler or table");
    VLA_REQUIRE(host_overhead_ns >= 0, "negative overhead");
    const size_t n = (size_t)s->n_models * s->n_buckets * s->n_models * s->n_buckets;
    for (size_t i = 0; i < n; ++i) VLA_REQUIRE(dur_ns[i] >= 0, "negative duration");
    s->dur_ns.assign(dur_ns, dur_ns + n);
    s->host_overhead_ns = host_overhead_ns;
    s->exec_kind = 1;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

vla_status vla_sched_set_gpu_executor(vla_sched s, const vla_sched_model_io* io, hipStream_t join) {
  try {
    vla_clear_error();
    VLA_REQUIRE(s && io, "null scheduler or io");
    for (int m = 0; m < s->n_models; ++m) {
      const vla_sched_model_io& x = io[m];
      VLA_REQUIRE(x.model && x.pixels && x.text_ids && x.noise && x.kv[0] && x.kv[1] && x.actions[0] && x.actions[1],
                  "model " + std::to_string(m) + ": null model or buffer");
      VLA_REQUIRE(x.kv[0] != x.kv[1] && x.actions[0] != x.actions[1], "the two hand-off slots must differ");
      VLA_REQUIRE(x.model->cfg.max_batch >= s->max_batch, "model max_batch below the scheduler's");
      VLA_REQUIRE(x.steps >= 1 && x.steps <= 1000, "steps must be in [1, 1000]");
    }
    s->io.assign(io, io + s->n_models);
    s->join = join;
    s->exec_kind = 2;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

vla_status vla_sched_set_mode(vla_sched s, int mode) {
  try {
    vla_clear_error();
    VLA_REQUIRE(s, "null scheduler");
    VLA_REQUIRE(mode == VLA_SCHED_LOCKSTEP || mode == VLA_SCHED_MONOLITHIC, "unknown execution mode");
    s->mode = mode;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

vla_status vla_sched_set_cu(vla_sched s, int default_cu, const int* cu_table) {
  try {
    vla_clear_error();
    VLA_REQUIRE(s, "null scheduler");
    auto ok = [](int c) { return c >= 8 && c <= 256 && c % 8 == 0; };
    VLA_REQUIRE(ok(default_cu), "default_cu must be a multiple of 8 in [8, 256]");
    s->default_cu = default_cu;
    s->cu_table.clear();
    if (cu_table) {
      const size_t n = (size_t)s->n_models * s->n_buckets * s->n_models * s->n_buckets;
      for (size_t i = 0; i < n; ++i) VLA_REQUIRE(cu_table[i] == 0 || ok(cu_table[i]), "bad cu_table entry");
      s->cu_table.assign(cu_table, cu_table + n);
    }
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

vla_status vla_sched_run(vla_sched s, const int64_t* t_arr, const int32_t* model, int n, int64_t drain_ns,
                         vla_request_rec* req_out, vla_lockstep_rec* ls_out, int ls_cap, int* n_ls_out) {
  try {
    vla_clear_error();
    VLA_REQUIRE(s && (n == 0 || (t_arr && model && req_out)) && n_ls_out && (ls_cap == 0 || ls_out),
                "null argument");
    VLA_REQUIRE(n >= 0 && ls_cap >= 0 && drain_ns >= 0, "negative size");
    VLA_REQUIRE(s->exec_kind != 0, "no executor set");
    for (int i = 0; i < n; ++i) {
      VLA_REQUIRE(model[i] >= 0 && model[i] < s->n_models, "request model index out of range");
      VLA_REQUIRE(t_arr[i] >= 0 && (i == 0 || t_arr[i] >= t_arr[i - 1]), "arrivals must be sorted and >= 0");
      req_out[i] = vla_request_rec{t_arr[i], -1, -1, model[i], 0};
    }
    const bool sim = s->exec_kind == 1;
    const int64_t horizon = (n ? t_arr[n - 1] : 0) + drain_ns;
    const auto wall0 = std::chrono::steady_clock::now();
    auto wall_ns = [&] {
      return (int64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - wall0)
          .count();
    };
    int64_t t_sim = 0;
    auto now_ns = [&] { return sim ? t_sim : wall_ns(); };

    std::vector<std::deque<int>> q(s->n_models);
    int next = 0, rr = 0, k = 0, n_ls = 0;
    int buf_model = -1, buf_slot = 0;
    std::vector<int> buf;                     // requests waiting for the action stage
    while (true) {
      int64_t now = now_ns();
      while (next < n && t_arr[next] <= now) q[model[next]].push_back(next), ++next;
      bool any_q = false;
      for (auto& d : q) any_q |= !d.empty();
      if (!any_q && buf.empty()) {
        if (next >= n) break;                 // everything served
        // idle until the next arrival
        if (sim) t_sim = t_arr[next];
        else {
          const int64_t wait = t_arr[next] - wall_ns();
          if (wait > 0) std::this_thread::sleep_for(std::chrono::nanoseconds(wait));
        }
        continue;
      }
      if (now > horizon) break;               // drain budget exhausted
      // ---- VLM batch: queue choice and power-of-two admission
      int mv = -1, bv = 0;
      if (any_q) {
        if (s->policy == VLA_SCHED_ESF) {
          int64_t best = 0;
          for (int m = 0; m < s->n_models; ++m) {
            if (q[m].empty()) continue;
            const int64_t rem = s->slo_ns[m] - (now - t_arr[q[m].front()]);
            if (mv < 0 || rem < best) { mv = m; best = rem; }
          }
        } else if (s->policy == VLA_SCHED_RR) {
          for (int j = 0; j < s->n_models; ++j) {
            const int m = (rr + j) % s->n_models;
            if (!q[m].empty()) { mv = m; break; }
          }
          rr = (mv + 1) % s->n_models;
        } else {
          size_t best = 0;
          for (int m = 0; m < s->n_models; ++m)
            if (q[m].size() > best) { best = q[m].size(); mv = m; }
        }
        bv = pow2_floor(std::min<int>((int)q[mv].size(), s->max_batch));
      }
      std::vector<int> vreq;
      for (int j = 0; j < bv; ++j) vreq.push_back(q[mv].front()), q[mv].pop_front();
      if (s->mode == VLA_SCHED_MONOLITHIC) {
        // the batch runs both stages back to back, unrestricted, and completes
        int64_t t_end;
        if (sim) {
          t_end = now + s->dur_ns[s->combo(mv, bv, -1, 0)] + s->dur_ns[s->combo(-1, 0, mv, bv)] +
                  2 * s->host_overhead_ns;
        } else {
          const vla_sched_model_io& x = s->io[mv];
          vla_step_args a{};
          a.vlm_model = x.model; a.vlm_batch = bv;
          a.pixels = x.pixels; a.text_ids = x.text_ids; a.state = x.state; a.kv_out = x.kv[0];
          a.vlm_cu_count = 256;
          vla_status st = vla_step(&a, s->join);
          if (st == VLA_OK) {
            vla_step_args d{};
            d.adit_model = x.model; d.adit_batch = bv;
            d.kv_in = x.kv[0]; d.noise = x.noise; d.steps = x.steps; d.actions_out = x.actions[0];
            d.vlm_cu_count = 256;
            st = vla_step(&d, s->join);
          }
          if (st != VLA_OK) throw VlaError{(int)st, std::string("monolithic step: ") + vla_last_error()};
          VLA_HIP(hipStreamSynchronize(s->join));
          t_end = wall_ns();
        }
        for (int r : vreq) req_out[r].t_vlm_start_ns = now, req_out[r].t_done_ns = t_end;
        if (n_ls < ls_cap) ls_out[n_ls] = vla_lockstep_rec{now, t_end, mv, bv, mv, bv, 256, 0};
        ++n_ls;
        ++k;
        if (sim) t_sim = t_end;
        continue;
      }
      const int ma = buf.empty() ? -1 : buf_model, ba = (int)buf.size();
      const int slot = k & 1;
      int cu = s->default_cu;
      const size_t ci = s->combo(mv, bv, ma, ba);
      if (!s->cu_table.empty() && s->cu_table[ci] > 0) cu = s->cu_table[ci];
      // ---- execute the lockstep
      int64_t t_end;
      if (sim) {
        t_end = now + s->dur_ns[ci] + s->host_overhead_ns;
      } else {
        vla_step_args a{};
        if (bv > 0) {
          const vla_sched_model_io& x = s->io[mv];
          a.vlm_model = x.model; a.vlm_batch = bv;
          a.pixels = x.pixels; a.text_ids = x.text_ids; a.state = x.state; a.kv_out = x.kv[slot];
        }
        if (ba > 0) {
          const vla_sched_model_io& x = s->io[ma];
          a.adit_model = x.model; a.adit_batch = ba;
          a.kv_in = x.kv[buf_slot]; a.noise = x.noise; a.steps = x.steps; a.actions_out = x.actions[buf_slot];
        }
        a.vlm_cu_count = cu;
        vla_status st = vla_step(&a, s->join);
        if (st != VLA_OK) throw VlaError{(int)st, std::string("lockstep: ") + vla_last_error()};
        VLA_HIP(hipStreamSynchronize(s->join));
        t_end = wall_ns();
      }
      for (int r : buf) req_out[r].t_done_ns = t_end;
      for (int r : vreq) req_out[r].t_vlm_start_ns = now;
      if (n_ls < ls_cap) ls_out[n_ls] = vla_lockstep_rec{now, t_end, mv, bv, ma, ba, cu, slot};
      ++n_ls;
      buf = vreq;
      buf_model = mv;
      buf_slot = slot;
      ++k;
      if (sim) t_sim = t_end;
    }
    for (int i = 0; i < n; ++i) {
      vla_request_rec& r = req_out[i];
      r.met_slo = r.t_done_ns >= 0 && r.t_done_ns - r.t_arrival_ns <= s->slo_ns[r.model];
    }
    *n_ls_out = n_ls;
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  }
}

}  // extern "C"
