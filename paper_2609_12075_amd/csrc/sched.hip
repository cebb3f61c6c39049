// Host-side serving scheduler (paper Section 4.1.2 lockstep execution and
// Section 4.1.3 SLO-aware multi-model serving): per-model FIFO queues,
// earliest-SLO-first queue choice, power-of-two fixed batches, a two-slot
// VLM -> action-stage hand-off, and SLO accounting. Requests arrive online
// (submit / run_lockstep / poll) or as a whole trace; locksteps execute on the
// GPU (vla_step, wall clock) or against a lockstep-duration table (simulated
// clock). The online GPU executor gathers every admitted request's inputs
// into library-owned stage rows and scatters each finished action chunk back
// to its request.
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

enum { EXEC_NONE = 0, EXEC_SIM = 1, EXEC_GPU_FIXED = 2, EXEC_GPU_ONLINE = 3 };

struct Req {
  int64_t id = 0;
  int model = 0;
  int64_t t_arr = 0, t_vlm = -1;
  vla_request_io io{};
};

// Stage buffers of one model for the online GPU executor (max_batch rows).
struct StageBufs {
  vla_model m = nullptr;
  int steps = 1;
  float* pixels = nullptr; int32_t* ids = nullptr; float* state = nullptr;
  float* noise[2] = {nullptr, nullptr}; void* kv[2] = {nullptr, nullptr}; float* act[2] = {nullptr, nullptr};
  size_t pix_row = 0, ids_row = 0, state_row = 0, chunk_row = 0;   // bytes per request
};

template <typename F>
vla_status guard(F&& f) {
  try {
    vla_clear_error();
    f();
    return VLA_OK;
  } catch (const VlaError& e) {
    vla_set_error(e.msg);
    return (vla_status)e.status;
  } catch (const std::bad_alloc&) {
    vla_set_error("host allocation failed");
    return VLA_ENOMEM;
  }
}

}  // namespace

struct vla_sched_s {
  int n_models = 0, max_batch = 1, policy = VLA_SCHED_ESF, n_buckets = 2;
  int mode = VLA_SCHED_LOCKSTEP;
  std::vector<int64_t> slo_ns;
  // executor
  int exec_kind = EXEC_NONE;
  std::vector<int64_t> dur_ns;
  int64_t host_overhead_ns = 0;
  std::vector<vla_sched_model_io> io;        // fixed-buffer GPU executor
  std::vector<StageBufs> stage;              // online GPU executor
  std::vector<void*> dev_allocs;
  CopySeg* seg_host = nullptr;               // pinned descriptor staging
  CopySeg* seg_dev = nullptr;
  int seg_cap = 0, device = 0;
  hipStream_t join = nullptr;
  int default_cu = 256;
  std::vector<int> cu_table;
  int disjoint = 0;                          // action half on the complement of the VLM's CUs
  // chunk delivery: at the lockstep end, or when the action half ends
  // (GPU executors: events; the online executor copies the chunks out on
  // its own stream as soon as the action half is done)
  int deliver = VLA_SCHED_DONE_LOCKSTEP;
  std::vector<int64_t> adit_ns;              // simulated executor, time to the action half's end
  hipEvent_t ev_adit = nullptr, ev_scat = nullptr, ev_end = nullptr;
  hipStream_t scat = nullptr;
  // serving state
  std::vector<std::deque<Req>> q;
  std::vector<Req> buf;                      // admitted one lockstep ago, waiting for the action stage
  int buf_model = -1, buf_slot = 0, k = 0, rr = 0;
  std::deque<vla_completion> done;
  int64_t t_sim = 0;
  std::chrono::steady_clock::time_point epoch = std::chrono::steady_clock::now();

  size_t combo(int mv, int bv, int ma, int ba) const {
    const int bkv = bucket_of(bv), bka = bucket_of(ba);
    const int iv = mv < 0 ? 0 : mv, ia = ma < 0 ? 0 : ma;
    return (((size_t)iv * n_buckets + bkv) * n_models + ia) * n_buckets + bka;
  }
  bool sim() const { return exec_kind == EXEC_SIM; }
  int64_t wall_ns() const {
    return (int64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(std::chrono::steady_clock::now() - epoch)
        .count();
  }
  int64_t clock() const { return sim() ? t_sim : wall_ns(); }
  void reset_state() {
    q.assign(n_models, {});
    buf.clear();
    done.clear();
    buf_model = -1; buf_slot = 0; k = 0; rr = 0; t_sim = 0;
    epoch = std::chrono::steady_clock::now();
  }
  int pending() const {
    size_t n = buf.size();
    for (auto& d : q) n += d.size();
    return (int)n;
  }
  void free_online() {
    if (dev_allocs.empty() && !seg_host && !ev_adit) return;
    DeviceGuard g(device);
    (void)hipDeviceSynchronize();
    for (void* p : dev_allocs) (void)hipFree(p);
    dev_allocs.clear();
    if (seg_host) (void)hipHostFree(seg_host);
    seg_host = nullptr; seg_dev = nullptr; seg_cap = 0;
    stage.clear();
    for (hipEvent_t* e : {&ev_adit, &ev_scat, &ev_end})
      if (*e) { (void)hipEventDestroy(*e); *e = nullptr; }
    if (scat) { (void)hipStreamDestroy(scat); scat = nullptr; }
  }
  // events and the delivery stream of the GPU executors (on `device`, current)
  void make_events() {
    for (hipEvent_t* e : {&ev_adit, &ev_scat, &ev_end}) VLA_HIP(hipEventCreate(e));
    VLA_HIP(hipStreamCreateWithFlags(&scat, hipStreamNonBlocking));
  }
  // GPU milliseconds from event a to event b (both completed)
  static double gap_ms(hipEvent_t a, hipEvent_t b) {
    float ms = 0.f;
    VLA_HIP(hipEventElapsedTime(&ms, a, b));
    return ms > 0.f ? ms : 0.0;
  }
  void* dalloc(size_t bytes) {
    void* p = nullptr;
    VLA_HIP(hipMalloc(&p, bytes > 0 ? bytes : 16));
    dev_allocs.push_back(p);
    return p;
  }
  void complete(const std::vector<Req>& rs, int64_t t_end) {
    for (const Req& r : rs)
      done.push_back(vla_completion{r.id, r.model, t_end - r.t_arr <= slo_ns[r.model] ? 1 : 0, r.t_arr, r.t_vlm, t_end});
  }
  // One lockstep at `now` (a whole batch in Monolithic mode). Appends the
  // admitted requests' indices into their queue order to `admitted`.
  void lockstep(int64_t now, vla_lockstep_rec& rec, std::vector<Req>* admitted);
  // returns, with chunk delivery at the action half's end and an action half,
  // how long before the lockstep's end the chunks were delivered (ms), else -1
  double gpu_online_exec(int mv, const std::vector<Req>& vreq, int ma, int cu, int slot, bool monolithic);
};

double vla_sched_s::gpu_online_exec(int mv, const std::vector<Req>& vreq, int ma, int cu, int slot, bool monolithic) {
  DeviceGuard g(device);
  const int bv = (int)vreq.size(), ba = monolithic ? bv : (int)buf.size();
  // descriptors: gather (VLM batch inputs), then scatter (finished chunks)
  int n = 0;
  long long gmax = 0, smax = 0;
  const int nslot = monolithic ? 0 : slot;
  if (bv > 0) {
    const StageBufs& sb = stage[mv];
    const bool dit = sb.m->cfg.head_kind == VLA_HEAD_DIT;
    for (int j = 0; j < bv; ++j) {
      const vla_request_io& x = vreq[j].io;
      seg_host[n++] = CopySeg{x.pixels, (char*)sb.pixels + j * sb.pix_row, (long long)sb.pix_row};
      seg_host[n++] = CopySeg{x.text_ids, (char*)sb.ids + j * sb.ids_row, (long long)sb.ids_row};
      seg_host[n++] = CopySeg{x.noise, (char*)sb.noise[nslot] + j * sb.chunk_row, (long long)sb.chunk_row};
      if (dit) seg_host[n++] = CopySeg{x.state, (char*)sb.state + j * sb.state_row, (long long)sb.state_row};
    }
    gmax = (long long)sb.pix_row;
  }
  const int ng = n;
  const std::vector<Req>& fin = monolithic ? vreq : buf;
  const int mf = monolithic ? mv : ma, fslot = monolithic ? 0 : buf_slot;
  if (ba > 0) {
    const StageBufs& sb = stage[mf];
    for (int j = 0; j < ba; ++j)
      seg_host[n++] = CopySeg{(char*)sb.act[fslot] + j * sb.chunk_row, fin[j].io.actions_out, (long long)sb.chunk_row};
    smax = (long long)sb.chunk_row;
  }
  if (n > 0) VLA_HIP(hipMemcpyAsync(seg_dev, seg_host, (size_t)n * sizeof(CopySeg), hipMemcpyHostToDevice, join));
  launch_batched_copy(seg_dev, ng, gmax, join);
  auto vlm_half = [&](vla_step_args& a, int s_kv) {
    const StageBufs& sb = stage[mv];
    a.vlm_model = sb.m; a.vlm_batch = bv;
    a.pixels = sb.pixels; a.text_ids = sb.ids;
    a.state = sb.m->cfg.head_kind == VLA_HEAD_DIT ? sb.state : nullptr;
    a.kv_out = sb.kv[s_kv];
  };
  auto act_half = [&](vla_step_args& a, int m, int b, int s) {
    const StageBufs& sb = stage[m];
    a.adit_model = sb.m; a.adit_batch = b;
    a.kv_in = sb.kv[s]; a.noise = sb.noise[s]; a.steps = sb.steps; a.actions_out = sb.act[s];
  };
  vla_status st = VLA_OK;
  if (monolithic) {
    vla_step_args a{};
    vlm_half(a, 0);
    a.vlm_cu_count = 256;
    st = vla_step(&a, join);
    if (st == VLA_OK) {
      vla_step_args d{};
      act_half(d, mv, bv, 0);
      d.vlm_cu_count = 256;
      st = vla_step(&d, join);
    }
  }
  const bool early = !monolithic && ba > 0 && deliver == VLA_SCHED_DONE_ADIT;
  if (!monolithic) {
    vla_step_args a{};
    if (bv > 0) vlm_half(a, slot);
    if (ba > 0) act_half(a, ma, ba, buf_slot);
    a.vlm_cu_count = cu;
    a.adit_cu_count = disjoint && cu < 256 ? 256 - cu : 0;
    a.adit_done = early ? ev_adit : nullptr;
    st = vla_step(&a, join);
  }
  if (st != VLA_OK) throw VlaError{(int)st, std::string("lockstep: ") + vla_last_error()};
  if (early) {
    // the chunks leave as soon as the action half is done; the lockstep
    // still ends when both halves (and this copy) have finished
    VLA_HIP(hipStreamWaitEvent(scat, ev_adit, 0));
    launch_batched_copy(seg_dev + ng, n - ng, smax, scat);
    VLA_HIP(hipEventRecord(ev_scat, scat));
    VLA_HIP(hipStreamWaitEvent(join, ev_scat, 0));
  } else {
    launch_batched_copy(seg_dev + ng, n - ng, smax, join);
  }
  VLA_HIP(hipGetLastError());
  VLA_HIP(hipEventRecord(ev_end, join));
  VLA_HIP(hipStreamSynchronize(join));
  return early ? gap_ms(ev_scat, ev_end) : -1.0;
}

void vla_sched_s::lockstep(int64_t now, vla_lockstep_rec& rec, std::vector<Req>* admitted) {
  // ---- VLM batch: queue choice and power-of-two admission
  int mv = -1, bv = 0;
  bool any_q = false;
  for (auto& d : q) any_q |= !d.empty();
  if (any_q) {
    if (policy == VLA_SCHED_ESF) {
      int64_t best = 0;
      for (int m = 0; m < n_models; ++m) {
        if (q[m].empty()) continue;
        const int64_t rem = slo_ns[m] - (now - q[m].front().t_arr);
        if (mv < 0 || rem < best) { mv = m; best = rem; }
      }
    } else if (policy == VLA_SCHED_RR) {
      for (int j = 0; j < n_models; ++j) {
        const int m = (rr + j) % n_models;
        if (!q[m].empty()) { mv = m; break; }
      }
      rr = (mv + 1) % n_models;
    } else {
      size_t best = 0;
      for (int m = 0; m < n_models; ++m)
        if (q[m].size() > best) { best = q[m].size(); mv = m; }
    }
    bv = pow2_floor(std::min<int>((int)q[mv].size(), max_batch));
  }
  std::vector<Req> vreq;
  for (int j = 0; j < bv; ++j) {
    vreq.push_back(q[mv].front());
    q[mv].pop_front();
    vreq.back().t_vlm = now;
  }
  if (admitted) admitted->insert(admitted->end(), vreq.begin(), vreq.end());
  if (mode == VLA_SCHED_MONOLITHIC) {
    // the batch runs both stages back to back, unrestricted, and completes
    int64_t t_end;
    if (sim()) {
      t_end = now + dur_ns[combo(mv, bv, -1, 0)] + dur_ns[combo(-1, 0, mv, bv)] + 2 * host_overhead_ns;
    } else if (exec_kind == EXEC_GPU_ONLINE) {
      (void)gpu_online_exec(mv, vreq, -1, 256, 0, true);
      t_end = wall_ns();
    } else {
      const vla_sched_model_io& x = io[mv];
      vla_step_args a{};
      a.vlm_model = x.model; a.vlm_batch = bv;
      a.pixels = x.pixels; a.text_ids = x.text_ids; a.state = x.state; a.kv_out = x.kv[0];
      a.vlm_cu_count = 256;
      vla_status st = vla_step(&a, join);
      if (st == VLA_OK) {
        vla_step_args d{};
        d.adit_model = x.model; d.adit_batch = bv;
        d.kv_in = x.kv[0]; d.noise = x.noise; d.steps = x.steps; d.actions_out = x.actions[0];
        d.vlm_cu_count = 256;
        st = vla_step(&d, join);
      }
      if (st != VLA_OK) throw VlaError{(int)st, std::string("monolithic step: ") + vla_last_error()};
      VLA_HIP(hipStreamSynchronize(join));
      t_end = wall_ns();
    }
    complete(vreq, t_end);
    rec = vla_lockstep_rec{now, t_end, mv, bv, mv, bv, 256, 0, t_end};
    ++k;
    if (sim()) t_sim = t_end;
    return;
  }
  const int ma = buf.empty() ? -1 : buf_model, ba = (int)buf.size();
  const int slot = k & 1;
  int cu = default_cu;
  const size_t ci = combo(mv, bv, ma, ba);
  if (!cu_table.empty() && cu_table[ci] > 0) cu = cu_table[ci];
  // ---- execute the lockstep
  int64_t t_end, t_chunks;
  const bool early = ba > 0 && deliver == VLA_SCHED_DONE_ADIT;
  if (sim()) {
    t_end = now + dur_ns[ci] + host_overhead_ns;
    t_chunks = early ? std::min(t_end, now + adit_ns[ci]) : t_end;
  } else if (exec_kind == EXEC_GPU_ONLINE) {
    const double before_ms = gpu_online_exec(mv, vreq, ma, cu, slot, false);
    t_end = wall_ns();
    t_chunks = before_ms >= 0.0 ? std::max(now, t_end - (int64_t)(before_ms * 1e6)) : t_end;
  } else {
    vla_step_args a{};
    if (bv > 0) {
      const vla_sched_model_io& x = io[mv];
      a.vlm_model = x.model; a.vlm_batch = bv;
      a.pixels = x.pixels; a.text_ids = x.text_ids; a.state = x.state; a.kv_out = x.kv[slot];
    }
    if (ba > 0) {
      const vla_sched_model_io& x = io[ma];
      a.adit_model = x.model; a.adit_batch = ba;
      a.kv_in = x.kv[buf_slot]; a.noise = x.noise; a.steps = x.steps; a.actions_out = x.actions[buf_slot];
    }
    a.vlm_cu_count = cu;
    a.adit_cu_count = disjoint && cu < 256 ? 256 - cu : 0;
    a.adit_done = early ? ev_adit : nullptr;
    vla_status st = vla_step(&a, join);
    if (st != VLA_OK) throw VlaError{(int)st, std::string("lockstep: ") + vla_last_error()};
    VLA_HIP(hipEventRecord(ev_end, join));
    VLA_HIP(hipStreamSynchronize(join));
    t_end = wall_ns();
    t_chunks = early ? std::max(now, t_end - (int64_t)(gap_ms(ev_adit, ev_end) * 1e6)) : t_end;
  }
  complete(buf, t_chunks);
  rec = vla_lockstep_rec{now, t_end, mv, bv, ma, ba, cu, slot, t_chunks};
  buf = std::move(vreq);
  buf_model = mv;
  buf_slot = slot;
  ++k;
  if (sim()) t_sim = t_end;
}

extern "C" {

vla_status vla_sched_create(const vla_sched_config* cfg, vla_sched* out) {
  return guard([&] {
    VLA_REQUIRE(cfg && out, "null config or out");
    *out = nullptr;
    VLA_REQUIRE(cfg->n_models >= 1 && cfg->n_models <= 16, "n_models must be in [1, 16]");
    VLA_REQUIRE(cfg->slo_ms, "null slo_ms");
    VLA_REQUIRE(cfg->max_batch >= 1 && cfg->max_batch <= 64 && (cfg->max_batch & (cfg->max_batch - 1)) == 0,
                "max_batch must be a power of two in [1, 64]");
    VLA_REQUIRE(cfg->policy >= VLA_SCHED_ESF && cfg->policy <= VLA_SCHED_LQF, "unknown policy");
    for (int m = 0; m < cfg->n_models; ++m) VLA_REQUIRE(cfg->slo_ms[m] > 0, "slo_ms must be > 0");
    auto* s = new vla_sched_s();
    s->n_models = cfg->n_models;
    s->max_batch = cfg->max_batch;
    s->policy = cfg->policy;
    s->n_buckets = bucket_of(cfg->max_batch) + 1;
    for (int m = 0; m < cfg->n_models; ++m) s->slo_ns.push_back((int64_t)(cfg->slo_ms[m] * 1e6 + 0.5));
    s->reset_state();
    *out = s;
  });
}

void vla_sched_destroy(vla_sched s) {
  if (!s) return;
  try { s->free_online(); } catch (...) {}
  delete s;
}

vla_status vla_sched_set_sim_executor(vla_sched s, const int64_t* dur_ns, int64_t host_overhead_ns) {
  return guard([&] {
    VLA_REQUIRE(s && dur_ns, "null scheduler or table");
    VLA_REQUIRE(host_overhead_ns >= 0, "negative overhead");
    const size_t n = (size_t)s->n_models * s->n_buckets * s->n_models * s->n_buckets;
    for (size_t i = 0; i < n; ++i) VLA_REQUIRE(dur_ns[i] >= 0, "negative duration");
    s->free_online();
    s->dur_ns.assign(dur_ns, dur_ns + n);
    s->host_overhead_ns = host_overhead_ns;
    s->exec_kind = EXEC_SIM;
    s->reset_state();
  });
}

vla_status vla_sched_set_gpu_executor(vla_sched s, const vla_sched_model_io* io, hipStream_t join) {
  return guard([&] {
    VLA_REQUIRE(s && io, "null scheduler or io");
    for (int m = 0; m < s->n_models; ++m) {
      const vla_sched_model_io& x = io[m];
      VLA_REQUIRE(x.model && x.pixels && x.text_ids && x.noise && x.kv[0] && x.kv[1] && x.actions[0] && x.actions[1],
                  "model " + std::to_string(m) + ": null model or buffer");
      VLA_REQUIRE(x.kv[0] != x.kv[1] && x.actions[0] != x.actions[1], "the two hand-off slots must differ");
      VLA_REQUIRE(x.model->cfg.max_batch >= s->max_batch, "model max_batch below the scheduler's");
      VLA_REQUIRE(x.steps >= 1 && x.steps <= 1000, "steps must be in [1, 1000]");
    }
    s->free_online();
    s->device = io[0].model->device;
    {
      DeviceGuard g(s->device);
      s->make_events();
    }
    s->io.assign(io, io + s->n_models);
    s->join = join;
    s->exec_kind = EXEC_GPU_FIXED;
    s->reset_state();
  });
}

vla_status vla_sched_set_gpu_online(vla_sched s, const vla_model* models, const int* steps, hipStream_t join) {
  return guard([&] {
    VLA_REQUIRE(s && models && steps, "null scheduler, models or steps");
    for (int m = 0; m < s->n_models; ++m) {
      VLA_REQUIRE(models[m], "model " + std::to_string(m) + " is null");
      VLA_REQUIRE(models[m]->cfg.max_batch >= s->max_batch, "model max_batch below the scheduler's");
      VLA_REQUIRE(models[m]->device == models[0]->device, "models on different devices");
      VLA_REQUIRE(steps[m] >= 1 && steps[m] <= 1000, "steps must be in [1, 1000]");
    }
    s->free_online();
    s->exec_kind = EXEC_NONE;
    s->device = models[0]->device;
    DeviceGuard g(s->device);
    const size_t B = (size_t)s->max_batch;
    try {
      for (int m = 0; m < s->n_models; ++m) {
        const vla_config& c = models[m]->cfg;
        StageBufs sb;
        sb.m = models[m];
        sb.steps = steps[m];
        sb.pix_row = (size_t)c.n_img * 3 * c.img_hw * c.img_hw * 4;
        sb.ids_row = (size_t)c.n_text * 4;
        sb.state_row = (size_t)std::max(c.state_dim, 1) * 4;
        sb.chunk_row = (size_t)c.horizon * c.action_dim * 4;
        sb.pixels = (float*)s->dalloc(B * sb.pix_row);
        sb.ids = (int32_t*)s->dalloc(B * sb.ids_row);
        sb.state = (float*)s->dalloc(B * sb.state_row);
        for (int i = 0; i < 2; ++i) {
          sb.noise[i] = (float*)s->dalloc(B * sb.chunk_row);
          sb.act[i] = (float*)s->dalloc(B * sb.chunk_row);
          sb.kv[i] = s->dalloc(models[m]->kv_bytes((int)B));
        }
        s->stage.push_back(sb);
      }
      s->seg_cap = 5 * s->max_batch;
      s->seg_dev = (CopySeg*)s->dalloc((size_t)s->seg_cap * sizeof(CopySeg));
      VLA_HIP(hipHostMalloc((void**)&s->seg_host, (size_t)s->seg_cap * sizeof(CopySeg), hipHostMallocDefault));
      s->make_events();
    } catch (...) {
      s->free_online();
      throw;
    }
    s->join = join;
    s->exec_kind = EXEC_GPU_ONLINE;
    s->reset_state();
  });
}

vla_status vla_sched_set_mode(vla_sched s, int mode) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    VLA_REQUIRE(mode == VLA_SCHED_LOCKSTEP || mode == VLA_SCHED_MONOLITHIC, "unknown execution mode");
    s->mode = mode;
  });
}

vla_status vla_sched_set_delivery(vla_sched s, int when, const int64_t* adit_ns) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    VLA_REQUIRE(when == VLA_SCHED_DONE_LOCKSTEP || when == VLA_SCHED_DONE_ADIT, "unknown delivery point");
    if (adit_ns) {
      const size_t n = (size_t)s->n_models * s->n_buckets * s->n_models * s->n_buckets;
      for (size_t i = 0; i < n; ++i) VLA_REQUIRE(adit_ns[i] >= 0, "negative action-half time");
      s->adit_ns.assign(adit_ns, adit_ns + n);
    }
    s->deliver = when;
  });
}

vla_status vla_sched_set_disjoint(vla_sched s, int disjoint) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    s->disjoint = disjoint != 0;
  });
}

vla_status vla_sched_set_cu(vla_sched s, int default_cu, const int* cu_table) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    auto ok = [](int c) { return c >= 8 && c <= 256 && c % 8 == 0; };
    VLA_REQUIRE(ok(default_cu), "default_cu must be a multiple of 8 in [8, 256]");
    std::vector<int> t;
    if (cu_table) {
      const size_t n = (size_t)s->n_models * s->n_buckets * s->n_models * s->n_buckets;
      for (size_t i = 0; i < n; ++i) VLA_REQUIRE(cu_table[i] == 0 || ok(cu_table[i]), "bad cu_table entry");
      t.assign(cu_table, cu_table + n);
    }
    s->default_cu = default_cu;
    s->cu_table = std::move(t);
  });
}

int64_t vla_sched_clock_ns(vla_sched s) { return s ? s->clock() : 0; }

vla_status vla_sched_reset(vla_sched s) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    s->reset_state();
  });
}

vla_status vla_sched_submit(vla_sched s, int64_t id, int model, int64_t t_arrival_ns, const vla_request_io* io) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    VLA_REQUIRE(model >= 0 && model < s->n_models, "request model index out of range");
    VLA_REQUIRE(t_arrival_ns >= 0, "negative arrival time");
    Req r;
    r.id = id; r.model = model; r.t_arr = t_arrival_ns;
    if (s->exec_kind == EXEC_GPU_ONLINE) {
      VLA_REQUIRE(io && io->pixels && io->text_ids && io->noise && io->actions_out,
                  "the online GPU executor needs the request's pixels, text_ids, noise and actions_out");
      VLA_REQUIRE((const void*)io->noise != (const void*)io->actions_out, "actions_out may not alias noise");
    }
    if (io) r.io = *io;
    s->q[model].push_back(r);
  });
}

int vla_sched_pending(vla_sched s) { return s ? s->pending() : 0; }

vla_status vla_sched_run_lockstep(vla_sched s, vla_lockstep_rec* rec, int* ran) {
  return guard([&] {
    VLA_REQUIRE(s && ran, "null scheduler or ran");
    VLA_REQUIRE(s->exec_kind != EXEC_NONE, "no executor set");
    VLA_REQUIRE(!(s->sim() && s->deliver == VLA_SCHED_DONE_ADIT && s->adit_ns.empty()),
                "delivery at the action half's end needs its time table for the simulated executor");
    *ran = 0;
    if (s->pending() == 0) return;
    vla_lockstep_rec r{};
    s->lockstep(s->clock(), r, nullptr);
    if (rec) *rec = r;
    *ran = 1;
  });
}

vla_status vla_sched_wait_until(vla_sched s, int64_t t_ns) {
  return guard([&] {
    VLA_REQUIRE(s, "null scheduler");
    if (s->sim()) {
      s->t_sim = std::max(s->t_sim, t_ns);
    } else {
      const int64_t wait = t_ns - s->wall_ns();
      if (wait > 0) std::this_thread::sleep_for(std::chrono::nanoseconds(wait));
    }
  });
}

int vla_sched_poll(vla_sched s, vla_completion* out, int cap) {
  if (!s || !out || cap <= 0) return 0;
  int n = 0;
  while (n < cap && !s->done.empty()) {
    out[n++] = s->done.front();
    s->done.pop_front();
  }
  return n;
}

vla_status vla_sched_run_trace(vla_sched s, const int64_t* t_arr, const int32_t* model, const vla_request_io* io,
                               int n, int64_t drain_ns, vla_request_rec* req_out, vla_lockstep_rec* ls_out, int ls_cap,
                               int* n_ls_out) {
  return guard([&] {
    VLA_REQUIRE(s && (n == 0 || (t_arr && model && req_out)) && n_ls_out && (ls_cap == 0 || ls_out),
                "null argument");
    VLA_REQUIRE(n >= 0 && ls_cap >= 0 && drain_ns >= 0, "negative size");
    VLA_REQUIRE(s->exec_kind != EXEC_NONE, "no executor set");
    VLA_REQUIRE(s->exec_kind != EXEC_GPU_ONLINE || io, "the online GPU executor needs per-request inputs");
    VLA_REQUIRE(!(s->sim() && s->deliver == VLA_SCHED_DONE_ADIT && s->adit_ns.empty()),
                "delivery at the action half's end needs its time table for the simulated executor");
    for (int i = 0; i < n; ++i) {
      VLA_REQUIRE(model[i] >= 0 && model[i] < s->n_models, "request model index out of range");
      VLA_REQUIRE(t_arr[i] >= 0 && (i == 0 || t_arr[i] >= t_arr[i - 1]), "arrivals must be sorted and >= 0");
      req_out[i] = vla_request_rec{t_arr[i], -1, -1, model[i], 0};
    }
    s->reset_state();
    const int64_t horizon = (n ? t_arr[n - 1] : 0) + drain_ns;
    int next = 0, n_ls = 0;
    std::vector<Req> admitted;
    std::vector<vla_completion> got(64);
    auto collect = [&] {
      int c;
      while ((c = vla_sched_poll(s, got.data(), (int)got.size())) > 0)
        for (int j = 0; j < c; ++j) {
          vla_request_rec& r = req_out[got[j].id];
          r.t_done_ns = got[j].t_done_ns;
          r.met_slo = got[j].met_slo;
        }
    };
    while (true) {
      const int64_t now = s->clock();
      while (next < n && t_arr[next] <= now) {
        Req r;
        r.id = next; r.model = model[next]; r.t_arr = t_arr[next];
        if (io) r.io = io[next];
        s->q[r.model].push_back(r);
        ++next;
      }
      if (s->pending() == 0) {
        if (next >= n) break;                 // everything served
        const int64_t t = t_arr[next];        // idle until the next arrival
        if (s->sim()) s->t_sim = t;
        else {
          const int64_t wait = t - s->wall_ns();
          if (wait > 0) std::this_thread::sleep_for(std::chrono::nanoseconds(wait));
        }
        continue;
      }
      if (now > horizon) break;               // drain budget exhausted
      vla_lockstep_rec rec{};
      admitted.clear();
      s->lockstep(now, rec, &admitted);
      for (const Req& r : admitted) req_out[r.id].t_vlm_start_ns = r.t_vlm;
      if (n_ls < ls_cap) ls_out[n_ls] = rec;
      ++n_ls;
      collect();
    }
    collect();
    *n_ls_out = n_ls;
  });
}

vla_status vla_sched_run(vla_sched s, const int64_t* t_arr, const int32_t* model, int n, int64_t drain_ns,
                         vla_request_rec* req_out, vla_lockstep_rec* ls_out, int ls_cap, int* n_ls_out) {
  return vla_sched_run_trace(s, t_arr, model, nullptr, n, drain_ns, req_out, ls_out, ls_cap, n_ls_out);
}

}  // extern "C"
