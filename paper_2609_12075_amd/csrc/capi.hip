// C ABI of libvla: argument validation, error reporting, and stage
// co-execution on CU-masked streams (paper Section 4.1.2: the VLM stage's
// stream is restricted to a subset of the compute units so the action stage
// always finds free units; one lockstep = one VLM batch alongside one action
// batch).
#include <cstring>
#include <list>
#include <map>
#include <mutex>
#include <set>

#include "../../include/vla.h"
#include "../../include/vla_debug.h"
#include "model.h"

// ---------------------------------------------------------------- errors
static thread_local std::string g_last_error;
void vla_set_error(const std::string& m) { g_last_error = m; }
void vla_clear_error() { g_last_error.clear(); }

template <typename F>
static vla_status guarded(F&& f) {
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
  } catch (const std::exception& e) {
    vla_set_error(e.what());
    return VLA_EINVAL;
  }
}

// ---------------------------------------------------------------- static scratch
// Scratch of the allocation-free projection entry point (vla_gemm_noalloc):
// split-K partial products, then a block of zero bytes that the staged
// kernels read for operand chunks past the end of K. Every device the library
// runs on holds its own copy for the life of the process.
constexpr long kScratchPartialBytes = 16L << 20;
constexpr long kScratchZeroBytes = 256;
static __device__ __align__(256) unsigned char scratch[kScratchPartialBytes + kScratchZeroBytes];

__global__ void zero_bytes_kernel(uint4* p, int n16) {
  for (int i = threadIdx.x; i < n16; i += blockDim.x) p[i] = make_uint4(0, 0, 0, 0);
}

namespace {

// ---------------------------------------------------------------- stream pool
// Streams are created once per (device, mask) and live until vla_shutdown.
// Mask bit i selects one compute unit; the driver spreads consecutive bits
// over the accelerator dies (XCDs) first, so the lowest k bits give k/8
// units on each of the 8 XCDs.
struct DevicePool {
  std::map<int, hipStream_t> vlm;     // key: cu count (256 = unrestricted)
  std::map<int, hipStream_t> adit;    // key: cu count from the top of the mask
  std::list<std::pair<bool, int>> masked_lru;   // (is adit, cu count) of live masked streams, most recent first
  hipEvent_t ev_start = nullptr, ev_v = nullptr, ev_a = nullptr;
  int cu_total = 0;
};

// At most this many CU-masked streams are alive per device. Measured on
// MI355X (ROCm 7, four hardware queues per process): with a fourth masked
// stream alive, every kernel replayed from a graph on the streams sharing its
// hardware queue costs ~20 us more (the action stage's ~1200 kernels per
// denoise went from 13.8 to 36 ms); with three or fewer there is no cost. A
// request for a further CU count first retires the least recently used one.
constexpr int kMaxMaskedStreams = 3;

std::mutex g_pool_mu;
std::map<int, DevicePool> g_pools;

// Models alive (created and not yet destroyed), so that vla_shutdown can
// release them and vla_destroy_model ignores handles it already released.
std::mutex g_models_mu;
std::set<vla_model_s*> g_models;

int device_cu_count(int dev) {
  hipDeviceProp_t p;
  VLA_HIP(hipGetDeviceProperties(&p, dev));
  return p.multiProcessorCount;
}

hipStream_t make_masked(int total, int count, bool from_top) {
  hipStream_t s = nullptr;
  if (count >= total) {
    VLA_HIP(hipStreamCreateWithFlags(&s, hipStreamNonBlocking));
    return s;
  }
  const int words = (total + 31) / 32;
  std::vector<uint32_t> mask(words, 0u);
  for (int i = 0; i < count; ++i) {
    const int bit = from_top ? total - 1 - i : i;
    mask[bit / 32] |= 1u << (bit % 32);
  }
  VLA_HIP(hipExtStreamCreateWithCUMask(&s, (uint32_t)words, mask.data()));
  return s;
}

DevicePool& pool(int dev) {
  auto& p = g_pools[dev];
  if (!p.ev_start) {
    p.cu_total = device_cu_count(dev);
    VLA_HIP(hipEventCreateWithFlags(&p.ev_start, hipEventDisableTiming));
    VLA_HIP(hipEventCreateWithFlags(&p.ev_v, hipEventDisableTiming));
    VLA_HIP(hipEventCreateWithFlags(&p.ev_a, hipEventDisableTiming));
    // The two unrestricted streams are created before any CU-masked one.
    // Measured on MI355X (ROCm 7): when a masked stream is created first,
    // every kernel later replayed from a graph, on any stream of the
    // process, costs ~20 us more; created in this order, up to
    // kMaxMaskedStreams masked streams cost nothing extra.
    p.vlm[256] = make_masked(p.cu_total, 256, false);
    p.adit[256] = make_masked(p.cu_total, 256, true);
  }
  return p;
}

// The stream restricted to `count` CUs (from the bottom of the mask for the
// VLM side, from the top for the action side); count >= the device's CUs is
// the unrestricted stream. Caller holds g_pool_mu.
hipStream_t pool_stream(int dev, int count, bool adit) {
  auto& p = pool(dev);
  if (count >= p.cu_total) count = 256;
  auto& m = adit ? p.adit : p.vlm;
  auto it = m.find(count);
  if (count == 256) return it->second;
  const std::pair<bool, int> key{adit, count};
  if (it != m.end()) {
    p.masked_lru.remove(key);
    p.masked_lru.push_front(key);
    return it->second;
  }
  while ((int)p.masked_lru.size() >= kMaxMaskedStreams) {
    const auto old = p.masked_lru.back();
    p.masked_lru.pop_back();
    auto& om = old.first ? p.adit : p.vlm;
    hipStream_t os = om[old.second];
    VLA_HIP(hipStreamSynchronize(os));
    VLA_HIP(hipStreamDestroy(os));
    om.erase(old.second);
  }
  hipStream_t s = make_masked(p.cu_total, count, adit);
  m[count] = s;
  p.masked_lru.push_front(key);
  return s;
}

hipStream_t vlm_stream(int dev, int count) { return pool_stream(dev, count, false); }
hipStream_t adit_stream(int dev, int count) { return pool_stream(dev, count <= 0 ? 256 : count, true); }

void check_model(vla_model m) { VLA_REQUIRE(m != nullptr, "null model"); }

// Split workspaces of the single-kernel test hooks: one per (device, kind),
// allocated on first use and kept until vla_shutdown.
std::mutex g_ws_mu;
std::map<std::pair<int, int>, float*> g_ws;

float* debug_ws(int kind, long floats) {
  auto& mu = g_ws_mu;
  auto& ws = g_ws;
  std::lock_guard<std::mutex> lk(mu);
  int dev = 0;
  VLA_HIP(hipGetDevice(&dev));
  auto it = ws.find({dev, kind});
  if (it != ws.end()) return it->second;
  float* p = nullptr;
  VLA_HIP(hipMalloc(&p, (size_t)floats * 4));
  VLA_HIP(hipMemset(p, 0, (size_t)floats * 4));   // zero (kind 2 is the operand zero buffer)
  ws[{dev, kind}] = p;
  return p;
}

void check_prefill(vla_model m, int B, const float* pix, const int32_t* ids, void* kv) {
  check_model(m);
  VLA_REQUIRE(B >= 1 && B <= m->cfg.max_batch,
              "batch " + std::to_string(B) + " outside [1, " + std::to_string(m->cfg.max_batch) + "]");
  VLA_REQUIRE(pix && ids && kv, "null pixels, text_ids or kv_out");
}

void check_denoise(vla_model m, int B, const void* kv, const float* noise, int steps, float* act) {
  check_model(m);
  VLA_REQUIRE(B >= 1 && B <= m->cfg.max_batch,
              "batch " + std::to_string(B) + " outside [1, " + std::to_string(m->cfg.max_batch) + "]");
  VLA_REQUIRE(steps >= 1 && steps <= 1000, "steps must be in [1, 1000]");
  VLA_REQUIRE(kv && noise && act, "null kv, noise or actions_out");
  VLA_REQUIRE((const void*)noise != (const void*)act, "actions_out may not alias noise");
}

// ---------------------------------------------------------------- static scratch address per device
std::mutex g_scratch_mu;
std::map<int, unsigned char*> g_scratch;     // device -> address of that device's scratch

// The device address of `scratch` on the current device, looked up once per
// device (the host-side name is not a device address).
unsigned char* scratch_ptr() {
  int dev = 0;
  VLA_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch.find(dev);
  if (it != g_scratch.end()) return it->second;
  void* p = nullptr;
  VLA_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
  VLA_REQUIRE(p != nullptr, "no device address for the static scratch");
  g_scratch[dev] = (unsigned char*)p;
  return (unsigned char*)p;
}

}  // namespace

// ---------------------------------------------------------------- model API
extern "C" {

size_t vla_weight_count(const vla_config* cfg) {
  if (!cfg) { vla_set_error("null config"); return 0; }
  std::string why = vla_config_check(*cfg);
  if (!why.empty()) { vla_set_error(why); return 0; }
  return vla_weight_count_impl(*cfg);
}

vla_status vla_create_model(const vla_config* cfg, const float* weights_host, size_t n_floats, int device,
                            vla_model* out) {
  return guarded([&] {
    VLA_REQUIRE(cfg && weights_host && out, "null config, weights or out");
    *out = nullptr;
    std::string why = vla_config_check(*cfg);
    VLA_REQUIRE(why.empty(), why);
    const size_t need = vla_weight_count_impl(*cfg);
    VLA_REQUIRE(n_floats == need, "parameter buffer has " + std::to_string(n_floats) + " values, shape needs " +
                                      std::to_string(need));
    int ndev = 0;
    VLA_HIP(hipGetDeviceCount(&ndev));
    VLA_REQUIRE(device >= 0 && device < ndev, "device " + std::to_string(device) + " not present");
    auto* m = new vla_model_s();
    try {
      m->init(*cfg, weights_host, n_floats, device);
    } catch (...) {
      try { m->destroy(); } catch (...) {}
      delete m;
      throw;
    }
    {
      std::lock_guard<std::mutex> lk(g_models_mu);
      g_models.insert(m);
    }
    *out = m;
  });
}

void vla_destroy_model(vla_model m) {
  if (!m) return;
  {
    std::lock_guard<std::mutex> lk(g_models_mu);
    if (!g_models.erase(m)) return;     // already released by vla_shutdown
  }
  try { m->destroy(); } catch (...) {}
  delete m;
}

void vla_shutdown(void) {
  std::set<int> devices;
  std::set<vla_model_s*> models;
  {
    std::lock_guard<std::mutex> lk(g_models_mu);
    models.swap(g_models);
  }
  for (vla_model_s* m : models) {
    devices.insert(m->device);
    try { m->destroy(); } catch (...) {}
    delete m;
  }
  std::lock_guard<std::mutex> lk(g_pool_mu);
  for (auto& kv : g_pools) devices.insert(kv.first);
  {
    std::lock_guard<std::mutex> wl(g_ws_mu);
    for (auto& kv : g_ws) devices.insert(kv.first.first);
  }
  int cur = -1;
  const bool have_cur = hipGetDevice(&cur) == hipSuccess;
  for (int d : devices) {
    if (hipSetDevice(d) == hipSuccess) (void)hipDeviceSynchronize();
  }
  for (auto& kv : g_pools) {
    if (hipSetDevice(kv.first) != hipSuccess) continue;
    DevicePool& p = kv.second;
    for (auto& s : p.vlm) (void)hipStreamDestroy(s.second);
    for (auto& s : p.adit) (void)hipStreamDestroy(s.second);
    for (hipEvent_t e : {p.ev_start, p.ev_v, p.ev_a})
      if (e) (void)hipEventDestroy(e);
  }
  g_pools.clear();
  {
    std::lock_guard<std::mutex> wl(g_ws_mu);
    for (auto& kv : g_ws) {
      if (hipSetDevice(kv.first.first) == hipSuccess) (void)hipFree(kv.second);
    }
    g_ws.clear();
  }
  if (have_cur) (void)hipSetDevice(cur);
}

vla_status vla_set_graphs(vla_model m, int enabled) {
  return guarded([&] {
    check_model(m);
    m->graphs = enabled != 0;
  });
}

size_t vla_kv_bytes(vla_model m, int batch) {
  if (!m) { vla_set_error("null model"); return 0; }
  if (batch < 1 || batch > m->cfg.max_batch) { vla_set_error("batch out of range"); return 0; }
  return m->kv_bytes(batch);
}

vla_status vla_prefill_ex(vla_model m, int batch, const float* pixels, const int32_t* text_ids, const float* state,
                          void* kv_out, hipStream_t stream) {
  return guarded([&] {
    check_prefill(m, batch, pixels, text_ids, kv_out);
    DeviceGuard g(m->device);
    m->prefill(batch, pixels, text_ids, m->cfg.head_kind == VLA_HEAD_DIT ? state : nullptr, kv_out, stream);
  });
}

vla_status vla_prefill(vla_model m, int batch, const float* pixels, const int32_t* text_ids, void* kv_out,
                       hipStream_t stream) {
  return vla_prefill_ex(m, batch, pixels, text_ids, nullptr, kv_out, stream);
}

vla_status vla_denoise(vla_model m, int batch, const void* kv, const float* noise, int steps, float* actions_out,
                       hipStream_t stream) {
  return guarded([&] {
    check_denoise(m, batch, kv, noise, steps, actions_out);
    DeviceGuard g(m->device);
    m->denoise(batch, kv, noise, steps, actions_out, stream);
  });
}

vla_status vla_step(const vla_step_args* a, hipStream_t join) {
  return guarded([&] {
    VLA_REQUIRE(a != nullptr, "null step args");
    const bool do_v = a->vlm_batch > 0, do_a = a->adit_batch > 0;
    VLA_REQUIRE(a->vlm_batch >= 0 && a->adit_batch >= 0, "negative batch");
    VLA_REQUIRE(do_v || do_a, "both halves empty");
    if (do_v) check_prefill(a->vlm_model, a->vlm_batch, a->pixels, a->text_ids, a->kv_out);
    if (do_a) check_denoise(a->adit_model, a->adit_batch, a->kv_in, a->noise, a->steps, a->actions_out);
    VLA_REQUIRE(a->vlm_cu_count >= 8 && a->vlm_cu_count <= 256 && a->vlm_cu_count % 8 == 0,
                "vlm_cu_count must be a multiple of 8 in [8, 256]");
    VLA_REQUIRE(a->adit_cu_count == 0 || (a->adit_cu_count >= 8 && a->adit_cu_count <= 256 && a->adit_cu_count % 8 == 0),
                "adit_cu_count must be 0 or a multiple of 8 in [8, 256]");
    const int dev = do_v ? a->vlm_model->device : a->adit_model->device;
    VLA_REQUIRE(!(do_v && do_a) || a->vlm_model->device == a->adit_model->device, "models on different devices");
    if (do_v && do_a && a->vlm_model == a->adit_model)
      VLA_REQUIRE(a->kv_out != a->kv_in, "kv_out and kv_in of one model must be different buffers");
    DeviceGuard g(dev);
    std::lock_guard<std::mutex> lk(g_pool_mu);
    DevicePool& p = pool(dev);
    hipStream_t vs = vlm_stream(dev, a->vlm_cu_count);
    // An unrestricted action half runs on the join stream itself when that is
    // a non-blocking stream: a stream waiting (from another hardware queue) on
    // an event recorded after a replayed graph slows every kernel of the graph
    // by ~0.7 us (0.57 ms per SmolVLA denoise, measured), while the join's wait
    // for this half, queued behind it on one queue, costs nothing. Blocking
    // join streams (the default stream among them) keep the separate action
    // stream: with the CU-masked VLM streams, which are blocking, they
    // serialised the two halves in measurements.
    unsigned join_flags = 0;
    const bool on_join = (a->adit_cu_count == 0 || a->adit_cu_count >= 256) && join != nullptr &&
                         hipStreamGetFlags(join, &join_flags) == hipSuccess && (join_flags & hipStreamNonBlocking);
    hipStream_t as = on_join ? join : adit_stream(dev, a->adit_cu_count);
    // both halves start after the work already queued on the join stream
    VLA_HIP(hipEventRecord(p.ev_start, join));
    if (do_v) VLA_HIP(hipStreamWaitEvent(vs, p.ev_start, 0));
    if (do_a && !on_join) VLA_HIP(hipStreamWaitEvent(as, p.ev_start, 0));
    if (do_v) a->vlm_model->prefill(a->vlm_batch, a->pixels, a->text_ids,
                                    a->vlm_model->cfg.head_kind == VLA_HEAD_DIT ? a->state : nullptr, a->kv_out, vs);
    if (do_a) a->adit_model->denoise(a->adit_batch, a->kv_in, a->noise, a->steps, a->actions_out, as);
    if (do_a && a->adit_done) VLA_HIP(hipEventRecord(a->adit_done, as));
    if (do_v) { VLA_HIP(hipEventRecord(p.ev_v, vs)); VLA_HIP(hipStreamWaitEvent(join, p.ev_v, 0)); }
    if (do_a && !on_join) { VLA_HIP(hipEventRecord(p.ev_a, as)); VLA_HIP(hipStreamWaitEvent(join, p.ev_a, 0)); }
  });
}

const char* vla_last_error(void) { return g_last_error.c_str(); }

// ---------------------------------------------------------------- test hooks
vla_status vla_debug_gemm(int M, int N, int K, const void* A, int lda, int a_type, const void* Wt, int ldw, int w_type,
                          const float* bias, int act, float* out, int ldo, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 0 && N >= 0 && K >= 0 && A && Wt && out, "bad gemm arguments");
    VLA_REQUIRE(a_type == ET_F32 || a_type == ET_BF16, "bad a_type");
    VLA_REQUIRE(w_type == ET_F32 || w_type == ET_BF16, "bad w_type");
    VLA_REQUIRE(lda >= K && ldw >= K && ldo >= N, "leading dimensions too small");
    if (w_type == ET_BF16) {
      VLA_REQUIRE(K % 8 == 0 && lda % 8 == 0 && ldw % 8 == 0, "bf16 path needs K, lda, ldw % 8 == 0");
    } else {
      VLA_REQUIRE(a_type == ET_F32, "fp32 weights need fp32 activations");
    }
    VLA_REQUIRE(act >= ACT_NONE && act <= ACT_GELU, "bad act");
    GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.A = A; g.lda = lda; g.a_type = a_type; g.W = Wt; g.ldw = ldw; g.w_type = w_type;
    g.mode = EPI_STORE; g.act = act; g.bias = bias; g.tab_period = 1; g.out = out; g.ldo = ldo; g.out_type = ET_F32;
    g.ws = debug_ws(0, vla_model_s::kSplitKFloats); g.ws_floats = vla_model_s::kSplitKFloats;
    g.zeros = debug_ws(2, 64);
    launch_gemm(g, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_gemm_bf16(int M, int N, int K, const void* A, int lda, const void* Wt, int ldw, const float* bias,
                               int glu, int act, int rms, float eps, void* out, int ldo, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 0 && N >= 0 && K >= 0 && A && Wt && out, "bad gemm arguments");
    VLA_REQUIRE(glu == 0 || glu == 1, "glu must be 0 or 1");
    VLA_REQUIRE(rms == 0 || (rms == 1 && K >= 8 && eps > 0.f), "rms must be 0, or 1 with K >= 8 and eps > 0");
    VLA_REQUIRE(act >= ACT_NONE && act <= ACT_GELU && !(glu && act), "bad act");
    VLA_REQUIRE(!glu || N % 2 == 0, "gate/up rows come in pairs: N must be even");
    VLA_REQUIRE(K % 8 == 0 && lda % 8 == 0 && ldw % 8 == 0, "bf16 path needs K, lda, ldw % 8 == 0");
    VLA_REQUIRE(lda >= K && ldw >= K && ldo >= (glu ? N / 2 : N), "leading dimensions too small");
    GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.A = A; g.lda = lda; g.a_type = ET_BF16; g.W = Wt; g.ldw = ldw; g.w_type = ET_BF16;
    g.mode = glu ? EPI_GEGLU : EPI_STORE; g.act = act; g.bias = bias; g.tab_period = 1; g.out = out; g.ldo = ldo;
    g.out_type = ET_BF16;
    g.ws = debug_ws(0, vla_model_s::kSplitKFloats); g.ws_floats = vla_model_s::kSplitKFloats;
    g.zeros = debug_ws(2, 64);
    if (rms) { g.rms_in = K; g.rms_eps = eps; }
    launch_gemm(g, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_gemm_noalloc(int M, int N, int K, const void* A, int lda, int a_type, const void* Wt, int ldw,
                            int w_type, const float* bias, int act, float* out, int ldo, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 0 && N >= 0 && K >= 0 && A && Wt && out, "bad gemm arguments");
    VLA_REQUIRE(a_type == ET_F32 || a_type == ET_BF16, "bad a_type");
    VLA_REQUIRE(w_type == ET_F32 || w_type == ET_BF16, "bad w_type");
    VLA_REQUIRE(lda >= K && ldw >= K && ldo >= N, "leading dimensions too small");
    if (w_type == ET_BF16) {
      VLA_REQUIRE(K % 8 == 0 && lda % 8 == 0 && ldw % 8 == 0, "bf16 path needs K, lda, ldw % 8 == 0");
    } else {
      VLA_REQUIRE(a_type == ET_F32, "fp32 weights need fp32 activations");
    }
    VLA_REQUIRE(act >= ACT_NONE && act <= ACT_GELU, "bad act");
    GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.A = A; g.lda = lda; g.a_type = a_type; g.W = Wt; g.ldw = ldw; g.w_type = w_type;
    g.mode = EPI_STORE; g.act = act; g.bias = bias; g.tab_period = 1; g.out = out; g.ldo = ldo; g.out_type = ET_F32;
    // The plan vla_debug_gemm would choose (its workspace holds
    // kSplitKFloats partials) must fit the static scratch: then this call
    // launches the same kernels over the same K ranges, with the same results.
    g.zeros = (const void*)&g;                 // planning only: any non-null address
    g.ws = (float*)&g;
    g.ws_floats = vla_model_s::kSplitKFloats;
    const GemmPlan want = gemm_plan(g);
    const long ldp = (N + 3) & ~3;
    const long need = want.splits > 1 ? (long)want.splits * M * ldp * 4 : 0;
    VLA_REQUIRE(need <= kScratchPartialBytes,
                "projection needs " + std::to_string(need) + " bytes of split-K partials; the static scratch holds " +
                    std::to_string(kScratchPartialBytes) + " (use vla_debug_gemm, which allocates)");
    g.ws_floats = kScratchPartialBytes / 4;
    const GemmPlan got = gemm_plan(g);
    VLA_REQUIRE(got.splits == want.splits && got.kind == want.kind && got.bn == want.bn && got.bm == want.bm,
                "projection plan does not fit the static scratch");
    unsigned char* p = scratch_ptr();
    g.ws = (float*)p;
    g.zeros = p + kScratchPartialBytes;
    zero_bytes_kernel<<<1, 64, 0, s>>>((uint4*)(p + kScratchPartialBytes), (int)(kScratchZeroBytes / 16));
    VLA_HIP(hipGetLastError());
    launch_gemm(g, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_resid_norm(int M, int N, int K, const void* A, const void* Wt, const float* bias, const float* gate,
                                float* x, int kind, const float* g, const float* b, float eps, void* z,
                                hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 1 && N >= 4 && K >= 8 && A && Wt && x && z, "bad resid_norm arguments");
    VLA_REQUIRE(K % 8 == 0 && N % 4 == 0 && N <= 2048, "resid_norm needs K % 8 == 0, N % 4 == 0, N <= 2048");
    VLA_REQUIRE(kind >= 0 && kind <= 2 && (kind != 2 || (g && b)), "bad norm kind");
    GemmArgs a{};
    a.M = M; a.N = N; a.K = K; a.A = A; a.lda = K; a.a_type = ET_BF16; a.W = Wt; a.ldw = K; a.w_type = ET_BF16;
    a.mode = EPI_RESID; a.bias = bias; a.gate = gate; a.tab_period = 1; a.out = x; a.ldo = N; a.out_type = ET_F32;
    a.ws = debug_ws(0, vla_model_s::kSplitKFloats); a.ws_floats = vla_model_s::kSplitKFloats;
    a.zeros = debug_ws(2, 64);
    NormArgs n{};
    n.rows = M; n.d = N; n.kind = kind; n.in = x; n.ld_in = N; n.out = z; n.ld_out = N; n.out_type = ET_BF16;
    n.g = g; n.b = b; n.eps = eps;
    launch_gemm_norm(a, n, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_gemm_rms(int M, int N, int K, const void* A, const void* Wt, const float* bias, float eps,
                              float* out, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 0 && N >= 0 && K >= 8 && A && Wt && out, "bad gemm_rms arguments");
    VLA_REQUIRE(K % 8 == 0, "gemm_rms needs K % 8 == 0");
    GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.A = A; g.lda = K; g.a_type = ET_BF16; g.W = Wt; g.ldw = K; g.w_type = ET_BF16;
    g.mode = EPI_STORE; g.bias = bias; g.tab_period = 1; g.out = out; g.ldo = N; g.out_type = ET_F32;
    g.ws = debug_ws(0, vla_model_s::kSplitKFloats); g.ws_floats = vla_model_s::kSplitKFloats;
    g.zeros = debug_ws(2, 64);
    g.rms_in = K; g.rms_eps = eps;
    launch_gemm(g, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_resid_copy(int M, int N, int K, const void* A, const void* Wt, const float* bias,
                                const float* gate, float* x, int ldx, void* xb, int ldxb, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(M >= 0 && N >= 0 && K >= 8 && A && Wt && x && xb, "bad resid_copy arguments");
    VLA_REQUIRE(K % 8 == 0, "resid_copy needs K % 8 == 0");
    VLA_REQUIRE(ldx >= N && ldxb >= N, "leading dimensions too small");
    GemmArgs a{};
    a.M = M; a.N = N; a.K = K; a.A = A; a.lda = K; a.a_type = ET_BF16; a.W = Wt; a.ldw = K; a.w_type = ET_BF16;
    a.mode = EPI_RESID; a.bias = bias; a.gate = gate; a.tab_period = 1; a.out = x; a.ldo = ldx; a.out_type = ET_F32;
    a.out2 = xb; a.ldo2 = ldxb;
    a.ws = debug_ws(0, vla_model_s::kSplitKFloats); a.ws_floats = vla_model_s::kSplitKFloats;
    a.zeros = debug_ws(2, 64);
    launch_gemm(a, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_attention(int B, int Hq, int Hkv, int Lq, int hd, int et, const void* q, const void* k0,
                               const void* v0, int len0, const void* k1, const void* v1, int len1, void* o,
                               hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(B >= 1 && Hq >= 1 && Hkv >= 1 && Hq % Hkv == 0 && Lq >= 1, "bad attention shape");
    VLA_REQUIRE(hd >= 8 && hd <= 256 && hd % 8 == 0, "hd must be a multiple of 8 in [8, 256]");
    VLA_REQUIRE(len0 >= 1 && len1 >= 0, "segment 0 needs a key");
    VLA_REQUIRE(q && k0 && v0 && o && (len1 == 0 || (k1 && v1)), "null attention buffer");
    VLA_REQUIRE(et == ET_F32 || et == ET_BF16, "bad element type");
    AttnArgs a{};
    a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.Lq = Lq; a.hd = hd; a.et = et; a.scale = 1.0f / sqrtf((float)hd);
    a.q = q; a.q_sb = (long)Hq * Lq * hd; a.q_sh = (long)Lq * hd; a.q_si = hd;
    a.seg[0] = AttnSeg{k0, (long)Hkv * len0 * hd, (long)len0 * hd, hd, v0, (long)Hkv * len0 * hd, (long)len0 * hd, hd, len0};
    a.seg[1] = AttnSeg{k1, (long)Hkv * len1 * hd, (long)len1 * hd, hd, v1, (long)Hkv * len1 * hd, (long)len1 * hd, hd, len1};
    a.o = o; a.o_sb = (long)Lq * Hq * hd; a.o_sh = hd; a.o_si = (long)Hq * hd;   // [B][Lq][Hq*hd]
    a.ws = debug_ws(1, vla_model_s::kAttnFloats); a.ws_floats = vla_model_s::kAttnFloats;
    a.zeros = debug_ws(2, 64);
    launch_attention(a, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_cu_probe(int device, int cu_count, int from_top, int blocks, int spin, int via_graph,
                              uint32_t* out, hipStream_t join) {
  return guarded([&] {
    VLA_REQUIRE(blocks >= 1 && blocks <= 65536 && spin >= 0 && spin <= 100000 && out, "bad probe arguments");
    VLA_REQUIRE(cu_count >= 8 && cu_count <= 256 && cu_count % 8 == 0, "cu_count must be a multiple of 8 in [8, 256]");
    DeviceGuard g(device);
    std::lock_guard<std::mutex> lk(g_pool_mu);
    DevicePool& p = pool(device);
    hipStream_t s = from_top ? adit_stream(device, cu_count) : vlm_stream(device, cu_count);
    VLA_HIP(hipEventRecord(p.ev_start, join));
    VLA_HIP(hipStreamWaitEvent(s, p.ev_start, 0));
    if (!via_graph) {
      launch_cu_probe(out, blocks, spin, s);
      VLA_HIP(hipGetLastError());
    } else {
      // as the stages run: captured on an unrestricted stream, replayed on
      // the restricted one
      hipStream_t cs = nullptr;
      hipGraph_t graph = nullptr;
      hipGraphExec_t exec = nullptr;
      VLA_HIP(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));
      hipError_t e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
      if (e == hipSuccess) {
        launch_cu_probe(out, blocks, spin, cs);
        e = hipStreamEndCapture(cs, &graph);
      }
      if (e == hipSuccess) e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      if (e == hipSuccess) e = hipGraphLaunch(exec, s);
      if (e == hipSuccess) e = hipStreamSynchronize(s);
      if (exec) (void)hipGraphExecDestroy(exec);
      if (graph) (void)hipGraphDestroy(graph);
      (void)hipStreamDestroy(cs);
      VLA_HIP(e);
    }
    VLA_HIP(hipEventRecord(p.ev_v, s));
    VLA_HIP(hipStreamWaitEvent(join, p.ev_v, 0));
  });
}

vla_status vla_debug_sync_probe(int kind, int grid, int iters, int words, int spin_limit, float* buf, unsigned* ctr,
                                int* err, float* sink, hipStream_t s) {
  return guarded([&] {
    VLA_REQUIRE(kind >= 0 && kind <= 2, "kind must be 0 (empty kernels), 1 (writing kernels) or 2 (grid barriers)");
    VLA_REQUIRE(grid >= 1 && grid <= 256, "grid must be in [1, 256] (the barrier needs every block resident)");
    VLA_REQUIRE(iters >= 1 && iters <= 1000 && words >= 0 && words <= 16384, "iters or words out of range");
    VLA_REQUIRE(spin_limit >= 1 && spin_limit <= 1000000, "spin_limit out of range");
    VLA_REQUIRE(sink && (words == 0 || buf) && (kind != 2 || (ctr && err)), "missing buffer");
    launch_sync_probe(kind, grid, iters, words, spin_limit, buf, ctr, err, sink, s);
    VLA_HIP(hipGetLastError());
  });
}

vla_status vla_debug_gemm_plan(int M, int N, int K, int mode, int out_bf16, int rms, int norm_follows, int* plan) {
  return guarded([&] {
    VLA_REQUIRE(M >= 1 && N >= 1 && K >= 8 && K % 8 == 0 && plan, "bad gemm_plan arguments");
    VLA_REQUIRE(mode >= EPI_STORE && mode <= EPI_EULER, "bad mode");
    VLA_REQUIRE(mode != EPI_GEGLU || N % 2 == 0, "GeGLU needs an even N");
    VLA_REQUIRE(!rms || mode != EPI_RESID, "a folded RMSNorm needs a store, QKV, GeGLU or Euler epilogue");
    // planning only: nothing below is dereferenced; the addresses are
    // 256-byte aligned stand-ins for the output, workspace and zero buffer
    const auto fake = reinterpret_cast<void*>(uintptr_t{256});
    GemmArgs g{};
    g.M = M; g.N = N; g.K = K; g.A = fake; g.lda = K; g.a_type = ET_BF16; g.W = fake; g.ldw = K; g.w_type = ET_BF16;
    g.mode = mode; g.tab_period = 1; g.out = fake; g.out_type = out_bf16 ? ET_BF16 : ET_F32;
    g.ldo = mode == EPI_GEGLU ? N / 2 : N;
    g.ws = static_cast<float*>(fake); g.ws_floats = vla_model_s::kSplitKFloats; g.zeros = fake;
    g.rms_in = rms ? K : 0; g.rms_eps = 1e-6f; g.norm_follows = norm_follows ? 1 : 0;
    const GemmPlan p = gemm_plan(g);
    plan[0] = p.bn; plan[1] = p.bm; plan[2] = p.splits; plan[3] = p.ksplit; plan[4] = p.kind;
    plan[5] = p.stages; plan[6] = p.bk; plan[7] = p.kg;
  });
}

vla_status vla_debug_replay_gemm(vla_model m, int which, int batch, int iters, hipStream_t s, double* flops,
                                 int* plan) {
  return guarded([&] {
    check_model(m);
    VLA_REQUIRE(batch >= 1 && batch <= m->cfg.max_batch, "batch out of range");
    VLA_REQUIRE(iters >= 0 && iters <= 1000000, "iters out of range");
    DeviceGuard g(m->device);
    GemmArgs a = m->stage_gemm(which, batch);
    if (flops) *flops = 2.0 * a.M * (double)a.N * (double)a.K;
    if (plan) {
      const GemmPlan p = gemm_plan(a);
      plan[0] = p.bn; plan[1] = p.bm; plan[2] = p.splits; plan[3] = a.mode; plan[4] = p.kind;
      plan[5] = p.stages; plan[6] = p.bk; plan[7] = p.kg; plan[8] = a.rms_in > 0 ? 1 : 0;
    }
    // launch i uses layer i's weights (cycling), so weights are re-read from
    // memory as in a pass over the stage rather than served from cache
    for (int i = 0; i < iters; ++i) launch_gemm(m->stage_gemm(which, batch, i), s);
    VLA_HIP(hipGetLastError());
  });
}

}  // extern "C"
