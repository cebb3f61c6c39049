// Model runtime: device parameters, per-stage workspaces, stage
// orchestration (VLM prefill, action-stage Euler loop) and the graph cache.
#pragma once
#include <functional>
#include <list>
#include <map>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/vla.h"
#include "common.h"

struct Mat {              // transposed weight [N][ldk] on the device
  void* p = nullptr;
  int N = 0, K = 0, ldk = 0;
};

struct VitLayer { float *ln1g, *ln1b, *ln2g, *ln2b, *bqkv, *bo, *b1, *b2; Mat qkv, wo, w1, w2; };
struct LlmLayer { float *ln1, *ln2; Mat qkv, wo, gu, wd; };
struct DitLayer { float *bqkv, *bo, *bcq, *bco, *b1, *b2; Mat qkv, wo, cq, co, w1, w2; };

struct CondCache {        // batch-independent per-step conditioning, keyed by steps
  float* phi = nullptr;   // [N][tdim]
  float* tb = nullptr;    // joint: [N][act_d] time bias of the concat MLP
  float* c1 = nullptr;    // DiT: hidden of the time MLP [N][act_d]
  float* c = nullptr;     // DiT: conditioning [N][act_d]
  float* sc = nullptr;    // DiT: SiLU(c)
  float* mods = nullptr;  // DiT: [N][L][6][act_d] (shift1, scale1, gate1, shift2, scale2, gate2)
  float* modf = nullptr;  // DiT: [N][2][act_d] (shift, scale)
};

enum Stage { STAGE_PREFILL = 0, STAGE_DENOISE = 1 };

struct GraphKey {
  int B, N;
  const void *p0, *p1, *p2, *p3;
  bool operator<(const GraphKey& o) const {
    return std::tie(B, N, p0, p1, p2, p3) < std::tie(o.B, o.N, o.p0, o.p1, o.p2, o.p3);
  }
  bool operator==(const GraphKey& o) const {
    return std::tie(B, N, p0, p1, p2, p3) == std::tie(o.B, o.N, o.p0, o.p1, o.p2, o.p3);
  }
};

struct vla_model_s {
  vla_config cfg{};
  int et = ET_F32;
  int device = 0;
  // derived sizes
  // T: image tokens per image in the prefix; Tv: patch tokens per image (the
  // ViT's sequence); S: side of the merged token blocks (1: no merge)
  int T = 0, Tv = 0, S = 1, P = 0, E = 0, Kp = 0, D = 0, Hq = 0, Hk = 0, hd = 0, Da = 0, A = 0, H = 0;
  int vhd = 0, dhd = 0, tdim = 0, Ltok = 0;

  std::vector<void*> allocs;   // every device allocation, freed on destroy

  // ---- parameters
  Mat patch; float *patch_b = nullptr, *pos = nullptr;
  std::vector<VitLayer> vit; float *vit_lnf_g = nullptr, *vit_lnf_b = nullptr; Mat proj; float* proj_b = nullptr;
  void* embed = nullptr;
  std::vector<LlmLayer> llm;
  // joint action expert
  Mat ain, t1a, t1t, t2, out; float *ain_b = nullptr, *t1_b = nullptr, *t2_b = nullptr, *lnf = nullptr, *out_b = nullptr;
  // bf16 joint expert: the action-in projection composed with the time MLP's
  // action half (W_ain W_t1a, [A] -> [Da]) and the bias that absorbs b_ain
  Mat ain_t1; float* t1_b1 = nullptr;
  std::vector<LlmLayer> act;
  // bf16 joint expert: each layer's RMSNorm gains are folded into the columns
  // of the projection that reads the normalised rows (ln1 into qkv, ln2 into
  // gu), and those projections normalise their input rows themselves
  bool act_fold = false;
  // DiT head
  float* llm_lnf = nullptr; Mat vp; float* vp_b = nullptr; Mat xkv; float* xkv_b = nullptr;
  Mat state_w; float* state_b = nullptr;
  Mat dt1, dt2, dain; float *dt1_b = nullptr, *dt2_b = nullptr, *dain_b = nullptr, *dpos = nullptr;
  Mat mod_all; float* mod_b = nullptr; std::vector<DitLayer> dit; Mat modf; float* modf_b = nullptr;
  Mat dout; float* dout_b = nullptr;
  float* rope_cs = nullptr;    // [P + horizon][hd/2][2]

  // ---- prefill workspace
  void* patches = nullptr;
  void* vshuf = nullptr;      // merged image tokens [B*n_img*T][S*S*vit_d] (S > 1)
  float* vx = nullptr; void *vz = nullptr, *vq = nullptr, *vk = nullptr, *vv = nullptr, *vo = nullptr, *vmlp = nullptr;
  float* h = nullptr; void *z = nullptr, *q = nullptr, *o = nullptr, *gu = nullptr, *kbuf = nullptr, *vbuf = nullptr;
  void* feat = nullptr; float* zero_state = nullptr;
  // ---- denoise workspace
  void *e = nullptr, *u = nullptr, *za = nullptr, *qa = nullptr, *ks = nullptr, *vs = nullptr, *oa = nullptr, *gua = nullptr;
  float* ha = nullptr;
  float* X = nullptr; void *zd = nullptr, *qd = nullptr, *kd = nullptr, *vd = nullptr, *qc = nullptr, *od = nullptr,
                          *mlp = nullptr, *zf = nullptr;

  std::map<int, CondCache> cond;
  std::mutex cond_mu;

  // split-K partial products, one workspace per stage (fp32)
  static constexpr long kSplitKFloats = 16L << 20;
  float* splitk_ws[2] = {nullptr, nullptr};
  // split-KV attention partials (fp32), one workspace per stage
  static constexpr long kAttnFloats = 8L << 20;
  float* attn_ws[2] = {nullptr, nullptr};
  void* zeros = nullptr;       // 256 zero bytes (operand zero fill of the multi-stage projection)


  // ---- graphs
  bool graphs = true;
  hipStream_t cap_stream[2] = {nullptr, nullptr};
  std::mutex graph_mu[2];
  std::map<GraphKey, hipGraphExec_t> graph_cache[2];
  std::list<GraphKey> graph_lru[2];
  static constexpr size_t kMaxGraphs = 32;

  // methods
  void init(const vla_config& c, const float* w, size_t n, int dev);
  void destroy();
  void* dalloc(size_t bytes);
  size_t kv_bytes(int B) const;
  void prefill(int B, const float* pix, const int32_t* ids, const float* state, void* kv, hipStream_t s);
  void denoise(int B, const void* kv, const float* noise, int N, float* act, hipStream_t s);
  void enqueue_prefill(int B, const float* pix, const int32_t* ids, const float* state, void* kv, hipStream_t s);
  void enqueue_denoise(int B, const void* kv, const float* noise, int N, float* act, const CondCache& cc,
                       hipStream_t s);
  const CondCache& cond_for(int N, hipStream_t s);
  void run_graph(int stage, const GraphKey& key, hipStream_t s, const std::function<void(hipStream_t)>& body);
  // One projection of a stage exactly as the stage launches it (for timing).
  GemmArgs stage_gemm(int which, int B, int layer = 0) const;
};

// Host-side validation of a shape; returns "" if valid, else the reason.
std::string vla_config_check(const vla_config& c);
size_t vla_weight_count_impl(const vla_config& c);

struct DeviceGuard {
  int old = -1;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&old) != hipSuccess) old = -1;
    if (old != dev) VLA_HIP(hipSetDevice(dev));
  }
  ~DeviceGuard() {
    int cur = -1;
    if (old >= 0 && hipGetDevice(&cur) == hipSuccess && cur != old) (void)hipSetDevice(old);
  }
};
