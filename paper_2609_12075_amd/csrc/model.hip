// Model runtime: parameter upload, workspaces and the two stages of one
// batched VLA inference (paper Section 2.1: VLM -> per-layer prefix state ->
// action diffusion transformer running a fixed number of denoising steps).
// Stages are recorded once per (batch, steps, buffers) into a HIP graph and
// replayed (Section 4.1.1 records one graph per stage and batch size).
#include <algorithm>
#include <cstring>
#include <functional>

#include "model.h"

namespace {

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- shape walk
// Walks the canonical parameter order; `take(n)` is called once per tensor
// with its element count. The same walk sizes the buffer and loads it.
template <typename Take>
void walk_params(const vla_config& c, Take&& take) {
  const int E = c.vit_layers > 0 ? c.vit_d : c.llm_d;
  const int Tv = (c.img_hw / c.patch) * (c.img_hw / c.patch);    // patch tokens per image
  const long S = c.pix_shuffle > 1 ? c.pix_shuffle : 1;
  const long pd = 3L * c.patch * c.patch;
  take(pd * E); take(E); take((long)Tv * E);
  for (int l = 0; l < c.vit_layers; ++l) {
    const long d = c.vit_d, f = c.vit_mlp;
    take(d); take(d);                       // ln1
    take(d * d); take(d); take(d * d); take(d); take(d * d); take(d);   // q, k, v
    take(d * d); take(d);                   // o
    take(d); take(d);                       // ln2
    take(d * f); take(f); take(f * d); take(d);
  }
  if (c.vit_layers > 0) { take(c.vit_d); take(c.vit_d); take(S * S * c.vit_d * c.llm_d); take(c.llm_d); }
  take((long)c.vocab * c.llm_d);
  const long D = c.llm_d, Hq = (long)c.n_q * c.head_dim, Hk = (long)c.n_kv * c.head_dim, F = c.llm_mlp;
  for (int l = 0; l < c.llm_layers; ++l) {
    take(D); take(D * Hq); take(D * Hk); take(D * Hk); take(Hq * D); take(D); take(D * F); take(D * F); take(F * D);
  }
  const long A = c.action_dim, Da = c.act_d, Fa = c.act_mlp, td = c.time_dim > 0 ? c.time_dim : c.act_d;
  if (c.head_kind == VLA_HEAD_JOINT) {
    take(A * Da); take(Da); take(Da * Da); take(td * Da); take(Da); take(Da * Da); take(Da);
    for (int l = 0; l < c.act_layers; ++l) {
      take(Da); take(Da * Hq); take(Da * Hk); take(Da * Hk); take(Hq * Da); take(Da); take(Da * Fa); take(Da * Fa);
      take(Fa * Da);
    }
    take(Da); take(Da * A); take(A);
  } else {
    take(D); take(D * Da); take(Da);
    for (int l = 0; l < c.act_layers; ++l) { take(Da * Da); take(Da); take(Da * Da); take(Da); }
    take((long)c.state_dim * Da); take(Da);
    take(td * Da); take(Da); take(Da * Da); take(Da); take(A * Da); take(Da); take((long)(c.horizon + 1) * Da);
    for (int l = 0; l < c.act_layers; ++l) {
      take(Da * 6 * Da); take(6 * Da);
      for (int j = 0; j < 6; ++j) { take(Da * Da); take(Da); }   // q, k, v, o, cross q, cross o
      take(Da * Fa); take(Fa); take(Fa * Da); take(Da);
    }
    take(Da * 2 * Da); take(2 * Da); take(Da * A); take(A);
  }
}

}  // namespace

std::string vla_config_check(const vla_config& c) {
  auto pos = [](int v) { return v > 0; };
  if (c.dtype != VLA_F32 && c.dtype != VLA_BF16) return "dtype must be VLA_F32 or VLA_BF16";
  if (c.head_kind != VLA_HEAD_JOINT && c.head_kind != VLA_HEAD_DIT) return "head_kind must be JOINT or DIT";
  if (!pos(c.n_img) || !pos(c.img_hw) || !pos(c.patch) || c.img_hw % c.patch) return "image size must be a multiple of patch";
  if (c.vit_layers < 0 || (c.vit_layers > 0 && (!pos(c.vit_d) || !pos(c.vit_heads) || !pos(c.vit_mlp) || c.vit_d % c.vit_heads)))
    return "bad ViT shape";
  if (c.vit_layers > 0 && ((c.vit_d / c.vit_heads) % 8 || c.vit_d / c.vit_heads > 256)) return "ViT head dim must be a multiple of 8, <= 256";
  if (c.pix_shuffle < 0) return "pix_shuffle must be >= 0";
  if (c.pix_shuffle > 1 && (c.vit_layers == 0 || (c.img_hw / c.patch) % c.pix_shuffle))
    return "pix_shuffle > 1 needs a ViT and must divide img_hw / patch";
  if (!pos(c.n_text) || !pos(c.vocab)) return "bad text shape";
  if (!pos(c.llm_layers) || !pos(c.llm_d) || !pos(c.n_q) || !pos(c.n_kv) || !pos(c.head_dim) || !pos(c.llm_mlp)) return "bad LLM shape";
  if (c.n_q % c.n_kv) return "n_q must be a multiple of n_kv";
  if (c.head_dim % 8 || c.head_dim > 256) return "head_dim must be a multiple of 8, <= 256";
  if (!pos(c.act_layers) || !pos(c.act_d) || !pos(c.act_mlp) || !pos(c.horizon) || !pos(c.action_dim)) return "bad action shape";
  if (!pos(c.max_batch) || c.max_batch > 4096) return "max_batch must be in [1, 4096]";
  if (c.time_dim < 0 || (c.time_dim > 0 && c.time_dim % 2)) return "time_dim must be even";
  const int td = c.time_dim > 0 ? c.time_dim : c.act_d;
  if (td % 2) return "time embedding width must be even";
  if (c.head_kind == VLA_HEAD_JOINT) {
    if (c.act_layers != c.llm_layers) return "joint head: act_layers must equal llm_layers";
  } else {
    if (!pos(c.act_heads) || c.act_d % c.act_heads) return "DiT: act_d must be a multiple of act_heads";
    if ((c.act_d / c.act_heads) % 8 || c.act_d / c.act_heads > 256) return "DiT head dim must be a multiple of 8, <= 256";
    if (c.state_dim < 0) return "bad state_dim";
  }
  if (c.dtype == VLA_BF16) {
    // matrix-core path: every reduction length (except the zero-padded patch
    // vector) must be a multiple of 8 elements
    const int ks[] = {c.llm_d, c.n_q * c.head_dim, c.llm_mlp, c.act_d, c.act_mlp, c.action_dim, td};
    for (int k : ks) if (k % 8) return "bf16 models need llm_d, n_q*head_dim, llm_mlp, act_d, act_mlp, action_dim, time_dim % 8 == 0";
    if (c.vit_layers > 0 && (c.vit_d % 8 || c.vit_mlp % 8)) return "bf16 ViT widths must be multiples of 8";
    if (c.head_kind == VLA_HEAD_DIT && c.state_dim % 8) return "bf16 DiT state_dim must be a multiple of 8";
  }
  if (!(c.norm_eps >= 0.f) || !(c.rope_base > 0.f)) return "bad norm_eps / rope_base";
  // normalised widths: one wavefront holds a row in registers
  for (int d : {c.llm_d, c.act_d, c.vit_layers > 0 ? c.vit_d : 4})
    if (d % 4 || d > 2048) return "llm_d, act_d and vit_d must be multiples of 4 and <= 2048";
  return "";
}

size_t vla_weight_count_impl(const vla_config& c) {
  size_t n = 0;
  walk_params(c, [&](long k) { n += (size_t)k; });
  return n;
}

void* vla_model_s::dalloc(size_t bytes) {
  void* p = nullptr;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) throw VlaError{2, "hipMalloc(" + std::to_string(bytes) + "): " + hipGetErrorString(e)};
  allocs.push_back(p);
  return p;
}

size_t vla_model_s::kv_bytes(int B) const {
  const size_t es = elem_size(et);
  if (cfg.head_kind == VLA_HEAD_JOINT) return (size_t)cfg.llm_layers * 2 * B * cfg.n_kv * P * cfg.head_dim * es;
  return ((size_t)B * P * cfg.act_layers * 2 * Da + (size_t)B * Da) * es;
}

// ---------------------------------------------------------------- parameter upload
namespace {

struct Loader {
  vla_model_s* m;
  const float* host;
  size_t off = 0, n = 0;
  float* stage = nullptr;       // device fp32 staging
  size_t stage_cap = 0;
  int* rowmap = nullptr;        // device row map staging
  size_t rowmap_cap = 0;
  hipStream_t s = nullptr;

  const float* next(size_t cnt) {
    if (off + cnt > n) throw VlaError{1, "parameter buffer too short"};
    const float* p = host + off;
    off += cnt;
    return p;
  }
  float* upload(const float* h, size_t cnt) {
    if (cnt > stage_cap) throw VlaError{1, "internal: staging too small"};
    VLA_HIP(hipMemcpyAsync(stage, h, cnt * sizeof(float), hipMemcpyHostToDevice, s));
    return stage;
  }
  // vector parameter (gain, bias, table) -> fp32 device copy, rounded to bf16 for bf16 models
  float* vec(size_t cnt, float* dst = nullptr) {
    const float* h = next(cnt);
    if (!dst) dst = (float*)m->dalloc(cnt * 4);
    float* d = upload(h, cnt);
    if (m->et == ET_BF16) launch_round_bf16_f32(d, (long)cnt, dst, s);
    else VLA_HIP(hipMemcpyAsync(dst, d, cnt * 4, hipMemcpyDeviceToDevice, s));
    VLA_HIP(hipStreamSynchronize(s));
    return dst;
  }
  // matrix [K][N] (row-major [in, out]) -> rows of dst (transposed, ldk) via rowmap
  void mat_into(Mat& dst, int K, int N, const std::vector<int>& rows) {
    const float* h = next((size_t)K * N);
    if ((size_t)K * N == 0) return;
    float* d = upload(h, (size_t)K * N);
    if (rows.size() > rowmap_cap) throw VlaError{1, "internal: rowmap staging too small"};
    VLA_HIP(hipMemcpyAsync(rowmap, rows.data(), rows.size() * sizeof(int), hipMemcpyHostToDevice, s));
    launch_transpose_convert(d, K, N, dst.p, dst.ldk, m->et, rowmap, s);
    VLA_HIP(hipGetLastError());
    VLA_HIP(hipStreamSynchronize(s));
  }
  Mat alloc_mat(int N, int K) {
    Mat w;
    w.N = N; w.K = K;
    w.ldk = m->et == ET_BF16 ? round_up(K, 8) : K;
    w.p = m->dalloc((size_t)N * w.ldk * elem_size(m->et));
    VLA_HIP(hipMemsetAsync(w.p, 0, (size_t)N * w.ldk * elem_size(m->et), s));
    return w;
  }
  static std::vector<int> iota(int n, int base) {
    std::vector<int> r(n);
    for (int i = 0; i < n; ++i) r[i] = base + i;
    return r;
  }
  // RoPE pair interleave within each head: column h*hd + t -> row h*hd + 2t
  // (t < hd/2) or h*hd + 2(t - hd/2) + 1.
  static std::vector<int> rope_rows(int heads, int hd, int base) {
    std::vector<int> r(heads * hd);
    const int half = hd / 2;
    for (int h = 0; h < heads; ++h)
      for (int t = 0; t < hd; ++t) r[h * hd + t] = base + h * hd + (t < half ? 2 * t : 2 * (t - half) + 1);
    return r;
  }
  static std::vector<int> stride_rows(int n, int stride, int base) {
    std::vector<int> r(n);
    for (int i = 0; i < n; ++i) r[i] = base + i * stride;
    return r;
  }
  Mat mat(int K, int N) {
    Mat w = alloc_mat(N, K);
    mat_into(w, K, N, iota(N, 0));
    return w;
  }
  // matrix [K][N] computed on the host (not read from the parameter buffer)
  Mat mat_host(int K, int N, const float* h) {
    Mat w = alloc_mat(N, K);
    float* d = upload(h, (size_t)K * N);
    const std::vector<int> rows = iota(N, 0);
    if (rows.size() > rowmap_cap) throw VlaError{1, "internal: rowmap staging too small"};
    VLA_HIP(hipMemcpyAsync(rowmap, rows.data(), rows.size() * sizeof(int), hipMemcpyHostToDevice, s));
    launch_transpose_convert(d, K, N, w.p, w.ldk, m->et, rowmap, s);
    VLA_HIP(hipGetLastError());
    VLA_HIP(hipStreamSynchronize(s));
    return w;
  }
};

// round-to-nearest-even to bf16, kept in an fp32 (host side; finite inputs)
static double host_bf16(float x) {
  uint32_t u;
  std::memcpy(&u, &x, 4);
  u = (u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u;
  float y;
  std::memcpy(&y, &u, 4);
  return y;
}

}  // namespace

void vla_model_s::init(const vla_config& c, const float* w, size_t n, int dev) {
  cfg = c;
  device = dev;
  et = c.dtype == VLA_BF16 ? ET_BF16 : ET_F32;
  Tv = (c.img_hw / c.patch) * (c.img_hw / c.patch);
  S = c.pix_shuffle > 1 ? c.pix_shuffle : 1;
  T = Tv / (S * S);
  P = c.n_img * T + c.n_text;
  E = c.vit_layers > 0 ? c.vit_d : c.llm_d;
  const int pd = 3 * c.patch * c.patch;
  Kp = et == ET_BF16 ? round_up(pd, 8) : pd;
  D = c.llm_d; hd = c.head_dim; Hq = c.n_q * hd; Hk = c.n_kv * hd;
  Da = c.act_d; A = c.action_dim; H = c.horizon;
  vhd = c.vit_layers > 0 ? c.vit_d / c.vit_heads : 0;
  dhd = c.head_kind == VLA_HEAD_DIT ? c.act_d / c.act_heads : 0;
  tdim = c.time_dim > 0 ? c.time_dim : c.act_d;
  Ltok = H + (c.head_kind == VLA_HEAD_DIT ? 1 : 0);
  const int Bm = c.max_batch;
  const bool dit_head = c.head_kind == VLA_HEAD_DIT;

  DeviceGuard g(dev);
  Loader L{this, w};
  L.n = n;
  VLA_HIP(hipStreamCreateWithFlags(&L.s, hipStreamNonBlocking));
  size_t max_t = 0;
  walk_params(c, [&](long k) { max_t = std::max(max_t, (size_t)k); });
  L.stage_cap = max_t;
  L.stage = (float*)dalloc(max_t * 4);
  L.rowmap_cap = (size_t)std::max({Hq + 2 * Hk, 2 * c.llm_mlp, 2 * c.act_mlp, 6 * Da, 2 * Da, c.vit_mlp, c.vocab, D, 3 * E, 64});
  L.rowmap = (int*)dalloc(L.rowmap_cap * 4);

  try {
    // ---- vision front-end
    patch = L.alloc_mat(E, pd);
    patch.ldk = Kp;
    L.mat_into(patch, pd, E, Loader::iota(E, 0));
    patch.K = Kp;                     // the patch rows are zero-padded to Kp
    patch_b = L.vec(E);
    pos = L.vec((size_t)Tv * E);
    for (int l = 0; l < c.vit_layers; ++l) {
      VitLayer v{};
      const int d = c.vit_d, f = c.vit_mlp;
      v.ln1g = L.vec(d); v.ln1b = L.vec(d);
      v.qkv = L.alloc_mat(3 * d, d);
      v.bqkv = (float*)dalloc(3 * d * 4);
      for (int j = 0; j < 3; ++j) {
        L.mat_into(v.qkv, d, d, Loader::iota(d, j * d));
        L.vec(d, v.bqkv + j * d);
      }
      v.wo = L.mat(d, d); v.bo = L.vec(d);
      v.ln2g = L.vec(d); v.ln2b = L.vec(d);
      v.w1 = L.mat(d, f); v.b1 = L.vec(f);
      v.w2 = L.mat(f, d); v.b2 = L.vec(d);
      vit.push_back(v);
    }
    if (c.vit_layers > 0) {
      vit_lnf_g = L.vec(c.vit_d); vit_lnf_b = L.vec(c.vit_d);
      proj = L.mat(S * S * c.vit_d, D); proj_b = L.vec(D);
    }
    {   // token embedding table, kept in the model dtype
      const size_t cnt = (size_t)c.vocab * D;
      const float* h = L.next(cnt);
      float* d = L.upload(h, cnt);
      embed = dalloc(cnt * elem_size(et));
      launch_convert(d, (long)cnt, embed, et, L.s);
      VLA_HIP(hipStreamSynchronize(L.s));
    }
    // ---- LLM
    auto gemma_layer = [&](int din, int F) {
      LlmLayer y{};
      y.ln1 = L.vec(din);
      y.qkv = L.alloc_mat(Hq + 2 * Hk, din);
      L.mat_into(y.qkv, din, Hq, Loader::rope_rows(c.n_q, hd, 0));
      L.mat_into(y.qkv, din, Hk, Loader::rope_rows(c.n_kv, hd, Hq));
      L.mat_into(y.qkv, din, Hk, Loader::iota(Hk, Hq + Hk));
      y.wo = L.mat(Hq, din);
      y.ln2 = L.vec(din);
      y.gu = L.alloc_mat(2 * F, din);
      L.mat_into(y.gu, din, F, Loader::stride_rows(F, 2, 0));
      L.mat_into(y.gu, din, F, Loader::stride_rows(F, 2, 1));
      y.wd = L.mat(F, din);
      return y;
    };
    for (int l = 0; l < c.llm_layers; ++l) llm.push_back(gemma_layer(D, c.llm_mlp));
    // ---- action stage
    const int Fa = c.act_mlp;
    if (!dit_head) {
      const float* h_ain = L.host + L.off;
      ain = L.mat(A, Da);
      const float* h_ain_b = L.host + L.off;
      ain_b = L.vec(Da);
      const float* h_t1a = L.host + L.off;
      t1a = L.mat(Da, Da); t1t = L.mat(tdim, Da);
      const float* h_t1_b = L.host + L.off;
      t1_b = L.vec(Da);
      if (et == ET_BF16) {
        // no nonlinearity between the action-in projection and the time MLP's
        // action half: u = SiLU((x W_ain + b_ain) W_t1a + tau-part + b_t1)
        // = SiLU(x (W_ain W_t1a) + tau-part + (b_ain W_t1a + b_t1)), composed
        // once from the bf16 parameters in double precision (one projection
        // per Euler step instead of two)
        std::vector<double> w((size_t)A * Da, 0.0), bb(Da, 0.0);
        std::vector<double> t1r((size_t)Da * Da);
        for (size_t i = 0; i < t1r.size(); ++i) t1r[i] = host_bf16(h_t1a[i]);
        for (int a = 0; a < A; ++a)
          for (int k = 0; k < Da; ++k) {
            const double v = host_bf16(h_ain[(size_t)a * Da + k]);
            const double* row = &t1r[(size_t)k * Da];
            double* o = &w[(size_t)a * Da];
            for (int n = 0; n < Da; ++n) o[n] += v * row[n];
          }
        for (int k = 0; k < Da; ++k) {
          const double v = host_bf16(h_ain_b[k]);
          for (int n = 0; n < Da; ++n) bb[n] += v * t1r[(size_t)k * Da + n];
        }
        std::vector<float> wf(w.begin(), w.end()), bf(Da);
        for (int n = 0; n < Da; ++n) bf[n] = (float)(bb[n] + host_bf16(h_t1_b[n]));
        ain_t1 = L.mat_host(A, Da, wf.data());
        t1_b1 = (float*)dalloc((size_t)Da * 4);
        VLA_HIP(hipMemcpy(t1_b1, bf.data(), (size_t)Da * 4, hipMemcpyHostToDevice));
      }
      t2 = L.mat(Da, Da); t2_b = L.vec(Da);
      for (int l = 0; l < c.act_layers; ++l) act.push_back(gemma_layer(Da, Fa));
      act_fold = et == ET_BF16;
      if (act_fold) {
        for (LlmLayer& y : act) {
          launch_scale_cols_bf16(y.qkv.p, y.qkv.N, Da, y.qkv.ldk, y.ln1, L.s);
          launch_scale_cols_bf16(y.gu.p, y.gu.N, Da, y.gu.ldk, y.ln2, L.s);
        }
        VLA_HIP(hipGetLastError());
        VLA_HIP(hipStreamSynchronize(L.s));
      }
      lnf = L.vec(Da);
      out = L.mat(Da, A); out_b = L.vec(A);
      if (act_fold) {
        // the final RMSNorm's gain, folded like the layers' into the output
        // projection's columns
        launch_scale_cols_bf16(out.p, out.N, Da, out.ldk, lnf, L.s);
        VLA_HIP(hipGetLastError());
        VLA_HIP(hipStreamSynchronize(L.s));
      }
    } else {
      llm_lnf = L.vec(D);
      vp = L.mat(D, Da); vp_b = L.vec(Da);
      const int NL = c.act_layers;
      xkv = L.alloc_mat(NL * 2 * Da, Da);
      xkv_b = (float*)dalloc((size_t)NL * 2 * Da * 4);
      for (int l = 0; l < NL; ++l) {
        L.mat_into(xkv, Da, Da, Loader::iota(Da, (2 * l) * Da)); L.vec(Da, xkv_b + (2 * l) * Da);
        L.mat_into(xkv, Da, Da, Loader::iota(Da, (2 * l + 1) * Da)); L.vec(Da, xkv_b + (2 * l + 1) * Da);
      }
      state_w = L.mat(std::max(c.state_dim, 0), Da); state_b = L.vec(Da);
      dt1 = L.mat(tdim, Da); dt1_b = L.vec(Da);
      dt2 = L.mat(Da, Da); dt2_b = L.vec(Da);
      dain = L.mat(A, Da); dain_b = L.vec(Da);
      dpos = L.vec((size_t)(H + 1) * Da);
      mod_all = L.alloc_mat(NL * 6 * Da, Da);
      mod_b = (float*)dalloc((size_t)NL * 6 * Da * 4);
      for (int l = 0; l < NL; ++l) {
        DitLayer y{};
        L.mat_into(mod_all, Da, 6 * Da, Loader::iota(6 * Da, l * 6 * Da));
        L.vec(6 * Da, mod_b + (size_t)l * 6 * Da);
        y.qkv = L.alloc_mat(3 * Da, Da);
        y.bqkv = (float*)dalloc(3 * Da * 4);
        for (int j = 0; j < 3; ++j) { L.mat_into(y.qkv, Da, Da, Loader::iota(Da, j * Da)); L.vec(Da, y.bqkv + j * Da); }
        y.wo = L.mat(Da, Da); y.bo = L.vec(Da);
        y.cq = L.mat(Da, Da); y.bcq = L.vec(Da);
        y.co = L.mat(Da, Da); y.bco = L.vec(Da);
        y.w1 = L.mat(Da, Fa); y.b1 = L.vec(Fa);
        y.w2 = L.mat(Fa, Da); y.b2 = L.vec(Da);
        dit.push_back(y);
      }
      modf = L.mat(Da, 2 * Da); modf_b = L.vec(2 * Da);
      dout = L.mat(Da, A); dout_b = L.vec(A);
    }
    if (L.off != n) throw VlaError{1, "parameter buffer has " + std::to_string(n) + " values, shape needs " +
                                          std::to_string(L.off)};
    // RoPE table for positions 0 .. P + horizon - 1
    rope_cs = (float*)dalloc((size_t)(P + H) * (hd / 2) * 2 * 4);
    launch_rope_table(P + H, hd, (double)c.rope_base, rope_cs, L.s);

    // ---- workspaces (sized for max_batch)
    const size_t es = elem_size(et);
    const size_t Mi = (size_t)Bm * c.n_img * Tv, Mp = (size_t)Bm * P;
    patches = dalloc(Mi * Kp * es);
    if (c.vit_layers > 0) {
      const size_t d = c.vit_d;
      if (S > 1) vshuf = dalloc(Mi * d * es);
      vx = (float*)dalloc(Mi * d * 4);
      vz = dalloc(Mi * d * es); vq = dalloc(Mi * d * es); vk = dalloc(Mi * d * es); vv = dalloc(Mi * d * es);
      vo = dalloc(Mi * d * es); vmlp = dalloc(Mi * c.vit_mlp * es);
    }
    h = (float*)dalloc(Mp * D * 4);
    z = dalloc(Mp * D * es);
    q = dalloc(Mp * Hq * es);
    o = dalloc(Mp * Hq * es);
    gu = dalloc(Mp * c.llm_mlp * es);
    if (dit_head) {
      kbuf = dalloc(Mp * Hk * es); vbuf = dalloc(Mp * Hk * es);
      feat = dalloc(Mp * Da * es);
      zero_state = (float*)dalloc((size_t)Bm * std::max(c.state_dim, 1) * 4);
      VLA_HIP(hipMemsetAsync(zero_state, 0, (size_t)Bm * std::max(c.state_dim, 1) * 4, L.s));
      const size_t Mt = (size_t)Bm * Ltok;
      X = (float*)dalloc(Mt * Da * 4);
      zd = dalloc(Mt * Da * es); qd = dalloc(Mt * Da * es); kd = dalloc(Mt * Da * es); vd = dalloc(Mt * Da * es);
      qc = dalloc(Mt * Da * es); od = dalloc(Mt * Da * es); mlp = dalloc(Mt * Fa * es);
      zf = dalloc((size_t)Bm * H * Da * es);
    } else {
      const size_t Ma = (size_t)Bm * H;
      e = dalloc(Ma * Da * es); u = dalloc(Ma * Da * es);
      ha = (float*)dalloc(Ma * Da * 4);
      za = dalloc(Ma * Da * es);
      qa = dalloc(Ma * Hq * es); ks = dalloc(Ma * Hk * es); vs = dalloc(Ma * Hk * es);
      oa = dalloc(Ma * Hq * es); gua = dalloc(Ma * Fa * es);
    }
    for (int i = 0; i < 2; ++i) {
      splitk_ws[i] = (float*)dalloc((size_t)kSplitKFloats * 4);
      attn_ws[i] = (float*)dalloc((size_t)kAttnFloats * 4);
    }
    zeros = dalloc(256);
    VLA_HIP(hipMemsetAsync(zeros, 0, 256, L.s));
    VLA_HIP(hipStreamSynchronize(L.s));
    for (int i = 0; i < 2; ++i) VLA_HIP(hipStreamCreateWithFlags(&cap_stream[i], hipStreamNonBlocking));
  } catch (...) {
    (void)hipStreamDestroy(L.s);
    throw;
  }
  (void)hipStreamDestroy(L.s);
}

void vla_model_s::destroy() {
  DeviceGuard g(device);
  // every launch of this model's graphs and kernels must have finished before
  // the executables, the capture streams and the memory they use go away
  (void)hipDeviceSynchronize();
  for (int st = 0; st < 2; ++st) {
    for (auto& kv : graph_cache[st]) (void)hipGraphExecDestroy(kv.second);
    graph_cache[st].clear();
    graph_lru[st].clear();
    if (cap_stream[st]) (void)hipStreamDestroy(cap_stream[st]);
    cap_stream[st] = nullptr;
  }
  for (void* p : allocs) (void)hipFree(p);
  allocs.clear();
}

// ---------------------------------------------------------------- GEMM helpers
namespace {

// A projection of stage `st` of the model (each stage has its own split-K
// workspace, so the two stages may run concurrently on different streams).
GemmArgs gm(const vla_model_s& m, int st, const Mat& w, int M, const void* A, int lda, int a_type) {
  GemmArgs g{};
  g.M = M; g.N = w.N; g.K = (m.et == ET_BF16) ? w.ldk : w.K;
  g.A = A; g.lda = lda; g.a_type = a_type;
  g.W = w.p; g.ldw = w.ldk; g.w_type = m.et;
  g.mode = EPI_STORE; g.act = ACT_NONE;
  g.tab_period = 1;
  g.ws = m.splitk_ws[st]; g.ws_floats = vla_model_s::kSplitKFloats;
  g.zeros = m.zeros;
  return g;
}

void store(GemmArgs g, void* out, int ldo, int out_type, const float* bias, int act, hipStream_t s) {
  g.mode = EPI_STORE; g.out = out; g.ldo = ldo; g.out_type = out_type; g.bias = bias; g.act = act;
  launch_gemm(g, s);
}

void resid(GemmArgs g, float* out, int ldo, const float* bias, const float* gate, hipStream_t s) {
  g.mode = EPI_RESID; g.out = out; g.ldo = ldo; g.out_type = ET_F32; g.bias = bias; g.gate = gate;
  launch_gemm(g, s);
}

NormArgs nargs(int rows, int d, int kind, const float* in, int ld_in, void* out, int ld_out, int out_type,
               const float* g, const float* b, float eps, int skip = 0, int skip_group = 1) {
  NormArgs a{};
  a.rows = rows; a.d = d; a.kind = kind; a.in = in; a.ld_in = ld_in; a.out = out; a.ld_out = ld_out;
  a.out_type = out_type; a.g = g; a.b = b; a.eps = eps; a.skip = skip; a.skip_group = skip_group;
  return a;
}

void norm(int rows, int d, int kind, const float* in, int ld_in, void* out, int ld_out, int out_type, const float* g,
          const float* b, float eps, hipStream_t s, int skip = 0, int skip_group = 1) {
  launch_norm(nargs(rows, d, kind, in, ld_in, out, ld_out, out_type, g, b, eps, skip, skip_group), s);
}

// residual projection into out, then the row norm n of the updated rows
void resid_norm(GemmArgs g, float* out, int ldo, const float* bias, const float* gate, const NormArgs& n,
                hipStream_t s) {
  g.mode = EPI_RESID; g.out = out; g.ldo = ldo; g.out_type = ET_F32; g.bias = bias; g.gate = gate;
  launch_gemm_norm(g, n, s);
}

AttnArgs attn(const vla_model_s& m, int st, int B, int Hq, int Hkv, int Lq, int hd, int et) {
  AttnArgs a{};
  a.B = B; a.Hq = Hq; a.Hkv = Hkv; a.Lq = Lq; a.hd = hd; a.et = et;
  a.scale = 1.0f / sqrtf((float)hd);
  a.ws = m.attn_ws[st]; a.ws_floats = vla_model_s::kAttnFloats;
  a.zeros = m.zeros;
  return a;
}

}  // namespace

// ---------------------------------------------------------------- VLM stage
void vla_model_s::enqueue_prefill(int B, const float* pix, const int32_t* ids, const float* state, void* kv,
                                  hipStream_t s) {
  constexpr int ST = STAGE_PREFILL;
  const vla_config& c = cfg;
  const size_t es = elem_size(et);
  const int nimg = B * c.n_img, Mi = nimg * Tv, Mp = B * P;
  const float eps = c.norm_eps;
  const bool dit_head = c.head_kind == VLA_HEAD_DIT;

  launch_im2col(pix, nimg, c.img_hw, c.patch, patches, Kp, et, s);
  if (c.vit_layers == 0) {
    // patch embedding + position table straight into the prefix rows b*P + t
    GemmArgs g = gm(*this, ST,patch, Mi, patches, Kp, et);
    g.tab = pos; g.tab_period = T; g.ldtab = E;
    g.row_group = c.n_img * T; g.row_group_stride = (long)P * D;
    store(g, h, D, ET_F32, patch_b, ACT_NONE, s);
  } else {
    const int d = c.vit_d, nh = c.vit_heads;
    GemmArgs g = gm(*this, ST,patch, Mi, patches, Kp, et);
    g.tab = pos; g.tab_period = Tv; g.ldtab = E;
    store(g, vx, d, ET_F32, patch_b, ACT_NONE, s);
    norm(Mi, d, 1, vx, d, vz, d, et, vit[0].ln1g, vit[0].ln1b, eps, s);
    for (int l = 0; l < c.vit_layers; ++l) {
      const VitLayer& y = vit[l];
      // vz holds LN1(vx) of this layer (written by the previous step)
      GemmArgs q3 = gm(*this, ST,y.qkv, Mi, vz, d, et);
      q3.mode = EPI_QKV; q3.bias = y.bqkv; q3.out_type = et;
      QkvEpi& e3 = q3.qkv;
      e3.n_q = nh; e3.n_kv = nh; e3.hd = vhd; e3.n_off = 0; e3.seq = Tv; e3.pos0 = -1;
      e3.q = vq; e3.q_sb = (long)nh * Tv * vhd; e3.q_sh = (long)Tv * vhd; e3.q_si = vhd;
      e3.k = vk; e3.k_sb = e3.q_sb; e3.k_sh = e3.q_sh; e3.k_si = vhd;
      e3.v = vv; e3.v_sb = e3.q_sb; e3.v_sh = e3.q_sh; e3.v_si = vhd;
      launch_gemm(q3, s);
      AttnArgs at = attn(*this, ST,nimg, nh, nh, Tv, vhd, et);
      at.q = vq; at.q_sb = e3.q_sb; at.q_sh = e3.q_sh; at.q_si = vhd;
      at.seg[0] = AttnSeg{vk, e3.k_sb, e3.k_sh, vhd, vv, e3.v_sb, e3.v_sh, vhd, Tv};
      at.seg[1].len = 0;
      at.o = vo; at.o_sb = (long)Tv * d; at.o_sh = vhd; at.o_si = d;
      launch_attention(at, s);
      resid_norm(gm(*this, ST,y.wo, Mi, vo, d, et), vx, d, y.bo, nullptr,
                 nargs(Mi, d, 1, vx, d, vz, d, et, y.ln2g, y.ln2b, eps), s);
      store(gm(*this, ST,y.w1, Mi, vz, d, et), vmlp, c.vit_mlp, et, y.b1, ACT_GELU, s);
      // then LN1 of the next layer, or the final LN
      const bool last = l + 1 == c.vit_layers;
      resid_norm(gm(*this, ST,y.w2, Mi, vmlp, c.vit_mlp, et), vx, d, y.b2, nullptr,
                 nargs(Mi, d, 1, vx, d, vz, d, et, last ? vit_lnf_g : vit[l + 1].ln1g,
                       last ? vit_lnf_b : vit[l + 1].ln1b, eps), s);
    }
    // vz holds the final LayerNorm of every patch token; with S > 1 each S x S
    // block of them becomes one token of width S*S*d first
    const void* pin = vz;
    if (S > 1) {
      launch_pixel_shuffle(vz, nimg, c.img_hw / c.patch, S, d, et, vshuf, s);
      pin = vshuf;
    }
    GemmArgs gp = gm(*this, ST,proj, nimg * T, pin, S * S * d, et);
    gp.row_group = c.n_img * T; gp.row_group_stride = (long)P * D;
    store(gp, h, D, ET_F32, proj_b, ACT_NONE, s);
  }
  launch_embed(ids, B, c.n_text, c.vocab, embed, et, D, h, P, c.n_img * T, s);

  const int nq = c.n_q, nkv = c.n_kv;
  norm(Mp, D, 0, h, D, z, D, et, llm[0].ln1, nullptr, eps, s);
  for (int l = 0; l < c.llm_layers; ++l) {
    const LlmLayer& y = llm[l];
    const bool last_kv_only = !dit_head && l == c.llm_layers - 1;
    void *kd_, *vd_;
    if (!dit_head) {
      const size_t per = (size_t)B * nkv * P * hd * es;
      kd_ = (char*)kv + (size_t)(2 * l) * per;
      vd_ = (char*)kv + (size_t)(2 * l + 1) * per;
    } else {
      kd_ = kbuf; vd_ = vbuf;
    }
    // z holds RMSNorm(h) with this layer's gain (written by the previous step)
    GemmArgs q3 = gm(*this, ST,y.qkv, Mp, z, D, et);
    q3.mode = EPI_QKV; q3.out_type = et;
    QkvEpi& e3 = q3.qkv;
    e3.n_q = nq; e3.n_kv = nkv; e3.hd = hd; e3.seq = P; e3.pos0 = 0; e3.rope_cs = rope_cs;
    e3.q = q; e3.q_sb = (long)nq * P * hd; e3.q_sh = (long)P * hd; e3.q_si = hd;
    e3.k = kd_; e3.k_sb = (long)nkv * P * hd; e3.k_sh = (long)P * hd; e3.k_si = hd;
    e3.v = vd_; e3.v_sb = e3.k_sb; e3.v_sh = e3.k_sh; e3.v_si = hd;
    if (last_kv_only) {
      // only this layer's keys and values are consumed downstream
      q3.W = (const char*)y.qkv.p + (size_t)Hq * y.qkv.ldk * es;
      q3.N = 2 * Hk; e3.n_off = Hq;
    }
    launch_gemm(q3, s);
    if (last_kv_only) continue;
    AttnArgs at = attn(*this, ST,B, nq, nkv, P, hd, et);
    at.q = q; at.q_sb = e3.q_sb; at.q_sh = e3.q_sh; at.q_si = hd;
    at.seg[0] = AttnSeg{kd_, e3.k_sb, e3.k_sh, hd, vd_, e3.v_sb, e3.v_sh, hd, P};
    at.seg[1].len = 0;
    at.o = o; at.o_sb = (long)P * Hq; at.o_sh = hd; at.o_si = Hq;
    launch_attention(at, s);
    resid_norm(gm(*this, ST,y.wo, Mp, o, Hq, et), h, D, nullptr, nullptr,
               nargs(Mp, D, 0, h, D, z, D, et, y.ln2, nullptr, eps), s);
    GemmArgs gg = gm(*this, ST,y.gu, Mp, z, D, et);
    gg.mode = EPI_GEGLU; gg.out = gu; gg.ldo = c.llm_mlp; gg.out_type = et;
    launch_gemm(gg, s);
    // then the next layer's RMSNorm (the DiT head's final one after the last)
    const bool last = l + 1 == c.llm_layers;
    if (!last || dit_head)
      resid_norm(gm(*this, ST,y.wd, Mp, gu, c.llm_mlp, et), h, D, nullptr, nullptr,
                 nargs(Mp, D, 0, h, D, z, D, et, last ? llm_lnf : llm[l + 1].ln1, nullptr, eps), s);
    else
      resid(gm(*this, ST,y.wd, Mp, gu, c.llm_mlp, et), h, D, nullptr, nullptr, s);
  }
  if (dit_head) {
    const int NL = c.act_layers;
    store(gm(*this, ST,vp, Mp, z, D, et), feat, Da, et, vp_b, ACT_NONE, s);
    store(gm(*this, ST,xkv, Mp, feat, Da, et), kv, NL * 2 * Da, et, xkv_b, ACT_NONE, s);
    void* st_out = (char*)kv + (size_t)B * P * NL * 2 * Da * es;
    const float* st_in = state ? state : zero_state;
    if (c.state_dim > 0) store(gm(*this, ST,state_w, B, st_in, c.state_dim, ET_F32), st_out, Da, et, state_b, ACT_NONE, s);
    else {
      // no state input: the token is the bias alone (a K = 0 product)
      GemmArgs g0 = gm(*this, ST,state_w, B, zero_state, 1, ET_F32);
      g0.K = 0;
      store(g0, st_out, Da, et, state_b, ACT_NONE, s);
    }
  }
}

// ---------------------------------------------------------------- action stage
const CondCache& vla_model_s::cond_for(int N, hipStream_t s) {
  constexpr int ST = STAGE_DENOISE;
  std::lock_guard<std::mutex> lk(cond_mu);
  auto it = cond.find(N);
  if (it != cond.end()) return it->second;
  CondCache cc;
  const bool dit_head = cfg.head_kind == VLA_HEAD_DIT;
  cc.phi = (float*)dalloc((size_t)N * tdim * 4);
  launch_time_embed(N, tdim, cc.phi, s);
  if (!dit_head) {
    cc.tb = (float*)dalloc((size_t)N * Da * 4);
    store(gm(*this, ST,t1t, N, cc.phi, tdim, ET_F32), cc.tb, Da, ET_F32, ain_t1.p ? t1_b1 : t1_b, ACT_NONE, s);
  } else {
    const int NL = cfg.act_layers;
    cc.c1 = (float*)dalloc((size_t)N * Da * 4);
    cc.c = (float*)dalloc((size_t)N * Da * 4);
    cc.sc = (float*)dalloc((size_t)N * Da * 4);
    cc.mods = (float*)dalloc((size_t)N * NL * 6 * Da * 4);
    cc.modf = (float*)dalloc((size_t)N * 2 * Da * 4);
    store(gm(*this, ST,dt1, N, cc.phi, tdim, ET_F32), cc.c1, Da, ET_F32, dt1_b, ACT_SILU, s);
    store(gm(*this, ST,dt2, N, cc.c1, Da, ET_F32), cc.c, Da, ET_F32, dt2_b, ACT_NONE, s);
    launch_silu_f32(cc.c, cc.sc, (long)N * Da, s);
    store(gm(*this, ST,mod_all, N, cc.sc, Da, ET_F32), cc.mods, NL * 6 * Da, ET_F32, mod_b, ACT_NONE, s);
    store(gm(*this, ST,modf, N, cc.sc, Da, ET_F32), cc.modf, 2 * Da, ET_F32, modf_b, ACT_NONE, s);
  }
  VLA_HIP(hipGetLastError());
  VLA_HIP(hipStreamSynchronize(s));
  return cond.emplace(N, cc).first->second;
}

void vla_model_s::enqueue_denoise(int B, const void* kv, const float* noise, int N, float* x, const CondCache& cc,
                                  hipStream_t s) {
  constexpr int ST = STAGE_DENOISE;
  const vla_config& c = cfg;
  const size_t es = elem_size(et);
  const float eps = c.norm_eps;
  const float dt = -1.0f / (float)N;
  launch_copy_f32(noise, x, (long)B * H * A, s);

  if (c.head_kind == VLA_HEAD_JOINT) {
    const int M = B * H, nq = c.n_q, nkv = c.n_kv, Fa = c.act_mlp;
    const size_t per = (size_t)B * nkv * P * hd * es;
    for (int k = 0; k < N; ++k) {
      if (ain_t1.p) {
        store(gm(*this, ST,ain_t1, M, x, A, ET_F32), u, Da, et, cc.tb + (size_t)k * Da, ACT_SILU, s);
      } else {
        store(gm(*this, ST,ain, M, x, A, ET_F32), e, Da, et, ain_b, ACT_NONE, s);
        store(gm(*this, ST,t1a, M, e, Da, et), u, Da, et, cc.tb + (size_t)k * Da, ACT_SILU, s);
      }
      // za holds RMSNorm(ha) with the next projection's gain, or with the
      // gains folded into the projections (act_fold) bf16(ha), which the
      // projection normalises row by row
      GemmArgs g2 = gm(*this, ST,t2, M, u, Da, et);
      if (act_fold) { g2.out2 = za; g2.ldo2 = Da; }
      store(g2, ha, Da, ET_F32, t2_b, ACT_NONE, s);
      if (!act_fold) norm(M, Da, 0, ha, Da, za, Da, et, act[0].ln1, nullptr, eps, s);
      for (int l = 0; l < c.act_layers; ++l) {
        const LlmLayer& y = act[l];
        GemmArgs q3 = gm(*this, ST,y.qkv, M, za, Da, et);
        q3.mode = EPI_QKV; q3.out_type = et;
        if (act_fold) { q3.rms_in = Da; q3.rms_eps = eps; }
        QkvEpi& e3 = q3.qkv;
        e3.n_q = nq; e3.n_kv = nkv; e3.hd = hd; e3.seq = H; e3.pos0 = P; e3.rope_cs = rope_cs;
        e3.q = qa; e3.q_sb = (long)nq * H * hd; e3.q_sh = (long)H * hd; e3.q_si = hd;
        e3.k = ks; e3.k_sb = (long)nkv * H * hd; e3.k_sh = (long)H * hd; e3.k_si = hd;
        e3.v = vs; e3.v_sb = e3.k_sb; e3.v_sh = e3.k_sh; e3.v_si = hd;
        launch_gemm(q3, s);
        AttnArgs at = attn(*this, ST,B, nq, nkv, H, hd, et);
        at.q = qa; at.q_sb = e3.q_sb; at.q_sh = e3.q_sh; at.q_si = hd;
        const char* kl = (const char*)kv + (size_t)(2 * l) * per;
        const char* vl = (const char*)kv + (size_t)(2 * l + 1) * per;
        at.seg[0] = AttnSeg{kl, (long)nkv * P * hd, (long)P * hd, hd, vl, (long)nkv * P * hd, (long)P * hd, hd, P};
        at.seg[1] = AttnSeg{ks, e3.k_sb, e3.k_sh, hd, vs, e3.v_sb, e3.v_sh, hd, H};
        at.o = oa; at.o_sb = (long)H * Hq; at.o_sh = hd; at.o_si = Hq;
        launch_attention(at, s);
        GemmArgs go = gm(*this, ST,y.wo, M, oa, Hq, et);
        if (act_fold) {
          go.out2 = za; go.ldo2 = Da;
          resid(go, ha, Da, nullptr, nullptr, s);
        } else {
          resid_norm(go, ha, Da, nullptr, nullptr, nargs(M, Da, 0, ha, Da, za, Da, et, y.ln2, nullptr, eps), s);
        }
        GemmArgs gg = gm(*this, ST,y.gu, M, za, Da, et);
        gg.mode = EPI_GEGLU; gg.out = gua; gg.ldo = Fa; gg.out_type = et;
        if (act_fold) { gg.rms_in = Da; gg.rms_eps = eps; }
        launch_gemm(gg, s);
        // then the next layer's RMSNorm, or the final one
        GemmArgs gd = gm(*this, ST,y.wd, M, gua, Fa, et);
        if (act_fold) {
          gd.out2 = za; gd.ldo2 = Da;
          resid(gd, ha, Da, nullptr, nullptr, s);
        } else {
          const float* gn = l + 1 < c.act_layers ? act[l + 1].ln1 : lnf;
          resid_norm(gd, ha, Da, nullptr, nullptr, nargs(M, Da, 0, ha, Da, za, Da, et, gn, nullptr, eps), s);
        }
      }
      GemmArgs go = gm(*this, ST,out, M, za, Da, et);
      go.mode = EPI_EULER; go.out = x; go.ldo = A; go.out_type = ET_F32; go.bias = out_b; go.dt = dt;
      if (act_fold) { go.rms_in = Da; go.rms_eps = eps; }   // the final norm, folded
      launch_gemm(go, s);
    }
    return;
  }

  // ---- DiT head
  const int NL = c.act_layers, nh = c.act_heads, S = Ltok, M = B * S, Fa = c.act_mlp;
  const char* xkv_base = (const char*)kv;
  const void* st_tok = (const char*)kv + (size_t)B * P * NL * 2 * Da * es;
  const long kv_row = (long)NL * 2 * Da;
  for (int k = 0; k < N; ++k) {
    const float* mk = cc.mods + (size_t)k * NL * 6 * Da;
    launch_dit_state_rows(st_tok, et, B, Da, S, dpos, X, s);
    GemmArgs ga = gm(*this, ST,dain, B * H, x, A, ET_F32);
    ga.tab = dpos + Da; ga.tab_period = H; ga.ldtab = Da;
    ga.row_group = H; ga.row_group_stride = (long)S * Da;
    store(ga, X + Da, Da, ET_F32, dain_b, ACT_NONE, s);
    norm(M, Da, 2, X, Da, zd, Da, et, mk + 1 * Da, mk + 0 * Da, eps, s);
    for (int l = 0; l < NL; ++l) {
      const DitLayer& y = dit[l];
      const float* m6 = mk + (size_t)l * 6 * Da;
      // zd holds the adaLN-modulated LN of X for this layer's self-attention
      GemmArgs q3 = gm(*this, ST,y.qkv, M, zd, Da, et);
      q3.mode = EPI_QKV; q3.out_type = et; q3.bias = y.bqkv;
      QkvEpi& e3 = q3.qkv;
      e3.n_q = nh; e3.n_kv = nh; e3.hd = dhd; e3.seq = S; e3.pos0 = -1;
      e3.q = qd; e3.q_sb = (long)nh * S * dhd; e3.q_sh = (long)S * dhd; e3.q_si = dhd;
      e3.k = kd; e3.k_sb = e3.q_sb; e3.k_sh = e3.q_sh; e3.k_si = dhd;
      e3.v = vd; e3.v_sb = e3.q_sb; e3.v_sh = e3.q_sh; e3.v_si = dhd;
      launch_gemm(q3, s);
      AttnArgs at = attn(*this, ST,B, nh, nh, S, dhd, et);
      at.q = qd; at.q_sb = e3.q_sb; at.q_sh = e3.q_sh; at.q_si = dhd;
      at.seg[0] = AttnSeg{kd, e3.k_sb, e3.k_sh, dhd, vd, e3.v_sb, e3.v_sh, dhd, S};
      at.seg[1].len = 0;
      at.o = od; at.o_sb = (long)S * Da; at.o_sh = dhd; at.o_si = Da;
      launch_attention(at, s);
      resid_norm(gm(*this, ST,y.wo, M, od, Da, et), X, Da, y.bo, m6 + 2 * Da,
                 nargs(M, Da, 1, X, Da, zd, Da, et, nullptr, nullptr, eps), s);
      // cross-attention to the VLM features of the paired layer
      store(gm(*this, ST,y.cq, M, zd, Da, et), qc, Da, et, y.bcq, ACT_NONE, s);
      AttnArgs ac = attn(*this, ST,B, nh, nh, S, dhd, et);
      ac.q = qc; ac.q_sb = (long)S * Da; ac.q_sh = dhd; ac.q_si = Da;
      const char* kl = xkv_base + (size_t)(2 * l) * Da * es;
      const char* vl = xkv_base + (size_t)(2 * l + 1) * Da * es;
      ac.seg[0] = AttnSeg{kl, (long)P * kv_row, dhd, kv_row, vl, (long)P * kv_row, dhd, kv_row, P};
      ac.seg[1].len = 0;
      ac.o = od; ac.o_sb = (long)S * Da; ac.o_sh = dhd; ac.o_si = Da;
      launch_attention(ac, s);
      resid_norm(gm(*this, ST,y.co, M, od, Da, et), X, Da, y.bco, nullptr,
                 nargs(M, Da, 2, X, Da, zd, Da, et, m6 + 4 * Da, m6 + 3 * Da, eps), s);
      store(gm(*this, ST,y.w1, M, zd, Da, et), mlp, Fa, et, y.b1, ACT_GELU, s);
      if (l + 1 < NL) {
        // then the next layer's self-attention adaLN
        const float* n6 = m6 + 6 * Da;
        resid_norm(gm(*this, ST,y.w2, M, mlp, Fa, et), X, Da, y.b2, m6 + 5 * Da,
                   nargs(M, Da, 2, X, Da, zd, Da, et, n6 + 1 * Da, n6 + 0 * Da, eps), s);
      } else {
        resid(gm(*this, ST,y.w2, M, mlp, Fa, et), X, Da, y.b2, m6 + 5 * Da, s);
      }
    }
    const float* mf = cc.modf + (size_t)k * 2 * Da;
    norm(B * H, Da, 2, X, Da, zf, Da, et, mf + Da, mf, eps, s, /*skip=*/1, /*skip_group=*/H);
    GemmArgs go = gm(*this, ST,dout, B * H, zf, Da, et);
    go.mode = EPI_EULER; go.out = x; go.ldo = A; go.out_type = ET_F32; go.bias = dout_b; go.dt = dt;
    launch_gemm(go, s);
  }
}

// ---------------------------------------------------------------- graphs
void vla_model_s::run_graph(int stage, const GraphKey& key, hipStream_t s,
                            const std::function<void(hipStream_t)>& body) {
  if (!graphs) {
    body(s);
    VLA_HIP(hipGetLastError());
    return;
  }
  std::lock_guard<std::mutex> lk(graph_mu[stage]);
  auto& cache = graph_cache[stage];
  auto& lru = graph_lru[stage];
  auto it = cache.find(key);
  if (it == cache.end()) {
    hipStream_t cs = cap_stream[stage];
    hipGraph_t graph = nullptr;
    VLA_HIP(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal));
    try {
      body(cs);
    } catch (...) {
      (void)hipStreamEndCapture(cs, &graph);
      if (graph) (void)hipGraphDestroy(graph);
      throw;
    }
    VLA_HIP(hipStreamEndCapture(cs, &graph));
    hipGraphExec_t exec = nullptr;
    hipError_t e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    VLA_HIP(e);
    if (cache.size() >= kMaxGraphs && !lru.empty()) {
      auto old = cache.find(lru.back());
      if (old != cache.end()) {
        VLA_HIP(hipDeviceSynchronize());    // the evicted graph may still be queued
        (void)hipGraphExecDestroy(old->second);
        cache.erase(old);
      }
      lru.pop_back();
    }
    it = cache.emplace(key, exec).first;
    lru.push_front(key);
  } else {
    lru.remove(key);
    lru.push_front(key);
  }
  VLA_HIP(hipGraphLaunch(it->second, s));
}

void vla_model_s::prefill(int B, const float* pix, const int32_t* ids, const float* state, void* kv, hipStream_t s) {
  GraphKey key{B, 0, pix, ids, state, kv};
  run_graph(STAGE_PREFILL, key, s, [&](hipStream_t cs) { enqueue_prefill(B, pix, ids, state, kv, cs); });
}

void vla_model_s::denoise(int B, const void* kv, const float* noise, int N, float* act, hipStream_t s) {
  const CondCache& cc = cond_for(N, s);
  GraphKey key{B, N, kv, noise, act, nullptr};
  run_graph(STAGE_DENOISE, key, s, [&](hipStream_t cs) { enqueue_denoise(B, kv, noise, N, act, cc, cs); });
}

// ---------------------------------------------------------------- timing hook
GemmArgs vla_model_s::stage_gemm(int which, int B, int layer) const {
  const int ST = (which == 2 || which == 3) ? STAGE_DENOISE : STAGE_PREFILL;
  const vla_config& c = cfg;
  GemmArgs g{};
  const int ll = layer % std::max(1, c.llm_layers), la = layer % std::max(1, c.act_layers);
  const int lv = layer % std::max(1, c.vit_layers);
  switch (which) {
    case 0:   // VLM stage: LLM layer MLP gate/up (GeGLU epilogue)
      g = gm(*this, ST,llm[ll].gu, B * P, z, D, et);
      g.mode = EPI_GEGLU; g.out = gu; g.ldo = c.llm_mlp; g.out_type = et;
      break;
    case 1:   // VLM stage: LLM layer MLP down projection (+ residual)
      g = gm(*this, ST,llm[ll].wd, B * P, gu, c.llm_mlp, et);
      g.mode = EPI_RESID; g.out = h; g.ldo = D; g.out_type = ET_F32;
      g.norm_follows = 1;     // the stage runs it with the next layer's norm fused
      break;
    case 2:   // action stage: layer MLP up (GeGLU for the joint expert, GELU for the DiT)
      if (c.head_kind == VLA_HEAD_JOINT) {
        g = gm(*this, ST,act[la].gu, B * H, za, Da, et);
        g.mode = EPI_GEGLU; g.out = gua; g.ldo = c.act_mlp; g.out_type = et;
        if (act_fold) { g.rms_in = Da; g.rms_eps = c.norm_eps; }
      } else {
        g = gm(*this, ST,dit[la].w1, B * Ltok, zd, Da, et);
        g.mode = EPI_STORE; g.act = ACT_GELU; g.bias = dit[la].b1; g.out = mlp; g.ldo = c.act_mlp; g.out_type = et;
      }
      break;
    case 3:   // action stage: layer MLP down projection (+ residual)
      if (c.head_kind == VLA_HEAD_JOINT) {
        g = gm(*this, ST,act[la].wd, B * H, gua, c.act_mlp, et);
        g.mode = EPI_RESID; g.out = ha; g.ldo = Da; g.out_type = ET_F32;
        // with folded gains the layers write the bf16 copy that the next
        // layer's QKV (the last: the output projection) normalises; without
        // them a norm follows
        if (act_fold) { g.out2 = za; g.ldo2 = Da; }
        else g.norm_follows = 1;
      } else {
        g = gm(*this, ST,dit[la].w2, B * Ltok, mlp, c.act_mlp, et);
        g.mode = EPI_RESID; g.bias = dit[la].b2; g.out = X; g.ldo = Da; g.out_type = ET_F32;
        g.norm_follows = 1;
      }
      break;
    case 4:   // VLM stage: ViT layer MLP up (GELU)
      VLA_REQUIRE(c.vit_layers > 0, "model has no ViT");
      g = gm(*this, ST,vit[lv].w1, B * c.n_img * Tv, vz, c.vit_d, et);
      g.mode = EPI_STORE; g.act = ACT_GELU; g.bias = vit[lv].b1; g.out = vmlp; g.ldo = c.vit_mlp; g.out_type = et;
      break;
    default:
      throw VlaError{1, "unknown projection index"};
  }
  return g;
}
