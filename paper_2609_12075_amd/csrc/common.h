// Shared definitions for libvla: element types, error plumbing and the
// launcher interfaces of the gfx950 kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include <string>

typedef __bf16 bf16;

// ---------------------------------------------------------------- errors
// Thread-local message of the last failed C-ABI call.
void vla_set_error(const std::string& msg);
void vla_clear_error();

struct VlaError {
  int status;
  std::string msg;
};

#define VLA_HIP(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      throw VlaError{3, std::string(#expr) + ": " + hipGetErrorString(e_)};        \
  } while (0)

#define VLA_REQUIRE(cond, msg)                                                     \
  do {                                                                             \
    if (!(cond)) throw VlaError{1, std::string(msg)};                              \
  } while (0)

// ---------------------------------------------------------------- kernels
enum ElemType { ET_F32 = 0, ET_BF16 = 1 };

// XCD-aware block order. The dispatcher hands workgroup L (linear id) to
// accelerator die L % 8, and each die has its own L2. This returns the
// logical block index u for L such that each die receives one contiguous run
// of logical indices (x fastest, then y, then z): blocks that share an
// operand (consecutive x) then share that die's L2. A bijection on [0, T).
__device__ __forceinline__ void xcd_remap(int& bx, int& by, int& bz) {
  const long gx = gridDim.x, gy = gridDim.y, T = gx * gy * (long)gridDim.z;
  const long L = blockIdx.x + gx * (blockIdx.y + gy * (long)blockIdx.z);
  const long q = T / 8, r = T % 8, x = L % 8, j = L / 8;
  const long u = x * q + (x < r ? x : r) + j;
  bx = (int)(u % gx);
  by = (int)((u / gx) % gy);
  bz = (int)(u / (gx * gy));
}

// The same die assignment for a matrix product's (M tile, N tile, K range)
// grid, with the logical order grouped: GM M tiles at a time, N tiles within
// a group, M fastest within a column of the group. A die's contiguous run of
// logical blocks, and so the ~64 blocks it holds at once, then covers a
// compact GM x (64 / GM) patch of output tiles, whose operand slices its L2
// shares, instead of every M tile of a few columns (which would stream all
// of A through the L2 again for every few columns).
__device__ __forceinline__ void xcd_remap_grouped(int& bx, int& by, int& bz, int GM) {
  const long gx = gridDim.x, gy = gridDim.y, T = gx * gy * (long)gridDim.z;
  const long L = blockIdx.x + gx * (blockIdx.y + gy * (long)blockIdx.z);
  const long q = T / 8, r = T % 8, x = L % 8, j = L / 8;
  const long u = x * q + (x < r ? x : r) + j;
  const long plane = gx * gy, v = u % plane;
  bz = (int)(u / plane);
  const long g = v / (GM * gy), m0 = g * GM, gm = gx - m0 < GM ? gx - m0 : GM;
  const long local = v - g * GM * gy;
  bx = (int)(m0 + local % gm);
  by = (int)(local / gm);
}

static inline size_t elem_size(int et) { return et == ET_BF16 ? 2 : 4; }

// GEMM: D[m][n] = sum_k A[m][k] * W[n][k] for m < M, n < N.
// A: row-major, element type a_type (fp32 or bf16; fp32 A is rounded to the
//    weight type on load), leading dimension lda (elements).
// W: the weight, stored transposed [N][ldw] (K contiguous) in w_type.
// The epilogue turns D into the stored result (see EpiMode).
enum EpiMode {
  EPI_STORE = 0,   // out[row(m)][n] = act(D + bias[n] + tab[m % tab_period][n]), type out_type
  EPI_RESID = 1,   // out_f32[row(m)][n] += gate[n] * (D + bias[n])  (gate optional)
  EPI_GEGLU = 2,   // W rows interleaved (gate f, up f): out[m][f] = gelu(D_2f) * D_2f+1
  EPI_QKV = 3,     // split into q / k / v heads (+bias), optional RoPE; see QkvEpi
  EPI_EULER = 4,   // x_f32[m][n] += dt * (D + bias[n])
};
enum ActMode { ACT_NONE = 0, ACT_SILU = 1, ACT_GELU = 2 };

struct QkvEpi {
  int n_q, n_kv, hd;        // heads; N = (n_q + 2 n_kv) * hd (or a suffix, see n_off)
  int n_off;                // first logical column this GEMM produces (skip q: n_q*hd)
  int seq;                  // tokens per request: m = b*seq + i
  int pos0;                 // RoPE position of token 0 (-1: no RoPE)
  const float* rope_cs;     // [pos][hd/2][2] (cos, sin) fp32, or null
  // destinations, element type = out_type; index (b, head, i, d) at
  // b*s_b + head*s_h + i*s_i + d
  void* q; long q_sb, q_sh, q_si;
  void* k; long k_sb, k_sh, k_si;
  void* v; long v_sb, v_sh, v_si;
};

struct GemmArgs {
  int M, N, K;
  const void* A; int lda; int a_type;
  const void* W; int ldw; int w_type;
  int mode, act;
  const float* bias;        // [N] or null
  const float* gate;        // [N] or null (EPI_RESID)
  const float* tab; int tab_period; int ldtab;   // additive row table (EPI_STORE) or null
  void* out; int ldo; int out_type;
  int row_group; long row_group_stride;          // out row of m: (m/g)*stride + (m%g)*ldo
  float dt;                                       // EPI_EULER
  QkvEpi qkv;
  // Optional split-K workspace (fp32). When the output tiles alone would
  // leave most compute units idle (few activation rows, as in the action
  // stage), launch_gemm cuts K into `splits` ranges: one kernel stores each
  // range's fp32 partial product in ws[split][m][n], a second kernel adds the
  // partials in split order and runs the epilogue (deterministic; no
  // inter-block synchronisation).
  float* ws; long ws_floats;
  int splits, ksplit;                             // set by launch_gemm
  // >= 16 zero bytes in device memory: operand chunks outside [0,M)x[0,K) or
  // [0,N)x[0,K) are read from here (exact zero fill, no out-of-range reads)
  const void* zeros;
  // set by launch_gemm: every epilogue access of four consecutive columns is
  // a single aligned vector access (N % 4 == 0, aligned bases and strides)
  int epi_vec;
  // planner hint: a row norm of this residual projection's output follows
  // (launch_gemm_norm); with K ranges it runs inside the reduce, without
  // them it costs a kernel of its own
  int norm_follows;
  // optional bf16 copy of an fp32 result (EPI_RESID, or EPI_STORE with fp32
  // out, no row groups): out2[m * ldo2 + n] = bf16(out value)
  void* out2; int ldo2;
  // RMSNorm folded into this projection (rms_in = d > 0): A holds rows x not
  // yet normalised and W the weights with the norm's gain folded into their
  // columns; row m of the product is scaled by rsqrt(sum_k x[m][k]^2 / d +
  // rms_eps) before the epilogue, the sum taken from the bf16 A tiles the
  // product reads (bf16 A and W, no K ranges)
  int rms_in; float rms_eps;
  // set by the launcher: the tile epilogue runs from the accumulators
  // (GeGLU or plain bf16 store on the 128-column staged tiles; no LDS pass)
  int epi_reg;
};

void launch_gemm(const GemmArgs& a, hipStream_t s);

// Launch plan of a bf16 projection: tile (bn weight rows x bm activation
// rows), number of K ranges and the K length per range.
// kind 0: register-pipelined, 1: multi-stage (K-steps of 64), 2: small-M,
// 3: large-tile, 4: multi-stage 64 x 64 or 128 x 128 tiles with K-steps of 128
// (stages 2 or 3); kg: wave groups sharing each K-step (4 waves each)
struct GemmPlan { int bn, bm, splits, ksplit, kind, stages = 2, bk = 64, kg = 1; };
GemmPlan gemm_plan(const GemmArgs& a);

// Attention: O = softmax(Q K^T * scale) V with grouped KV heads, keys drawn
// from up to two segments (e.g. the prefix cache and the action tokens' own
// keys) without concatenation. Element (b, h, i, d) of a tensor X sits at
// X + b*sb + h*sh + i*si + d.
struct AttnSeg {
  const void* k; long k_sb, k_sh, k_si;
  const void* v; long v_sb, v_sh, v_si;
  int len;
};
struct AttnArgs {
  int B, Hq, Hkv, Lq, hd;
  float scale;
  const void* q; long q_sb, q_sh, q_si;
  AttnSeg seg[2];
  void* o; long o_sb, o_sh, o_si;
  int et;                   // element type of q, k, v, o
  // Optional fp32 workspace for splitting the keys over blocks when the
  // (row tile, KV head, request) blocks alone would leave the chip idle
  // (decode at small batch): each key range stores its unnormalised output
  // and softmax statistics, and a second kernel merges them in range order.
  float* ws; long ws_floats;
  int splits, kchunk;       // set by launch_attention
  const void* zeros;        // >= 16 zero bytes (fill of chunks past hd); required for bf16
};
void launch_attention(const AttnArgs& a, hipStream_t s);

// Row normalisation of an fp32 [rows][d] stream into `out` (type out_type).
// kind 0: RMSNorm * g;  kind 1: LayerNorm * g + b (g, b optional);
// kind 2: LayerNorm * (1 + scale) + shift (adaLN modulation, vectors [d]).
// Row r is read from in + rin(r)*ld_in and written to out + rout(r)*ld_out with
// rin(r) = r + (r / skip_group + 1) * skip when skip > 0 (skip the leading
// `skip` rows of each group of skip_group + skip input rows), else r.
struct NormArgs {
  int rows, d, kind;
  const float* in; int ld_in;
  void* out; int ld_out; int out_type;
  const float* g; const float* b;
  float eps;
  int skip, skip_group;
};
void launch_norm(const NormArgs& a, hipStream_t s);

// A residual projection (mode EPI_RESID into a.out) followed by the row norm
// n of its output (n.in == a.out). When the projection splits K, the norm
// runs inside the split-K reduce (one kernel fewer); otherwise the two run
// back to back. Either way the results are those of launch_gemm then
// launch_norm with the same plan.
void launch_gemm_norm(const GemmArgs& a, const NormArgs& n, hipStream_t s);

// Patch extraction: pixels [n_images][3][hw][hw] fp32 -> rows
// [n_images * (hw/p)^2][ldo] of type out_type in (c, dy, dx) order; columns
// >= 3 p^2 are zero-filled.
void launch_im2col(const float* pix, int n_images, int hw, int p, void* out, int ldo, int out_type,
                   hipStream_t s);

// Token embedding: rows b*P + first + j of the fp32 stream h (ld d) get
// table[clamp(ids[b*n + j])] for j < n.
void launch_embed(const int32_t* ids, int B, int n, int vocab, const void* table, int table_type,
                  int d, float* h, long P, int first, hipStream_t s);

// Sinusoid of the flow time for each Euler step: out[k][i] for k < steps,
// t_k = 1 - k/steps: [sin(1000 t w_i), cos(1000 t w_i)], w_i = 10000^(-i/(dim/2)).
void launch_time_embed(int steps, int dim, float* out, hipStream_t s);

// RoPE (cos, sin) table [npos][hd/2][2] for angles pos * base^(-2i/hd),
// evaluated in double precision.
void launch_rope_table(int npos, int hd, double base, float* out, hipStream_t s);

// Elementwise helpers.
void launch_copy_f32(const float* src, float* dst, long n, hipStream_t s);
void launch_silu_f32(const float* src, float* dst, long n, hipStream_t s);
// DiT token rows: X[b][0][:] = state_tok[b][:] + pos[0][:] (fp32 out).
void launch_dit_state_rows(const void* state_tok, int et, int B, int d, int seq, const float* pos,
                           float* X, hipStream_t s);
// Parameter conversion: src fp32 [K][N] (row-major, [in, out]) -> dst [N][ldk]
// of type et, transposed, rounded (bf16: nearest even), columns >= K zero.
// perm (optional, length N): dst row n takes source column perm[n].
void launch_transpose_convert(const float* src, int K, int N, void* dst, int ldk, int et,
                              const int* perm, hipStream_t s);
void launch_convert(const float* src, long n, void* dst, int et, hipStream_t s);
void launch_round_bf16_f32(const float* src, long n, float* dst, hipStream_t s);
// W[n][k] = bf16(W[n][k] * g[k]) for n < N, k < K (bf16 rows of stride ldk)
void launch_scale_cols_bf16(void* W, long N, int K, int ldk, const float* g, hipStream_t s);

// Debug probe: each workgroup writes its hardware placement (XCC id, SE id,
// CU id) to out[block] as one word: xcc << 16 | se << 8 | cu.
void launch_cu_probe(uint32_t* out, int blocks, int spin, hipStream_t s);
void launch_sync_probe(int kind, int grid, int iters, int words, int spin_limit, float* buf, unsigned* ctr, int* err,
                       float* sink, hipStream_t s);
// Merge s x s blocks of each image's g x g patch tokens ([n_img][g*g][d],
// raster order) into [n_img][(g/s)^2][s*s*d]: block (I, J) in raster order,
// its tokens (s*I + di, s*J + dj) in (di, dj) order, channels innermost.
void launch_pixel_shuffle(const void* src, int n_img, int g, int s, int d, int et, void* dst, hipStream_t st);

// One segment of a batched copy: `bytes` bytes from src to dst (src NULL:
// zero fill). Used by the serving scheduler to gather admitted requests'
// inputs into a model's stage rows and to scatter finished action chunks.
struct CopySeg { const void* src; void* dst; long long bytes; };
// Copies n segments whose descriptors sit in device memory (segs), each cut
// into chunks of kCopyChunk bytes; max_bytes bounds every segment's size.
constexpr long long kCopyChunk = 65536;
void launch_batched_copy(const CopySeg* segs, int n, long long max_bytes, hipStream_t s);
