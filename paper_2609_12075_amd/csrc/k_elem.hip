// Row-wise and element-wise kernels of the VLA path on gfx950: RMSNorm /
// LayerNorm / adaLN modulation (one to four wavefronts per row, wave64 reductions),
// patch extraction, token embedding, the flow-time sinusoid, RoPE tables,
// parameter conversion and a placement probe for CU-masked streams.
#include "common.h"
#include "rownorm.h"

namespace {

__device__ __forceinline__ float round_bf16(float x) { return (float)(bf16)x; }

// ---------------------------------------------------------------- norms
// A row per WPR wavefronts (rownorm::waves_per_row), each holding NVW
// 16-byte vectors per lane. The row is read once into registers with loads
// that are all issued before the first reduction (one memory round trip);
// statistics and output as in rownorm::store_row. Requires d % 4 == 0 and
// d <= 256 * NVW * WPR.
template <int NVW, int WPR>
__global__ void __launch_bounds__(256) norm_kernel(NormArgs a) {
  constexpr int RPB = 4 / WPR;
  __shared__ float red[4][2];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, w = wv % WPR;
  const int r = blockIdx.x * RPB + wv / WPR;
  if (WPR == 1 && r >= a.rows) return;              // (no barrier with one wave per row)
  const bool rok = r < a.rows;
  const int rr = rok ? r : 0;
  const int rin = a.skip > 0 ? rr + (rr / a.skip_group + 1) * a.skip : rr;
  const float* x = a.in + (long)rin * a.ld_in;
  rownorm::f4 v[NVW], g[NVW], b[NVW];
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = rownorm::col<NVW>(w, j, lane);
    v[j] = i < a.d ? *reinterpret_cast<const rownorm::f4*>(x + i) : rownorm::f4{0.f, 0.f, 0.f, 0.f};
  }
  rownorm::load_params<NVW>(a, w, lane, g, b);
  rownorm::store_row<NVW, WPR>(a, r, rok, v, wv, w, lane, g, b, red);
}

// ---------------------------------------------------------------- staging
// One thread per output element of [n_images * T][ldo].
__global__ void im2col_kernel(const float* pix, int n_images, int hw, int p, void* out, int ldo, int out_type) {
  const int gp = hw / p, T = gp * gp, kdim = 3 * p * p;
  const long total = (long)n_images * T * ldo;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total; e += (long)gridDim.x * blockDim.x) {
    const int col = (int)(e % ldo);
    const long row = e / ldo;
    float v = 0.f;
    if (col < kdim) {
      const int img = (int)(row / T), t = (int)(row % T);
      const int py = t / gp, px = t % gp;
      const int c = col / (p * p), dy = (col / p) % p, dx = col % p;
      v = pix[(((long)img * 3 + c) * hw + (py * p + dy)) * hw + px * p + dx];
    }
    if (out_type == ET_BF16) reinterpret_cast<bf16*>(out)[e] = (bf16)v;
    else reinterpret_cast<float*>(out)[e] = v;
  }
}

__global__ void embed_kernel(const int32_t* ids, int B, int n, int vocab, const void* table, int table_type,
                             int d, float* h, long P, int first) {
  const long total = (long)B * n * d;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total; e += (long)gridDim.x * blockDim.x) {
    const int i = (int)(e % d);
    const long tok = e / d;
    const int b = (int)(tok / n), j = (int)(tok % n);
    int id = ids[(long)b * n + j];
    id = id < 0 ? 0 : (id >= vocab ? vocab - 1 : id);
    const float v = table_type == ET_BF16 ? (float)reinterpret_cast<const bf16*>(table)[(long)id * d + i]
                                          : reinterpret_cast<const float*>(table)[(long)id * d + i];
    h[((long)b * P + first + j) * d + i] = v;
  }
}

// out[k][i], k < steps: angle = 1000 * t_k * 10000^(-i/half), in double.
__global__ void time_embed_kernel(int steps, int dim, float* out) {
  const int half = dim / 2;
  const int k = blockIdx.x;
  for (int i = threadIdx.x; i < half; i += blockDim.x) {
    const double t = 1.0 - (double)k / steps;
    const double w = pow(10000.0, -(double)i / half);
    const double ang = 1000.0 * t * w;
    out[(long)k * dim + i] = (float)sin(ang);
    out[(long)k * dim + half + i] = (float)cos(ang);
  }
}

__global__ void rope_table_kernel(int npos, int hd, double base, float* out) {
  const int half = hd / 2;
  const long total = (long)npos * half;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total; e += (long)gridDim.x * blockDim.x) {
    const int pos = (int)(e / half), i = (int)(e % half);
    const double ang = pos * pow(base, -2.0 * i / hd);
    out[e * 2 + 0] = (float)cos(ang);
    out[e * 2 + 1] = (float)sin(ang);
  }
}

__global__ void copy_f32_kernel(const float* src, float* dst, long n) {
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) dst[e] = src[e];
}

__global__ void silu_f32_kernel(const float* src, float* dst, long n) {
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
    const float x = src[e];
    dst[e] = x * __builtin_amdgcn_rcpf(1.0f + __expf(-x));
  }
}

__global__ void dit_state_rows_kernel(const void* st, int et, int B, int d, int seq, const float* pos, float* X) {
  const long total = (long)B * d;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total; e += (long)gridDim.x * blockDim.x) {
    const int b = (int)(e / d), i = (int)(e % d);
    const float v = et == ET_BF16 ? (float)reinterpret_cast<const bf16*>(st)[e] : reinterpret_cast<const float*>(st)[e];
    X[(long)b * seq * d + i] = v + pos[i];
  }
}

// ---------------------------------------------------------------- parameters
// 32 x 32 tiles through LDS: src [K][N] -> dst[rowmap(n)][k] (ldk), zero k >= K.
__global__ void transpose_convert_kernel(const float* src, int K, int N, void* dst, int ldk, int et, const int* rowmap) {
  __shared__ float tile[32][33];
  const int n0 = blockIdx.x * 32, k0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;   // 256 threads: 32 x 8
  for (int j = ty; j < 32; j += 8) {
    const int k = k0 + j, n = n0 + tx;
    tile[j][tx] = (k < K && n < N) ? src[(long)k * N + n] : 0.f;
  }
  __syncthreads();
  for (int j = ty; j < 32; j += 8) {
    const int n = n0 + j, k = k0 + tx;
    if (n < N && k < ldk) {
      const long row = rowmap ? rowmap[n] : n;
      const float v = tile[tx][j];
      if (et == ET_BF16) reinterpret_cast<bf16*>(dst)[row * ldk + k] = (bf16)v;
      else reinterpret_cast<float*>(dst)[row * ldk + k] = v;
    }
  }
}

__global__ void convert_kernel(const float* src, long n, void* dst, int et) {
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x) {
    if (et == ET_BF16) reinterpret_cast<bf16*>(dst)[e] = (bf16)src[e];
    else reinterpret_cast<float*>(dst)[e] = src[e];
  }
}

__global__ void round_bf16_kernel(const float* src, long n, float* dst) {
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < n; e += (long)gridDim.x * blockDim.x)
    dst[e] = round_bf16(src[e]);
}

// W[n][k] *= g[k] for the bf16 weight rows of a projection whose input row
// norm is folded into it (k < K; row stride ldk), rounded back to bf16
__global__ void scale_cols_bf16_kernel(bf16* W, long N, int K, int ldk, const float* g) {
  const long total = N * (long)K;
  for (long e = blockIdx.x * (long)blockDim.x + threadIdx.x; e < total; e += (long)gridDim.x * blockDim.x) {
    const long n = e / K;
    const int k = (int)(e % K);
    bf16& w = W[n * ldk + k];
    w = (bf16)((float)w * g[k]);
  }
}

// ---------------------------------------------------------------- probe
__global__ void cu_probe_kernel(uint32_t* out, int spin) {
  // HW_ID (hwreg 4) and XCC_ID (hwreg 20), read whole (size 32, offset 0)
  const uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);
  const uint32_t xcc = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 20);
  for (int i = 0; i < spin; ++i) __builtin_amdgcn_s_sleep(64);
  if (threadIdx.x == 0) {
    out[2 * blockIdx.x + 0] = hw;
    out[2 * blockIdx.x + 1] = xcc;
  }
}

inline int grid_for(long n, int block = 256) {
  long g = (n + block - 1) / block;
  return (int)(g < 1 ? 1 : (g > 65536 ? 65536 : g));
}

}  // namespace

// Token merge: thread i writes 16-byte chunk c of block slot k of merged token
// r (destination order), read from the source token that slot holds.
__global__ void pixel_shuffle_kernel(const uint4* src, uint4* dst, long total, int g, int s, int cpt) {
  const int G = g / s, ss = s * s;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const int c = (int)(i % cpt);
    const long t = i / cpt;
    const int kk = (int)(t % ss);
    const long r = t / ss;
    const int J = (int)(r % G);
    const long r2 = r / G;
    const int I = (int)(r2 % G);
    const long img = r2 / G;
    const long sr = img * g * g + (long)(s * I + kk / s) * g + s * J + kk % s;
    dst[i] = src[sr * cpt + c];
  }
}

// Batched copy: block (x, y) copies chunk x of segment y. 16-byte vector
// accesses when source, destination and size allow them, else 4-byte, else
// single bytes; a null source writes zeros.
__global__ void __launch_bounds__(256) batched_copy_kernel(const CopySeg* segs) {
  const CopySeg sg = segs[blockIdx.y];
  const long long off = (long long)blockIdx.x * kCopyChunk;
  if (off >= sg.bytes) return;
  const long long n = sg.bytes - off < kCopyChunk ? sg.bytes - off : kCopyChunk;
  const char* src = (const char*)sg.src;
  char* dst = (char*)sg.dst + off;
  const uintptr_t al = (uintptr_t)dst | (uintptr_t)(src ? src + off : nullptr) | (uintptr_t)n;
  if ((al & 15) == 0) {
    uint4* d = (uint4*)dst;
    const uint4* s4 = src ? (const uint4*)(src + off) : nullptr;
    for (long long i = threadIdx.x; i < n / 16; i += blockDim.x) d[i] = s4 ? s4[i] : make_uint4(0, 0, 0, 0);
  } else if ((al & 3) == 0) {
    uint32_t* d = (uint32_t*)dst;
    const uint32_t* s1 = src ? (const uint32_t*)(src + off) : nullptr;
    for (long long i = threadIdx.x; i < n / 4; i += blockDim.x) d[i] = s1 ? s1[i] : 0u;
  } else {
    for (long long i = threadIdx.x; i < n; i += blockDim.x) dst[i] = src ? src[off + i] : (char)0;
  }
}

// 256-thread blocks of 4 / WPR rows
template <int NV>
static void launch_norm_nv(const NormArgs& a, hipStream_t s) {
  constexpr int W = NV >= 4 ? 4 : NV;
  if (rownorm::waves_per_row(NV, a.rows) == 1) {
    hipLaunchKernelGGL((norm_kernel<NV, 1>), dim3((a.rows + 3) / 4), dim3(256), 0, s, a);
  } else {
    hipLaunchKernelGGL((norm_kernel<NV / W, W>), dim3((a.rows + 4 / W - 1) / (4 / W)), dim3(256), 0, s, a);
  }
}

void launch_norm(const NormArgs& a, hipStream_t s) {
  if (a.rows <= 0) return;
  if (a.d % 4 || a.ld_in % 4 || a.ld_out % 4 || a.d > 2048) throw VlaError{4, "norm: d, ld must be multiples of 4, d <= 2048"};
  if (a.d <= 256) launch_norm_nv<1>(a, s);
  else if (a.d <= 512) launch_norm_nv<2>(a, s);
  else if (a.d <= 1024) launch_norm_nv<4>(a, s);
  else launch_norm_nv<8>(a, s);
}

void launch_im2col(const float* pix, int n_images, int hw, int p, void* out, int ldo, int out_type, hipStream_t s) {
  const long total = (long)n_images * (hw / p) * (hw / p) * ldo;
  hipLaunchKernelGGL(im2col_kernel, dim3(grid_for(total)), dim3(256), 0, s, pix, n_images, hw, p, out, ldo, out_type);
}

void launch_embed(const int32_t* ids, int B, int n, int vocab, const void* table, int table_type, int d, float* h,
                  long P, int first, hipStream_t s) {
  const long total = (long)B * n * d;
  hipLaunchKernelGGL(embed_kernel, dim3(grid_for(total)), dim3(256), 0, s, ids, B, n, vocab, table, table_type, d, h, P,
                     first);
}

void launch_time_embed(int steps, int dim, float* out, hipStream_t s) {
  hipLaunchKernelGGL(time_embed_kernel, dim3(steps), dim3(128), 0, s, steps, dim, out);
}

void launch_rope_table(int npos, int hd, double base, float* out, hipStream_t s) {
  hipLaunchKernelGGL(rope_table_kernel, dim3(grid_for((long)npos * hd / 2)), dim3(256), 0, s, npos, hd, base, out);
}

void launch_copy_f32(const float* src, float* dst, long n, hipStream_t s) {
  hipLaunchKernelGGL(copy_f32_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, dst, n);
}

void launch_silu_f32(const float* src, float* dst, long n, hipStream_t s) {
  hipLaunchKernelGGL(silu_f32_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, dst, n);
}

void launch_dit_state_rows(const void* st, int et, int B, int d, int seq, const float* pos, float* X, hipStream_t s) {
  hipLaunchKernelGGL(dit_state_rows_kernel, dim3(grid_for((long)B * d)), dim3(256), 0, s, st, et, B, d, seq, pos, X);
}

void launch_transpose_convert(const float* src, int K, int N, void* dst, int ldk, int et, const int* rowmap,
                              hipStream_t s) {
  dim3 grid((N + 31) / 32, (ldk + 31) / 32);
  hipLaunchKernelGGL(transpose_convert_kernel, grid, dim3(256), 0, s, src, K, N, dst, ldk, et, rowmap);
}

void launch_convert(const float* src, long n, void* dst, int et, hipStream_t s) {
  hipLaunchKernelGGL(convert_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, n, dst, et);
}

void launch_scale_cols_bf16(void* W, long N, int K, int ldk, const float* g, hipStream_t s) {
  hipLaunchKernelGGL(scale_cols_bf16_kernel, dim3(grid_for(N * (long)K)), dim3(256), 0, s, reinterpret_cast<bf16*>(W), N,
                     K, ldk, g);
}

void launch_round_bf16_f32(const float* src, long n, float* dst, hipStream_t s) {
  hipLaunchKernelGGL(round_bf16_kernel, dim3(grid_for(n)), dim3(256), 0, s, src, n, dst);
}

void launch_pixel_shuffle(const void* src, int n_img, int g, int s, int d, int et, void* dst, hipStream_t st) {
  const long row_bytes = (long)d * (et == ET_BF16 ? 2 : 4);
  VLA_REQUIRE(row_bytes % 16 == 0 && g % s == 0, "token merge needs 16-byte rows and s | g");
  const int cpt = (int)(row_bytes / 16);
  const long total = (long)n_img * g * g * cpt;
  const long blocks = std::min<long>((total + 255) / 256, 65536);
  pixel_shuffle_kernel<<<(unsigned)blocks, 256, 0, st>>>((const uint4*)src, (uint4*)dst, total, g, s, cpt);
}

void launch_batched_copy(const CopySeg* segs, int n, long long max_bytes, hipStream_t s) {
  if (n <= 0 || max_bytes <= 0) return;
  const long long chunks = (max_bytes + kCopyChunk - 1) / kCopyChunk;
  VLA_REQUIRE(n <= 65535 && chunks <= (1LL << 31) - 1, "batched copy too large");
  batched_copy_kernel<<<dim3((unsigned)chunks, (unsigned)n), 256, 0, s>>>(segs);
}

void launch_cu_probe(uint32_t* out, int blocks, int spin, hipStream_t s) {
  hipLaunchKernelGGL(cu_probe_kernel, dim3(blocks), dim3(64), 0, s, out, spin);
}

// Synchronisation-cost probes. sync_empty_kernel does nothing (a kernel
// boundary alone); sync_write_kernel has every block write `words` floats of
// its own slice (a boundary after a tile's worth of stores).
__global__ void __launch_bounds__(256) sync_empty_kernel(float* sink) {
  if (sink && threadIdx.x > 1024) sink[0] = 0.f;   // never taken
}

__global__ void __launch_bounds__(256) sync_write_kernel(float* buf, int words) {
  float* b = buf + (long)blockIdx.x * words;
  for (int i = threadIdx.x; i < words; i += 256) b[i] = (float)i;
}

// `iters` grid-wide barriers inside one kernel. Before each, every block
// writes `words` floats of its own slice; after it, the block reads the slice
// of another block (a hand-off between XCDs). Slices alternate between two
// halves of buf by round, so a block that runs ahead into the next round
// never overwrites what a slower block still reads. Thread 0 adds to a monotone
// counter with release semantics at agent scope and polls it with acquire
// loads until every block of the round has arrived; past `spin_limit` polls
// it counts an overrun in *err and goes on, so every block always finishes.
// Needs every block resident at once (grid <= the CUs).
__global__ void __launch_bounds__(256) sync_barrier_kernel(unsigned* ctr, int iters, int spin_limit, int* err,
                                                           float* buf, int words, float* sink) {
  __shared__ int overrun;
  float acc = 0.f;
  const unsigned G = gridDim.x;
  for (int it = 0; it < iters; ++it) {
    float* half = buf + (long)(it & 1) * G * words;
    float* mine = half + (long)blockIdx.x * words;
    for (int i = threadIdx.x; i < words; i += 256) mine[i] = (float)(i + it);
    __syncthreads();
    if (threadIdx.x == 0) {
      overrun = 0;
      __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
      const unsigned target = (unsigned)(it + 1) * G;
      int n = 0;
      while (__hip_atomic_load(ctr, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (++n > spin_limit) { overrun = 1; break; }
        __builtin_amdgcn_s_sleep(1);
      }
      if (overrun) __hip_atomic_fetch_add(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const float* other = half + (long)((blockIdx.x + 37) % G) * words;
    for (int i = threadIdx.x; i < words; i += 256) acc += other[i];
    __syncthreads();
  }
  sink[(long)blockIdx.x * 256 + threadIdx.x] = acc;
}

void launch_sync_probe(int kind, int grid, int iters, int words, int spin_limit, float* buf, unsigned* ctr, int* err,
                       float* sink, hipStream_t s) {
  if (kind == 0) {
    for (int i = 0; i < iters; ++i) hipLaunchKernelGGL(sync_empty_kernel, dim3(grid), dim3(256), 0, s, sink);
  } else if (kind == 1) {
    for (int i = 0; i < iters; ++i) hipLaunchKernelGGL(sync_write_kernel, dim3(grid), dim3(256), 0, s, buf, words);
  } else {
    hipLaunchKernelGGL(sync_barrier_kernel, dim3(grid), dim3(256), 0, s, ctr, iters, spin_limit, err, buf, words, sink);
  }
}
