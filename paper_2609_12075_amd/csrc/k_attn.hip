// Prefix-KV attention for both VLA stages on gfx950.
//
// One kernel serves every attention of the path: bidirectional prefill over
// the image+text prefix (grouped-query heads), the ViT's per-image attention,
// the action tokens' attention over [prefix K,V of the paired LLM layer ;
// their own K,V] (two key segments, no concatenation copy), and the DiT's
// self- and cross-attention. Keys/values stream through LDS in tiles of 64;
// softmax is online in fp32 (exp2 domain); both products run on the matrix
// cores (v_mfma_f32_16x16x32_bf16).
//
// Work decomposition: rows of a block are (query head within its KV group,
// query position) pairs, so all query heads sharing a KV head read each K/V
// tile once. Block = 4 waves x 16 rows. The score tile is computed
// transposed (S^T = K Q^T) so a lane holds four keys of one query; the
// probabilities then feed P V as the B operand without leaving registers,
// with the key order inside each 32-key chunk permuted consistently on the
// V side.
#include <algorithm>

#include "common.h"

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;

namespace {

constexpr int BQ = 64;    // rows per block
constexpr int BKV = 64;   // keys per tile

__device__ __forceinline__ const bf16* seg_row(const AttnArgs& a, int which, int b, int g, int key, bool is_v) {
  const AttnSeg& s = a.seg[which];
  const bf16* base = reinterpret_cast<const bf16*>(is_v ? s.v : s.k);
  long off = is_v ? ((long)b * s.v_sb + (long)g * s.v_sh + (long)key * s.v_si)
                  : ((long)b * s.k_sb + (long)g * s.k_sh + (long)key * s.k_si);
  return base + off;
}

template <int HDP>
__global__ void __launch_bounds__(256) attn_mfma_kernel(AttnArgs a) {
  constexpr int LDK = HDP + 8;       // K tile row stride (elements)
  constexpr int LDV = BKV + 8;       // V^T tile row stride
  constexpr int NC = HDP / 32;       // 32-wide chunks of the head dimension
  constexpr int ND = HDP / 16;       // 16-wide output subtiles
  constexpr int CH = HDP / 8;        // 8-element chunks per key row
  __shared__ __attribute__((aligned(16))) bf16 Ks[BKV][LDK];
  __shared__ __attribute__((aligned(16))) bf16 Vt[HDP][LDV];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int S = a.splits > 1 ? a.splits : 1;      // key ranges (split-KV)
  // die-aware order: the row tiles sharing one (request, KV head) K/V stream
  // are consecutive logical blocks and so share one die's L2
  int bx, by, bz;
  xcd_remap(bx, by, bz);
  const int b = bz / S, split = bz % S, g = by;
  const int G = a.Hq / a.Hkv;
  const int rows = G * a.Lq;
  const int hd = a.hd;
  const int lq = lane & 15, grp = lane >> 4;

  // this lane's query row
  const int r = bx * BQ + wave * 16 + lq;
  const bool rvalid = r < rows;
  const int jh = rvalid ? r / a.Lq : 0, qi = rvalid ? r % a.Lq : 0;
  const int h = g * G + jh;

  bf16x8 qf[NC];
  {
    const bf16* qp = reinterpret_cast<const bf16*>(a.q) + (long)b * a.q_sb + (long)h * a.q_sh + (long)qi * a.q_si;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int d = c * 32 + grp * 8;
      qf[c] = (rvalid && d < hd) ? *reinterpret_cast<const bf16x8*>(qp + d) : bf16x8{};
    }
  }

  f32x4 o[ND];
#pragma unroll
  for (int t = 0; t < ND; ++t) o[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;   // scale * log2(e)

  const int len0 = a.seg[0].len;
  const int kbeg = S > 1 ? split * a.kchunk : 0;
  const int kend = S > 1 ? min(len0 + a.seg[1].len, kbeg + a.kchunk) : len0 + a.seg[1].len;
  // K/V tile chunks (8 elements) handled by this thread; with PREFETCH the
  // next tile's chunks are loaded into registers while the current tile is
  // consumed, hiding the global-load latency behind the matrix work.
  constexpr int PER = BKV * CH / 256;
  constexpr bool PREFETCH = HDP <= 128;
  // Chunk j of this thread: key row kr, dims d8..d8+7. When the chunk count
  // divides by 4, a thread owns R = CH/4 consecutive keys of one 8-dim chunk,
  // so its V^T values for one dim are R consecutive bf16 (one vector store).
  constexpr bool GROUPED = CH % 4 == 0 && 256 % CH == 0;
  constexpr int R = GROUPED ? CH / 4 : 1;
  auto chunk_of = [&](int j, int& kr, int& d8) {
    if constexpr (GROUPED) {
      d8 = (tid % CH) * 8;
      kr = (tid / CH) * R + j;
    } else {
      const int c = tid + 256 * j;
      kr = c / CH;
      d8 = (c % CH) * 8;
    }
  };
  auto load_chunk = [&](int k0, int kr, int d8, bool is_v) {
    const int kg = k0 + kr;
    if (kg < kend && d8 < hd) {
      const int which = kg < len0 ? 0 : 1;
      const int key = which ? kg - len0 : kg;
      return *reinterpret_cast<const bf16x8*>(seg_row(a, which, b, g, key, is_v) + d8);
    }
    return bf16x8{};
  };
  // V^T store of this thread's PER chunks (R keys per dim when grouped)
  auto store_vt = [&](const bf16x8 (&vr)[PER]) {
    int kr, d8;
    if constexpr (GROUPED) {
      chunk_of(0, kr, d8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if constexpr (R == 1) {
          Vt[d8 + e][kr] = vr[0][e];
        } else if constexpr (R == 2) {
          typedef __attribute__((ext_vector_type(2))) __bf16 v2;
          *reinterpret_cast<v2*>(&Vt[d8 + e][kr]) = v2{vr[0][e], vr[1][e]};
        } else {
          static_assert(R == 8, "grouped staging supports 1, 2 or 8 keys per thread");
          *reinterpret_cast<bf16x8*>(&Vt[d8 + e][kr]) =
              bf16x8{vr[0][e], vr[1][e], vr[2][e], vr[3][e], vr[4][e], vr[5][e], vr[6][e], vr[7][e]};
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        chunk_of(j, kr, d8);
#pragma unroll
        for (int e = 0; e < 8; ++e) Vt[d8 + e][kr] = vr[j][e];
      }
    }
  };
  bf16x8 kreg[PER], vreg[PER];
  auto load_regs = [&](int k0) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      int kr, d8;
      chunk_of(j, kr, d8);
      kreg[j] = load_chunk(k0, kr, d8, false);
      vreg[j] = load_chunk(k0, kr, d8, true);
    }
  };
  if constexpr (PREFETCH) load_regs(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += BKV) {
    // ---- stage K (row-major) and V (transposed) tiles into LDS
    if constexpr (PREFETCH) {
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        int kr, d8;
        chunk_of(j, kr, d8);
        *reinterpret_cast<bf16x8*>(&Ks[kr][d8]) = kreg[j];
      }
      store_vt(vreg);
    } else {
      // K then V, PER chunks each in flight at once
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        int kr, d8;
        chunk_of(j, kr, d8);
        kreg[j] = load_chunk(k0, kr, d8, false);
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        int kr, d8;
        chunk_of(j, kr, d8);
        *reinterpret_cast<bf16x8*>(&Ks[kr][d8]) = kreg[j];
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        int kr, d8;
        chunk_of(j, kr, d8);
        vreg[j] = load_chunk(k0, kr, d8, true);
      }
      store_vt(vreg);
    }
    __syncthreads();
    if constexpr (PREFETCH) {
      if (k0 + BKV < kend) load_regs(k0 + BKV);
    }

    // ---- S^T = K Q^T for 4 subtiles of 16 keys
    f32x4 s[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      s[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Ks[st * 16 + lq][c * 32 + grp * 8]);
        s[st] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[c], s[st], 0, 0, 0);
      }
    }
    // lane holds scores of query lq for keys st*16 + 4*grp + i
    float mx = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kg = k0 + st * 16 + grp * 4 + i;
        float v = kg < kend ? s[st][i] * sl2 : -INFINITY;
        s[st][i] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float p = exp2f(s[st][i] - m_new);
        s[st][i] = p;
        psum += p;
      }
    psum += __shfl_xor(psum, 16);
    psum += __shfl_xor(psum, 32);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int t = 0; t < ND; ++t) o[t] *= alpha;

    // ---- O^T += V^T P^T over two 32-key chunks. K-slot jj of lane group grp
    // is key 4*grp + jj (jj < 4) or 16 + 4*grp + jj - 4 (jj >= 4) of the chunk.
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      bf16x8 pf = {(bf16)s[2 * kc][0], (bf16)s[2 * kc][1], (bf16)s[2 * kc][2], (bf16)s[2 * kc][3],
                   (bf16)s[2 * kc + 1][0], (bf16)s[2 * kc + 1][1], (bf16)s[2 * kc + 1][2], (bf16)s[2 * kc + 1][3]};
#pragma unroll
      for (int t = 0; t < ND; ++t) {
        const bf16* vr = &Vt[t * 16 + lq][kc * 32 + grp * 4];
        bf16x4 lo = *reinterpret_cast<const bf16x4*>(vr);
        bf16x4 hi = *reinterpret_cast<const bf16x4*>(vr + 16);
        bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[t], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  if (!rvalid) return;
  if (S > 1) {
    // split-KV: unnormalised output and (max, sum) of this key range, fp32
    const long row = ((long)b * a.Hq + h) * a.Lq + qi;
    float* po = a.ws + (row * S + split) * hd;
#pragma unroll
    for (int t = 0; t < ND; ++t) {
      const int d = t * 16 + grp * 4;
      if (d < hd) *reinterpret_cast<f32x4*>(po + d) = o[t];
    }
    if (grp == 0) {
      float* st = a.ws + (long)a.B * a.Hq * a.Lq * S * hd + (row * S + split) * 2;
      st[0] = m_run;
      st[1] = l_run;
    }
    return;
  }
  const float inv = 1.0f / l_run;
  bf16* op = reinterpret_cast<bf16*>(a.o) + (long)b * a.o_sb + (long)h * a.o_sh + (long)qi * a.o_si;
#pragma unroll
  for (int t = 0; t < ND; ++t) {
    const int d = t * 16 + grp * 4;
    if (d < hd) {
      bf16x4 w = {(bf16)(o[t][0] * inv), (bf16)(o[t][1] * inv), (bf16)(o[t][2] * inv), (bf16)(o[t][3] * inv)};
      *reinterpret_cast<bf16x4*>(op + d) = w;
    }
  }
}

// Split-KV merge: one wavefront per query row combines the key ranges in
// order: m = max m_s, l = sum l_s 2^(m_s - m), o = sum o_s 2^(m_s - m) / l.
// Each lane owns four consecutive dims; all (<= 16) partial loads of a lane
// are issued before any is used.
constexpr int MAX_SPLITS = 16;
__global__ void __launch_bounds__(256) attn_combine_kernel(AttnArgs a) {
  const int lane = threadIdx.x & 63;
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  if (row >= (long)a.B * a.Hq * a.Lq) return;
  const int S = a.splits, hd = a.hd;
  const float* st = a.ws + (long)a.B * a.Hq * a.Lq * S * hd + row * S * 2;
  float ms[MAX_SPLITS], w[MAX_SPLITS];
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s) ms[s] = s < S ? st[2 * s] : -INFINITY;
  float m = -INFINITY;
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s) m = fmaxf(m, ms[s]);
  float l = 0.f;
#pragma unroll
  for (int s = 0; s < MAX_SPLITS; ++s) {
    w[s] = s < S ? exp2f(ms[s] - m) : 0.f;
    l += s < S ? st[2 * s + 1] * w[s] : 0.f;
  }
  const float inv = 1.0f / l;
  const int qi = (int)(row % a.Lq), h = (int)((row / a.Lq) % a.Hq), b = (int)(row / ((long)a.Lq * a.Hq));
  bf16* op = reinterpret_cast<bf16*>(a.o) + (long)b * a.o_sb + (long)h * a.o_sh + (long)qi * a.o_si;
  const float* po = a.ws + row * S * hd;
  for (int d = lane * 4; d < hd; d += 256) {
    f32x4 part[MAX_SPLITS];
#pragma unroll
    for (int s = 0; s < MAX_SPLITS; ++s)
      part[s] = s < S ? *reinterpret_cast<const f32x4*>(po + (long)s * hd + d) : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < MAX_SPLITS; ++s) acc += part[s] * w[s];
    *reinterpret_cast<bf16x4*>(op + d) =
        bf16x4{(bf16)(acc[0] * inv), (bf16)(acc[1] * inv), (bf16)(acc[2] * inv), (bf16)(acc[3] * inv)};
  }
}

// fp32 attention: one wave per (query, head, request); keys in chunks of 64
// (one per lane), online softmax; each lane accumulates hd/64 output dims.
__global__ void __launch_bounds__(64) attn_f32_kernel(AttnArgs a) {
  __shared__ float p[64];
  const int lane = threadIdx.x;
  const int qi = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int g = h / (a.Hq / a.Hkv);
  const int hd = a.hd;
  const float* q = reinterpret_cast<const float*>(a.q) + (long)b * a.q_sb + (long)h * a.q_sh + (long)qi * a.q_si;
  constexpr int MAXD = 4;   // hd <= 256
  float acc[MAXD] = {0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const int len0 = a.seg[0].len, total = len0 + a.seg[1].len;
  for (int k0 = 0; k0 < total; k0 += 64) {
    const int kg = k0 + lane;
    float sc = -INFINITY;
    if (kg < total) {
      const int which = kg < len0 ? 0 : 1, key = which ? kg - len0 : kg;
      const AttnSeg& s = a.seg[which];
      const float* kp = reinterpret_cast<const float*>(s.k) + (long)b * s.k_sb + (long)g * s.k_sh + (long)key * s.k_si;
      float dot = 0.f;
      for (int d = 0; d < hd; ++d) dot = fmaf(q[d], kp[d], dot);
      sc = dot * a.scale;
    }
    float mx = sc;
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    const float m_new = fmaxf(m_run, mx);
    const float pe = kg < total ? __expf(sc - m_new) : 0.f;
    float ps = pe;
    for (int o = 32; o > 0; o >>= 1) ps += __shfl_xor(ps, o);
    const float alpha = __expf(m_run - m_new);
    l_run = l_run * alpha + ps;
    m_run = m_new;
    p[lane] = pe;
    __syncthreads();
    for (int j = 0; j < MAXD; ++j) acc[j] *= alpha;
    const int nk = min(64, total - k0);
    for (int kk = 0; kk < nk; ++kk) {
      const int kg2 = k0 + kk;
      const int which = kg2 < len0 ? 0 : 1, key = which ? kg2 - len0 : kg2;
      const AttnSeg& s = a.seg[which];
      const float* vp = reinterpret_cast<const float*>(s.v) + (long)b * s.v_sb + (long)g * s.v_sh + (long)key * s.v_si;
      const float pk = p[kk];
#pragma unroll
      for (int j = 0; j < MAXD; ++j) {
        const int d = lane + 64 * j;
        if (d < hd) acc[j] = fmaf(pk, vp[d], acc[j]);
      }
    }
    __syncthreads();
  }
  float* op = reinterpret_cast<float*>(a.o) + (long)b * a.o_sb + (long)h * a.o_sh + (long)qi * a.o_si;
  const float inv = 1.0f / l_run;
#pragma unroll
  for (int j = 0; j < MAXD; ++j) {
    const int d = lane + 64 * j;
    if (d < hd) op[d] = acc[j] * inv;
  }
}

}  // namespace

void launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.Lq <= 0) return;
  if (a.et == ET_F32) {
    hipLaunchKernelGGL(attn_f32_kernel, dim3(a.Lq, a.Hq, a.B), dim3(64), 0, s, a);
    return;
  }
  AttnArgs b = a;
  const int rows = (a.Hq / a.Hkv) * a.Lq;
  const long blocks = (long)((rows + BQ - 1) / BQ) * a.Hkv * a.B;
  const int total = a.seg[0].len + a.seg[1].len, ntiles = (total + BKV - 1) / BKV;
  // split the keys when the blocks alone would leave most CUs idle
  b.splits = 1;
  b.kchunk = ntiles * BKV;
  if (a.ws && blocks < 128 && ntiles >= 2) {
    int sp = (int)std::min<long>({(256 + blocks - 1) / blocks, (long)ntiles, 16L});
    while (sp > 1 && (long)a.B * a.Hq * a.Lq * sp * (a.hd + 2) > a.ws_floats) --sp;
    const int per = (ntiles + sp - 1) / sp;
    b.kchunk = per * BKV;
    b.splits = (ntiles + per - 1) / per;            // every range holds keys
  }
  dim3 grid((rows + BQ - 1) / BQ, a.Hkv, a.B * b.splits);
  if (a.hd <= 32) hipLaunchKernelGGL(attn_mfma_kernel<32>, grid, dim3(256), 0, s, b);
  else if (a.hd <= 64) hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, s, b);
  else if (a.hd <= 96) hipLaunchKernelGGL(attn_mfma_kernel<96>, grid, dim3(256), 0, s, b);
  else hipLaunchKernelGGL(attn_mfma_kernel<256>, grid, dim3(256), 0, s, b);
  if (b.splits > 1) {
    const long nrows = (long)a.B * a.Hq * a.Lq;
    hipLaunchKernelGGL(attn_combine_kernel, dim3((unsigned)((nrows + 3) / 4)), dim3(256), 0, s, b);
  }
}
