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

// Split-KV merge: LPR lanes per query row (the fewest of 16, 32, 64 whose
// four dims each cover the head dim, so 64 / LPR rows share a wavefront)
// combine the key ranges in order: m = max m_s, l = sum l_s 2^(m_s - m),
// o = sum o_s 2^(m_s - m) / l. Each lane owns four consecutive dims; its
// range statistics and all (<= 16) partial loads are issued together before
// any is used (one memory round trip instead of two: 7.6 -> 6.4 us for the
// pi0-shaped action attention at batch 8, four ranges).
constexpr int MAX_SPLITS = 16;
template <int LPR>
__global__ void __launch_bounds__(256) attn_combine_kernel(AttnArgs a) {
  constexpr int RPW = 64 / LPR;
  const int lane = threadIdx.x & 63, sub = lane % LPR;
  const long row = (blockIdx.x * 4L + (threadIdx.x >> 6)) * RPW + lane / LPR;
  if (row >= (long)a.B * a.Hq * a.Lq) return;
  const int S = a.splits, hd = a.hd, d = sub * 4;
  const bool dok = d < hd;
  const float* st = a.ws + (long)a.B * a.Hq * a.Lq * S * hd + row * S * 2;
  const float* po = a.ws + row * S * hd + (dok ? d : 0);
  float ms[MAX_SPLITS], ls[MAX_SPLITS], w[MAX_SPLITS];
  f32x4 part[MAX_SPLITS];
#pragma unroll
  for (int q = 0; q < MAX_SPLITS; ++q) {
    ms[q] = q < S ? st[2 * q] : -INFINITY;
    ls[q] = q < S ? st[2 * q + 1] : 0.f;
    part[q] = (q < S && dok) ? *reinterpret_cast<const f32x4*>(po + (long)q * hd) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  float m = -INFINITY;
#pragma unroll
  for (int q = 0; q < MAX_SPLITS; ++q) m = fmaxf(m, ms[q]);
  float l = 0.f;
#pragma unroll
  for (int q = 0; q < MAX_SPLITS; ++q) {
    w[q] = q < S ? exp2f(ms[q] - m) : 0.f;
    l += q < S ? ls[q] * w[q] : 0.f;
  }
  const float inv = 1.0f / l;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < MAX_SPLITS; ++q) acc += part[q] * w[q];
  if (!dok) return;
  const int qi = (int)(row % a.Lq), h = (int)((row / a.Lq) % a.Hq), b = (int)(row / ((long)a.Lq * a.Hq));
  bf16* op = reinterpret_cast<bf16*>(a.o) + (long)b * a.o_sb + (long)h * a.o_sh + (long)qi * a.o_si;
  *reinterpret_cast<bf16x4*>(op + d) =
      bf16x4{(bf16)(acc[0] * inv), (bf16)(acc[1] * inv), (bf16)(acc[2] * inv), (bf16)(acc[3] * inv)};
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


// ---------------------------------------------------------------- v2 kernel
// Same row decomposition, softmax and products as attn_mfma_kernel, with the
// K/V staging of the multi-stage projection kernel: tiles move global -> LDS
// with the CDNA4 direct loads (global_load_lds_dwordx4, lane l's 16 bytes at
// LDS base + 16 l) through a ring of NS tiles, so the next round of tiles
// loads while this one is consumed, without registers. Rows are unpadded and
// key-major for both K and V; the 16-byte chunk c of row r sits in slot
// c ^ swz(r), which makes the 16-row fragment reads conflict-free. The P V
// product needs V^T fragments (one dimension, 8 keys per lane); they come
// from the transposing LDS read (ds_read_b64_tr_b16): within each 16-lane
// group, source lane s points at 4 dimensions of one key row (row
// 4-block + s / 4, dims 4 (s % 4) ..), and lane i receives dimension i of the
// group's 4 keys. Chunks past hd and keys past the range read zeros.
//
// KS > 1 splits the block's key range over KS groups of 4 waves (tile t goes
// to group t % KS), so short decode ranges run KS tiles at a time with KS
// waves per SIMD; the groups' (max, sum, output) are merged through LDS at
// the end in group order (as the split-KV combine does across blocks).
typedef short v4s __attribute__((ext_vector_type(4)));

// A row statistic combined with the value of lane l ^ 16 (l ^ 32): one CDNA4
// permlane swap of a value with itself exchanges the 16-lane rows (32-lane
// halves), and its two results hold the lane's own value and its partner's.
__device__ __forceinline__ float max_x16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_x32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_x16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_x32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int HDP>
struct V2 {
  static constexpr int BKV = HDP >= 256 ? 32 : 64;          // keys per tile
  static constexpr int CR = HDP / 8;                          // 16-byte chunks per row
  static constexpr int ROWB = HDP * 2;
  static constexpr int TILE = BKV * ROWB;                     // bytes of a K (or V) tile
  static constexpr int NS = 2 * TILE <= 16384 ? 4 : 2;        // ring depth in tiles (KS = 1)
  static constexpr int RP = CR >= 16 ? 1 : 16 / CR;           // rows per 256 bytes (one bank cycle)
  static constexpr int SWM = (CR >= 16 ? 16 : CR) - 1;
  __device__ static constexpr int swz(int r) { return (r / RP) & SWM; }
};

template <int HDP, int KS>
__global__ void __launch_bounds__(256 * KS) attn_v2_kernel(AttnArgs a) {
  using C = V2<HDP>;
  constexpr int BKV = C::BKV, ROWB = C::ROWB, TILE = C::TILE, CR = C::CR;
  constexpr int NW = 4 * KS;                       // waves per block
  constexpr int IW = TILE / 1024 / NW;             // 1 KiB direct loads per wave per tile (K or V)
  static_assert(IW >= 1 && IW * NW * 1024 == TILE, "tile loads must spread evenly over the waves");
  constexpr int NR = KS == 1 ? C::NS : 2;          // ring depth in rounds of KS tiles
  constexpr int NC = HDP / 32, ND = HDP / 16;
  constexpr int RING = NR * KS * 2 * TILE;
  constexpr int MST = ND * 4 + 4;                   // merge record: o, m, l, pad (16-byte aligned)
  constexpr int MERGE = KS > 1 ? (KS - 1) * 256 * MST * 4 : 0;
  __shared__ __attribute__((aligned(1024))) char smem[RING > MERGE ? RING : MERGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int kg = wave >> 2, wrow = wave & 3;       // key group, row group
  const int S = a.splits > 1 ? a.splits : 1;
  int bx, by, bz;
  xcd_remap(bx, by, bz);
  const int b = bz / S, split = bz % S, g = by;
  const int G = a.Hq / a.Hkv;
  const int rows = G * a.Lq;
  const int hd = a.hd;
  const int lq = lane & 15, grp = lane >> 4;

  const int r = bx * BQ + wrow * 16 + lq;
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

  const int len0 = a.seg[0].len;
  const int kbeg = S > 1 ? split * a.kchunk : 0;
  const int kend = S > 1 ? min(len0 + a.seg[1].len, kbeg + a.kchunk) : len0 + a.seg[1].len;
  const int nt = kend > kbeg ? (kend - kbeg + BKV - 1) / BKV : 0;
  const int nrounds = (nt + KS - 1) / KS;
  const bf16* Z = reinterpret_cast<const bf16*>(a.zeros);

  // Loop-invariant addressing: the (request, KV head) base of each segment's
  // K and V rows in bytes and, per lane and load, the byte offset of its row
  // and chunk; per tile only the segment bases move (scalar work) and each
  // lane picks its row's segment.
  const long kbase0 = (long)a.seg[0].k + ((long)b * a.seg[0].k_sb + (long)g * a.seg[0].k_sh) * 2;
  const long kbase1 = (long)a.seg[1].k + ((long)b * a.seg[1].k_sb + (long)g * a.seg[1].k_sh) * 2;
  const long vbase0 = (long)a.seg[0].v + ((long)b * a.seg[0].v_sb + (long)g * a.seg[0].v_sh) * 2;
  const long vbase1 = (long)a.seg[1].v + ((long)b * a.seg[1].v_sb + (long)g * a.seg[1].v_sh) * 2;
  const long kst0 = a.seg[0].k_si * 2, kst1 = a.seg[1].k_si * 2, vst0 = a.seg[0].v_si * 2, vst1 = a.seg[1].v_si * 2;
  // (head dim 256 with one key group keeps the per-tile computation: the
  // hoisted offsets would cost it half its occupancy)
  constexpr bool HOIST = !(HDP >= 256 && KS == 1);
  constexpr int IWH = HOIST ? IW : 1;
  int lrow[IWH], lok[IWH];
  unsigned rk0[IWH], rk1[IWH], rv0[IWH], rv1[IWH];  // < 2^32 (checked by the launcher)
#pragma unroll
  for (int i = 0; i < IWH; ++i) {
    const int u = (i * NW + wave) * 64 + lane, row = u / CR, c = (u % CR) ^ C::swz(row), d8 = c * 8;
    lrow[i] = row;
    lok[i] = d8 < hd;
    rk0[i] = (unsigned)(row * kst0 + d8 * 2); rk1[i] = (unsigned)(row * kst1 + d8 * 2);
    rv0[i] = (unsigned)(row * vst0 + d8 * 2); rv1[i] = (unsigned)(row * vst1 + d8 * 2);
  }

  // round p holds tiles p KS .. p KS + KS - 1 in ring slot p % NR; each tile
  // is its K tile then its V tile. 16-byte unit u of a tile is (row u / CR,
  // slot u % CR); wave w loads units [(i NW + w) 64, + 64) for i < IW.
  auto issue = [&](int p) {
    char* base = smem + (p % NR) * KS * 2 * TILE;
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      const int t = p * KS + q;
      char* kt = base + q * 2 * TILE;
      const int k0 = kbeg + t * BKV;
      // row k0 + r of segment 1 is its row k0 - len0 + r (used only for rows >= len0)
      const long tk0 = kbase0 + k0 * kst0, tk1 = kbase1 + (long)(k0 - len0) * kst1;
      const long tv0 = vbase0 + k0 * vst0, tv1 = vbase1 + (long)(k0 - len0) * vst1;
#pragma unroll
      for (int i = 0; i < IW; ++i) {
        const bf16 *ks = Z, *vs = Z;
        if constexpr (HOIST) {
          const int kk = k0 + lrow[i];
          if (t < nt && kk < kend && lok[i]) {
            const bool s1 = kk >= len0;
            ks = reinterpret_cast<const bf16*>(s1 ? tk1 + rk1[i] : tk0 + rk0[i]);
            vs = reinterpret_cast<const bf16*>(s1 ? tv1 + rv1[i] : tv0 + rv0[i]);
          }
        } else {
          const int u = (i * NW + wave) * 64 + lane, row = u / CR, c = (u % CR) ^ C::swz(row), d8 = c * 8;
          const int kk = k0 + row;
          if (t < nt && kk < kend && d8 < hd) {
            const int which = kk < len0 ? 0 : 1;
            const int key = which ? kk - len0 : kk;
            ks = seg_row(a, which, b, g, key, false) + d8;
            vs = seg_row(a, which, b, g, key, true) + d8;
          }
        }
        __builtin_amdgcn_global_load_lds(ks, kt + (i * NW + wave) * 1024, 16, 0, 0);
        __builtin_amdgcn_global_load_lds(vs, kt + TILE + (i * NW + wave) * 1024, 16, 0, 0);
      }
    }
  };

  f32x4 o[ND];
#pragma unroll
  for (int u = 0; u < ND; ++u) o[u] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float sl2 = a.scale * 1.4426950408889634f;   // scale * log2(e)
  constexpr int PER_ROUND = KS * 2 * IW;             // direct loads per wave per round

#pragma unroll
  for (int p = 0; p < NR - 1; ++p)
    if (p < nrounds) issue(p);
  for (int p = 0; p < nrounds; ++p) {
    // round p has landed once at most the NR - 2 later rounds' loads are
    // pending; the barrier (no fence) then also guarantees every wave is done
    // with round p - 1, whose slot the next issue overwrites
    if (p + NR - 2 < nrounds) {
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"((NR - 2) * PER_ROUND) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    if (p + NR - 1 < nrounds) issue(p + NR - 1);
    const int t = p * KS + kg;
    if (t >= nt) continue;
    const char* Kt = smem + (p % NR) * KS * 2 * TILE + kg * 2 * TILE;
    const char* Vt = Kt + TILE;
    const int k0 = kbeg + t * BKV;

    // ---- S^T = K Q^T over BKV / 16 subtiles of 16 keys
    constexpr int NST = BKV / 16;
    f32x4 sc[NST];
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      sc[st] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int row = st * 16 + lq;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int cc = c * 4 + grp;
        bf16x8 kf = *reinterpret_cast<const bf16x8*>(Kt + row * ROWB + ((cc ^ C::swz(row)) << 4));
        sc[st] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[c], sc[st], 0, 0, 0);
      }
    }
    // keys past the range exist only in a range's last tile (a block-uniform
    // test): they get score -inf. The running max is kept in log2 units
    // (scores times scale log2 e, positive), so each probability is one fused
    // multiply-add and the hardware exp2, whose argument is <= 0 or -inf.
    if (k0 + BKV > kend) {
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (k0 + st * 16 + grp * 4 + i >= kend) sc[st][i] = -INFINITY;
    }
    float mx = fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3]));
#pragma unroll
    for (int st = 1; st < NST; ++st)
      mx = fmaxf(mx, fmaxf(fmaxf(sc[st][0], sc[st][1]), fmaxf(sc[st][2], sc[st][3])));
    mx = max_x32(max_x16(mx));
    const float m_new = fmaxf(m_run, mx * sl2);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[st][i], sl2, -m_new));
        sc[st][i] = pv;
        ps[i] += pv;
      }
    const float psum = sum_x32(sum_x16((ps[0] + ps[1]) + (ps[2] + ps[3])));
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int u = 0; u < ND; ++u) o[u] *= alpha;

    // ---- O^T += V^T P^T per 32-key chunk; K-slot jj of lane group grp is key
    // 4 grp + jj (jj < 4) or 16 + 4 grp + jj - 4 (jj >= 4) of the chunk
    const int s4 = lane & 15;
#pragma unroll
    for (int kc = 0; kc < BKV / 32; ++kc) {
      bf16x8 pf = {(bf16)sc[2 * kc][0], (bf16)sc[2 * kc][1], (bf16)sc[2 * kc][2], (bf16)sc[2 * kc][3],
                   (bf16)sc[2 * kc + 1][0], (bf16)sc[2 * kc + 1][1], (bf16)sc[2 * kc + 1][2], (bf16)sc[2 * kc + 1][3]};
      const int r_lo = kc * 32 + 4 * grp + (s4 >> 2), r_hi = r_lo + 16;
#pragma unroll
      for (int u = 0; u < ND; ++u) {
        const int cc = 2 * u + ((s4 & 3) >> 1), off = (s4 & 1) << 3;
        const char* plo = Vt + r_lo * ROWB + ((cc ^ C::swz(r_lo)) << 4) + off;
        const char* phi = Vt + r_hi * ROWB + ((cc ^ C::swz(r_hi)) << 4) + off;
        const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(plo));
        const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4s*)(phi));
        const bf16x4 l4 = __builtin_bit_cast(bf16x4, lo), h4 = __builtin_bit_cast(bf16x4, hi);
        const bf16x8 vf = {l4[0], l4[1], l4[2], l4[3], h4[0], h4[1], h4[2], h4[3]};
        o[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf, o[u], 0, 0, 0);
      }
    }
  }

  if constexpr (KS > 1) {
    // merge the key groups into group 0, in group order: m = max m_q,
    // l = sum l_q 2^(m_q - m), o = sum o_q 2^(m_q - m)
    __syncthreads();                               // the ring is free from here on
    float* mg = reinterpret_cast<float*>(smem);
    const int slot = wrow * 64 + lane;             // lane of a row group
    if (kg > 0) {
      float* dst = mg + ((kg - 1) * 256 + slot) * MST;
#pragma unroll
      for (int u = 0; u < ND; ++u) *reinterpret_cast<f32x4*>(dst + 4 * u) = o[u];
      dst[ND * 4] = m_run;
      dst[ND * 4 + 1] = l_run;
    }
    __syncthreads();
    if (kg > 0) return;
    float mq[KS], lq_[KS];
    mq[0] = m_run; lq_[0] = l_run;
#pragma unroll
    for (int q = 1; q < KS; ++q) {
      const float* src = mg + ((q - 1) * 256 + slot) * MST;
      mq[q] = src[ND * 4]; lq_[q] = src[ND * 4 + 1];
    }
    float m = mq[0];
#pragma unroll
    for (int q = 1; q < KS; ++q) m = fmaxf(m, mq[q]);
    float l = 0.f, w[KS];
#pragma unroll
    for (int q = 0; q < KS; ++q) {
      w[q] = __builtin_amdgcn_exp2f(mq[q] - m);
      l += lq_[q] * w[q];
    }
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      f32x4 acc = o[u] * w[0];
#pragma unroll
      for (int q = 1; q < KS; ++q)
        acc += *reinterpret_cast<const f32x4*>(mg + ((q - 1) * 256 + slot) * MST + 4 * u) * w[q];
      o[u] = acc;
    }
    m_run = m;
    l_run = l;
  }

  if (!rvalid) return;
  if (S > 1) {
    const long row = ((long)b * a.Hq + h) * a.Lq + qi;
    float* po = a.ws + (row * S + split) * hd;
#pragma unroll
    for (int u = 0; u < ND; ++u) {
      const int d = u * 16 + grp * 4;
      if (d < hd) *reinterpret_cast<f32x4*>(po + d) = o[u];
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
  for (int u = 0; u < ND; ++u) {
    const int d = u * 16 + grp * 4;
    if (d < hd) {
      bf16x4 wv = {(bf16)(o[u][0] * inv), (bf16)(o[u][1] * inv), (bf16)(o[u][2] * inv), (bf16)(o[u][3] * inv)};
      *reinterpret_cast<bf16x4*>(op + d) = wv;
    }
  }
}

}  // namespace

// Launch plan of a bf16 attention. Direct-load kernel: key groups inside a
// block (KS = 2) whenever the grid leaves CUs without a second block (short
// decode and small prefill grids), and key ranges over blocks (split-KV,
// merged by attn_combine_kernel) only when the rounds of tiles they save
// outweigh the merge: the count S minimises rounds x tile time + merge time
// (measured on MI355X: a round of 64 keys ~0.8 us at head dim 32, ~1.4 us
// at 64, of 32 keys ~2.1 us at 256; the merge ~3.5 us), at most one block
// per CU.
// Register-staged kernel (head dim 72): split when fewer than 128 blocks.
static void attn_plan(const AttnArgs& a, int& splits, int& kchunk, int& ks) {
  const int rows = (a.Hq / a.Hkv) * a.Lq;
  const long blocks = (long)((rows + BQ - 1) / BQ) * a.Hkv * a.B;
  const int total = a.seg[0].len + a.seg[1].len, ntiles = (total + BKV - 1) / BKV;
  const bool v2 = a.zeros != nullptr;
  // two key groups per block when the grid leaves CUs free, and always at
  // head dim 256, where the second group of waves hides the per-tile latency
  // of the large output accumulators (bidirectional pi0-shaped prefill over
  // 816 keys: 155 -> 115 us at batch 8)
  ks = (v2 && a.hd > 32 && (blocks < 256 || a.hd > 128)) ? 2 : 1;
  splits = 1;
  kchunk = ntiles * BKV;
  if (!a.ws || ntiles < 2) return;
  int best = 1;
  if (v2) {
    const int tile = a.hd >= 256 ? 32 : 64;                      // keys per kernel tile
    const double t_tile = a.hd <= 32 ? 0.8 : (a.hd <= 64 ? 1.4 : (a.hd <= 128 ? 1.7 : 2.1)), t_merge = 3.5;
    const int smax = (int)std::min<long>(16, std::max<long>(1, 256 / blocks));
    double best_t = 1e30;
    for (int sp = 1; sp <= std::min(smax, ntiles); ++sp) {
      const int per = (ntiles + sp - 1) / sp;                   // 64-key units per range
      const int rounds = ((per * BKV + tile - 1) / tile + ks - 1) / ks;
      const double t = rounds * t_tile + (sp > 1 ? t_merge : 0.0);
      if (t < best_t - 1e-9) { best_t = t; best = sp; }
    }
  } else if (blocks < 128) {
    best = (int)std::min<long>({(256 + blocks - 1) / blocks, (long)ntiles, 16L});
  }
  while (best > 1 && (long)a.B * a.Hq * a.Lq * best * (a.hd + 2) > a.ws_floats) --best;
  const int per = (ntiles + best - 1) / best;
  kchunk = per * BKV;
  splits = (ntiles + per - 1) / per;              // every range holds keys
}

void launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.B <= 0 || a.Lq <= 0) return;
  if (a.et == ET_F32) {
    hipLaunchKernelGGL(attn_f32_kernel, dim3(a.Lq, a.Hq, a.B), dim3(64), 0, s, a);
    return;
  }
  // the direct-load kernel keeps scores in log2 units scaled by a positive
  // factor and 32-bit offsets of a tile's rows within a segment
  VLA_REQUIRE(a.scale > 0.f, "attention scale must be positive");
  for (const AttnSeg& sg : a.seg)
    VLA_REQUIRE(64L * 2 * std::max(std::labs(sg.k_si), std::labs(sg.v_si)) + 2L * a.hd < (1L << 32),
                "attention key row stride too large");
  AttnArgs b = a;
  int ks;
  attn_plan(a, b.splits, b.kchunk, ks);
  const int rows = (a.Hq / a.Hkv) * a.Lq;
  dim3 grid((rows + BQ - 1) / BQ, a.Hkv, a.B * b.splits);
  // the direct-load kernel serves every head dim (a multiple of 8) with a
  // zero buffer, padded to the next of 32, 64, 128, 256 (chunks past hd load
  // zeros and are not stored): the ViT's 72 runs on the 128-wide variant
  // (54.8 -> 33.4 us per pi0-shaped layer at batch 8 against the
  // register-staged kernel padded to 96); callers without a zero buffer use
  // the register-staged one
  const bool v2 = a.zeros != nullptr;
  if (v2 && a.hd <= 32) hipLaunchKernelGGL((attn_v2_kernel<32, 1>), grid, dim3(256), 0, s, b);
  else if (v2 && a.hd <= 64 && ks == 2) hipLaunchKernelGGL((attn_v2_kernel<64, 2>), grid, dim3(512), 0, s, b);
  else if (v2 && a.hd <= 64) hipLaunchKernelGGL((attn_v2_kernel<64, 1>), grid, dim3(256), 0, s, b);
  else if (v2 && a.hd <= 128 && ks == 2) hipLaunchKernelGGL((attn_v2_kernel<128, 2>), grid, dim3(512), 0, s, b);
  else if (v2 && a.hd <= 128) hipLaunchKernelGGL((attn_v2_kernel<128, 1>), grid, dim3(256), 0, s, b);
  else if (v2 && ks == 2) hipLaunchKernelGGL((attn_v2_kernel<256, 2>), grid, dim3(512), 0, s, b);
  else if (v2) hipLaunchKernelGGL((attn_v2_kernel<256, 1>), grid, dim3(256), 0, s, b);
  else if (a.hd <= 32) hipLaunchKernelGGL(attn_mfma_kernel<32>, grid, dim3(256), 0, s, b);
  else if (a.hd <= 64) hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, s, b);
  else if (a.hd <= 96) hipLaunchKernelGGL(attn_mfma_kernel<96>, grid, dim3(256), 0, s, b);
  else hipLaunchKernelGGL(attn_mfma_kernel<256>, grid, dim3(256), 0, s, b);
  if (b.splits > 1) {
    // 256-thread blocks of 4 wavefronts x 64 / LPR rows
    const long nrows = (long)a.B * a.Hq * a.Lq;
    auto blocks = [&](int lpr) { const long rpb = 4L * (64 / lpr); return dim3((unsigned)((nrows + rpb - 1) / rpb)); };
    if (a.hd <= 64) hipLaunchKernelGGL(attn_combine_kernel<16>, blocks(16), dim3(256), 0, s, b);
    else if (a.hd <= 128) hipLaunchKernelGGL(attn_combine_kernel<32>, blocks(32), dim3(256), 0, s, b);
    else hipLaunchKernelGGL(attn_combine_kernel<64>, blocks(64), dim3(256), 0, s, b);
  }
}
