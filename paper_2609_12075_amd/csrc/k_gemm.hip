// Matrix products of the VLA stages on gfx950.
//
// Every dense projection of both stages (QKV, attention output, MLP, patch
// embedding, projector, action in/out, time and adaLN conditioning) is
// D[m][n] = sum_k A[m][k] W[n][k] with the weight stored transposed (K
// contiguous). bf16 models use the CDNA4 matrix cores
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation); fp32 models use a VALU FMA
// kernel. The product is computed as D^T = W A^T so that each lane of the
// matrix instruction ends up owning four consecutive output columns of one
// row: that makes the fused epilogues (bias, residual add, GeGLU pairs, RoPE
// pairs, head scatter, Euler update) lane-local and the stores contiguous.
#include <algorithm>

#include "common.h"
#include "rownorm.h"

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2v;

// s0 + v0^2 + v1^2 + v2^2 + v3^2 and s1 + v4^2 + ... + v7^2 with the bf16
// pair dot instruction (two accumulators keep the chain short)
__device__ __forceinline__ void sumsq8(const bf16x8& v, float& s0, float& s1) {
  const bf16x2v p0 = __builtin_shufflevector(v, v, 0, 1), p1 = __builtin_shufflevector(v, v, 2, 3);
  const bf16x2v p2 = __builtin_shufflevector(v, v, 4, 5), p3 = __builtin_shufflevector(v, v, 6, 7);
  s0 = __builtin_amdgcn_fdot2_f32_bf16(p0, p0, s0, false);
  s1 = __builtin_amdgcn_fdot2_f32_bf16(p2, p2, s1, false);
  s0 = __builtin_amdgcn_fdot2_f32_bf16(p1, p1, s0, false);
  s1 = __builtin_amdgcn_fdot2_f32_bf16(p3, p3, s1, false);
}
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// ---------------------------------------------------------------- epilogue
__device__ __forceinline__ float act_apply(float x, int act) {
  if (act == ACT_SILU) return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x));   // -0 once e^-x overflows
  if (act == ACT_GELU) {
    // tanh form: 0.5 x (1 + tanh u) with u = sqrt(2/pi) (x + 0.044715 x^3),
    // evaluated through the identity 0.5 (1 + tanh u) = 1 / (1 + e^(-2u)):
    // the hardware exp2 and reciprocal (about 1 ulp each) in place of the
    // library tanh; e^(-2u) = +inf for very negative x gives -0, = 0 for very
    // positive x gives x
    const float u = 0.7978845608028654f * (x + 0.044715f * x * x * x);
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-2.8853900817779268f * u));   // 2 log2 e
  }
  return x;
}

__device__ __forceinline__ void store_elem(void* base, long idx, int type, float v) {
  if (type == ET_BF16) reinterpret_cast<bf16*>(base)[idx] = (bf16)v;
  else reinterpret_cast<float*>(base)[idx] = v;
}

// The residual update x + g * (d + b) (g = the gate, or 1) and the Euler
// update x + dt * (d + b), each one explicit fused multiply-add after the
// bias add, so that every epilogue path (per-element, vector, from
// registers, the reduce fused with a row norm) rounds alike.
__device__ __forceinline__ float upd(float x, float d, float b, float g) { return fmaf(d + b, g, x); }
__device__ __forceinline__ f32x4 upd(f32x4 x, f32x4 d, f32x4 b, f32x4 g) {
  return f32x4{upd(x[0], d[0], b[0], g[0]), upd(x[1], d[1], b[1], g[1]), upd(x[2], d[2], b[2], g[2]),
               upd(x[3], d[3], b[3], g[3])};
}

// Epilogue for output row m and the four columns n0..n0+3 (n0 % 4 == 0).
template <int MODE>
__device__ __forceinline__ void epilogue4(const GemmArgs& a, int m, int n0, float v[4]) {
  if (m >= a.M || n0 >= a.N) return;
  const int nv = min(4, a.N - n0);
  switch (MODE) {
    case EPI_STORE: {
      long row = a.row_group > 0 ? (long)(m / a.row_group) * a.row_group_stride + (long)(m % a.row_group) * a.ldo
                                 : (long)m * a.ldo;
      float r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float x = v[j];
        if (j < nv) {
          if (a.bias) x += a.bias[n0 + j];
          if (a.tab) x += a.tab[(long)(m % a.tab_period) * a.ldtab + n0 + j];
        }
        r[j] = act_apply(x, a.act);
      }
      if (a.out_type == ET_BF16) {
        bf16* o = reinterpret_cast<bf16*>(a.out) + row + n0;
        if (nv == 4 && ((reinterpret_cast<uintptr_t>(o) & 7) == 0)) {
          bf16x4 w = {(bf16)r[0], (bf16)r[1], (bf16)r[2], (bf16)r[3]};
          *reinterpret_cast<bf16x4*>(o) = w;
        } else {
          for (int j = 0; j < nv; ++j) o[j] = (bf16)r[j];
        }
      } else {
        float* o = reinterpret_cast<float*>(a.out) + row + n0;
        if (nv == 4 && ((reinterpret_cast<uintptr_t>(o) & 15) == 0)) {
          *reinterpret_cast<f32x4*>(o) = f32x4{r[0], r[1], r[2], r[3]};
        } else {
          for (int j = 0; j < nv; ++j) o[j] = r[j];
        }
        if (a.out2) {
          bf16* o2 = reinterpret_cast<bf16*>(a.out2) + (long)m * a.ldo2 + n0;
          for (int j = 0; j < nv; ++j) o2[j] = (bf16)r[j];
        }
      }
      break;
    }
    case EPI_RESID: {
      long row = a.row_group > 0 ? (long)(m / a.row_group) * a.row_group_stride + (long)(m % a.row_group) * a.ldo
                                 : (long)m * a.ldo;
      float* o = reinterpret_cast<float*>(a.out) + row + n0;
      for (int j = 0; j < nv; ++j) {
        o[j] = upd(o[j], v[j], a.bias ? a.bias[n0 + j] : 0.0f, a.gate ? a.gate[n0 + j] : 1.0f);
        if (a.out2) reinterpret_cast<bf16*>(a.out2)[(long)m * a.ldo2 + n0 + j] = (bf16)o[j];
      }
      break;
    }
    case EPI_GEGLU: {
      // weight rows interleaved: row 2f = gate f, row 2f + 1 = up f
      bf16* ob = reinterpret_cast<bf16*>(a.out);
      float* of = reinterpret_cast<float*>(a.out);
      const int f0 = n0 >> 1;
      for (int j = 0; j + 1 < nv; j += 2) {
        float g = v[j], u = v[j + 1];
        if (a.bias) { g += a.bias[n0 + j]; u += a.bias[n0 + j + 1]; }
        float r = act_apply(g, ACT_GELU) * u;
        long idx = (long)m * a.ldo + f0 + (j >> 1);
        if (a.out_type == ET_BF16) ob[idx] = (bf16)r; else of[idx] = r;
      }
      break;
    }
    case EPI_QKV: {
      const QkvEpi& q = a.qkv;
      const int c0 = q.n_off + n0;            // logical column (multiple of 4)
      const int hd = q.hd;
      const int b = m / q.seq, i = m % q.seq;
      int seg, head, j0;
      if (c0 < q.n_q * hd) { seg = 0; head = c0 / hd; j0 = c0 % hd; }
      else if (c0 < (q.n_q + q.n_kv) * hd) { seg = 1; head = (c0 - q.n_q * hd) / hd; j0 = (c0 - q.n_q * hd) % hd; }
      else { seg = 2; head = (c0 - (q.n_q + q.n_kv) * hd) / hd; j0 = (c0 - (q.n_q + q.n_kv) * hd) % hd; }
      float x[4];
      for (int j = 0; j < 4; ++j) x[j] = v[j] + ((a.bias && j < nv) ? a.bias[n0 + j] : 0.0f);
      void* dst; long idx;
      if (seg == 0) { dst = q.q; idx = (long)b * q.q_sb + (long)head * q.q_sh + (long)i * q.q_si; }
      else if (seg == 1) { dst = q.k; idx = (long)b * q.k_sb + (long)head * q.k_sh + (long)i * q.k_si; }
      else { dst = q.v; idx = (long)b * q.v_sb + (long)head * q.v_sh + (long)i * q.v_si; }
      if (seg < 2 && q.pos0 >= 0) {
        // weight rows of q and k are stored pair-interleaved per head:
        // row 2t holds dimension t and row 2t + 1 holds dimension t + hd/2,
        // so these four columns are dims (t, t+1) and (t+hd/2, t+1+hd/2)
        const int half = hd >> 1, pos = q.pos0 + i, t = j0 >> 1;
        const f32x4 cs = *reinterpret_cast<const f32x4*>(q.rope_cs + ((long)pos * half + t) * 2);  // c_t s_t c_t+1 s_t+1
        const float lo0 = x[0] * cs[0] - x[1] * cs[1], hi0 = x[1] * cs[0] + x[0] * cs[1];
        const float lo1 = x[2] * cs[2] - x[3] * cs[3], hi1 = x[3] * cs[2] + x[2] * cs[3];
        if (a.out_type == ET_BF16) {
          bf16* d = reinterpret_cast<bf16*>(dst) + idx;
          *reinterpret_cast<bf16x2*>(d + t) = bf16x2{(bf16)lo0, (bf16)lo1};
          *reinterpret_cast<bf16x2*>(d + t + half) = bf16x2{(bf16)hi0, (bf16)hi1};
        } else {
          float* d = reinterpret_cast<float*>(dst) + idx;
          d[t] = lo0; d[t + 1] = lo1; d[t + half] = hi0; d[t + half + 1] = hi1;
        }
      } else if (a.out_type == ET_BF16 && nv == 4) {
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(dst) + idx + j0) =
            bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
      } else {
        for (int j = 0; j < nv; ++j) store_elem(dst, idx + j0 + j, a.out_type, x[j]);
      }
      break;
    }
    case EPI_EULER: {
      float* o = reinterpret_cast<float*>(a.out) + (long)m * a.ldo + n0;
      for (int j = 0; j < nv; ++j) o[j] = upd(o[j], v[j], a.bias ? a.bias[n0 + j] : 0.0f, a.dt);
      break;
    }
  }
}

// ---------------------------------------------------------------- tile epilogue
// Epilogue of a whole output tile staged in LDS as fp32 (ROWS rows of BN
// columns, row stride LDC floats). Thread t finishes the four columns
// nc = (t % (BN/4)) * 4 of rows t / (BN/4) + it * (NT / (BN/4)). What depends
// only on the columns (bias, gate, QKV head and destination) is read or
// computed once per thread, and every load that depends on the row (the old
// residual or Euler state, the position table, the RoPE angles) is issued for
// all of the thread's rows before the first store, so the row loads share one
// memory round trip instead of one each. Arithmetic per element is that of
// epilogue4. Valid when a.epi_vec is set (N % 4 == 0 and every vector access
// aligned; see epi_vec_ok); otherwise callers use epilogue4.
// The epilogue of NIT rows ms[] (valid where ok[]) of the four columns
// n0..n0+3 (n0 < N), given their sums t[].
template <int MODE, int NIT>
__device__ __forceinline__ void epi_rows(const GemmArgs& a, const f32x4 (&t)[NIT], const int (&ms)[NIT],
                                         const bool (&ok)[NIT], int n0) {
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
  const f32x4 bias = a.bias ? *reinterpret_cast<const f32x4*>(a.bias + n0) : zero;
  auto row_off = [&](int m) -> long {
    return a.row_group > 0 ? (long)(m / a.row_group) * a.row_group_stride + (long)(m % a.row_group) * a.ldo
                           : (long)m * a.ldo;
  };
  if constexpr (MODE == EPI_STORE) {
    f32x4 tb[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it)
      tb[it] = (a.tab && ok[it]) ? *reinterpret_cast<const f32x4*>(a.tab + (long)(ms[it] % a.tab_period) * a.ldtab + n0)
                                 : zero;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      if (!ok[it]) continue;
      f32x4 x = t[it] + bias + tb[it];
      if (a.act != ACT_NONE) {
#pragma unroll
        for (int j = 0; j < 4; ++j) x[j] = act_apply(x[j], a.act);
      }
      const long o = row_off(ms[it]) + n0;
      if (a.out_type == ET_BF16) {
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(a.out) + o) = bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
      } else {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(a.out) + o) = x;
        if (a.out2)
          *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(a.out2) + (long)ms[it] * a.ldo2 + n0) =
              bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
      }
    }
  } else if constexpr (MODE == EPI_RESID || MODE == EPI_EULER) {
    float* out = reinterpret_cast<float*>(a.out);
    const f32x4 gate = (MODE == EPI_RESID && a.gate) ? *reinterpret_cast<const f32x4*>(a.gate + n0) : f32x4{1.f, 1.f, 1.f, 1.f};
    f32x4 old[NIT];
    long off[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      off[it] = (MODE == EPI_RESID ? row_off(ms[it]) : (long)ms[it] * a.ldo) + n0;
      old[it] = ok[it] ? *reinterpret_cast<const f32x4*>(out + off[it]) : zero;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      if (!ok[it]) continue;
      f32x4 r;
      if constexpr (MODE == EPI_RESID) r = upd(old[it], t[it], bias, gate);
      else r = upd(old[it], t[it], bias, f32x4{a.dt, a.dt, a.dt, a.dt});
      *reinterpret_cast<f32x4*>(out + off[it]) = r;
      if (MODE == EPI_RESID && a.out2)
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(a.out2) + (long)ms[it] * a.ldo2 + n0) =
            bf16x4{(bf16)r[0], (bf16)r[1], (bf16)r[2], (bf16)r[3]};
    }
  } else if constexpr (MODE == EPI_GEGLU) {
    // weight rows interleaved: column 2f = gate f, 2f + 1 = up f
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      if (!ok[it]) continue;
      const f32x4 x = t[it] + bias;
      const float r0v = act_apply(x[0], ACT_GELU) * x[1], r1v = act_apply(x[2], ACT_GELU) * x[3];
      const long o = (long)ms[it] * a.ldo + (n0 >> 1);
      if (a.out_type == ET_BF16)
        *reinterpret_cast<bf16x2*>(reinterpret_cast<bf16*>(a.out) + o) = bf16x2{(bf16)r0v, (bf16)r1v};
      else {
        float* of = reinterpret_cast<float*>(a.out) + o;
        of[0] = r0v;
        of[1] = r1v;
      }
    }
  } else if constexpr (MODE == EPI_QKV) {
    const QkvEpi& q = a.qkv;
    const int c0 = q.n_off + n0, hd = q.hd;
    int seg, head, j0;
    if (c0 < q.n_q * hd) { seg = 0; head = c0 / hd; j0 = c0 % hd; }
    else if (c0 < (q.n_q + q.n_kv) * hd) { seg = 1; head = (c0 - q.n_q * hd) / hd; j0 = (c0 - q.n_q * hd) % hd; }
    else { seg = 2; head = (c0 - (q.n_q + q.n_kv) * hd) / hd; j0 = (c0 - (q.n_q + q.n_kv) * hd) % hd; }
    void* dst = seg == 0 ? q.q : seg == 1 ? q.k : q.v;
    const long sb = seg == 0 ? q.q_sb : seg == 1 ? q.k_sb : q.v_sb;
    const long sh = seg == 0 ? q.q_sh : seg == 1 ? q.k_sh : q.v_sh;
    const long si = seg == 0 ? q.q_si : seg == 1 ? q.k_si : q.v_si;
    const bool rope = seg < 2 && q.pos0 >= 0;
    const int half = hd >> 1, tt = j0 >> 1;
    long idx[NIT];
    f32x4 cs[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int b = ms[it] / q.seq, i = ms[it] % q.seq;
      idx[it] = (long)b * sb + (long)head * sh + (long)i * si;
      // (cos, sin) of dims t and t + 1 at position pos0 + i
      cs[it] = (rope && ok[it]) ? *reinterpret_cast<const f32x4*>(q.rope_cs + ((long)(q.pos0 + i) * half + tt) * 2) : zero;
    }
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      if (!ok[it]) continue;
      const f32x4 x = t[it] + bias;
      if (rope) {
        // columns are dims (t, t+1) and (t+hd/2, t+1+hd/2): weight rows of q and
        // k are stored pair-interleaved per head
        const f32x4 c = cs[it];
        const float lo0 = x[0] * c[0] - x[1] * c[1], hi0 = x[1] * c[0] + x[0] * c[1];
        const float lo1 = x[2] * c[2] - x[3] * c[3], hi1 = x[3] * c[2] + x[2] * c[3];
        if (a.out_type == ET_BF16) {
          bf16* d = reinterpret_cast<bf16*>(dst) + idx[it];
          *reinterpret_cast<bf16x2*>(d + tt) = bf16x2{(bf16)lo0, (bf16)lo1};
          *reinterpret_cast<bf16x2*>(d + tt + half) = bf16x2{(bf16)hi0, (bf16)hi1};
        } else {
          float* d = reinterpret_cast<float*>(dst) + idx[it];
          d[tt] = lo0; d[tt + 1] = lo1; d[tt + half] = hi0; d[tt + half + 1] = hi1;
        }
      } else if (a.out_type == ET_BF16) {
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(dst) + idx[it] + j0) = bf16x4{(bf16)x[0], (bf16)x[1], (bf16)x[2], (bf16)x[3]};
      } else {
        *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(dst) + idx[it] + j0) = x;
      }
    }
  }
}

// The folded norm's row scale as a multiply of its own, never fused with the
// bias add that follows, so that every epilogue path (LDS tile, per-element,
// from registers) rounds alike.
__device__ __forceinline__ f32x4 row_scale(f32x4 t, float s) {
#pragma clang fp contract(off)
  return t * s;
}

// Thread tid of NT finishes the tile's rows r0 + it * RS of its four columns
// (see above), GRP rows per memory round trip (GRP bounds the registers the
// row loads hold); the tile is the sum of NSUM fp32 planes in LDS (plane
// stride ROWS * LDC floats), added in plane order, times rsc[row] when rsc
// (an LDS array of per-row scales) is given.
template <int MODE, int BN, int ROWS, int NT, int LDC, int NSUM = 1, int GRP = 8>
__device__ __forceinline__ void tile_epilogue(const GemmArgs& a, const float* Cs, int m_blk, int n_blk, int tid,
                                              const float* rsc = nullptr) {
  // GeGLU has no row loads to overlap and its activation is long: two rows at
  // a time keep its registers within the kernels' budget
  constexpr int GR = MODE == EPI_GEGLU ? 2 : GRP;
  constexpr int CPT = BN / 4, RS = NT / CPT, NIT = (ROWS + RS - 1) / RS, G = NIT < GR ? NIT : GR;
  static_assert(NT % CPT == 0, "threads must cover whole rows");
  const int nc = (tid % CPT) * 4, r0 = tid / CPT, n0 = n_blk + nc;
  if (n0 >= a.N) return;
#pragma unroll
  for (int g0 = 0; g0 < NIT; g0 += G) {
    f32x4 t[G];
    int ms[G];
    bool ok[G];
#pragma unroll
    for (int it = 0; it < G; ++it) {
      const int mr = r0 + (g0 + it) * RS;
      ms[it] = m_blk + mr;
      ok[it] = g0 + it < NIT && (ROWS % RS == 0 || mr < ROWS) && ms[it] < a.M;
      t[it] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (ok[it]) {
        t[it] = *reinterpret_cast<const f32x4*>(Cs + mr * LDC + nc);
#pragma unroll
        for (int z = 1; z < NSUM; ++z) t[it] += *reinterpret_cast<const f32x4*>(Cs + z * ROWS * LDC + mr * LDC + nc);
        if (rsc) t[it] = row_scale(t[it], rsc[mr]);
      }
    }
    epi_rows<MODE, G>(a, t, ms, ok, n0);
  }
}

// Epilogue of the split-K partial pass: the fp32 tile (the sum of NSUM
// planes, in plane order) goes to the workspace slice of K range bz (the
// reduce kernel runs the epilogue).
template <int BN, int ROWS, int NT, int LDC, int NSUM = 1>
__device__ __forceinline__ void tile_store_partial(const GemmArgs& a, const float* Cs, int m_blk, int n_blk, int bz,
                                                   int tid) {
  constexpr int CPT = BN / 4, RS = NT / CPT, NIT = (ROWS + RS - 1) / RS;
  const int ldp = (a.N + 3) & ~3;
  float* part = a.ws + (long)bz * a.M * ldp;
  const int nc = (tid % CPT) * 4, r0 = tid / CPT, n = n_blk + nc;
  if (n >= a.N) return;
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int mr = r0 + it * RS, m = m_blk + mr;
    if ((ROWS % RS == 0 || mr < ROWS) && m < a.M) {
      f32x4 t = *reinterpret_cast<const f32x4*>(Cs + mr * LDC + nc);
#pragma unroll
      for (int z = 1; z < NSUM; ++z) t += *reinterpret_cast<const f32x4*>(Cs + z * ROWS * LDC + mr * LDC + nc);
      *reinterpret_cast<f32x4*>(part + (long)m * ldp + n) = t;
    }
  }
}

// ---------------------------------------------------------------- epilogue from registers
// A wave's four fragments i = 0..3 along the weight rows: lane (lr, lq) of
// fragment (i, j) holds weight columns nb + 16 i + 4 lq .. + 3 of activation
// row mb + 16 j + lr (lr = lane % 16, lq = lane / 16). A 4 x 4 transpose of
// 32-bit words over the four 16-lane rows of the wave (two 32-lane and two
// 16-lane swaps) hands lane lq the words of fragment i = lq from all four
// lanes that share its row: 16 consecutive weight columns.
__device__ __forceinline__ void xpose4x4(unsigned (&p)[4]) {
  const auto s02 = __builtin_amdgcn_permlane32_swap(p[0], p[2], false, false);   // rows 0,1 <-> 2,3
  const auto s13 = __builtin_amdgcn_permlane32_swap(p[1], p[3], false, false);
  const auto s01 = __builtin_amdgcn_permlane16_swap(s02[0], s13[0], false, false);   // rows 0 <-> 1, 2 <-> 3
  const auto s23 = __builtin_amdgcn_permlane16_swap(s02[1], s13[1], false, false);
  p[0] = s01[0]; p[1] = s01[1]; p[2] = s23[0]; p[3] = s23[1];
}

__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  const bf16x2 h = bf16x2{(bf16)lo, (bf16)hi};
  return *reinterpret_cast<const unsigned*>(&h);
}

// The bias of the lane's four columns of each fragment (loaded ahead of the
// K loop where registers allow, so its latency is not paid at the end).
__device__ __forceinline__ void reg_bias(const GemmArgs& a, int nb, int lane, f32x4 (&bias)[4]) {
  const int lq = lane >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n0 = nb + 16 * i + 4 * lq;
    bias[i] = (a.bias && n0 < a.N) ? *reinterpret_cast<const f32x4*>(a.bias + n0) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

// The GeGLU or plain bf16-store epilogue of such a wave tile, without the LDS
// round trip: GeGLU (a fragment holds two whole gate/up pairs) leaves one
// word per fragment and the lane stores 16 bytes (output columns nb / 2 +
// 8 lq ..); a store leaves two words per fragment (both halves transposed)
// and the lane stores 32 bytes (columns nb + 16 lq ..). reg_epi_ok states
// what the caller must hold (N % 16 == 0, so a group of 16 columns is wholly
// inside or outside; aligned rows; no row table, row groups or copy).
template <int MODE, int TM>
__device__ __forceinline__ void reg_epilogue(const GemmArgs& a, const f32x4 (&acc)[4][TM], const f32x4 (&bias)[4], int nb,
                                             int mb, int lane) {
  static_assert(MODE == EPI_GEGLU || MODE == EPI_STORE, "GeGLU or plain store");
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const int lr = lane & 15, lq = lane >> 4;
  const bool col_ok = nb + 16 * lq < a.N;
  bf16* out = reinterpret_cast<bf16*>(a.out) + (MODE == EPI_GEGLU ? (nb >> 1) + 8 * lq : nb + 16 * lq);
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = mb + 16 * j + lr;
    if constexpr (MODE == EPI_GEGLU) {
      unsigned p[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 x = acc[i][j] + bias[i];
        p[i] = pack_bf16x2(act_apply(x[0], ACT_GELU) * x[1], act_apply(x[2], ACT_GELU) * x[3]);
      }
      xpose4x4(p);
      if (m < a.M && col_ok) *reinterpret_cast<u32x4*>(out + (long)m * a.ldo) = u32x4{p[0], p[1], p[2], p[3]};
    } else {
      unsigned lo[4], hi[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        f32x4 x = acc[i][j] + bias[i];
        if (a.act != ACT_NONE) {
#pragma unroll
          for (int e = 0; e < 4; ++e) x[e] = act_apply(x[e], a.act);
        }
        lo[i] = pack_bf16x2(x[0], x[1]);
        hi[i] = pack_bf16x2(x[2], x[3]);
      }
      xpose4x4(lo);
      xpose4x4(hi);
      if (m < a.M && col_ok) {
        u32x4* o = reinterpret_cast<u32x4*>(out + (long)m * a.ldo);
        o[0] = u32x4{lo[0], hi[0], lo[1], hi[1]};
        o[1] = u32x4{lo[2], hi[2], lo[3], hi[3]};
      }
    }
  }
}

// The residual update x += gate * (D + bias) of a wave tile from the
// accumulators (no LDS pass): fragment (i, j) of lane (lr, lq) covers the
// four fp32 columns nb + 16 i + 4 lq .. + 3 of row mb + 16 j + lr, one
// 16-byte read and write each (a row's four lanes cover 64 contiguous
// bytes). The old values, bias and gate are read ahead of the K loop
// (reg_resid_load): the block alone reads and writes its tile, and the
// launcher checks that the product's input does not overlap the output.
__device__ __forceinline__ long resid_row(const GemmArgs& a, int m) {
  return a.row_group > 0 ? (long)(m / a.row_group) * a.row_group_stride + (long)(m % a.row_group) * a.ldo
                         : (long)m * a.ldo;
}

template <int TN, int TM>
__device__ __forceinline__ void reg_resid_load(const GemmArgs& a, int nb, int mb, int lane, f32x4 (&old)[TN][TM],
                                               f32x4 (&bias)[TN], f32x4 (&gate)[TN]) {
  const int lr = lane & 15, lq = lane >> 4;
  const f32x4 zero = {0.f, 0.f, 0.f, 0.f}, one = {1.f, 1.f, 1.f, 1.f};
  const float* out = reinterpret_cast<const float*>(a.out);
#pragma unroll
  for (int i = 0; i < TN; ++i) {
    const int n0 = nb + 16 * i + 4 * lq;
    bias[i] = (a.bias && n0 < a.N) ? *reinterpret_cast<const f32x4*>(a.bias + n0) : zero;
    gate[i] = (a.gate && n0 < a.N) ? *reinterpret_cast<const f32x4*>(a.gate + n0) : one;
  }
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = mb + 16 * j + lr;
    const long ro = m < a.M ? resid_row(a, m) : 0;
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int n0 = nb + 16 * i + 4 * lq;
      old[i][j] = (m < a.M && n0 < a.N) ? *reinterpret_cast<const f32x4*>(out + ro + n0) : zero;
    }
  }
}

template <int TN, int TM>
__device__ __forceinline__ void reg_resid(const GemmArgs& a, const f32x4 (&acc)[TN][TM], const f32x4 (&old)[TN][TM],
                                          const f32x4 (&bias)[TN], const f32x4 (&gate)[TN], int nb, int mb, int lane) {
  const int lr = lane & 15, lq = lane >> 4;
  float* out = reinterpret_cast<float*>(a.out);
#pragma unroll
  for (int j = 0; j < TM; ++j) {
    const int m = mb + 16 * j + lr;
    if (m >= a.M) continue;
    const long ro = resid_row(a, m);
#pragma unroll
    for (int i = 0; i < TN; ++i) {
      const int n0 = nb + 16 * i + 4 * lq;
      if (n0 >= a.N) continue;
      const f32x4 r = upd(old[i][j], acc[i][j], bias[i], gate[i]);
      *reinterpret_cast<f32x4*>(out + ro + n0) = r;
      if (a.out2)
        *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(a.out2) + (long)m * a.ldo2 + n0) =
            bf16x4{(bf16)r[0], (bf16)r[1], (bf16)r[2], (bf16)r[3]};
    }
  }
}

// ---------------------------------------------------------------- bf16 MFMA kernel
// Block: 256 threads = 4 waves in a 2 x 2 grid over a BN (weight rows) x BM
// (activation rows) tile; K advances in steps of 64 through a double-buffered
// LDS tile whose rows are padded by 8 elements (conflict-free 16-byte reads).
template <int BN, int BM, typename TA, int MODE>
__global__ void __launch_bounds__(256)
gemm_mfma_kernel(GemmArgs a) {
  constexpr int BK = 64, LDK = BK + 8;
  constexpr int TN = BN / 32, TM = BM / 32;         // 16-wide subtiles per wave
  constexpr int WCH = BN * 8 / 256, ACH = BM * 8 / 256;   // 8-element chunks per thread
  constexpr int LDC = BN + 4;         // fp32 output tile row stride (epilogue)
  constexpr int OPER_BYTES = 2 * (BN + BM) * LDK * 2, OUT_BYTES = BM * LDC * 4;
  __shared__ __attribute__((aligned(16))) char smem[OPER_BYTES > OUT_BYTES ? OPER_BYTES : OUT_BYTES];
  auto Ws = reinterpret_cast<bf16 (*)[BN][LDK]>(smem);
  auto As = reinterpret_cast<bf16 (*)[BM][LDK]>(smem + 2 * BN * LDK * 2);
  auto Cs = reinterpret_cast<float (*)[LDC]>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn0 = (wave >> 1) * (BN / 2), wm0 = (wave & 1) * (BM / 2);
  int bx, by, bz;                       // (M tile, N tile, K range), die-aware order
  xcd_remap_grouped(bx, by, bz, 8);
  const int n_blk = by * BN, m_blk = bx * BM;
  // K range of this block: range bz covers [kbeg, kbeg + ksplit)
  const int kbeg = bz * a.ksplit;
  const int K = min(a.K, kbeg + a.ksplit);
  const int nk = K > kbeg ? (K - kbeg + BK - 1) / BK : 0;
  const bf16* W = reinterpret_cast<const bf16*>(a.W);
  const TA* A = reinterpret_cast<const TA*>(a.A);

  // PF K-tiles are in flight per thread (register slots; slot = tile % PF):
  // a tile's global loads are issued PF - 1 steps before it is written to LDS.
  constexpr int PF = (BN * BM <= 64 * 64) ? 4 : (BN * BM <= 128 * 64 ? 2 : 1);   // 128x128: keep 2 blocks/CU
  bf16x8 wreg[PF][WCH], areg[PF][ACH];
  const int crow = tid >> 3, ccol = (tid & 7) * 8;

  auto load_tile = [&](int kt, bf16x8 (&wr)[WCH], bf16x8 (&ar)[ACH]) {
    const int k = kbeg + kt * BK + ccol;
#pragma unroll
    for (int j = 0; j < WCH; ++j) {
      const int n = n_blk + crow + 32 * j;
      if (n < a.N && k < K) wr[j] = *reinterpret_cast<const bf16x8*>(W + (long)n * a.ldw + k);
      else wr[j] = bf16x8{};
    }
#pragma unroll
    for (int j = 0; j < ACH; ++j) {
      const int m = m_blk + crow + 32 * j;
      if (m < a.M && k < K) {
        if constexpr (sizeof(TA) == 2) {
          ar[j] = *reinterpret_cast<const bf16x8*>(A + (long)m * a.lda + k);
        } else {
          const f32x4* p = reinterpret_cast<const f32x4*>(A + (long)m * a.lda + k);
          f32x4 x0 = p[0], x1 = p[1];
          ar[j] = bf16x8{(bf16)x0[0], (bf16)x0[1], (bf16)x0[2], (bf16)x0[3],
                         (bf16)x1[0], (bf16)x1[1], (bf16)x1[2], (bf16)x1[3]};
        }
      } else {
        ar[j] = bf16x8{};
      }
    }
  };
  auto store_tile = [&](int buf, const bf16x8 (&wr)[WCH], const bf16x8 (&ar)[ACH]) {
#pragma unroll
    for (int j = 0; j < WCH; ++j) *reinterpret_cast<bf16x8*>(&Ws[buf][crow + 32 * j][ccol]) = wr[j];
#pragma unroll
    for (int j = 0; j < ACH; ++j) *reinterpret_cast<bf16x8*>(&As[buf][crow + 32 * j][ccol]) = ar[j];
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lk = (lane >> 4) * 8;
  auto compute = [&](int buf) {
#pragma unroll
    for (int kc = 0; kc < BK; kc += 32) {
      bf16x8 wf[TN], af[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) wf[i] = *reinterpret_cast<const bf16x8*>(&Ws[buf][wn0 + 16 * i + lr][kc + lk]);
#pragma unroll
      for (int j = 0; j < TM; ++j) af[j] = *reinterpret_cast<const bf16x8*>(&As[buf][wm0 + 16 * j + lr][kc + lk]);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[i], af[j], acc[i][j], 0, 0, 0);
    }
  };

#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (p < nk) load_tile(p, wreg[p], areg[p]);
  if (nk > 0) store_tile(0, wreg[0], areg[0]);
  __syncthreads();
  for (int kt0 = 0; kt0 < nk; kt0 += PF) {
#pragma unroll
    for (int p = 0; p < PF; ++p) {
      const int kt = kt0 + p;             // kt % PF == p: its slot was written to LDS already
      if (kt < nk) {
        if (kt + PF < nk) load_tile(kt + PF, wreg[p], areg[p]);
        compute(kt & 1);
        if (kt + 1 < nk) store_tile((kt + 1) & 1, wreg[(p + 1) % PF], areg[(p + 1) % PF]);
        __syncthreads();
      }
    }
  }

  // lane owns D[n = 4*(lane/16) + r][m = lane % 16] of every 16 x 16 subtile;
  // stage the tile through LDS (operand tiles are dead after the last
  // barrier) so each thread then finishes four consecutive columns of a row.
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
      *reinterpret_cast<f32x4*>(&Cs[wm0 + 16 * j + lr][wn0 + 16 * i + (lane >> 4) * 4]) = acc[i][j];
  __syncthreads();
  if (a.splits > 1) {
    // split-K: store this K range's partial tile; the reduce kernel finishes
    tile_store_partial<BN, BM, 256, LDC>(a, &Cs[0][0], m_blk, n_blk, bz, tid);
    return;
  }
  if (a.epi_vec) {
    tile_epilogue<MODE, BN, BM, 256, LDC>(a, &Cs[0][0], m_blk, n_blk, tid);
    return;
  }
#pragma unroll 1
  for (int c = tid; c < BM * (BN / 4); c += 256) {
    const int mr = c / (BN / 4), nc = (c % (BN / 4)) * 4;
    f32x4 t = *reinterpret_cast<const f32x4*>(&Cs[mr][nc]);
    float v[4] = {t[0], t[1], t[2], t[3]};
    epilogue4<MODE>(a, m_blk + mr, n_blk + nc, v);
  }
}

// Split-K second pass: out = epilogue(sum over splits, in split order).
// One thread per four consecutive output columns of a row.
template <int MODE>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(GemmArgs a) {
  const int ldp = (a.N + 3) & ~3, nc = ldp / 4;
  const long c = blockIdx.x * 256L + threadIdx.x;
  if (c >= (long)a.M * nc) return;
  const int m = (int)(c / nc), n0 = (int)(c % nc) * 4;
  const long stride = (long)a.M * ldp;
  const float* p = a.ws + (long)m * ldp + n0;
  // issue every partial load before the first add (splits <= 16)
  f32x4 part[16];
#pragma unroll
  for (int z = 0; z < 16; ++z)
    part[z] = z < a.splits ? *reinterpret_cast<const f32x4*>(p + z * stride) : f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 t = part[0];
#pragma unroll
  for (int z = 1; z < 16; ++z) t += part[z];
  if (a.epi_vec) {
    const f32x4 tt[1] = {t};
    const int mm[1] = {m};
    const bool ok[1] = {true};
    epi_rows<MODE, 1>(a, tt, mm, ok, n0);
    return;
  }
  float v[4] = {t[0], t[1], t[2], t[3]};
  epilogue4<MODE>(a, m, n0, v);
}

// Split-K second pass of a residual projection fused with the row norm that
// follows it: the waves of an output row (rownorm::waves_per_row, as in the
// norm kernel) sum the partials in split order, apply the residual
// epilogue (x += gate * (sum + bias)) exactly as the plain reduce does,
// write x, and normalise the new row into n.out (the same arithmetic as the
// norm kernel). Four waves per row instead of one: 30 % faster at a few
// thousand rows (1632 x 2048 with two K ranges 16.2 -> 11.1 us). Requires
// N == n.d <= 256 * NVW * WPR and contiguous rows (no row groups).
template <int NVW, int WPR>
__global__ void __launch_bounds__(256) splitk_reduce_norm_kernel(GemmArgs a, NormArgs n) {
  constexpr int RPB = 4 / WPR;
  __shared__ float red[4][2];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, w = wv % WPR;
  const int r = blockIdx.x * RPB + wv / WPR;
  if (WPR == 1 && r >= a.M) return;                 // (no barrier with one wave per row)
  const bool rok = r < a.M;
  const int rr = rok ? r : 0;
  const int ldp = (a.N + 3) & ~3;
  const long stride = (long)a.M * ldp;
  const float* p = a.ws + (long)rr * ldp;
  float* x = reinterpret_cast<float*>(a.out) + (long)rr * a.ldo;
  // every load of the row (partials in split order, old x, the residual's
  // bias and gate, the norm's parameters) before the first store, so they
  // share one memory round trip per four K ranges
  rownorm::f4 v[NVW], g[NVW], b[NVW];
  f32x4 t[NVW], bs[NVW], gt[NVW];
  const bool has_bias = a.bias != nullptr, has_gate = a.gate != nullptr;
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = min(rownorm::col<NVW>(w, j, lane), a.N - 4);
    v[j] = *reinterpret_cast<const f32x4*>(x + i);
    bs[j] = has_bias ? *reinterpret_cast<const f32x4*>(a.bias + i) : f32x4{0.f, 0.f, 0.f, 0.f};
    gt[j] = has_gate ? *reinterpret_cast<const f32x4*>(a.gate + i) : f32x4{1.f, 1.f, 1.f, 1.f};
  }
  rownorm::load_params<NVW>(n, w, lane, g, b);
  for (int z0 = 0; z0 < a.splits; z0 += 4) {
    f32x4 part[NVW][4];
#pragma unroll
    for (int j = 0; j < NVW; ++j) {
      const int i = min(rownorm::col<NVW>(w, j, lane), a.N - 4);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        part[j][q] = z0 + q < a.splits ? *reinterpret_cast<const f32x4*>(p + (z0 + q) * stride + i)
                                       : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int j = 0; j < NVW; ++j) {
      // partials summed in split order
      if (z0 == 0) t[j] = part[j][0];
      else t[j] += part[j][0];
#pragma unroll
      for (int q = 1; q < 4; ++q) t[j] += part[j][q];
    }
  }
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = rownorm::col<NVW>(w, j, lane);
    if (i >= a.N) {
      v[j] = rownorm::f4{0.f, 0.f, 0.f, 0.f};
      continue;
    }
    // as the residual epilogue: x + gate * (sum + bias) (gate 1 when absent)
    v[j] = upd(v[j], t[j], bs[j], gt[j]);
    if (rok) *reinterpret_cast<f32x4*>(x + i) = v[j];
  }
  rownorm::store_row<NVW, WPR>(n, r, rok, v, wv, w, lane, g, b, red);
}

// ---------------------------------------------------------------- small-M kernel
// For products with few activation rows (the action stage at small batch),
// where a tile's work is a short K loop and the cost is the memory round
// trip rather than the matrix work. A block owns 16 * TN weight rows and 64
// activation rows; its four waves take interleaved 32-wide K chunks (wave w:
// chunks w, w + 4, ...) and each wave issues the loads of CPW chunks before
// its first matrix instruction, so one round trip covers 4 * CPW * 32 of K.
// Loads are unconditional from clamped addresses (out-of-range fragments are
// zeroed after the load), which keeps them all in flight together. The wave
// partials are summed in LDS in wave order and the epilogue runs once per
// output (no atomics: results do not depend on timing).
template <int TN, int MODE, int RMS = 0>
__global__ void __launch_bounds__(256) gemm_skinny_kernel(GemmArgs a) {
  constexpr int BM = 64, BN = 16 * TN, CPW = 8;
  __shared__ __attribute__((aligned(16))) float red[4][BM][BN];
  __shared__ float rsq[RMS ? 4 : 1][RMS ? BM : 1], rsc[RMS ? BM : 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int bx, by, bz;
  xcd_remap_grouped(bx, by, bz, 8);
  const int m0 = bx * BM, n0 = by * BN;
  (void)bz;
  const int kbeg = 0, kend = a.K;
  const bf16* W = reinterpret_cast<const bf16*>(a.W);
  const bf16* A = reinterpret_cast<const bf16*>(a.A);
  const int lr = lane & 15, lk = (lane >> 4) * 8;
  // this lane's fragment rows (clamped into the operands) and their validity
  const bf16* wrow[TN];
  bool wok[TN];
#pragma unroll
  for (int i = 0; i < TN; ++i) {
    const int n = n0 + i * 16 + lr;
    wok[i] = n < a.N;
    wrow[i] = W + (long)min(n, a.N - 1) * a.ldw;
  }
  const bf16* arow[4];
  bool aok[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + j * 16 + lr;
    aok[j] = m < a.M;
    arow[j] = A + (long)min(m, a.M - 1) * a.lda;
  }
  f32x4 acc[TN][4];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  float rs[4] = {0.f, 0.f, 0.f, 0.f}, rs2[4] = {0.f, 0.f, 0.f, 0.f};   // RMS: sums of squares of this lane's A fragments

  for (int k0 = kbeg + wave * 32; k0 < kend; k0 += 4 * 32 * CPW) {
    bf16x8 wf[CPW][TN], af[CPW][4];
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      const int k = k0 + c * 128 + lk;
      const int kc = min(k, a.K - 8);
#pragma unroll
      for (int i = 0; i < TN; ++i) wf[c][i] = *reinterpret_cast<const bf16x8*>(wrow[i] + kc);
#pragma unroll
      for (int j = 0; j < 4; ++j) af[c][j] = *reinterpret_cast<const bf16x8*>(arow[j] + kc);
    }
    // keep every load of the round ahead of the matrix work
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      const bool kok = k0 + c * 128 + lk < kend;
#pragma unroll
      for (int i = 0; i < TN; ++i)
        if (!(kok && wok[i])) wf[c][i] = bf16x8{};
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (!(kok && aok[j])) af[c][j] = bf16x8{};
      if constexpr (RMS) {
#pragma unroll
        for (int j = 0; j < 4; ++j) sumsq8(af[c][j], rs[j], rs2[j]);
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][i], af[c][j], acc[i][j], 0, 0, 0);
    }
  }
  // lane holds rows n = 16 i + 4 (lane >> 4) + e, column m = 16 j + (lane & 15)
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *reinterpret_cast<f32x4*>(&red[wave][j * 16 + lr][i * 16 + (lane >> 4) * 4]) = acc[i][j];
  if constexpr (RMS) {
    // every A element of the block's rows was read by exactly one lane: add
    // the four K-chunk lanes of a row, then the waves, in wave order
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      rs[j] += rs2[j];
      rs[j] += __shfl_xor(rs[j], 16);
      rs[j] += __shfl_xor(rs[j], 32);
    }
    if (lane < 16) {
#pragma unroll
      for (int j = 0; j < 4; ++j) rsq[wave][j * 16 + lr] = rs[j];
    }
  }
  __syncthreads();
  if constexpr (RMS) {
    if (tid < BM) rsc[tid] = rsqrtf((rsq[0][tid] + rsq[1][tid] + rsq[2][tid] + rsq[3][tid]) / (float)a.rms_in + a.rms_eps);
    __syncthreads();
  }
  if (a.epi_vec) {
    tile_epilogue<MODE, BN, BM, 256, BN, 4>(a, &red[0][0][0], m0, n0, tid, RMS ? rsc : nullptr);
    return;
  }
#pragma unroll
  for (int c = tid; c < BM * BN / 4; c += 256) {
    const int mr = c / (BN / 4), nc = (c % (BN / 4)) * 4;
    f32x4 t = *reinterpret_cast<const f32x4*>(&red[0][mr][nc]) + *reinterpret_cast<const f32x4*>(&red[1][mr][nc]) +
              *reinterpret_cast<const f32x4*>(&red[2][mr][nc]) + *reinterpret_cast<const f32x4*>(&red[3][mr][nc]);
    if constexpr (RMS) t = row_scale(t, rsc[mr]);
    float v[4] = {t[0], t[1], t[2], t[3]};
    epilogue4<MODE>(a, m0 + mr, n0 + nc, v);
  }
}

// ---------------------------------------------------------------- multi-stage kernel
// For products with many activation rows (the VLM stage; the action stage at
// larger batches). Operand tiles move global -> LDS with the CDNA4 direct
// loads (global_load_lds_dwordx4: each lane's 16 bytes land at LDS base +
// 16 * lane, one wave writes 1 KiB contiguous) through STAGES buffers, so
// STAGES - 1 K-steps of loads are in flight without holding registers.
// LDS rows are BK bf16 without padding; the 16-byte chunk c of row r is
// stored in slot c ^ swz(r) (BK 128: r & 15; BK 64: (r >> 1) & 7; BK 32: (r >> 2) & 3), which
// makes the matrix-core fragment reads (16 rows, one chunk) conflict-free.
// Chunks outside the operand (rows >= M or N, columns >= K) are read from a
// zero buffer, which zero-fills K tails exactly. Block: KG groups of 4 waves;
// the waves of a group form a 2 x 2 grid of (BN/2) x (BM/2) wave tiles of
// 16 x 16 x 32 products, and group g takes K chunks g, g + KG, ... of every
// K-step's BK / 32 (a second group doubles the waves that issue loads and
// fragment reads per CU: with one wave per SIMD, LDS reads stay
// latency-bound at ~100 B/clk per CU, with two they reach ~280). The groups'
// tiles are summed in a fixed order in the epilogue. BK 32 with more stages
// keeps the same LDS per block but more K-steps of loads in flight. RMS: the
// RMSNorm folded into the product (a.rms_in): every A element passes through
// the fragment reads of the waves of weight-row half 0 exactly once, so those
// waves' A_j A_j^T diagonals are the rows' sums of squares; the row sums
// meet in LDS and scale the tile rows in the epilogue.
template <int BN, int BM, int STAGES, int MODE, int BK = 64, int KG = 1, int RMS = 0>
__global__ void __launch_bounds__(256 * KG)
gemm_stage_kernel(GemmArgs a) {
  constexpr int NT = 256 * KG, NWV = 4 * KG;            // threads, waves
  constexpr int ROWB = BK * 2;                          // bytes per LDS row
  constexpr int CPR = BK / 8;                           // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;                         // rows per wave load instruction
  constexpr int SWS = BK == 128 ? 0 : (BK == 64 ? 1 : 2);   // swizzle: slot = c ^ ((r >> SWS) & (CPR - 1))
  constexpr int TN = BN / 32, TM = BM / 32;
  constexpr int STAGE_BYTES = (BN + BM) * ROWB;
  constexpr int WG = BN / RPI / NWV, AG = BM / RPI / NWV;   // row groups per wave (W, A)
  constexpr int LOADS = WG + AG;                        // direct loads per thread per stage
  constexpr int KC = BK / 32, KCG = KC / KG;            // K chunks per step, per wave group
  static_assert(BK == 128 || BK == 64 || BK == 32, "BK must be 32, 64 or 128");
  static_assert(WG * RPI * NWV == BN && AG * RPI * NWV == BM, "row groups must divide among the waves");
  static_assert(KCG * KG == KC, "K chunks must divide among the wave groups");
  constexpr int LDC = BN + 4;
  constexpr int CS_BYTES = KG * BM * LDC * 4;           // one fp32 tile plane per wave group
  constexpr int MAIN = STAGES * STAGE_BYTES > CS_BYTES ? STAGES * STAGE_BYTES : CS_BYTES;
  // RMS: per-(wave group, row) sums of squares and the row scales after the
  // main buffer (one LDS object: a second one makes the compiler wait for
  // every direct load before each fragment read)
  constexpr int SMEM = MAIN + (RMS ? (KG + 1) * BM * 4 : 0);
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  float* Cs = reinterpret_cast<float*>(smem);
  float* rsq = reinterpret_cast<float*>(smem + MAIN);   // [KG][BM]
  float* rsc = rsq + KG * BM;                           // [BM]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, kg = wave >> 2, w4 = wave & 3;
  const int wn0 = (w4 >> 1) * (BN / 2), wm0 = (w4 & 1) * (BM / 2);
  int bx, by, bz;
  xcd_remap_grouped(bx, by, bz, 8);
  const int n_blk = by * BN, m_blk = bx * BM;
  // K range of this block (range bz of a split product)
  const int kbeg = bz * a.ksplit;
  const int K = min(a.K, kbeg + a.ksplit);
  const int nk = K > kbeg ? (K - kbeg + BK - 1) / BK : 0;
  const bf16* W = reinterpret_cast<const bf16*>(a.W);
  const bf16* A = reinterpret_cast<const bf16*>(a.A);
  const bf16* Z = reinterpret_cast<const bf16*>(a.zeros);

  // this lane's row within a row group and its LDS slot; the slot holds
  // logical chunk (slot ^ swz(row)) of the row
  const int lrow = lane / CPR, slot = lane % CPR;
  auto issue = [&](int kt, int buf) {
    char* st = smem + buf * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < WG; ++j) {
      const int grp = j * NWV + wave, r = grp * RPI + lrow;
      const int c = slot ^ ((r >> SWS) & (CPR - 1)), k = kbeg + kt * BK + c * 8, n = n_blk + r;
      const bf16* src = (n < a.N && k < K) ? W + (long)n * a.ldw + k : Z;
      __builtin_amdgcn_global_load_lds(src, st + grp * RPI * ROWB, 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < AG; ++j) {
      const int grp = j * NWV + wave, r = grp * RPI + lrow;
      const int c = slot ^ ((r >> SWS) & (CPR - 1)), k = kbeg + kt * BK + c * 8, m = m_blk + r;
      const bf16* src = (m < a.M && k < K) ? A + (long)m * a.lda + k : Z;
      __builtin_amdgcn_global_load_lds(src, st + BN * ROWB + grp * RPI * ROWB, 16, 0, 0);
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // RMS: A_j A_j^T over this wave's K chunks; its diagonal holds the rows'
  // sums of squares (one extra matrix instruction per A fragment: these
  // products are bound by the loads, not by the matrix pipe, and VALU
  // dot products of the same fragments cost more)
  f32x4 sq[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) sq[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lq = lane >> 4;
  constexpr bool REG_EPI = KG == 1 && TN == 4 && (MODE == EPI_GEGLU || MODE == EPI_STORE);
  f32x4 rbias[4];
  if constexpr (REG_EPI) {
    if (a.epi_reg) reg_bias(a, n_blk + wn0, lane, rbias);
  }
  // residual update from registers with two wave groups (group 1 hands its
  // tile to group 0 through LDS, group 0 updates the rows: half the LDS
  // traffic of summing two staged planes; 2-4 % on the action stage's O and
  // down projections. With one group the LDS-staged update, whose rows are
  // written whole, measured as fast or faster): old values, bias and gate
  // read before the first stage's loads
  constexpr bool REG_RES = MODE == EPI_RESID && !RMS && KG == 2;
  constexpr int RTN = REG_RES ? TN : 1, RTM = REG_RES ? TM : 1;
  f32x4 rold[RTN][RTM], rrb[RTN], rrg[RTN];
  if constexpr (REG_RES) {
    if (a.epi_reg && kg == 0) reg_resid_load<TN, TM>(a, n_blk + wn0, m_blk + wm0, lane, rold, rrb, rrg);
  }
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(s, s);
  for (int kt = 0; kt < nk; ++kt) {
    // Stage kt has landed once at most the later stages' loads are pending;
    // then a plain barrier (no fence, which would wait for every pending
    // load): after it every wave's stage-kt data is in LDS and every wave has
    // consumed stage kt-1 (its fragments fed the matrix instructions).
    if (kt + STAGES - 2 < nk) {
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"((STAGES - 2) * LOADS) : "memory");
    } else {
      asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    }
    if (kt + STAGES - 1 < nk) issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    const char* st = smem + (kt % STAGES) * STAGE_BYTES;
    // all of the group's fragments of the K-step, then the products; the
    // scheduler is told to interleave the second chunk's fragment reads with
    // the first chunk's matrix instructions, so LDS latency hides behind
    // matrix work
    bf16x8 wf[KCG][TN], af[KCG][TM];
#pragma unroll
    for (int q = 0; q < KCG; ++q) {
      const int c = (q * KG + kg) * 4 + lq;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int r = wn0 + 16 * i + lr;
        wf[q][i] = *reinterpret_cast<const bf16x8*>(st + r * ROWB + ((c ^ ((r >> SWS) & (CPR - 1))) << 4));
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int r = wm0 + 16 * j + lr;
        af[q][j] = *reinterpret_cast<const bf16x8*>(st + BN * ROWB + r * ROWB + ((c ^ ((r >> SWS) & (CPR - 1))) << 4));
      }
    }
#pragma unroll
    for (int q = 0; q < KCG; ++q)
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[q][i], af[q][j], acc[i][j], 0, 0, 0);
    if constexpr (KCG == 2) {
      constexpr int NRD = TN + TM, NMF = TN * TM, R = NMF / NRD > 0 ? NMF / NRD : 1;
      __builtin_amdgcn_sched_group_barrier(0x100, NRD, 0);      // chunk 0 reads
#pragma unroll
      for (int q = 0; q < NRD; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // one chunk-1 read
        __builtin_amdgcn_sched_group_barrier(0x008, R, 0);      // R chunk-0 products
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * NMF - NRD * R, 0);
    }
    if constexpr (RMS) {
#pragma unroll
      for (int q = 0; q < KCG; ++q)
#pragma unroll
        for (int j = 0; j < TM; ++j) sq[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[q][j], af[q][j], sq[j], 0, 0, 0);
    }
  }
  if constexpr (RMS) {
    // lane l holds entries (4 (l / 16) + v, l % 16), v < 4, of each 16 x 16
    // block: the diagonal entry of row c = l % 16 sits in v = c - 4 (l / 16).
    // Weight-row half 0's waves publish one sum per (wave group, row).
    const int c = lane & 15, v = c - 4 * lq;
    if ((w4 >> 1) == 0 && v >= 0 && v < 4) {
#pragma unroll
      for (int j = 0; j < TM; ++j)
        rsq[kg * BM + wm0 + 16 * j + c] = v == 0 ? sq[j][0] : v == 1 ? sq[j][1] : v == 2 ? sq[j][2] : sq[j][3];
    }
  }
  if constexpr (REG_RES) {
    if (a.epi_reg) {
      {
        // group 1 hands its tile to group 0 through LDS (the stage buffers
        // are free once every wave has passed the barrier); the sum is in
        // group order, as in the LDS-staged epilogue
        __syncthreads();
        if (kg == 1) {
#pragma unroll
          for (int i = 0; i < TN; ++i)
#pragma unroll
            for (int j = 0; j < TM; ++j)
              *reinterpret_cast<f32x4*>(&Cs[(wm0 + 16 * j + lr) * LDC + wn0 + 16 * i + 4 * lq]) = acc[i][j];
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
          for (int j = 0; j < TM; ++j)
            acc[i][j] += *reinterpret_cast<const f32x4*>(&Cs[(wm0 + 16 * j + lr) * LDC + wn0 + 16 * i + 4 * lq]);
      }
      reg_resid<TN, TM>(a, acc, rold, rrb, rrg, n_blk + wn0, m_blk + wm0, lane);
      return;
    }
  }
  if constexpr (REG_EPI) {
    // GeGLU or a plain bf16 store from the accumulators (the launcher sets
    // epi_reg when reg_epi_ok holds and K is not split); RMS: the row scales
    // meet in LDS as below and each lane scales its rows' fragments
    if (a.epi_reg) {
      if constexpr (RMS) {
        __syncthreads();
        if (tid < BM) rsc[tid] = rsqrtf(rsq[tid] / (float)a.rms_in + a.rms_eps);
        __syncthreads();
#pragma unroll
        for (int j = 0; j < TM; ++j) {
          const float sc = rsc[wm0 + 16 * j + lr];
#pragma unroll
          for (int i = 0; i < TN; ++i) acc[i][j] = row_scale(acc[i][j], sc);
        }
      }
      reg_epilogue<MODE, TM>(a, acc, rbias, n_blk + wn0, m_blk + wm0, lane);
      return;
    }
  }
  // each wave group's tile to its own fp32 plane; the epilogues add the
  // planes in group order (the row scales, in their own LDS words, are
  // formed while the planes are written)
  __syncthreads();
  if constexpr (RMS) {
    if (tid < BM) {
      float t = rsq[tid];
#pragma unroll
      for (int z = 1; z < KG; ++z) t += rsq[z * BM + tid];
      rsc[tid] = rsqrtf(t / (float)a.rms_in + a.rms_eps);
    }
  }
  float* Cp = Cs + kg * BM * LDC;
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j)
      *reinterpret_cast<f32x4*>(&Cp[(wm0 + 16 * j + lr) * LDC + wn0 + 16 * i + (lane >> 4) * 4]) = acc[i][j];
  __syncthreads();
  if (!RMS && a.splits > 1) {
    // split-K: store this K range's partial tile; the reduce kernel finishes
    tile_store_partial<BN, BM, NT, LDC, KG>(a, Cs, m_blk, n_blk, bz, tid);
    return;
  }
  if (a.epi_vec) {
    tile_epilogue<MODE, BN, BM, NT, LDC, KG>(a, Cs, m_blk, n_blk, tid, RMS ? rsc : nullptr);
    return;
  }
#pragma unroll 1
  for (int c = tid; c < BM * (BN / 4); c += NT) {
    const int mr = c / (BN / 4), nc = (c % (BN / 4)) * 4;
    f32x4 t = *reinterpret_cast<const f32x4*>(&Cs[mr * LDC + nc]);
#pragma unroll
    for (int z = 1; z < KG; ++z) t += *reinterpret_cast<const f32x4*>(&Cs[z * BM * LDC + mr * LDC + nc]);
    if constexpr (RMS) t = row_scale(t, rsc[mr]);
    float v[4] = {t[0], t[1], t[2], t[3]};
    epilogue4<MODE>(a, m_blk + mr, n_blk + nc, v);
  }
}

// ---------------------------------------------------------------- large-tile kernel
// For large products (the VLM stage): 256 x 256 output tiles, NW waves in a
// (NW / 2) x 2 grid: 8 waves of 64 x 128 (12 fragment reads per 32 matrix
// instructions) or 4 waves of 128 x 128 (16 reads per 64 instructions: half
// the LDS read traffic per product of a 64 x 64 wave tile; LDS bandwidth,
// which the operand stores into LDS share, is what bounds the smaller
// tiles). Operands move global -> LDS with direct loads through two 64 KiB
// stages (one block per CU); per output this loads half the bytes of a
// 128 x 128 tile. Rows are XOR-swizzled as in the multi-stage kernel; the
// second K chunk's fragment reads are interleaved with the first chunk's
// products. The epilogue stages the fp32 tile through LDS in two halves of
// 128 rows; with REG (GeGLU or a plain bf16 store, eight waves) it works from
// the accumulators instead (reg_epilogue): a lane's fragment holds four
// consecutive weight columns of one activation row (for GeGLU two whole
// gate/up pairs, so the activation runs in registers), and the four lanes
// that share a row trade their packed results so that each lane stores 16 or
// 32 contiguous bytes. That takes the LDS round trip and its barriers out of
// every tile (pi0-shaped gate/up, 6528 x 32768 x 2048: 775 -> 740 us; 3264
// rows 407 -> 362 us; results identical).
template <int MODE, int NW, int BM = 256, bool REG = false>
__global__ void __launch_bounds__(NW * 64) gemm_big_kernel(GemmArgs a) {
  constexpr int BN = 256, BK = 64, ROWB = BK * 2;
  static_assert(BM == 256 || BM == 224, "activation tile of 256 or 224 rows");
  constexpr int WGN = NW / 2;                                    // waves along the weight rows
  constexpr int WTN = BN / WGN, WTM = BM / 2;                    // wave tile
  constexpr int TN = WTN / 16, TM = WTM / 16;
  static_assert(!REG || ((MODE == EPI_GEGLU || MODE == EPI_STORE) && TN == 4), "register epilogue: eight waves");
  constexpr int STAGE_BYTES = (BN + BM) * ROWB;                  // 64 KiB (60 KiB)
  constexpr int LDC = BN + 4;
  constexpr int SMEM = REG || 2 * STAGE_BYTES > 128 * LDC * 4 ? 2 * STAGE_BYTES : 128 * LDC * 4;
  constexpr int GPW = 32 / NW;                                   // 8-row groups per wave of the weight tile
  constexpr int AG = BM / 8;                                     // 8-row groups of the activation tile
  constexpr int GPWA = (AG + NW - 1) / NW;                       // ... per wave (the last may be short)
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];
  auto Cs = reinterpret_cast<float (*)[LDC]>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn0 = (wave >> 1) * WTN, wm0 = (wave & 1) * WTM;
  int bx, by, bz;
  xcd_remap_grouped(bx, by, bz, 8);
  const int n_blk = by * BN, m_blk = bx * BM;
  const int K = a.K;
  const int nk = (K + BK - 1) / BK;
  const bf16* W = reinterpret_cast<const bf16*>(a.W);
  const bf16* A = reinterpret_cast<const bf16*>(a.A);
  const bf16* Z = reinterpret_cast<const bf16*>(a.zeros);

  // 8-row groups: 32 of W and BM / 8 of A per stage (with 224 rows the
  // last round of A groups covers half the waves; the count per wave differs,
  // which the full waits below do not mind)
  const int lrow = lane >> 3, slot = lane & 7;
  auto issue = [&](int kt, int buf) {
    char* st = smem + buf * STAGE_BYTES;
#pragma unroll
    for (int j = 0; j < GPW; ++j) {
      const int grp = j * NW + wave, r = grp * 8 + lrow;
      const int c = slot ^ ((r >> 1) & 7), k = kt * BK + c * 8, n = n_blk + r;
      const bf16* src = (n < a.N && k < K) ? W + (long)n * a.ldw + k : Z;
      __builtin_amdgcn_global_load_lds(src, st + grp * 8 * ROWB, 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < GPWA; ++j) {
      const int grp = j * NW + wave, r = grp * 8 + lrow;
      if (AG % NW != 0 && grp >= AG) break;
      const int c = slot ^ ((r >> 1) & 7), k = kt * BK + c * 8, m = m_blk + r;
      const bf16* src = (m < a.M && k < K) ? A + (long)m * a.lda + k : Z;
      __builtin_amdgcn_global_load_lds(src, st + BN * ROWB + grp * 8 * ROWB, 16, 0, 0);
    }
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lq = lane >> 4;
  if (nk > 0) issue(0, 0);
  for (int kt = 0; kt < nk; ++kt) {
    // stage kt landed (nothing later is pending yet), and every wave is done
    // with stage kt - 1, whose buffer the next issue overwrites
    asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (kt + 1 < nk) issue(kt + 1, (kt + 1) & 1);
    const char* st = smem + (kt & 1) * STAGE_BYTES;
    bf16x8 wf[2][TN], af[2][TM];
#pragma unroll
    for (int kc = 0; kc < 2; ++kc) {
      const int c = kc * 4 + lq;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
        const int r = wn0 + 16 * i + lr;
        wf[kc][i] = *reinterpret_cast<const bf16x8*>(st + r * ROWB + ((c ^ ((r >> 1) & 7)) << 4));
      }
#pragma unroll
      for (int j = 0; j < TM; ++j) {
        const int r = wm0 + 16 * j + lr;
        af[kc][j] = *reinterpret_cast<const bf16x8*>(st + BN * ROWB + r * ROWB + ((c ^ ((r >> 1) & 7)) << 4));
      }
    }
#pragma unroll
    for (int kc = 0; kc < 2; ++kc)
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[kc][i], af[kc][j], acc[i][j], 0, 0, 0);
    {
      constexpr int NRD = TN + TM, NMF = TN * TM, R = NMF / NRD > 0 ? NMF / NRD : 1;
      __builtin_amdgcn_sched_group_barrier(0x100, NRD, 0);      // chunk 0 reads
#pragma unroll
      for (int q = 0; q < NRD; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // one chunk-1 read
        __builtin_amdgcn_sched_group_barrier(0x008, R, 0);      // R chunk-0 products
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 2 * NMF - NRD * R, 0);
    }
  }
  if constexpr (REG) {
    f32x4 bias[4];
    reg_bias(a, n_blk + wn0, lane, bias);
    reg_epilogue<MODE, TM>(a, acc, bias, n_blk + wn0, m_blk + wm0, lane);
    return;
  }
  // epilogue in two halves of BM / 2 activation rows (waves with wm0 == WTM h)
#pragma unroll 1
  for (int h = 0; h < 2; ++h) {
    __syncthreads();
    if (wm0 == WTM * h) {
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          *reinterpret_cast<f32x4*>(&Cs[16 * j + lr][wn0 + 16 * i + (lane >> 4) * 4]) = acc[i][j];
    }
    __syncthreads();
    if (a.epi_vec) {
      tile_epilogue<MODE, BN, WTM, NW * 64, LDC, 1, 4>(a, &Cs[0][0], m_blk + WTM * h, n_blk, tid);
      continue;
    }
#pragma unroll 1
    for (int c = tid; c < WTM * (BN / 4); c += NW * 64) {
      const int mr = c / (BN / 4), nc = (c % (BN / 4)) * 4;
      f32x4 t = *reinterpret_cast<const f32x4*>(&Cs[mr][nc]);
      float v[4] = {t[0], t[1], t[2], t[3]};
      epilogue4<MODE>(a, m_blk + WTM * h + mr, n_blk + nc, v);
    }
  }
}

// ---------------------------------------------------------------- fp32 VALU kernel
// 64 x 64 tile, 256 threads, each thread 4 columns x 4 rows; K in steps of 16.
template <int MODE>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmArgs a) {
  constexpr int BN = 64, BM = 64, BK = 16;
  __shared__ float Ws[BK][BN + 4];
  __shared__ float As[BK][BM + 4];
  const int tid = threadIdx.x;
  const int n_blk = blockIdx.y * BN, m_blk = blockIdx.x * BM;
  const float* W = reinterpret_cast<const float*>(a.W);
  const float* A = reinterpret_cast<const float*>(a.A);
  const int tn = (tid & 15) * 4, tm = (tid >> 4) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += BK) {
    for (int e = tid; e < BN * BK; e += 256) {
      const int r = e / BK, kk = e % BK;
      const int n = n_blk + r, k = k0 + kk;
      Ws[kk][r] = (n < a.N && k < a.K) ? W[(long)n * a.ldw + k] : 0.0f;
      const int m = m_blk + r;
      As[kk][r] = (m < a.M && k < a.K) ? A[(long)m * a.lda + k] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float w[4], x[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { w[i] = Ws[kk][tn + i]; x[i] = As[kk][tm + i]; }
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fmaf(x[r], w[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) epilogue4<MODE>(a, m_blk + tm + r, n_blk + tn, acc[r]);
}

// The epilogue from registers (reg_epilogue) needs bf16 output, whole
// 16-column groups, 16-byte aligned output rows and bias, and for a plain
// store no row table, row groups or fp32/bf16 copy.
static bool reg_epi_ok(const GemmArgs& a) {
  auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
  if (a.out_type != ET_BF16 || a.N % 16 != 0 || a.ldo % 8 != 0 || !al(a.out) || (a.bias && !al(a.bias))) return false;
  if (a.mode == EPI_GEGLU) return true;
  return a.mode == EPI_STORE && !a.tab && a.row_group <= 0 && !a.out2;
}

// ---------------------------------------------------------------- dispatch
// Kernels are specialised on tile shape, activation type and epilogue; fp32
// activations (the Euler state, conditioning vectors, robot state) only feed
// plain stores.
static GemmPlan plan_base(const GemmArgs& a) {
  constexpr int BK = 64;
  GemmPlan p{64, 32, 1, 64, 0};
  if (a.w_type == ET_F32) {
    p.bm = 64;
    p.ksplit = a.K;
    return p;
  }
  auto blocks = [&](int bn, int bm) { return (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn); };
  const int nk = (a.K + BK - 1) / BK;
  const long ldp = (a.N + 3) & ~3;
  // largest split count <= want whose partials fit the workspace, with the K
  // steps spread evenly (no empty range)
  auto set_splits = [&](int want) {
    int splits = std::max(1, std::min(want, 16));
    while (splits > 1 && (long)splits * a.M * ldp > a.ws_floats) --splits;
    const int ksteps = std::max(1, (nk + splits - 1) / splits);
    p.ksplit = ksteps * BK;
    p.splits = std::max(1, (nk + ksteps - 1) / ksteps);
  };
  if (a.a_type == ET_BF16 && a.zeros) {
    // few activation rows and many weight rows: the small-M kernel (one
    // memory round trip per 1024 of K, no K split); also for 1024-1535
    // weight rows when K fits one round trip, instead of K ranges and their
    // reduce (the DiT head's output and cross-attention projections at batch
    // 1-3: a DiT step at batch 1 1.110 -> 1.054 ms; narrower products such as
    // the SmolVLA-shaped O projection, 720 x 960, measured slower this way)
    if (a.M <= 64 && (a.N >= 1536 || (a.N >= 1024 && a.K <= 1024))) {
      p.kind = 2;
      p.bn = a.N >= 6144 ? 32 : 16;
      p.bm = 64;
      p.ksplit = a.K;
      return p;
    }
    // long-K products with enough 256 x 256 tiles: the large-tile kernel
    // (measured ahead of the staged tiles from K = 2048 on), unless its last
    // round of tiles leaves the chip mostly idle where the 128 x 128 staged
    // tiles fill theirs: per K-step of 64, a round of 256 large tiles (one
    // per CU) measured 2.1 us and a round of 512 staged tiles (two per CU)
    // 1.2 us (e.g. the 2560-wide QKV projection of 6528 rows: 260 large tiles
    // in two rounds, 124 us, against 1020 staged tiles in two rounds, 76 us)
    // The large tiles are 256 activation rows high, or 224 when no more
    // rounds of tiles result: a 224-row tile measured 3-7 % faster than a
    // 256-row one (not the 12.5 % of its area: each K-step's fixed costs
    // dominate), e.g. the pi0-shaped MLP down projection at 6528 rows, 240
    // such tiles in one round, 435 us against 450 us for 208 taller ones. The
    // accumulation order of every output, and so the result, is the same
    // for both heights.
    // Below K = 2048 the large tiles' fixed costs weigh more: they are taken
    // there only for an output stored from registers (reg_epi_ok) and a
    // margin of 10 % (measured: the SmolVLA-shaped vision encoder's MLP up,
    // 49152 x 3072 x 768, 270 -> 240 us; the pi0-shaped ViT MLP up at 6144
    // rows, 73 -> 70 us; half-filled last rounds stay on the staged tiles)
    const long t256 = blocks(256, 256), t224 = blocks(256, 224), t128 = blocks(128, 128);
    const double c256 = (t256 + 255) / 256 * 2.1, c224 = (t224 + 255) / 256 * 2.1 * 0.95;
    const double c_big = std::min(c256, c224), c_staged = (t128 + 511) / 512 * 1.2;
    const bool long_k = a.K >= 2048 && c_big <= c_staged;
    const bool short_k = a.K >= 512 && a.K < 2048 && reg_epi_ok(a) && c_big <= 0.9 * c_staged;
    if (a.M >= 256 && t256 >= 160 && (long_k || short_k)) {
      p.bn = 256; p.bm = c224 < c256 - 1e-9 ? 224 : 256; p.kind = 3;
      p.ksplit = nk * BK;
      return p;
    }
    // a few hundred activation rows (the action stage at batch 2-32, short
    // prefills): K-steps of 128 shared by two wave groups (8 waves). 64 x 64
    // tiles while they fit in one round of two blocks per CU (<= 512 blocks),
    // three stages (96 KiB of LDS, one block per CU) when the blocks fit in
    // kOneRoundCUs; the number of K ranges s from a cost model fitted to
    // measured sweeps: ceil(K-steps / s) x step time (0.48 us at one block per
    // CU, 0.9 us at two) + for s > 1 the reduce (~2.5 us + its fp32 partial
    // traffic at ~5 TB/s, 8 M N s bytes), or for s = 1 the row norm's own
    // kernel when one follows (~4 us). Wider products whose 128 x 128 tiles
    // (135 KiB of LDS) fill 160 to kOneRoundCUs CUs once take those tiles
    // (measured 10-15 % faster than 128 x 64 tiles with K-steps of 64 there).
    // kOneRoundCUs is below the chip's 256 because the action stage shares
    // the GPU with a VLM stage that holds some CUs' LDS: one-block-per-CU
    // launches sized for all 256 CUs ran a second round there.
    // Up to 36 K-steps (K <= 4608), but past 32 only with K ranges: the ViT
    // MLP down (K = 4304) with two ranges at 256-768 rows is faster than on
    // the staged tiles (GR00T-like prefill at batch 1 3.765 -> 3.703 ms, the
    // pi0-shaped one 7.327 -> 7.278 ms), with one range at 1024 rows slower
    // (7.38 -> 7.61 ms at batch 4).
    constexpr long kOneRoundCUs = 192;
    if (a.M <= 1024 && a.K <= 4608 && (a.M > 64 || (a.N < 1536 && a.K >= 2048))) {
      const long t64 = blocks(64, 64);
      const int nk128 = (a.K + 127) / 128;
      double best_t = 1e30;
      int best_s = 0;
      for (int sp = 1; sp <= 8; sp *= 2) {
        if (t64 * sp > 512 || (sp > 1 && (nk128 < 2 * sp || !a.ws || (long)sp * a.M * ldp > a.ws_floats))) continue;
        const int ksteps = (nk128 + sp - 1) / sp;
        double t = ksteps * (t64 * sp <= kOneRoundCUs ? 0.48 : 0.9);
        if (sp > 1) t += 2.5 + 8.0 * a.M * (double)a.N * sp / 5e6;
        else if (a.norm_follows) t += 4.0;
        if (t < best_t) { best_t = t; best_s = sp; }
      }
      if (best_s > 0 && (a.K <= 4096 || best_s > 1)) {
        const int ksteps = (nk128 + best_s - 1) / best_s;
        p.bn = 64; p.bm = 64; p.kind = 4; p.bk = 128; p.kg = 2;
        p.stages = t64 * best_s <= kOneRoundCUs ? 3 : 2;
        p.ksplit = ksteps * 128;
        p.splits = (nk128 + ksteps - 1) / ksteps;
        return p;
      }
      if (a.K <= 4096 && a.M >= 256 && t128 >= 160 && t128 <= kOneRoundCUs) {
        p.bn = 128; p.bm = 128; p.kind = 4; p.bk = 128; p.kg = 2; p.stages = 2;
        p.ksplit = nk128 * 128;
        p.splits = 1;
        return p;
      }
    }
    // many activation rows: the LDS-staged kernel (two stages, two blocks per
    // CU). Tile (128 x 128 or 128 x 64) and K ranges from a cost model fitted
    // to measured sweeps: K ranges until the blocks fill both slots of every
    // CU (>= 8 K-steps per range); time = rounds of resident blocks x K-steps
    // per range x step time (0.87 us for 128 x 128, 0.59 us for 128 x 64)
    // + the ordered reduce (its fp32 partial traffic at ~5 TB/s + 3 us).
    // Also a few hundred rows with K past the two-group kernel's 4096: there
    // the 64 x 32 register tiles, enough of them to skip K ranges, each ran
    // the whole K loop alone (the GR00T-like LLM MLP down at batch 1, 296 x
    // 2048 x 16384: 143 -> 38 us, that prefill 5.89 -> 3.78 ms).
    const bool staged = (a.M >= 64 && blocks(128, 64) >= 128) || (a.M > 64 && nk >= 24 && a.ws);
    // short K and under ~1.25 128 x 64 tiles per CU (the action stage at
    // batch 8-16): 64 x 64 tiles, up to four blocks per CU (measured 15-25 %
    // faster there)
    if (staged && a.M <= 1024 && nk <= 24 && blocks(128, 64) < 320) {
      p.bn = 64; p.bm = 64; p.kind = 1; p.splits = 1; p.ksplit = nk * BK;
      return p;
    }
    if (staged) {
      double best_t = 1e30;
      for (int bm = 128; bm >= 64; bm -= 64) {
        if (bm == 128 && a.M < 128) continue;
        const long tiles = blocks(128, bm);
        int sp = a.ws ? (int)std::max<long>(1, std::min<long>({512 / tiles, nk / 8, 16L})) : 1;
        while (sp > 1 && (long)sp * a.M * ldp > a.ws_floats) --sp;
        const int ksteps = (nk + sp - 1) / sp;
        sp = (nk + ksteps - 1) / ksteps;
        const long rounds = (tiles * sp + 511) / 512;
        double t = rounds * ksteps * (bm == 128 ? 0.87 : 0.59);
        if (sp > 1) t += 4.0 * sp * a.M * ldp / 5e6 + 3.0;
        else if (a.norm_follows) t += 4.0;
        if (t < best_t) {
          best_t = t;
          p.bn = 128; p.bm = bm; p.kind = 1; p.splits = sp; p.ksplit = ksteps * BK;
        }
      }
      return p;
    }
  }
  // otherwise the register-pipelined kernel: 128-row tiles only for large
  // products, else 64 x 32 tiles (measured best up to a few hundred rows);
  // split K when the tiles leave the CUs short of work, keeping >= 3 K steps
  // per range
  if (a.M >= 128 && blocks(128, 128) >= 256) p.bn = 128, p.bm = 128;
  p.ksplit = nk * BK;
  const long tiles = blocks(p.bn, p.bm);
  if (a.ws && tiles < 256 && nk >= 6) set_splits((int)std::min<long>((256 + tiles - 1) / tiles, nk / 3));
  return p;
}

// A product with a folded RMSNorm needs each row's whole K in one block: the
// plan without K ranges, on a kernel that sums the squares (LDS-staged or
// small-M).
GemmPlan gemm_plan(const GemmArgs& a) {
  if (!a.rms_in || a.w_type != ET_BF16) return plan_base(a);
  GemmArgs b = a;
  b.ws = nullptr;
  b.ws_floats = 0;
  GemmPlan p = plan_base(b);
  if (p.kind == 1 || p.kind == 2 || p.kind == 4) return p;
  const bool big = a.M >= 128 && (long)((a.M + 127) / 128) * ((a.N + 127) / 128) >= 128;
  return GemmPlan{big ? 128 : 64, big ? 128 : 64, 1, (a.K + 63) / 64 * 64, 1};
}


// The residual update from registers (reg_resid, the two-group staged tiles)
// needs the vector epilogue's alignment (epi_vec), fp32 output, and a product
// input that does not overlap the output rows (their old values are read
// before the K loop).
static bool reg_res_ok(const GemmArgs& a) {
  if (a.mode != EPI_RESID || !a.epi_vec || a.out_type != ET_F32 || a.rms_in || a.M <= 0) return false;
  const size_t esz = a.a_type == ET_BF16 ? 2 : 4;
  const char* ab = reinterpret_cast<const char*>(a.A);
  const char* ae = ab + ((size_t)(a.M - 1) * a.lda + a.K) * esz;
  const long last = a.row_group > 0 ? (long)((a.M - 1) / a.row_group) * a.row_group_stride + (long)(a.row_group - 1) * a.ldo
                                     : (long)(a.M - 1) * a.ldo;
  const char* ob = reinterpret_cast<const char*>(a.out);
  const char* oe = ob + ((size_t)last + a.N) * 4;
  return ae <= ob || oe <= ab;
}

// The fused reduce with a row norm over rows of N <= 256 * NV columns: the
// waves per row of the norm kernel's rule (rownorm::waves_per_row), 256-thread
// blocks of 4 / WPR rows.
template <int NV>
static void launch_reduce_norm(const GemmArgs& a, const NormArgs& n, hipStream_t s) {
  constexpr int W = NV >= 4 ? 4 : NV;
  if (rownorm::waves_per_row(NV, a.M) == 1) {
    hipLaunchKernelGGL((splitk_reduce_norm_kernel<NV, 1>), dim3((a.M + 3) / 4), dim3(256), 0, s, a, n);
  } else {
    hipLaunchKernelGGL((splitk_reduce_norm_kernel<NV / W, W>), dim3((a.M + 4 / W - 1) / (4 / W)), dim3(256), 0, s, a, n);
  }
}

// Second pass of a split product: the ordered reduce with the epilogue, or
// for a residual projection with a following row norm, the fused reduce.
template <int MODE>
static void launch_reduce(const GemmArgs& a, const NormArgs* fuse, hipStream_t s) {
  if constexpr (MODE == EPI_RESID) {
    if (fuse) {
      if (a.N <= 256) launch_reduce_norm<1>(a, *fuse, s);
      else if (a.N <= 512) launch_reduce_norm<2>(a, *fuse, s);
      else if (a.N <= 1024) launch_reduce_norm<4>(a, *fuse, s);
      else launch_reduce_norm<8>(a, *fuse, s);
      return;
    }
  }
  const long chunks = (long)a.M * (((a.N + 3) & ~3) / 4);
  hipLaunchKernelGGL(splitk_reduce_kernel<MODE>, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, s, a);
}

template <int BN, int BM, int MODE>
static void launch_staged(const GemmArgs& a0, const GemmPlan& p, const NormArgs* fuse, hipStream_t s) {
  GemmArgs a = a0;
  a.epi_reg = 0;
  a.ksplit = p.ksplit;
  a.splits = p.splits;
  dim3 grid((a.M + BM - 1) / BM, (a.N + BN - 1) / BN, a.splits);
  if (a.splits > 1) {
    // partial pass without epilogue, then the ordered reduce applies it
    hipLaunchKernelGGL((gemm_stage_kernel<BN, BM, 2, EPI_STORE>), grid, dim3(256), 0, s, a);
    launch_reduce<MODE>(a, fuse, s);
    return;
  }
  a.epi_reg = BN == 128 && reg_epi_ok(a) ? 1 : 0;
  if constexpr (MODE == EPI_STORE || MODE == EPI_QKV || MODE == EPI_GEGLU || MODE == EPI_EULER) {
    if (a.rms_in) {
      hipLaunchKernelGGL((gemm_stage_kernel<BN, BM, 2, MODE, 64, 1, 1>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_stage_kernel<BN, BM, 2, MODE>), grid, dim3(256), 0, s, a);
}

template <int BT, int ST, int MODE>
static void launch_staged128(const GemmArgs& a0, const GemmPlan& p, const NormArgs* fuse, hipStream_t s) {
  GemmArgs a = a0;
  a.epi_reg = 0;
  a.ksplit = p.ksplit;
  a.splits = p.splits;
  dim3 grid((a.M + BT - 1) / BT, (a.N + BT - 1) / BT, a.splits);
  if (a.splits > 1) {
    hipLaunchKernelGGL((gemm_stage_kernel<BT, BT, ST, EPI_STORE, 128, 2>), grid, dim3(512), 0, s, a);
    launch_reduce<MODE>(a, fuse, s);
    return;
  }
  a.epi_reg = reg_res_ok(a) ? 1 : 0;
  if constexpr (MODE == EPI_STORE || MODE == EPI_QKV || MODE == EPI_GEGLU || MODE == EPI_EULER) {
    if (a.rms_in) {
      hipLaunchKernelGGL((gemm_stage_kernel<BT, BT, ST, MODE, 128, 2, 1>), grid, dim3(512), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_stage_kernel<BT, BT, ST, MODE, 128, 2>), grid, dim3(512), 0, s, a);
}


template <int MODE, int NW = 8>
static void launch_big(const GemmArgs& a, int bm, hipStream_t s) {
  if constexpr ((MODE == EPI_GEGLU || MODE == EPI_STORE) && NW == 8) {
    if (reg_epi_ok(a)) {
      dim3 grid((a.M + bm - 1) / bm, (a.N + 255) / 256, 1);
      if (bm == 224) hipLaunchKernelGGL((gemm_big_kernel<MODE, NW, 224, true>), grid, dim3(NW * 64), 0, s, a);
      else hipLaunchKernelGGL((gemm_big_kernel<MODE, NW, 256, true>), grid, dim3(NW * 64), 0, s, a);
      return;
    }
  }
  if (bm == 224) {
    dim3 grid((a.M + 223) / 224, (a.N + 255) / 256, 1);
    hipLaunchKernelGGL((gemm_big_kernel<MODE, NW, 224>), grid, dim3(NW * 64), 0, s, a);
    return;
  }
  dim3 grid((a.M + 255) / 256, (a.N + 255) / 256, 1);
  hipLaunchKernelGGL((gemm_big_kernel<MODE, NW, 256>), grid, dim3(NW * 64), 0, s, a);
}

template <int TN, int MODE>
static void launch_skinny(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.M + 63) / 64, (a.N + 16 * TN - 1) / (16 * TN), 1);
  if constexpr (MODE == EPI_STORE || MODE == EPI_QKV || MODE == EPI_GEGLU || MODE == EPI_EULER) {
    if (a.rms_in) {
      hipLaunchKernelGGL((gemm_skinny_kernel<TN, MODE, 1>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_skinny_kernel<TN, MODE>), grid, dim3(256), 0, s, a);
}

template <int BN, int BM, int MODE>
static void launch_mfma(const GemmArgs& a0, const GemmPlan& p, const NormArgs* fuse, hipStream_t s) {
  GemmArgs a = a0;
  a.ksplit = p.ksplit;
  a.splits = p.splits;
  dim3 grid((a.M + BM - 1) / BM, (a.N + BN - 1) / BN, a.splits);
  bool f32a = false;
  if constexpr (MODE == EPI_STORE) f32a = a.a_type == ET_F32;
  if (a.splits > 1) {
    // the partial pass does not use the epilogue: one instantiation serves all modes
    if (f32a) hipLaunchKernelGGL((gemm_mfma_kernel<BN, BM, float, EPI_STORE>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((gemm_mfma_kernel<BN, BM, bf16, EPI_STORE>), grid, dim3(256), 0, s, a);
    launch_reduce<MODE>(a, fuse, s);
    return;
  }
  if constexpr (MODE == EPI_STORE) {
    if (f32a) {
      hipLaunchKernelGGL((gemm_mfma_kernel<BN, BM, float, MODE>), grid, dim3(256), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((gemm_mfma_kernel<BN, BM, bf16, MODE>), grid, dim3(256), 0, s, a);
}

// fuse: a row norm of the output to run inside the split-K reduce (only
// passed when the plan splits K and the product is a residual projection)
template <int MODE>
static void launch_mode(const GemmArgs& a, const GemmPlan& p, const NormArgs* fuse, hipStream_t s) {
  if (a.w_type == ET_F32) {
    dim3 grid((a.M + 63) / 64, (a.N + 63) / 64);
    hipLaunchKernelGGL(gemm_f32_kernel<MODE>, grid, dim3(256), 0, s, a);
    return;
  }
  if (p.kind == 3) {
    launch_big<MODE>(a, p.bm, s);
    return;
  }
  if (p.kind == 4) {
    if (p.bn == 128) launch_staged128<128, 2, MODE>(a, p, fuse, s);
    else if (p.stages == 3) launch_staged128<64, 3, MODE>(a, p, fuse, s);
    else launch_staged128<64, 2, MODE>(a, p, fuse, s);
    return;
  }
  if (p.kind == 2) {
    if (p.bn == 32) launch_skinny<2, MODE>(a, s);
    else launch_skinny<1, MODE>(a, s);
    return;
  }
  if (p.kind == 1) {
    if (p.bm == 128) launch_staged<128, 128, MODE>(a, p, fuse, s);
    else if (p.bn == 64) launch_staged<64, 64, MODE>(a, p, fuse, s);
    else launch_staged<128, 64, MODE>(a, p, fuse, s);
    return;
  }
  if (p.bn == 128) launch_mfma<128, 128, MODE>(a, p, fuse, s);
  else launch_mfma<64, 32, MODE>(a, p, fuse, s);
}

// True when the tile epilogue may use one vector access per four columns:
// N a multiple of 4 and every base address and stride it touches aligned.
static bool epi_vec_ok(const GemmArgs& a) {
  auto al = [](const void* p, uintptr_t b) { return (reinterpret_cast<uintptr_t>(p) & (b - 1)) == 0; };
  if (a.N % 4 != 0) return false;
  if (a.bias && !al(a.bias, 16)) return false;
  switch (a.mode) {
    case EPI_STORE:
      if (a.tab && (!al(a.tab, 16) || a.ldtab % 4 != 0 || a.tab_period <= 0)) return false;
      if (a.out2 && (!al(a.out2, 8) || a.ldo2 % 4 != 0)) return false;
      return al(a.out, 16) && a.ldo % 4 == 0 && (a.row_group <= 0 || a.row_group_stride % 4 == 0);
    case EPI_RESID:
      if (a.gate && !al(a.gate, 16)) return false;
      if (a.out2 && (!al(a.out2, 8) || a.ldo2 % 4 != 0)) return false;
      return al(a.out, 16) && a.ldo % 4 == 0 && (a.row_group <= 0 || a.row_group_stride % 4 == 0);
    case EPI_EULER:
      return al(a.out, 16) && a.ldo % 4 == 0;
    case EPI_GEGLU:
      return al(a.out, 8) && a.ldo % 2 == 0;
    case EPI_QKV: {
      const QkvEpi& q = a.qkv;
      const bool strides = q.q_sb % 4 == 0 && q.q_sh % 4 == 0 && q.q_si % 4 == 0 && q.k_sb % 4 == 0 &&
                           q.k_sh % 4 == 0 && q.k_si % 4 == 0 && q.v_sb % 4 == 0 && q.v_sh % 4 == 0 && q.v_si % 4 == 0;
      return strides && q.hd % 4 == 0 && q.n_off % 4 == 0 && q.seq > 0 && al(q.q, 16) && al(q.k, 16) && al(q.v, 16) &&
             (q.pos0 < 0 || al(q.rope_cs, 16));
    }
  }
  return false;
}

void launch_gemm(const GemmArgs& a0, hipStream_t s) {
  if (a0.M <= 0 || a0.N <= 0) return;
  if (a0.a_type == ET_F32 && a0.w_type == ET_BF16 && a0.mode != EPI_STORE)
    throw VlaError{4, "fp32 activations with bf16 weights only feed plain stores"};
  if (a0.rms_in && (a0.rms_in < 0 || a0.a_type != ET_BF16 || a0.w_type != ET_BF16 || !a0.zeros ||
                    (a0.mode != EPI_STORE && a0.mode != EPI_QKV && a0.mode != EPI_GEGLU && a0.mode != EPI_EULER)))
    throw VlaError{4, "a folded RMSNorm needs bf16 operands and a store, QKV, GeGLU or Euler epilogue"};
  if (a0.out2 && (a0.row_group > 0 || a0.ldo2 < a0.N || a0.out_type != ET_F32 ||
                  (a0.mode != EPI_STORE && a0.mode != EPI_RESID)))
    throw VlaError{4, "a bf16 copy needs an fp32 store or residual epilogue without row groups"};
  GemmArgs a = a0;
  a.epi_vec = epi_vec_ok(a) ? 1 : 0;
  const GemmPlan p = a.w_type == ET_F32 ? GemmPlan{} : gemm_plan(a);
  switch (a.mode) {
    case EPI_STORE: launch_mode<EPI_STORE>(a, p, nullptr, s); break;
    case EPI_RESID: launch_mode<EPI_RESID>(a, p, nullptr, s); break;
    case EPI_GEGLU: launch_mode<EPI_GEGLU>(a, p, nullptr, s); break;
    case EPI_QKV: launch_mode<EPI_QKV>(a, p, nullptr, s); break;
    case EPI_EULER: launch_mode<EPI_EULER>(a, p, nullptr, s); break;
  }
}

void launch_gemm_norm(const GemmArgs& a, const NormArgs& n, hipStream_t s) {
  const bool fusable = a.M > 0 && a.N > 0 && a.mode == EPI_RESID && a.w_type == ET_BF16 && a.row_group == 0 && !a.out2 &&
                       n.skip == 0 && n.rows == a.M && n.d == a.N && n.in == a.out && n.ld_in == a.ldo &&
                       a.N % 4 == 0 && a.ldo % 4 == 0 && n.ld_out % 4 == 0 && a.N <= 2048;
  if (fusable) {
    GemmArgs av = a;
    av.norm_follows = 1;
    av.epi_vec = epi_vec_ok(av) ? 1 : 0;
    const GemmPlan p = gemm_plan(av);
    launch_mode<EPI_RESID>(av, p, p.splits > 1 ? &n : nullptr, s);
    if (p.splits == 1) launch_norm(n, s);
    return;
  }
  launch_gemm(a, s);
  launch_norm(n, s);
}
