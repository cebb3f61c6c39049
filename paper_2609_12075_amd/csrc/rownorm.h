// Row normalisation shared by the norm kernel and the fused split-K reduce
// (device code). A row is held in registers by WPR wavefronts of one block
// (WPR = 1, 2 or 4; a 256-thread block holds 4 / WPR rows): lane l of the
// row's wave w holds columns col(w, j, l) .. + 3 in v[j], j < NVW; columns
// >= d hold zeros. Several waves per row keep more loads in flight than one
// wave per row would at a few thousand rows (the statistics then meet in
// LDS, in wave order).
#pragma once
#include "common.h"

namespace rownorm {

typedef __attribute__((ext_vector_type(4))) float f4;
typedef __attribute__((ext_vector_type(4))) __bf16 b4;

template <int NVW>
__device__ __forceinline__ int col(int w, int j, int lane) { return ((w * NVW + j) * 64 + lane) * 4; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// The row total of one statistic: each wave's sum, then (WPR > 1) the row's
// waves' sums added in wave order through red (one word per wave of the
// block and statistic). Every thread of the block calls it (it may hold a
// barrier).
template <int WPR>
__device__ __forceinline__ float row_total(float s, float (*red)[2], int stat, int wv, int w) {
  s = wave_sum(s);
  if constexpr (WPR == 1) {
    return s;
  } else {
    if ((threadIdx.x & 63) == 0) red[wv][stat] = s;
    __syncthreads();
    const int base = wv - w;
    float t = red[base][stat];
#pragma unroll
    for (int q = 1; q < WPR; ++q) t += red[base + q][stat];
    return t;
  }
}

// The norm's per-column parameters for this lane's columns: g (gain or
// adaLN scale, 1 when absent) and b (bias or adaLN shift, 0 when absent).
// Loaded together with the row itself, so both share one memory round trip.
template <int NVW>
__device__ __forceinline__ void load_params(const NormArgs& a, int w, int lane, f4 (&g)[NVW], f4 (&b)[NVW]) {
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = col<NVW>(w, j, lane);
    const bool ok = i < a.d;
    g[j] = (ok && a.g) ? *reinterpret_cast<const f4*>(a.g + i) : f4{a.kind == 2 ? 0.f : 1.f, a.kind == 2 ? 0.f : 1.f,
                                                                    a.kind == 2 ? 0.f : 1.f, a.kind == 2 ? 0.f : 1.f};
    b[j] = (ok && a.b) ? *reinterpret_cast<const f4*>(a.b + i) : f4{0.f, 0.f, 0.f, 0.f};
  }
}

// Statistics of the row (two passes over registers: mean for the LayerNorm
// kinds, then the centred second moment), then output row r of a (only when
// store is set; every thread of the block calls this):
// kind 0 RMSNorm * g; kind 1 LayerNorm * g + b (each optional);
// kind 2 LayerNorm * (1 + g) + b (adaLN modulation: g = scale, b = shift).
template <int NVW, int WPR>
__device__ __forceinline__ void store_row(const NormArgs& a, int r, bool store, const f4 (&v)[NVW], int wv, int w,
                                          int lane, const f4 (&g)[NVW], const f4 (&b)[NVW], float (*red)[2]) {
  const int d = a.d;
  float mean = 0.f;
  if (a.kind != 0) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NVW; ++j) s += (v[j][0] + v[j][1]) + (v[j][2] + v[j][3]);
    mean = row_total<WPR>(s, red, 0, wv, w) / d;
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = col<NVW>(w, j, lane);
    if (i < d)
#pragma unroll
      for (int e = 0; e < 4; ++e) { const float t = v[j][e] - mean; ss = fmaf(t, t, ss); }
  }
  const float rstd = rsqrtf(row_total<WPR>(ss, red, 1, wv, w) / d + a.eps);
  if (!store) return;
#pragma unroll
  for (int j = 0; j < NVW; ++j) {
    const int i = col<NVW>(w, j, lane);
    if (i >= d) continue;
    f4 y;
#pragma unroll
    for (int e = 0; e < 4; ++e) y[e] = (v[j][e] - mean) * rstd;
    if (a.kind == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e) y[e] = y[e] * (1.0f + g[j][e]) + b[j][e];
    } else {
      if (a.g) y *= g[j];
      if (a.b) y += b[j];
    }
    if (a.out_type == ET_BF16) {
      *reinterpret_cast<b4*>(reinterpret_cast<bf16*>(a.out) + (long)r * a.ld_out + i) =
          b4{(bf16)y[0], (bf16)y[1], (bf16)y[2], (bf16)y[3]};
    } else {
      *reinterpret_cast<f4*>(reinterpret_cast<float*>(a.out) + (long)r * a.ld_out + i) = y;
    }
  }
}

// Waves per row for a norm over `rows` rows of d <= 256 * nv columns: one
// for d <= 256 or for many rows (>= 8192, where one wave per row already
// keeps enough loads in flight and the LDS exchange only costs: 1-2 % slower
// measured at 12288 rows), else up to four. The norm kernel and the fused
// reduce use the same rule, so both give the same bits for the same rows.
__host__ __device__ inline int waves_per_row(int nv, int rows) { return nv == 1 || rows >= 8192 ? 1 : (nv >= 4 ? 4 : nv); }

}  // namespace rownorm
