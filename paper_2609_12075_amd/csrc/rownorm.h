// Row normalisation shared by the norm kernel and the fused split-K reduce
// (device code; one wavefront holds one row). Lane l holds columns
// (j * 64 + l) * 4 .. + 3 of the row in v[j]; columns >= d hold zeros.
#pragma once
#include "common.h"

namespace rownorm {

typedef __attribute__((ext_vector_type(4))) float f4;
typedef __attribute__((ext_vector_type(4))) __bf16 b4;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// The norm's per-column parameters for this lane's columns: g (gain or
// adaLN scale, 1 when absent) and b (bias or adaLN shift, 0 when absent).
// Loaded together with the row itself, so both share one memory round trip.
template <int NV>
__device__ __forceinline__ void load_params(const NormArgs& a, int lane, f4 (&g)[NV], f4 (&b)[NV]) {
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (j * 64 + lane) * 4;
    const bool ok = i < a.d;
    g[j] = (ok && a.g) ? *reinterpret_cast<const f4*>(a.g + i) : f4{a.kind == 2 ? 0.f : 1.f, a.kind == 2 ? 0.f : 1.f,
                                                                    a.kind == 2 ? 0.f : 1.f, a.kind == 2 ? 0.f : 1.f};
    b[j] = (ok && a.b) ? *reinterpret_cast<const f4*>(a.b + i) : f4{0.f, 0.f, 0.f, 0.f};
  }
}

// Statistics of the row (two passes over registers: mean for the LayerNorm
// kinds, then the centred second moment), then output row r of a:
// kind 0 RMSNorm * g; kind 1 LayerNorm * g + b (each optional);
// kind 2 LayerNorm * (1 + g) + b (adaLN modulation: g = scale, b = shift).
template <int NV>
__device__ __forceinline__ void store_row(const NormArgs& a, int r, const f4 (&v)[NV], int lane, const f4 (&g)[NV],
                                          const f4 (&b)[NV]) {
  const int d = a.d;
  float mean = 0.f;
  if (a.kind != 0) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NV; ++j) s += (v[j][0] + v[j][1]) + (v[j][2] + v[j][3]);
    mean = wave_sum(s) / d;
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (j * 64 + lane) * 4;
    if (i < d)
#pragma unroll
      for (int e = 0; e < 4; ++e) { const float t = v[j][e] - mean; ss = fmaf(t, t, ss); }
  }
  const float rstd = rsqrtf(wave_sum(ss) / d + a.eps);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = (j * 64 + lane) * 4;
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

}  // namespace rownorm
