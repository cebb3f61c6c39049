/*
 * vla_debug.h - test hooks of libvla.so: single kernels behind the C ABI, for
 * per-kernel parity tests and for checking where CU-masked streams place
 * work. Same conventions as vla.h (asynchronous, status + vla_last_error).
 */
#ifndef VLA_DEBUG_H
#define VLA_DEBUG_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "vla.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * out[m][n] = act(sum_k A[m][k] * Wt[n][k] + bias[n]) for m < M, n < N, fp32
 * out (leading dimension ldo). This is the projection kernel every dense
 * layer of both stages uses (the layers are plain matrix products).
 *  A   device [M][lda], a_type 0 = fp32, 1 = bf16 (fp32 A is rounded to bf16
 *      on load when the weight is bf16).
 *  Wt  device [N][ldw] weight, transposed (K contiguous), w_type 0/1.
 *  bias device fp32 [N] or NULL. act: 0 none, 1 SiLU, 2 tanh-GELU.
 * bf16 weights need K, lda, ldw multiples of 8; fp32 weights need fp32 A.
 */
vla_status vla_debug_gemm(int M, int N, int K, const void* A, int lda, int a_type, const void* Wt, int ldw,
                          int w_type, const float* bias, int act, float* out, int ldo, hipStream_t stream);

/*
 * Projection with bf16 output, as the model's bf16 layers run it:
 *  glu = 0: out[m][n] = act(D[m][n] + bias[n])  (act: 0 none, 1 SiLU,
 *           2 tanh-GELU), out [M][ldo] with ldo >= N;
 *  glu = 1: the gated-GELU MLP projection (the gate/up of the LLM and of the
 *           joint action expert, Section 2.1's VLM and action stages): weight
 *           rows interleaved, row 2f the gate and row 2f + 1 the up projection
 *           of feature f, out[m][f] = gelu(D[m][2f] + bias[2f]) *
 *           (D[m][2f + 1] + bias[2f + 1]), out [M][ldo] with ldo >= N / 2,
 *           N even, act 0;
 *  D = A Wt^T, or with rms = 1 D[m][n] = sum_k A[m][k] Wt[n][k] /
 *  sqrt(mean_k A[m][k]^2 + eps) (the RMSNorm of the input rows folded into
 *  the product, as the bf16 action experts run it; K >= 8).
 *  A device bf16 [M][lda]; Wt device bf16 [N][ldw] (K contiguous); bias
 *  device fp32 [N] or NULL. K, lda, ldw multiples of 8.
 * The same plan and kernels as a model projection of that shape: the
 * large-tile and 128-column staged kernels store from registers when N % 16
 * == 0, ldo % 8 == 0 and out and bias are 16-byte aligned, through LDS
 * otherwise (same results).
 */
vla_status vla_debug_gemm_bf16(int M, int N, int K, const void* A, int lda, const void* Wt, int ldw, const float* bias,
                               int glu, int act, int rms, float eps, void* out, int ldo, hipStream_t stream);

/*
 * vla_debug_gemm without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, hosts
 * that forbid allocation). Same arguments, kernels, K ranges and results as
 * vla_debug_gemm; its split-K partials and its zero block live in a static
 * device array of 16 MiB + 256 bytes that every device the library runs on
 * holds until the process ends. Returns VLA_EINVAL, enqueuing nothing, when
 * the projection's K-split plan needs more than 16 MiB of partials
 * (splits x M x round_up(N, 4) x 4 bytes; a plan without a K split needs
 * none). Calls on one device share that array: calls that overlap on one
 * device (different streams, or host threads) race and must be serialised
 * by the caller. Each call first rewrites the zero block on `stream`.
 */
vla_status vla_gemm_noalloc(int M, int N, int K, const void* A, int lda, int a_type, const void* Wt, int ldw,
                            int w_type, const float* bias, int act, float* out, int ldo, hipStream_t stream);

/*
 * Residual projection followed by the row norm of its output (every
 * transformer block: x += o W_o, then the next sublayer's norm):
 *   x[m][n] += gate[n] * (sum_k A[m][k] Wt[n][k] + bias[n])   (x in place)
 *   z[m][:] = norm(x[m][:])  kind 0: RMSNorm * g; 1: LayerNorm * g + b
 *                             (g, b optional); 2: LayerNorm * (1 + g) + b
 * A bf16 [M][K], Wt bf16 [N][K], bias/gate fp32 [N] or NULL, x fp32 [M][N],
 * z bf16 [M][N]. K % 8 == 0, N % 4 == 0, N <= 2048. When the projection is
 * split over K the norm runs inside the split reduce.
 */
vla_status vla_debug_resid_norm(int M, int N, int K, const void* A, const void* Wt, const float* bias, const float* gate,
                                float* x, int kind, const float* g, const float* b, float eps, void* z,
                                hipStream_t stream);

/*
 * Projection with the RMSNorm of its input rows folded in (the action
 * expert's QKV and MLP up projections read rows not yet normalised, with the
 * norm's gain folded into the weight columns):
 *   out[m][n] = rsqrt(sum_k A[m][k]^2 / K + eps) * sum_k A[m][k] Wt[n][k] + bias[n]
 * A bf16 [M][K], Wt bf16 [N][K], bias fp32 [N] or NULL, out fp32 [M][N].
 * K % 8 == 0. The sum of squares is taken from the bf16 A the product reads.
 */
vla_status vla_debug_gemm_rms(int M, int N, int K, const void* A, const void* Wt, const float* bias, float eps,
                              float* out, hipStream_t stream);

/*
 * Residual projection that also writes a bf16 copy of the updated rows (the
 * input of a projection with a folded RMSNorm):
 *   x[m][n] += gate[n] * (sum_k A[m][k] Wt[n][k] + bias[n]);  xb[m][n] = bf16(x[m][n])
 * A bf16 [M][K], Wt bf16 [N][K], bias/gate fp32 [N] or NULL, x fp32 [M][ldx]
 * (ldx >= N), xb bf16 [M][ldxb] (ldxb >= N). K % 8 == 0. Rows or strides
 * that are not 16-byte aligned take the per-element epilogue (same results).
 */
vla_status vla_debug_resid_copy(int M, int N, int K, const void* A, const void* Wt, const float* bias,
                                const float* gate, float* x, int ldx, void* xb, int ldxb, hipStream_t stream);

/*
 * o = softmax(q k^T / sqrt(hd)) v over the keys [k0 ; k1] (segment 1 may be
 * empty), grouped KV heads (query head h uses KV head h / (Hq / Hkv)).
 *  q  device [B][Hq][Lq][hd]; k0, v0 [B][Hkv][len0][hd]; k1, v1 [B][Hkv][len1][hd];
 *  o  device [B][Lq][Hq * hd]. et 0 = fp32, 1 = bf16 for every tensor.
 * hd a multiple of 8 up to 256; len0 >= 1.
 */
vla_status vla_debug_attention(int B, int Hq, int Hkv, int Lq, int hd, int et, const void* q, const void* k0,
                               const void* v0, int len0, const void* k1, const void* v1, int len1, void* o,
                               hipStream_t stream);

/*
 * Launch `blocks` one-wave workgroups on the pool stream restricted to
 * `cu_count` compute units (the VLM-side mask of vla_step, or the action-side
 * mask counted from the top when from_top != 0). Each workgroup sleeps
 * `spin` x 64 cycles-ish and writes out[2*i] = HW_ID, out[2*i+1] = XCC_ID
 * hardware register words. out: device uint32 [2 * blocks]. The join stream
 * waits for the probe. via_graph != 0: the launch is captured into a graph on
 * an unrestricted stream and the graph replayed on the restricted stream (as
 * vla_step replays the stages); the call then waits for the replay.
 */
vla_status vla_debug_cu_probe(int device, int cu_count, int from_top, int blocks, int spin, int via_graph,
                              uint32_t* out, hipStream_t join);

/*
 * Cost of handing data between workgroups on different XCDs: the kernel
 * boundary against a grid-wide barrier inside one kernel. kind 0: enqueue
 * `iters` launches of an empty kernel of `grid` 256-thread blocks; kind 1:
 * `iters` launches in which every block writes `words` floats of its slice of
 * buf; kind 2: one launch that runs `iters` grid barriers, each after the
 * blocks write their slices and followed by every block reading another
 * block's slice (release add / acquire polls of *ctr at agent scope). For
 * timing with events around the call (or around a graph that captured it).
 *  buf  device fp32 [2 * grid * words] (kind 2 alternates halves by round;
 *       kinds 0 and 1 use the first half; may be NULL when words == 0).
 *  ctr  device uint32, zero before a kind-2 call; ends at iters * grid.
 *  err  device int32: kind 2 adds the number of polls that passed spin_limit
 *       (the block then went on without the barrier; 0 on a correct run).
 *  sink device fp32 [grid * 256] (the reads' sums, so they are not elided).
 * grid <= 256 so that every block of the barrier kernel is resident at once on
 * an otherwise idle GPU; iters <= 1000, words <= 16384, spin_limit in
 * [1, 1e6] (polls ~64 cycles apart). Status 1 on bad arguments.
 */
vla_status vla_debug_sync_probe(int kind, int grid, int iters, int words, int spin_limit, float* buf, unsigned* ctr,
                                int* err, float* sink, hipStream_t stream);

/*
 * The launch plan of a bf16 projection (bf16 activations and weights, rows of
 * lengths K, the split-K workspace of a model's stage), as the model's
 * projections and vla_debug_gemm_bf16 choose it. Host only: no device is
 * touched, so it also answers on a machine without a GPU.
 *  mode: 0 store, 1 residual, 2 GeGLU (N even; the output has N / 2
 *  columns), 3 QKV, 4 Euler; out_bf16: bf16 rather than fp32 output;
 *  rms != 0: the RMSNorm of the input rows folded in (not with mode 1);
 *  norm_follows != 0: a row norm of the output follows (residual projections).
 *  plan: int[8] = weight rows and activation rows per tile, number of K
 *  ranges, K length per range, kernel kind (0 register-pipelined, 1
 *  LDS-staged, 2 small-M, 3 large-tile, 4 LDS-staged with K-steps of 128),
 *  LDS stages, K-step length, wave groups sharing each K-step.
 * Status 1 (VLA_EINVAL) on bad arguments.
 */
vla_status vla_debug_gemm_plan(int M, int N, int K, int mode, int out_bf16, int rms, int norm_follows, int* plan);

/*
 * Enqueue `iters` launches of one projection of a model's stage, exactly as
 * the stage launches it (same kernel, shape, epilogue, parameters and
 * workspace buffers), on `stream`, and store the algorithmic flops of one
 * launch (2 M N K) in *flops (may be NULL). For timing one kernel with events
 * around the loop. It overwrites the stage's workspace: do not overlap it
 * with that model's stages. which: 0 VLM LLM MLP gate/up (GeGLU), 1 VLM LLM
 * MLP down, 2 action-stage MLP up, 3 action-stage MLP down, 4 ViT MLP up;
 * launch i uses layer (i mod layer count)'s weights, so, as in a pass over
 * the stage, each launch reads weights the previous launches did not.
 * plan (may be NULL): int[9] set to
 * the kernel's tile (weight rows, activation rows), number of K ranges
 * (1 = one kernel, > 1 = partial + reduce kernels), epilogue mode, kernel
 * kind (0 register-pipelined, 1 LDS-staged, 2 small-M, 3 large-tile,
 * 4 LDS-staged with K-steps of 128), LDS stages, K-step length, the
 * number of 4-wave groups that share each K-step, and 1 when the
 * projection normalises its input rows (folded RMSNorm), else 0.
 */
vla_status vla_debug_replay_gemm(vla_model m, int which, int batch, int iters, hipStream_t stream, double* flops,
                                 int* plan);

#ifdef __cplusplus
}
#endif
#endif /* VLA_DEBUG_H */
