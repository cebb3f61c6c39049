/*
 * vla.h - C ABI of libvla.so: one batched VLA inference step on an MI355X.
 *
 * The paper's VLA models run in two stages (Section 2.1, Fig. 1): a VLM stage
 * encodes the robot's camera frames and its instruction text and hands the
 * action model either hidden states or a compact per-layer KV cache, and an
 * action diffusion transformer (ADiT) denoises for a set number of steps into
 * a chunk of actions. The
 * serving engine (Section 4.1) runs the two stages as separate fixed-size
 * batches on two GPU streams, one lockstep at a time, restricting the compute
 * units the VLM stream may occupy (Section 4.1.2) and ordering requests by
 * least remaining time to their SLO (Section 4.1.3).
 *
 * Conventions for every call:
 *  - Device buffers (pixels, text ids, noise, state, kv, actions) are owned by
 *    the caller and must stay alive until the work enqueued on the given
 *    stream has finished. The library owns the model's device parameters,
 *    its workspaces and its captured graphs.
 *  - Compute calls are asynchronous: they validate their arguments, enqueue
 *    work on the stream and return. On any error nothing is enqueued, the
 *    call returns a non-zero vla_status and vla_last_error() describes it.
 *    The library never aborts the process.
 *  - Results are deterministic: identical inputs give bit-identical outputs
 *    (no atomics in any reduction). Batch rows are independent: row r of
 *    every output depends only on row r of the inputs.
 *  - A model's prefill calls must be ordered among themselves (one stream, or
 *    externally synchronised), and so must its denoise calls: each stage has
 *    one workspace. A prefill and a denoise of the same model may overlap.
 *  - Numeric policy for VLA_BF16 models: parameters are rounded to bf16
 *    (round to nearest even) at creation; activations that feed matrix
 *    products are bf16; accumulation, norm statistics, softmax, RoPE angles,
 *    the residual streams and the Euler state are fp32; the prefix KV is bf16.
 *    VLA_F32 models compute in fp32 throughout.
 */
#ifndef VLA_H
#define VLA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>   /* hipStream_t */

#ifdef __cplusplus
extern "C" {
#endif

typedef struct vla_model_s* vla_model;       /* opaque, owned by the library */

typedef enum {
  VLA_OK = 0,
  VLA_EINVAL = 1,        /* bad argument: nothing was enqueued */
  VLA_ENOMEM = 2,        /* device or host allocation failed */
  VLA_EHIP = 3,          /* a HIP runtime call failed */
  VLA_EUNSUPPORTED = 4   /* valid request the library does not implement */
} vla_status;

enum { VLA_F32 = 0, VLA_BF16 = 1 };
enum { VLA_HEAD_JOINT = 0, VLA_HEAD_DIT = 1 };

/*
 * Model shape. Readings of the two-stage structure (Section 2.1):
 *  - vision: n_img images of 3 x img_hw x img_hw fp32 pixels, cut into
 *    patch x patch patches in raster order, each flattened (channel, row,
 *    column); a patch embedding (+ bias + learned position table shared by the
 *    images), then vit_layers pre-LN ViT blocks of width vit_d with vit_heads
 *    heads and a tanh-GELU MLP of vit_mlp, a final LayerNorm and a projection
 *    to llm_d. With vit_layers == 0 the patch embedding maps to llm_d directly.
 *  - text: n_text ids < vocab, embedded by table lookup.
 *  - LLM: llm_layers Gemma-style blocks (RMSNorm, grouped-query attention
 *    with n_q query and n_kv key/value heads of head_dim, half-split RoPE with
 *    rope_base, bidirectional over the prefix; GeGLU MLP of llm_mlp).
 *  - head_kind VLA_HEAD_JOINT: an action expert of act_layers (== llm_layers)
 *    blocks of width act_d in the LLM's head layout, whose action tokens
 *    attend over [LLM layer l's prefix K,V ; their own K,V]; time enters by a
 *    concat MLP over [action embedding ; sinusoid(t) of width time_dim].
 *  - head_kind VLA_HEAD_DIT: a DiT of act_layers blocks of width act_d with
 *    act_heads heads: adaLN-modulated self-attention over [state ; horizon
 *    action tokens], cross-attention to the projected final LLM states, and a
 *    tanh-GELU MLP of act_mlp; time enters through a sinusoid of width
 *    time_dim and an MLP.
 *    With pix_shuffle = s > 1 the image contributes (img_hw/patch/s)^2
 *    tokens to the prefix (P counts these), the ViT still runs over all
 *    (img_hw/patch)^2 patch tokens, and the position table has that many rows.
 *  - horizon actions of action_dim per chunk; state_dim robot state (DiT).
 *  - max_batch: the largest batch any call may use (workspaces are sized for
 *    it). norm_eps applies to every RMSNorm / LayerNorm.
 */
typedef struct {
  int dtype;                                   /* VLA_F32 | VLA_BF16 */
  int n_img, img_hw, patch;
  int vit_layers, vit_d, vit_heads, vit_mlp;
  int n_text, vocab;
  int llm_layers, llm_d, n_q, n_kv, head_dim, llm_mlp;
  int head_kind;                               /* VLA_HEAD_JOINT | VLA_HEAD_DIT */
  int act_layers, act_d, act_heads, act_mlp;
  int horizon, action_dim, state_dim, time_dim;
  int max_batch;
  float rope_base, norm_eps;
  int pix_shuffle;     /* s: after the ViT's final LayerNorm, each s x s block of
                          patch tokens (raster order) is merged into one token of
                          width s*s*vit_d (block rows then columns, channels
                          innermost) before the projection to llm_d; 0 or 1: none.
                          s > 1 needs vit_layers > 0 and s | img_hw/patch */
} vla_config;

/* Number of fp32 values the parameter buffer of this shape holds, 0 if the
 * shape is invalid (vla_last_error says why). Host-only, no GPU needed. */
size_t vla_weight_count(const vla_config* cfg);

/*
 * Create a model on `device` from host parameters: `n_floats` fp32 values in
 * the canonical order (tensors concatenated, matrices [in, out] row-major).
 * The library copies and converts them; the host buffer may be freed on
 * return. Captured graphs are enabled by default.
 */
vla_status vla_create_model(const vla_config* cfg, const float* weights_host, size_t n_floats,
                            int device, vla_model* out);
void vla_destroy_model(vla_model m);

/* Enable (1) or disable (0) graph capture/replay of whole stages (Section
 * 4.1.1: one graph per stage and batch size, replayed on the stage stream).
 * Graphs are keyed by (stage, batch, steps, buffer addresses). */
vla_status vla_set_graphs(vla_model m, int enabled);

/*
 * Bytes of the VLM -> action-stage hand-off for `batch` requests (0 on a bad
 * argument). Layout, element type = the model dtype:
 *  - VLA_HEAD_JOINT: the prefix KV cache [llm_layers][2][batch][n_kv][P][head_dim],
 *    index 0 = keys after RoPE, 1 = values; P = n_img*(img_hw/patch/s)^2 + n_text
 *    (s = pix_shuffle, 1 when unset).
 *  - VLA_HEAD_DIT: cross-attention keys/values [batch][P][act_layers][2][act_d]
 *    followed by the embedded state token [batch][act_d].
 */
size_t vla_kv_bytes(vla_model m, int batch);

/*
 * VLM stage (prefill) for `batch` requests (1 <= batch <= max_batch).
 *  pixels   device fp32 [batch][n_img][3][img_hw][img_hw], values as given
 *           (no normalisation).
 *  text_ids device int32 [batch][n_text]; ids outside [0, vocab) are clamped.
 *  kv_out   device buffer of vla_kv_bytes(m, batch) bytes, written.
 */
vla_status vla_prefill(vla_model m, int batch, const float* pixels, const int32_t* text_ids,
                       void* kv_out, hipStream_t stream);

/* As vla_prefill, with the robot state for VLA_HEAD_DIT models: device fp32
 * [batch][state_dim], or NULL for a zero state. Ignored for joint models. */
vla_status vla_prefill_ex(vla_model m, int batch, const float* pixels, const int32_t* text_ids,
                          const float* state, void* kv_out, hipStream_t stream);

/*
 * Action stage: `steps` explicit Euler steps of the flow field from the noise
 * at t = 1 to the action chunk at t = 0 (t_k = 1 - k/steps, dt = -1/steps).
 *  kv          the hand-off written by vla_prefill for the same `batch`.
 *  noise       device fp32 [batch][horizon][action_dim], read only.
 *  actions_out device fp32 [batch][horizon][action_dim], written (it holds the
 *              Euler state while the call runs). May not alias `noise`.
 */
vla_status vla_denoise(vla_model m, int batch, const void* kv, const float* noise, int steps,
                       float* actions_out, hipStream_t stream);

/*
 * One lockstep (Section 4.1.2): the VLM stage of one batch runs on a stream
 * restricted to `vlm_cu_count` compute units while the action stage of the
 * previous batch runs on an unrestricted stream. Either half may be skipped
 * with batch 0. Both halves wait for work already enqueued on `join_stream`,
 * and `join_stream` waits for both halves, so stream order is preserved.
 * vlm_cu_count: a multiple of 8 in [8, 256]; 256 means no restriction (on
 * MI355X multiples of 32 give every shader engine the same number of CUs; the
 * dispatcher shares workgroups equally between shader engines, so other counts
 * run at the speed of the next lower multiple of 32). The
 * restricted streams come from a per-device pool created on first use. When
 * `join_stream` is a non-blocking stream (hipStreamNonBlocking) and the action
 * half is unrestricted, the action half runs on `join_stream` itself (faster:
 * no cross-queue wait is pending while its kernels run); otherwise it runs on
 * a pool stream. `adit_done` (may be NULL) is recorded on the action half's
 * stream right after its last kernel, when there is an action half: a caller
 * can wait on it to use the action chunks (copy them out, return them)
 * before the VLM half ends; the event must belong to the models' device.
 */
typedef struct {
  vla_model vlm_model;  int vlm_batch;
  const float* pixels;  const int32_t* text_ids;  const float* state;  void* kv_out;
  vla_model adit_model; int adit_batch;
  const void* kv_in;    const float* noise;  int steps;  float* actions_out;
  int vlm_cu_count;
  int adit_cu_count;    /* 0 or 256: unrestricted; else the complement-style
                           disjoint baseline (multiple of 8) */
  hipEvent_t adit_done; /* NULL, or recorded after the action half */
} vla_step_args;
vla_status vla_step(const vla_step_args* args, hipStream_t join_stream);

/* Message of the last failed call on this thread ("" if none). */
const char* vla_last_error(void);

/*
 * Orderly teardown, for the end of a process (or before unloading the
 * library): waits for all work on every device the library used, then
 * releases every model still alive (its graphs, capture streams and device
 * memory; those handles become invalid and vla_destroy_model ignores them),
 * the CU-restricted stream pool and its events, and the workspaces of the
 * test hooks. Callers must not use the library concurrently with it. The
 * library stays usable afterwards (pools are re-created on demand). Call it
 * before the HIP runtime unloads, e.g. from an exit handler that runs before
 * the host framework's own teardown.
 */
void vla_shutdown(void);

#ifdef __cplusplus
}
#endif
#endif /* VLA_H */
