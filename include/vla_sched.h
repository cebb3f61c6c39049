/*
 * vla_sched.h - host-side serving scheduler of libvla.so (paper Section 4.1).
 *
 * Requests of co-located models wait in one FIFO queue per model. Work runs
 * in locksteps (Section 4.1.2): at the start of lockstep k the scheduler
 * picks a queue, dequeues a fixed batch of b_k requests for the VLM stage,
 * and the action stage runs the batch that finished the VLM stage in
 * lockstep k-1 (held in a two-slot hand-off buffer, slot = k mod 2). The
 * lockstep ends when both stages have finished. Queue choice (Section 4.1.3):
 * earliest-SLO-first picks the queue whose head request has the least time
 * left before its deadline (SLO minus time already waited); ties go to the
 * lowest model index. Batch size: the largest power of two not above
 * min(pending requests in that queue, max_batch), so every lockstep replays a
 * pre-captured graph (Section 4.1.2). A request meets its SLO when its
 * completion time minus its arrival time is at most the model's SLO.
 *
 * The scheduler runs a whole arrival trace against an executor: either the
 * GPU (vla_step on caller-provided buffers, wall-clock time) or a table of
 * lockstep durations (simulated time, deterministic, no GPU needed).
 * All calls are host calls; only vla_sched_run with the GPU executor touches
 * the device. Errors follow vla.h (status + vla_last_error).
 */
#ifndef VLA_SCHED_H
#define VLA_SCHED_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#include "vla.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct vla_sched_s* vla_sched;

/* queue-selection policies: earliest-SLO-first (the paper's), round robin,
 * largest queue first (the paper's comparison policies, Section 5.3) */
enum { VLA_SCHED_ESF = 0, VLA_SCHED_RR = 1, VLA_SCHED_LQF = 2 };

/* execution modes: stage-disaggregated locksteps (the paper's design, the
 * default) or Monolithic, the paper's control (Section 5): each admitted
 * batch runs the VLM stage then the action stage back to back on the whole
 * GPU and completes before the next batch starts (simulated duration: the
 * two stages' stand-alone table entries plus two host overheads). */
enum { VLA_SCHED_LOCKSTEP = 0, VLA_SCHED_MONOLITHIC = 1 };

typedef struct {
  int n_models;            /* 1 .. 16 */
  const double* slo_ms;    /* [n_models] per-model deadline (ms), copied */
  int max_batch;           /* a power of two, 1 .. 64 */
  int policy;              /* VLA_SCHED_ESF | VLA_SCHED_RR | VLA_SCHED_LQF */
} vla_sched_config;

/* Batch-size bucket used by the duration and CU tables: 0 = no batch,
 * j > 0 = batch 2^(j-1). n_buckets = log2(max_batch) + 2. Tables are indexed
 * [vlm_model][vlm_bucket][adit_model][adit_bucket] (row-major). */

typedef struct {           /* one executed lockstep */
  int64_t t_start_ns, t_end_ns;
  int vlm_model, vlm_batch;     /* -1, 0 when the VLM half is empty */
  int adit_model, adit_batch;   /* -1, 0 when the action half is empty */
  int cu_count;                 /* CU restriction applied to the VLM stream */
  int slot;                     /* hand-off slot written by the VLM half (k mod 2) */
} vla_lockstep_rec;

typedef struct {           /* outcome of one request */
  int64_t t_arrival_ns;
  int64_t t_vlm_start_ns;       /* start of its VLM lockstep, -1 if never admitted */
  int64_t t_done_ns;            /* end of its action lockstep, -1 if unfinished */
  int model;
  int met_slo;                  /* 1 if t_done - t_arrival <= SLO */
} vla_request_rec;

vla_status vla_sched_create(const vla_sched_config* cfg, vla_sched* out);
void vla_sched_destroy(vla_sched s);

/* Simulated executor: lockstep duration in ns from `dur_ns` (table above,
 * n_models^2 * n_buckets^2 entries, copied) plus `host_overhead_ns` per
 * lockstep. Durations must be >= 0. */
vla_status vla_sched_set_sim_executor(vla_sched s, const int64_t* dur_ns, int64_t host_overhead_ns);

/* GPU executor: per-model device buffers, each sized for max_batch requests.
 * kv[0], kv[1] hold vla_kv_bytes(model, max_batch) bytes each; actions[0..1]
 * [max_batch][horizon][action_dim] fp32; pixels, text_ids, noise (and state
 * for DiT models, may be NULL) are the inputs every batch reads (rows
 * 0 .. b-1). The arrays are copied. `join` is the stream each lockstep is
 * joined on; the host waits for it at every lockstep end. */
typedef struct {
  vla_model model;
  const float* pixels; const int32_t* text_ids; const float* state; const float* noise;
  void* kv[2];
  float* actions[2];
  int steps;               /* Euler steps of this model's action stage */
} vla_sched_model_io;
vla_status vla_sched_set_gpu_executor(vla_sched s, const vla_sched_model_io* io, hipStream_t join);

/* Execution mode (VLA_SCHED_LOCKSTEP or VLA_SCHED_MONOLITHIC); the default
 * is LOCKSTEP. Monolithic ignores the CU table. */
vla_status vla_sched_set_mode(vla_sched s, int mode);

/* CU restriction of the VLM stream per lockstep: `default_cu` (multiple of 8,
 * 8 .. 256) unless `cu_table` (same indexing as the duration table, entries 0
 * = use default) names another count for the batch combination (the
 * profiled lookup table of Section 4.1.2). The table is copied; NULL clears. */
vla_status vla_sched_set_cu(vla_sched s, int default_cu, const int* cu_table);

/*
 * Run an arrival trace: n requests with arrival times t_arrival_ns (sorted
 * ascending, relative to the run start) and model indices. Requests still
 * unfinished `drain_ns` after the last arrival are reported unfinished.
 * Writes req_out[n] and up to ls_cap lockstep records (*n_ls_out = count
 * executed, which may exceed ls_cap; records beyond it are dropped).
 */
vla_status vla_sched_run(vla_sched s, const int64_t* t_arrival_ns, const int32_t* model, int n,
                         int64_t drain_ns, vla_request_rec* req_out, vla_lockstep_rec* ls_out, int ls_cap,
                         int* n_ls_out);

/*
 * Adaptive traffic controller (Section 4.2.2): robot-to-GPU assignment for a
 * multi-GPU server, solved once at initialisation on the host.
 *   host      [n_models][n_gpus] placement, 1 where GPU j hosts model i
 *   n_robots  [n_models] robot population N_i (>= 0)
 *   limits    [n_models] C_i >= 1: robots of model i one GPU sustains at the
 *             SLO-attainment target (found by benchmarking the model alone)
 *   r_out     [n_models][n_gpus] robots of model i assigned to GPU j
 * Constraints: eq (1) sum_j r[i][j] = N_i; eq (2) sum_i r[i][j] / C_i <= 1
 * (exact rational test); r[i][j] = 0 where not hosted. Objective, eq (3):
 * minimise sum_j sum_{i<k} r[i][j] r[k][j] (per-GPU traffic concentrated on
 * few models). Exact branch and bound; it stops after max_nodes search nodes
 * and sets *optimal = 1 only when the optimum was proven. Optimal
 * assignments need not be unique (interchangeable GPUs); *objective is.
 * Returns VLA_EINVAL when no assignment satisfies the constraints ("change
 * the placement or add GPUs"), VLA_EUNSUPPORTED when the node limit is hit
 * before any feasible assignment is found. Host-only; no GPU is used.
 */
vla_status vla_traffic_assign(int n_models, int n_gpus, const int* host, const int* n_robots, const int* limits,
                              long long max_nodes, int* r_out, long long* objective, int* optimal);

#ifdef __cplusplus
}
#endif
#endif /* VLA_SCHED_H */
