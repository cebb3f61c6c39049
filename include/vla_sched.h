/*
 * vla_sched.h - host-side serving scheduler of libvla.so (paper Section 4.1).
 *
 * Requests of co-located models wait in one FIFO queue per model. Work runs
 * in locksteps (Section 4.1.2): when lockstep k begins, the scheduler
 * picks a queue, dequeues a fixed batch of b_k requests for the VLM stage,
 * and the action stage runs the batch that finished the VLM stage in
 * lockstep k-1 (held in a two-slot hand-off buffer, slot = k mod 2). The
 * lockstep ends when both stages have finished. Queue choice (Section 4.1.3):
 * earliest-SLO-first serves the queue whose oldest request is closest to
 * its deadline (SLO minus time already waited); ties go to the
 * lowest model index. Batch size: the largest power of two not above
 * min(pending requests in that queue, max_batch), so every lockstep replays a
 * pre-captured graph (Section 4.1.2). A request meets its SLO when its
 * completion time minus its arrival time is at most the model's SLO.
 *
 * The scheduler serves requests online (submit / run_lockstep / poll) or
 * runs a whole arrival trace, against an executor: the GPU (vla_step, wall
 * clock) with per-request inputs gathered into library-owned stage buffers,
 * the GPU on fixed caller buffers (every batch reads rows 0 .. b-1), or a
 * table of lockstep durations (simulated time, deterministic, no GPU).
 * All calls are host calls; only locksteps of a GPU executor touch the
 * device. A scheduler is used by one host thread at a time. Errors follow
 * vla.h (status + vla_last_error).
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
enum { VLA_SCHED_DONE_LOCKSTEP = 0, VLA_SCHED_DONE_ADIT = 1 };

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
  int64_t t_chunks_ns;          /* when the action half's chunks were delivered
                                   (t_end_ns without an action half, in Monolithic
                                   mode, and with delivery at the lockstep end) */
} vla_lockstep_rec;

typedef struct {           /* outcome of one request */
  int64_t t_arrival_ns;
  int64_t t_vlm_start_ns;       /* start of its VLM lockstep, -1 if never admitted */
  int64_t t_done_ns;            /* delivery of its chunk (see vla_sched_set_delivery),
                                   -1 if unfinished */
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

/*
 * When a request completes (lockstep mode). VLA_SCHED_DONE_LOCKSTEP (the
 * default): at the end of the lockstep in which its action stage ran.
 * VLA_SCHED_DONE_ADIT: when its action stage ends. The paper's lockstep
 * starts the next lockstep only once both halves have finished (Section
 * 4.1.2) and does not say when a finished chunk leaves the server; in this
 * mode the online GPU executor copies the chunks to the requests' buffers
 * as soon as the action half is done (on a stream of its own, while the VLM
 * half may still run), and the completion time is that copy's end, read
 * from GPU events; the fixed-buffer executor uses the action half's end. The
 * simulated executor takes it from `adit_ns` (same indexing as the duration
 * table: time from the lockstep's start to the end of its action half; an
 * entry above the lockstep's duration counts as the lockstep's end); the
 * table is copied, and is required before a simulated run in this mode
 * (NULL keeps the previous one). Monolithic mode always completes a batch at
 * its end.
 */
vla_status vla_sched_set_delivery(vla_sched s, int when, const int64_t* adit_ns);

/* Partition of the compute units between the two halves of a lockstep: 0
 * (the default, the paper's guarded restriction) restricts only the VLM half
 * and lets the action half use every CU; 1 (the disjoint partition the paper
 * compares against, Section 5.2) also restricts the action half, to the
 * 256 - k CUs the VLM half may not use (k = the lockstep's VLM restriction;
 * k = 256 leaves both halves unrestricted). Monolithic mode ignores it. */
vla_status vla_sched_set_disjoint(vla_sched s, int disjoint);

/* CU restriction of the VLM stream per lockstep: `default_cu` (multiple of 8,
 * 8 .. 256) unless `cu_table` (same indexing as the duration table, entries 0
 * = use default) names another count for the batch combination (the
 * profiled lookup table of Section 4.1.2). The table is copied; NULL clears. */
vla_status vla_sched_set_cu(vla_sched s, int default_cu, const int* cu_table);

/*
 * Run an arrival trace (vla_sched_run_trace without per-request inputs): n
 * requests with arrival times t_arrival_ns (sorted ascending, relative to the
 * run start) and model indices. Requests still
 * unfinished `drain_ns` after the last arrival are reported unfinished.
 * Writes req_out[n] and up to ls_cap lockstep records (*n_ls_out = count
 * executed, which may exceed ls_cap; records beyond it are dropped).
 */
vla_status vla_sched_run(vla_sched s, const int64_t* t_arrival_ns, const int32_t* model, int n,
                         int64_t drain_ns, vla_request_rec* req_out, vla_lockstep_rec* ls_out, int ls_cap,
                         int* n_ls_out);

/*
 * Online serving (Sections 4.1.2 and 4.1.3): requests arrive one at a time
 * with their own inputs, each lockstep admits a batch, and finished action
 * chunks are handed back per request.
 *
 * vla_sched_set_gpu_online selects the online GPU executor: for every model
 * the library allocates stage buffers of max_batch rows (pixels, text ids,
 * state, two noise slots, two hand-off slots, two action slots) and keeps
 * them until vla_sched_destroy. A lockstep then runs on `join`:
 *   1. one batched-copy kernel gathers the admitted requests' pixels, text
 *      ids, state (zeros when NULL) and noise into rows 0 .. b-1 of the VLM
 *      model's stage buffers (noise into the slot the next lockstep's action
 *      half reads);
 *   2. vla_step runs the VLM half on those rows, restricted by the CU table,
 *      beside the action half of the batch admitted one lockstep earlier;
 *   3. one batched-copy kernel scatters row i of that action batch to the
 *      actions_out buffer of the request that sat in row i;
 *   4. the host waits for `join`; the finished requests become completions.
 * steps[m]: Euler steps of model m's action stage.
 */
typedef struct {
  const float* pixels;     /* device fp32 [n_img][3][img_hw][img_hw] */
  const int32_t* text_ids; /* device int32 [n_text] */
  const float* state;      /* device fp32 [state_dim] (DiT models) or NULL for a zero state */
  const float* noise;      /* device fp32 [horizon][action_dim], read only */
  float* actions_out;      /* device fp32 [horizon][action_dim], written when the request completes */
} vla_request_io;

typedef struct {           /* a finished request, as returned by vla_sched_poll */
  int64_t id;
  int model;
  int met_slo;
  int64_t t_arrival_ns, t_vlm_start_ns, t_done_ns;
} vla_completion;

vla_status vla_sched_set_gpu_online(vla_sched s, const vla_model* models, const int* steps, hipStream_t join);

/* Scheduler clock in ns: wall time since the executor was set (or since the
 * last vla_sched_reset) for the GPU executors, the simulated time for the
 * simulated one. Arrival times passed to vla_sched_submit use this clock. */
int64_t vla_sched_clock_ns(vla_sched s);

/* Drop every queued, in-flight and unpolled request and restart the clock at
 * 0 (the lockstep counter restarts too). */
vla_status vla_sched_reset(vla_sched s);

/*
 * Queue a request of `model` that arrived at t_arrival_ns (scheduler clock)
 * at the tail of that model's FIFO. `io` is copied; the buffers it names
 * must stay valid until the request's completion has been polled. With the
 * online GPU executor io (pixels, text_ids, noise, actions_out) is required;
 * the simulated executor and the fixed-buffer GPU executor accept NULL.
 */
vla_status vla_sched_submit(vla_sched s, int64_t id, int model, int64_t t_arrival_ns, const vla_request_io* io);

/* Requests queued or waiting for the action stage. */
int vla_sched_pending(vla_sched s);

/*
 * Run one lockstep now (a whole batch in Monolithic mode): choose the queue,
 * admit a power-of-two batch, execute, and turn the batch whose action stage
 * finished into completions. With nothing queued and nothing waiting for the
 * action stage it does nothing and sets *ran = 0. rec (may be NULL) receives
 * the lockstep's record. The simulated clock advances by the lockstep's
 * duration; the GPU executors block until the lockstep has finished.
 */
vla_status vla_sched_run_lockstep(vla_sched s, vla_lockstep_rec* rec, int* ran);

/* Let the clock reach t_ns when idle: the simulated clock jumps there, the
 * GPU executors sleep until then. Earlier times do nothing. */
vla_status vla_sched_wait_until(vla_sched s, int64_t t_ns);

/* Move up to `cap` completions (oldest first) into out; returns how many. */
int vla_sched_poll(vla_sched s, vla_completion* out, int cap);

/*
 * Trace driver on the calls above: resets the scheduler, submits request i
 * (id i, io[i] when io is not NULL) once the clock reaches t_arrival_ns[i],
 * runs locksteps while work is pending, idles until the next arrival
 * otherwise, and stops drain_ns after the last arrival. Outputs as for
 * vla_sched_run.
 */
vla_status vla_sched_run_trace(vla_sched s, const int64_t* t_arrival_ns, const int32_t* model,
                               const vla_request_io* io, int n, int64_t drain_ns, vla_request_rec* req_out,
                               vla_lockstep_rec* ls_out, int ls_cap, int* n_ls_out);

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
