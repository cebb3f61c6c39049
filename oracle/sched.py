"""Reference serving scheduler in plain Python (test infrastructure).

Restates the serving rules of the paper for the scheduler tests; it shares
no code with the library's C++ scheduler.

* Section 4.1.2 (lockstep execution): work advances in locksteps. When
  lockstep k begins, a fixed batch is admitted to the VLM stage; the action
  stage runs, in the same lockstep, the batch that finished the VLM stage in
  lockstep k-1 (kept in a small hand-off buffer). The next lockstep starts
  when both stages of this one have finished. When fewer than max_batch
  requests are pending, the admitted batch is a power of two so a
  pre-recorded graph exists for it (reading: the largest power of two not
  above min(pending, max_batch); the printed sentence is garbled).
* Section 4.1.3 (several models on one VLM and one action stream): one FIFO
  queue per model; when a lockstep begins, the queue whose oldest request is
  closest to its deadline (SLO minus time already waited) is served
  (reading: ties go to the lowest model index). Round robin and
  largest-queue-first are the comparison policies of Section 5.3.
* Section 5.1: a request meets its SLO when its end-to-end latency is within
  the deadline (network latency taken as zero here).
* When a request's chunk is delivered (reading; the paper gates only the next
  lockstep's start on both halves and is silent on when a finished chunk
  leaves the server): by default at the end of the lockstep that ran its
  action stage; with delivery "adit", when that action half ends, given by a
  second table (time from the lockstep's start to its action half's end, same
  indexing), capped at the lockstep's end.
* Monolithic, the paper's control system (Section 5): no stage
  disaggregation; the admitted batch runs the VLM stage and then the action
  stage back to back on the whole GPU and completes before the next batch is
  admitted (duration: the two stand-alone table entries plus two host
  overheads).

The executor is a table of lockstep durations indexed by
(VLM model, VLM batch bucket, action model, action batch bucket), bucket 0 =
no batch and bucket j = batch 2**(j-1); time is simulated.
"""
from collections import deque


def bucket(b):
    if b <= 0:
        return 0
    j = 1
    while 2 ** (j - 1) < b:
        j += 1
    return j


def largest_pow2_at_most(x):
    p = 1
    while p * 2 <= x:
        p *= 2
    return p


def simulate(arrivals, slo_ms, max_batch, dur_ns, policy="esf", drain_ns=10 ** 9, overhead_ns=0,
             cu_default=256, cu_table=None, mode="lockstep", delivery="lockstep", adit_ns=None):
    """arrivals: list of (t_ns, model) sorted by time. dur_ns (and adit_ns
    for delivery "adit"): nested lists [mv][bv_bucket][ma][ba_bucket].
    Returns (requests, locksteps): requests = list of dicts (t_arrival,
    t_vlm_start, t_done, model, met), locksteps = list of tuples (t_start,
    t_end, vlm_model, vlm_batch, adit_model, adit_batch, cu, slot,
    t_chunks)."""
    n_models = len(slo_ms)
    slo_ns = [int(s * 1e6 + 0.5) for s in slo_ms]
    reqs = [{"t_arrival": t, "t_vlm_start": -1, "t_done": -1, "model": m, "met": 0} for t, m in arrivals]
    queues = [deque() for _ in range(n_models)]
    horizon = (arrivals[-1][0] if arrivals else 0) + drain_ns
    now, nxt, rr, k = 0, 0, 0, 0
    handoff, handoff_model, handoff_slot = [], -1, 0
    locksteps = []
    while True:
        while nxt < len(arrivals) and arrivals[nxt][0] <= now:
            queues[arrivals[nxt][1]].append(nxt)
            nxt += 1
        pending = any(queues)
        if not pending and not handoff:
            if nxt >= len(arrivals):
                break
            now = arrivals[nxt][0]
            continue
        if now > horizon:
            break
        # which queue feeds the VLM stage
        mv, bv = -1, 0
        if pending:
            candidates = [m for m in range(n_models) if queues[m]]
            if policy == "esf":
                mv = min(candidates, key=lambda m: (slo_ns[m] - (now - reqs[queues[m][0]]["t_arrival"]), m))
            elif policy == "rr":
                mv = next(m for m in [(rr + j) % n_models for j in range(n_models)] if queues[m])
                rr = (mv + 1) % n_models
            else:
                mv = min(candidates, key=lambda m: (-len(queues[m]), m))
            bv = largest_pow2_at_most(min(len(queues[mv]), max_batch))
        admitted = [queues[mv].popleft() for _ in range(bv)]
        if mode == "monolithic":
            end = now + dur_ns[mv][bucket(bv)][0][0] + dur_ns[0][0][mv][bucket(bv)] + 2 * overhead_ns
            for r in admitted:
                reqs[r]["t_vlm_start"] = now
                reqs[r]["t_done"] = end
            locksteps.append((now, end, mv, bv, mv, bv, 256, 0, end))
            k += 1
            now = end
            continue
        ma, ba = (handoff_model, len(handoff)) if handoff else (-1, 0)
        slot = k % 2
        iv, ia = bucket(bv), bucket(ba)
        d = dur_ns[max(mv, 0)][iv][max(ma, 0)][ia]
        cu = cu_default
        if cu_table is not None and cu_table[max(mv, 0)][iv][max(ma, 0)][ia] > 0:
            cu = cu_table[max(mv, 0)][iv][max(ma, 0)][ia]
        end = now + d + overhead_ns
        chunks = end
        if delivery == "adit" and handoff:
            chunks = min(end, now + adit_ns[max(mv, 0)][iv][max(ma, 0)][ia])
        for r in handoff:
            reqs[r]["t_done"] = chunks
        for r in admitted:
            reqs[r]["t_vlm_start"] = now
        locksteps.append((now, end, mv, bv, ma, ba, cu, slot, chunks))
        handoff, handoff_model, handoff_slot = admitted, mv, slot
        k += 1
        now = end
    for r in reqs:
        r["met"] = int(r["t_done"] >= 0 and r["t_done"] - r["t_arrival"] <= slo_ns[r["model"]])
    return reqs, locksteps
