"""Serving layer: ctypes binding of the host scheduler (include/vla_sched.h),
lockstep-duration profiling on the GPU, and robot-load sweeps.

The scheduler itself (queues, earliest-SLO-first choice, power-of-two
batches, lockstep pairing, SLO accounting) is C++ inside libvla.so; this
module marshals arguments and post-processes the records it returns.
"""
from __future__ import annotations

import ctypes
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import synth, vla

POLICIES = {"esf": 0, "rr": 1, "lqf": 2}
MODES = {"lockstep": 0, "monolithic": 1}
DELIVERY = {"lockstep": 0, "adit": 1}

REQ_DTYPE = np.dtype([("t_arrival_ns", np.int64), ("t_vlm_start_ns", np.int64), ("t_done_ns", np.int64),
                      ("model", np.int32), ("met_slo", np.int32)])
LS_DTYPE = np.dtype([("t_start_ns", np.int64), ("t_end_ns", np.int64), ("vlm_model", np.int32),
                     ("vlm_batch", np.int32), ("adit_model", np.int32), ("adit_batch", np.int32),
                     ("cu_count", np.int32), ("slot", np.int32), ("t_chunks_ns", np.int64)])


class _Cfg(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int), ("slo_ms", ctypes.POINTER(ctypes.c_double)),
                ("max_batch", ctypes.c_int), ("policy", ctypes.c_int)]


class _ReqIO(ctypes.Structure):
    _fields_ = [("pixels", ctypes.c_void_p), ("text_ids", ctypes.c_void_p), ("state", ctypes.c_void_p),
                ("noise", ctypes.c_void_p), ("actions_out", ctypes.c_void_p)]


COMP_DTYPE = np.dtype([("id", np.int64), ("model", np.int32), ("met_slo", np.int32), ("t_arrival_ns", np.int64),
                       ("t_vlm_start_ns", np.int64), ("t_done_ns", np.int64)])


class _IO(ctypes.Structure):
    _fields_ = [("model", ctypes.c_void_p), ("pixels", ctypes.c_void_p), ("text_ids", ctypes.c_void_p),
                ("state", ctypes.c_void_p), ("noise", ctypes.c_void_p), ("kv", ctypes.c_void_p * 2),
                ("actions", ctypes.c_void_p * 2), ("steps", ctypes.c_int)]


def _lib():
    L = vla.lib()
    if not getattr(L, "_sched_bound", False):
        vp, ci, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
        L.vla_sched_create.argtypes = [ctypes.POINTER(_Cfg), ctypes.POINTER(vp)]; L.vla_sched_create.restype = ci
        L.vla_sched_destroy.argtypes = [vp]; L.vla_sched_destroy.restype = None
        L.vla_sched_set_sim_executor.argtypes = [vp, vp, i64]; L.vla_sched_set_sim_executor.restype = ci
        L.vla_sched_set_gpu_executor.argtypes = [vp, vp, vp]; L.vla_sched_set_gpu_executor.restype = ci
        L.vla_sched_set_cu.argtypes = [vp, ci, vp]; L.vla_sched_set_cu.restype = ci
        L.vla_sched_set_mode.argtypes = [vp, ci]; L.vla_sched_set_mode.restype = ci
        L.vla_sched_run.argtypes = [vp, vp, vp, ci, i64, vp, vp, ci, ctypes.POINTER(ci)]
        L.vla_sched_run.restype = ci
        L.vla_sched_set_gpu_online.argtypes = [vp, vp, vp, vp]; L.vla_sched_set_gpu_online.restype = ci
        L.vla_sched_set_delivery.argtypes = [vp, ci, vp]; L.vla_sched_set_delivery.restype = ci
        L.vla_sched_set_disjoint.argtypes = [vp, ci]; L.vla_sched_set_disjoint.restype = ci
        L.vla_sched_clock_ns.argtypes = [vp]; L.vla_sched_clock_ns.restype = i64
        L.vla_sched_reset.argtypes = [vp]; L.vla_sched_reset.restype = ci
        L.vla_sched_submit.argtypes = [vp, i64, ci, i64, vp]; L.vla_sched_submit.restype = ci
        L.vla_sched_pending.argtypes = [vp]; L.vla_sched_pending.restype = ci
        L.vla_sched_run_lockstep.argtypes = [vp, vp, ctypes.POINTER(ci)]; L.vla_sched_run_lockstep.restype = ci
        L.vla_sched_wait_until.argtypes = [vp, i64]; L.vla_sched_wait_until.restype = ci
        L.vla_sched_poll.argtypes = [vp, vp, ci]; L.vla_sched_poll.restype = ci
        L.vla_sched_run_trace.argtypes = [vp, vp, vp, vp, ci, i64, vp, vp, ci, ctypes.POINTER(ci)]
        L.vla_sched_run_trace.restype = ci
        L.vla_traffic_assign.argtypes = [ci, ci, vp, vp, vp, ctypes.c_longlong, vp, ctypes.POINTER(ctypes.c_longlong),
                                         ctypes.POINTER(ci)]
        L.vla_traffic_assign.restype = ci
        L._sched_bound = True
    return L


def n_buckets(max_batch: int) -> int:
    """Batch buckets of the duration / CU tables: 0 (no batch), 1, 2, 4, ..., max_batch."""
    return int(np.log2(max_batch)) + 2


def bucket(b: int) -> int:
    return 0 if b <= 0 else int(np.log2(b)) + 1


def bucket_batches(max_batch: int) -> List[int]:
    return [0] + [1 << j for j in range(n_buckets(max_batch) - 1)]


class Scheduler:
    """One serving scheduler over co-located models (see include/vla_sched.h)."""

    def __init__(self, slo_ms: Sequence[float], max_batch: int, policy: str = "esf", mode: str = "lockstep"):
        self.n_models = len(slo_ms)
        self.max_batch = max_batch
        self._slo = (ctypes.c_double * self.n_models)(*[float(x) for x in slo_ms])
        cfg = _Cfg(self.n_models, self._slo, max_batch, POLICIES[policy])
        h = ctypes.c_void_p()
        vla._check(_lib().vla_sched_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.handle = h
        self._keep = []
        self.online = False
        vla._check(_lib().vla_sched_set_mode(self.handle, MODES[mode]))
        vla.register(self)

    def close(self):
        if getattr(self, "handle", None):
            _lib().vla_sched_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def table_shape(self):
        nb = n_buckets(self.max_batch)
        return (self.n_models, nb, self.n_models, nb)

    def set_sim(self, dur_ns: np.ndarray, host_overhead_ns: int = 0):
        t = np.ascontiguousarray(dur_ns, dtype=np.int64)
        assert t.shape == self.table_shape(), (t.shape, self.table_shape())
        vla._check(_lib().vla_sched_set_sim_executor(self.handle, t.ctypes.data, int(host_overhead_ns)))

    def set_cu(self, default_cu: int, table: Optional[np.ndarray] = None):
        ptr = None
        if table is not None:
            t = np.ascontiguousarray(table, dtype=np.int32)
            assert t.shape == self.table_shape()
            self._keep.append(t)
            ptr = t.ctypes.data
        vla._check(_lib().vla_sched_set_cu(self.handle, int(default_cu), ptr))

    def set_gpu(self, models: Sequence[vla.Model], bufs: Sequence[Dict], join_stream=None):
        """bufs[m]: dict of torch tensors pixels, text_ids, noise, (state), kv0, kv1, act0, act1 (max_batch rows)."""
        ios = (_IO * self.n_models)()
        for i, (m, b) in enumerate(zip(models, bufs)):
            io = ios[i]
            io.model = m.handle.value
            io.pixels, io.text_ids, io.noise = vla._ptr(b["pixels"]), vla._ptr(b["text_ids"]), vla._ptr(b["noise"])
            io.state = vla._ptr(b.get("state"))
            io.kv[0], io.kv[1] = vla._ptr(b["kv0"]), vla._ptr(b["kv1"])
            io.actions[0], io.actions[1] = vla._ptr(b["act0"]), vla._ptr(b["act1"])
            io.steps = m.cfg.steps
        self._keep.append((models, bufs))
        vla._check(_lib().vla_sched_set_gpu_executor(self.handle, ctypes.addressof(ios), vla._stream(join_stream)))

    def set_delivery(self, when: str = "lockstep", adit_ns: Optional[np.ndarray] = None):
        """When requests complete: "lockstep" (end of the lockstep that ran
        their action stage) or "adit" (end of that action half; adit_ns, the
        simulated executor's table of times from lockstep start to the action
        half's end, same shape as the duration table)."""
        ptr = None
        if adit_ns is not None:
            t = np.ascontiguousarray(adit_ns, dtype=np.int64)
            assert t.shape == self.table_shape(), (t.shape, self.table_shape())
            ptr = t.ctypes.data
        vla._check(_lib().vla_sched_set_delivery(self.handle, DELIVERY[when], ptr))

    def set_disjoint(self, enabled: bool):
        """Disjoint CU partition: the action half runs on the CUs the VLM half
        may not use (the paper's comparison point) instead of on all of them."""
        vla._check(_lib().vla_sched_set_disjoint(self.handle, int(bool(enabled))))

    def set_gpu_online(self, models: Sequence[vla.Model], join_stream=None):
        """Online GPU executor: the library allocates max_batch stage rows per
        model; requests bring their own device inputs (see submit)."""
        hs = (ctypes.c_void_p * self.n_models)(*[m.handle.value for m in models])
        st = (ctypes.c_int * self.n_models)(*[m.cfg.steps for m in models])
        self._keep.append((models, join_stream))
        vla._check(_lib().vla_sched_set_gpu_online(self.handle, hs, st, vla._stream(join_stream)))
        self.online = True

    @staticmethod
    def request_io(pixels, text_ids, noise, actions_out, state=None) -> _ReqIO:
        """Per-request device buffers: pixels [n_img,3,H,W] fp32, text_ids
        [n_text] int32, noise and actions_out [horizon, action_dim] fp32,
        state [state_dim] fp32 or None. Views of larger tensors are fine."""
        return _ReqIO(vla._ptr(pixels), vla._ptr(text_ids), vla._ptr(state), vla._ptr(noise), vla._ptr(actions_out))

    def clock_ns(self) -> int:
        return int(_lib().vla_sched_clock_ns(self.handle))

    def reset(self):
        vla._check(_lib().vla_sched_reset(self.handle))

    def submit(self, rid: int, model: int, t_arrival_ns: int, io: Optional[_ReqIO] = None):
        vla._check(_lib().vla_sched_submit(self.handle, int(rid), int(model), int(t_arrival_ns),
                                           ctypes.byref(io) if io is not None else None))

    def pending(self) -> int:
        return int(_lib().vla_sched_pending(self.handle))

    def run_lockstep(self):
        """One lockstep now; returns its record, or None when idle."""
        rec = np.zeros(1, dtype=LS_DTYPE)
        ran = ctypes.c_int(0)
        vla._check(_lib().vla_sched_run_lockstep(self.handle, rec.ctypes.data, ctypes.byref(ran)))
        return rec[0] if ran.value else None

    def wait_until(self, t_ns: int):
        vla._check(_lib().vla_sched_wait_until(self.handle, int(t_ns)))

    def poll(self, cap: int = 4096) -> np.ndarray:
        out = np.zeros(cap, dtype=COMP_DTYPE)
        n = int(_lib().vla_sched_poll(self.handle, out.ctypes.data, cap))
        return out[:n]

    def run(self, arrivals: np.ndarray, drain_ns: int, ls_cap: int = 1 << 20, ios=None):
        """arrivals: structured array with t_ns (sorted) and model. ios: array
        of per-request inputs (request_io, one per arrival; required with the
        online executor). Returns (request records, lockstep records) as numpy
        structured arrays."""
        t = np.ascontiguousarray(arrivals["t_ns"], dtype=np.int64)
        mo = np.ascontiguousarray(arrivals["model"], dtype=np.int32)
        n = len(t)
        req = np.zeros(n, dtype=REQ_DTYPE)
        ls = np.zeros(ls_cap, dtype=LS_DTYPE)
        nls = ctypes.c_int(0)
        io_arr = None
        if ios is not None:
            assert len(ios) == n, "one request_io per arrival"
            io_arr = (_ReqIO * n)(*ios)
        vla._check(_lib().vla_sched_run_trace(self.handle, t.ctypes.data if n else None,
                                              mo.ctypes.data if n else None,
                                              ctypes.addressof(io_arr) if io_arr is not None else None, n,
                                              int(drain_ns), req.ctypes.data if n else None, ls.ctypes.data, ls_cap,
                                              ctypes.byref(nls)))
        return req, ls[:min(nls.value, ls_cap)]


# ---------------------------------------------------------------- metrics
def attainment(req: np.ndarray) -> float:
    """Fraction of requests that met their SLO (unfinished requests miss)."""
    return float(req["met_slo"].mean()) if len(req) else 1.0


def latency_ms(req: np.ndarray) -> np.ndarray:
    done = req["t_done_ns"] >= 0
    return (req["t_done_ns"][done] - req["t_arrival_ns"][done]) / 1e6


def p99_ms(req: np.ndarray) -> float:
    lat = latency_ms(req)
    return float(np.percentile(lat, 99)) if len(lat) else float("inf")


# ---------------------------------------------------------------- GPU profiling
def alloc_io(models: Sequence[vla.Model], max_batch: int):
    """Per-model device buffers for the GPU executor (seeded inputs, max_batch rows)."""
    import torch
    bufs = []
    for m in models:
        inp = synth.make_inputs(m.cfg, max_batch)
        d = {k: torch.from_numpy(v).to(f"cuda:{m.device}") for k, v in inp.items()}
        d["kv0"], d["kv1"] = m.alloc_kv(max_batch), m.alloc_kv(max_batch)
        d["act0"], d["act1"] = torch.empty_like(d["noise"]), torch.empty_like(d["noise"])
        bufs.append(d)
    return bufs


def profile_locksteps(models: Sequence[vla.Model], bufs, max_batch: int, cu_counts: Sequence[int],
                      reps: int = 3, warmup: int = 1, log=None, join_stream=None, disjoint: bool = False,
                      with_adit: bool = False):
    """Median duration (ns) of one lockstep for every (VLM model, VLM batch,
    action model, action batch) combination and every CU restriction of the
    VLM stream, timed with HIP events on the join stream. Returns
    dur[k_index][mv][bv][ma][ba] (int64; combinations with both halves empty
    are 0) — the profiling pass behind the restriction lookup table. With
    disjoint=True the action half runs on the complementary 256 - k CUs. With
    with_adit=True also returns, same indexing, the median time from the
    lockstep's start to the end of its action half (the lockstep's duration
    when it has none): (dur, adit)."""
    import torch
    nm, nb = len(models), n_buckets(max_batch)
    bs = bucket_batches(max_batch)
    out = np.zeros((len(cu_counts), nm, nb, nm, nb), dtype=np.int64)
    adit = np.zeros_like(out)
    stream = join_stream if join_stream is not None else torch.cuda.current_stream()
    ev_a = torch.cuda.Event(enable_timing=True)
    ev_a.record(stream)                      # creates the event before its handle is passed on
    for ki, cu in enumerate(cu_counts):
        for mv in range(nm):
            for iv, bv in enumerate(bs):
                for ma in range(nm):
                    for ia, ba in enumerate(bs):
                        if bv == 0 and ba == 0:
                            continue
                        if bv == 0 and mv > 0:
                            out[ki, mv, iv, ma, ia] = out[ki, 0, iv, ma, ia]   # no VLM half: model irrelevant
                            adit[ki, mv, iv, ma, ia] = adit[ki, 0, iv, ma, ia]
                            continue
                        if ba == 0 and ma > 0:
                            out[ki, mv, iv, ma, ia] = out[ki, mv, iv, 0, ia]
                            adit[ki, mv, iv, ma, ia] = adit[ki, mv, iv, 0, ia]
                            continue
                        xv, xa = bufs[mv], bufs[ma]

                        def one():
                            vla.step(models[mv] if bv else None, bv, xv["pixels"], xv["text_ids"], xv["kv0"],
                                     models[ma] if ba else None, ba, xa["kv1"], xa["noise"], models[ma].cfg.steps,
                                     xa["act1"], vlm_cu_count=cu, state=xv.get("state"), join_stream=join_stream,
                                     adit_cu_count=256 - cu if disjoint and cu < 256 else 0,
                                     adit_done=ev_a if (with_adit and ba) else None)
                        for _ in range(warmup):
                            one()
                        ts, ta = [], []
                        for _ in range(reps):
                            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                            e0.record(stream)
                            one()
                            e1.record(stream)
                            e1.synchronize()
                            ts.append(e0.elapsed_time(e1))
                            ta.append(e0.elapsed_time(ev_a) if (with_adit and ba) else ts[-1])
                        out[ki, mv, iv, ma, ia] = int(np.median(ts) * 1e6)
                        adit[ki, mv, iv, ma, ia] = min(int(np.median(ta) * 1e6), out[ki, mv, iv, ma, ia])
        if log:
            log(f"[profile] cu={cu} done")
    return (out, adit) if with_adit else out


def best_cu_table(prof: np.ndarray, cu_counts: Sequence[int], adit: Optional[np.ndarray] = None):
    """Per combination, the CU restriction with the shortest lockstep, and
    the resulting duration table (and, given the profile's action-half
    times, those at the chosen restrictions: (table, dur, adit))."""
    best = np.argmin(np.where(prof > 0, prof, np.iinfo(np.int64).max), axis=0)
    table = np.asarray(cu_counts, dtype=np.int32)[best]
    dur = np.take_along_axis(prof, best[None], axis=0)[0]
    if adit is None:
        return table, dur
    return table, dur, np.take_along_axis(adit, best[None], axis=0)[0]


def expand_tables(dur_ns: np.ndarray, cu_table: np.ndarray, arch_of: Sequence[int]):
    """Duration and CU tables for co-located fine-tuned variants: models with
    the same architecture have the same shapes, so their lockstep entries are
    those of the architecture's profile (one profile serves every variant).
    arch_of[i] = index of model i's architecture in the profiled tables."""
    a = np.asarray(arch_of)
    return (np.ascontiguousarray(dur_ns[a][:, :, a]), np.ascontiguousarray(cu_table[a][:, :, a]))


def sweep_robots(dur_ns: np.ndarray, slo_ms: Sequence[float], max_batch: int, robots: Sequence[int], rate_hz,
                 duration_s: float, epochs: int, policy: str = "esf", host_overhead_ns: int = 0,
                 traffic: str = "poisson", target: float = 0.98, mode: str = "lockstep",
                 adit_ns: Optional[np.ndarray] = None):
    """Simulated robot-load sweep on a lockstep-duration table: for each robot
    count, the mean SLO attainment over `epochs` seeded traces. With adit_ns
    (time from lockstep start to the action half's end) requests complete
    when their action half ends, else at their lockstep's end. Returns
    (rows, max robots with attainment >= target)."""
    rows, best = [], 0
    gen = synth.poisson_arrivals if traffic == "poisson" else synth.periodic_arrivals
    for R in robots:
        att, p99 = [], []
        for e in range(epochs):
            arr = gen(R, rate_hz, duration_s, e, n_models=len(slo_ms))
            s = Scheduler(slo_ms, max_batch, policy, mode)
            s.set_sim(dur_ns, host_overhead_ns)
            if adit_ns is not None:
                s.set_delivery("adit", adit_ns)
            req, _ = s.run(arr, drain_ns=int(1e9), ls_cap=16)
            s.close()
            att.append(attainment(req))
            p99.append(p99_ms(req))
        a = float(np.mean(att))
        rows.append({"robots": int(R), "attainment": a, "p99_ms": float(np.mean(p99))})
        if a >= target:
            best = max(best, int(R))
    return rows, best


def max_robots(dur_ns: np.ndarray, slo_ms: Sequence[float], max_batch: int, rate_hz, duration_s: float,
               epochs: int, policy: str = "esf", traffic: str = "poisson", mode: str = "lockstep",
               target: float = 0.98, r_max: int = 256, patience: int = 3, host_overhead_ns: int = 0,
               adit_ns: Optional[np.ndarray] = None):
    """Largest robot count with mean simulated SLO attainment >= target,
    scanning upwards and stopping after `patience` consecutive failures.
    Returns (robots, rows)."""
    rows, best, fails = [], 0, 0
    for R in range(1, r_max + 1):
        r, _ = sweep_robots(dur_ns, slo_ms, max_batch, [R], rate_hz, duration_s, epochs, policy, host_overhead_ns,
                            traffic, target, mode, adit_ns)
        rows += r
        if r[0]["attainment"] >= target:
            best, fails = R, 0
        else:
            fails += 1
            if fails >= patience:
                break
    return best, rows


def robot_limit(dur_ns: np.ndarray, model: int, slo_ms: float, max_batch: int, rate_hz, duration_s: float,
                epochs: int, target: float = 0.98, max_robots: int = 256, policy: str = "esf",
                traffic: str = "poisson", host_overhead_ns: int = 0):
    """Robots one GPU sustains for `model` served alone (Section 4.2.2,
    finding GPU robot limits): raise the robot count until the simulated SLO
    attainment on the model's own lockstep durations falls below `target`;
    returns (limit, rows). dur_ns is a co-location table; its (model, model)
    slice is used."""
    sub = np.ascontiguousarray(dur_ns[model:model + 1, :, model:model + 1, :])
    rows, limit = [], 0
    for R in range(1, max_robots + 1):
        r, _ = sweep_robots(sub, [slo_ms], max_batch, [R], rate_hz, duration_s, epochs, policy, host_overhead_ns,
                            traffic, target)
        rows += r
        if r[0]["attainment"] < target:
            break
        limit = R
    return limit, rows


def traffic_assign(host, n_robots, limits, max_nodes: int = 10_000_000):
    """Robot-to-GPU assignment of the adaptive traffic controller (eqs (1)-(3)
    of Section 4.2.2) by the library's exact search. host: [models][gpus] 0/1;
    returns (r [models][gpus], objective, proven_optimal)."""
    host = np.ascontiguousarray(host, dtype=np.int32)
    n = np.ascontiguousarray(n_robots, dtype=np.int32)
    c = np.ascontiguousarray(limits, dtype=np.int32)
    M, G = host.shape
    if n.shape != (M,) or c.shape != (M,):
        raise ValueError("n_robots and limits need one entry per model")
    r = np.zeros((M, G), dtype=np.int32)
    obj, opt = ctypes.c_longlong(0), ctypes.c_int(0)
    vla._check(_lib().vla_traffic_assign(M, G, host.ctypes.data, n.ctypes.data, c.ctypes.data, int(max_nodes),
                                         r.ctypes.data, ctypes.byref(obj), ctypes.byref(opt)))
    return r, int(obj.value), bool(opt.value)
