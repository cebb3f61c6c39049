#!/usr/bin/env python3
"""Benchmark of the VLA serving hot path on one MI355X.

Default: the co-located serving workload, a pi0-shaped and a SmolVLA-shaped
model sharing one GPU (robot i -> model i mod 2), Poisson requests at
--rate Hz per robot, a --slo-ms deadline, earliest-SLO-first queues and
power-of-two batches up to a cap of 2, 4 or 8 (--serve-batches; paper
Sections 4.1.2-4.1.3). The
metric is the paper's robot-limit method (Section 4.2.2, Section 5.1): the
largest robot count whose SLO attainment is >= 98 %, times the rate, in
action chunks/s. It is found in three steps:

1. profile every lockstep combination (VLM model, batch, action model,
   batch) under each VLM CU restriction and keep the fastest restriction per
   combination (the lookup table of Section 4.1.2);
2. sweep the robot count on those durations in the simulated executor, for
   each batch cap, and keep the cap that sustains the most robots;
3. serve in real time on the GPU through the online scheduler (every request
   gathers its own robot's inputs into the stage rows and gets its chunk
   scattered back) at the simulated limit, then one robot more or fewer until
   the largest count with >= 98 % attainment is confirmed. ``value`` is that
   GPU-validated count times the rate.

A step (``--steps``/``--warmup``) is one lockstep of the saturated pipeline
at the serving batch, alternating (pi0 VLM || SmolVLA action stage) and
(SmolVLA VLM || pi0 action stage) at the table's CU restriction;
``ms_per_step`` is their mean. Also reported: stage times alone, ADiT step
ms and MFMA fractions, a roofline entry for the kernel with the most time in
this workload (timed with HIP events on the stream it runs on), and the CPU
oracle on a bounded sample of the same workload.

Other modes: --lockstep (one model, saturated locksteps), --serve (studies:
controls, policies, periodic traffic, traffic controller), --stages (stage
times per config and batch), --counters (hardware counter passes).

    python bench.py [--steps K] [--warmup W] [--rate 10] [--serve-batch 4]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "action chunks/s at 98% SLO per GPU; ADiT step ms; MFMA % of bf16 peak"
PEAK = {"bf16": 2500.0, "f32": 157.3}     # dense TFLOP/s (MFMA bf16, fp32 vector)
# per-chunk deadlines of the paper's models (Section 5.1), used for the closed-loop latency check
SLO_MS = {"smolvla": 50.0, "pi0": 156.0, "gr00t": 53.0, "tiny": 50.0}
GEMM_NAMES = {0: "VLM LLM MLP gate/up (GeGLU epilogue)", 1: "VLM LLM MLP down (+residual)",
              2: "action-stage MLP up", 3: "action-stage MLP down (+residual)", 4: "ViT MLP up (GELU)"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def cpu_baseline(cfg, weights, budget_s):
    """Time the CPU oracle (as it stands) on whole requests of the same
    workload until ~budget_s of work; returns the JSON object."""
    import numpy as np
    from oracle import vla as O
    from paper_2609_12075_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    W = O.params(cfg, weights)
    done, t0 = 0, time.perf_counter()
    while True:
        inp = synth.make_inputs(cfg, 1, first_row=done)
        O.run(cfg, W, inp)
        done += 1
        el = time.perf_counter() - t0
        if el >= budget_s or el / done * (done + 1) > 3 * budget_s:
            break
    return {"value": done / el, "unit": "action chunks/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{done} request(s) of the {cfg.name}-shaped model at batch 1 (prefill + {cfg.steps} Euler "
                      f"steps), numpy fp64, {el:.1f} s"}


class GpuValidator:
    """Real-time serving runs on the GPU for the robot-limit search: the
    online scheduler gathers each request's inputs from its robot's own
    device buffers (robot i -> model i mod n) and scatters its chunk to a
    buffer of its own; attainment counts unfinished requests as misses."""

    def __init__(self, models, cfgs, slo, f, seconds, join_stream, n_rob_max, log_prefix="[bench]"):
        import torch
        from paper_2609_12075_amd import synth
        self.models, self.cfgs, self.slo, self.f, self.seconds = models, cfgs, slo, f, seconds
        self.js, self.lp = join_stream, log_prefix
        self.rob_in = []
        for i, c in enumerate(cfgs):
            n = (n_rob_max + len(cfgs) - 1 - i) // len(cfgs)
            inp = synth.make_inputs(c, max(n, 1), first_row=100)
            self.rob_in.append({k: torch.from_numpy(v).to("cuda:0") for k, v in inp.items()})

    def run(self, R, epoch, mb, cu_table=None, default_cu=256, mode="lockstep", disjoint=False, policy="esf",
            traffic="poisson", slo=None, delivery="lockstep"):
        import torch
        from paper_2609_12075_amd import serve, synth
        slo = self.slo if slo is None else slo
        gen = synth.poisson_arrivals if traffic == "poisson" else synth.periodic_arrivals
        arr = gen(R, self.f, self.seconds, epoch=epoch, n_models=len(self.cfgs))
        outs = [torch.full((max(1, int((arr["model"] == i).sum())), c.horizon, c.action_dim), float("nan"),
                           device="cuda:0") for i, c in enumerate(self.cfgs)]
        cnt, ios = [0] * len(self.cfgs), []
        for j in range(len(arr)):
            mi, r = int(arr["model"][j]), int(arr["robot"][j]) // len(self.cfgs)
            d = self.rob_in[mi]
            ios.append(serve.Scheduler.request_io(d["pixels"][r], d["text_ids"][r], d["noise"][r], outs[mi][cnt[mi]],
                                                  d["state"][r] if "state" in d else None))
            cnt[mi] += 1
        sch = serve.Scheduler(slo, mb, policy, mode)
        sch.set_gpu_online(self.models, join_stream=self.js)
        sch.set_cu(default_cu, cu_table)
        sch.set_disjoint(disjoint)
        sch.set_delivery(delivery)
        torch.cuda.synchronize()
        req, ls = sch.run(arr, drain_ns=int(1e9), ios=ios)
        sch.close()
        done = req["t_done_ns"] >= 0
        finite = all(bool(torch.isfinite(o[:c]).all()) for o, c in zip(outs, cnt) if c) if done.all() else None
        dur = (ls["t_end_ns"] - ls["t_start_ns"]) / 1e6
        early = (ls["t_end_ns"] - ls["t_chunks_ns"])[ls["adit_batch"] > 0] / 1e6
        rec = {"robots": int(R), "requests": int(len(req)), "attainment": round(serve.attainment(req), 4),
               "p99_ms": round(serve.p99_ms(req), 2), "locksteps": int(len(ls)),
               "lockstep_ms_mean": round(float(dur.mean()), 3) if len(dur) else None,
               "chunks_before_lockstep_end_ms_mean": round(float(early.mean()), 3) if len(early) else None,
               "delivery": delivery, "outputs_finite": finite, "seconds": self.seconds}
        log(f"{self.lp} GPU R={R}: attainment {rec['attainment']:.4f}, p99 {rec['p99_ms']} ms, "
            f"{rec['requests']} requests, {rec['locksteps']} locksteps")
        return rec

    def search(self, R0, r_max, epoch0=100, target=0.98, **kw):
        """Largest robot count with GPU attainment >= target, starting from
        the simulated limit R0: up while it holds, else down until it does.
        Returns (robots, checks)."""
        checks, R = [], max(1, min(R0, r_max))
        rec = self.run(R, epoch0, **kw)
        checks.append(rec)
        ok = rec["attainment"] >= target
        best = R if ok else 0
        while ok and R < r_max:
            R += 1
            rec = self.run(R, epoch0 + R, **kw)
            checks.append(rec)
            ok = rec["attainment"] >= target
            if ok:
                best = R
        R = checks[0]["robots"]
        while best == 0 and R > 1:
            R -= 1
            rec = self.run(R, epoch0 + R, **kw)
            checks.append(rec)
            if rec["attainment"] >= target:
                best = R
        return best, checks


def serve_main(args):
    """Co-located serving studies (pi0-shaped + SmolVLA-shaped models on one
    GPU, batch cap --serve-batch, Poisson traffic at the first --serve-rates
    rate unless stated): every robot count reported is the largest one whose
    real-time GPU run reaches >= 98 % SLO attainment, searched from the
    simulated limit on the profiled lockstep durations (the simulated limit is
    reported beside it). Arms:

    * the paper's execution-mode ablation (Section 5.2, Fig. 7): Monolithic
      (no stage disaggregation), stage disaggregation only (two streams, no
      CU restriction), disjoint CU partition (VLM on k CUs, action stage on
      the other 256 - k, k from a lookup table), and the guarded restriction
      (VLM on k CUs, action stage on all; the default);
    * queue policies RR and LQF beside ESF (Section 5.3);
    * the paper's periodic 2 Hz traffic with per-model SLOs (Section 5.1);
    * two fine-tuned variants of each architecture co-located (4 models);
    * per-model GPU robot limits (simulated, each model alone) and the
      traffic controller's assignment for a two-GPU server (Section 4.2.2).

    Prints one JSON line."""
    import numpy as np
    import torch
    from paper_2609_12075_amd import serve, synth, vla

    names = args.serve_models.split(",")
    mb = args.serve_batch
    cfgs = [synth.CONFIGS[n].with_(max_batch=mb) for n in names]
    slo = [args.slo_ms] * len(cfgs)
    cus = [int(x) for x in args.serve_cus.split(",")]
    rates = [float(x) for x in args.serve_rates.split(",")]
    f0 = rates[0]
    T, E, RM = args.serve_seconds, args.serve_epochs, args.serve_max_robots
    t0 = time.perf_counter()
    models = [vla.Model(c, synth.make_weights(c), device=0) for c in cfgs]
    log(f"[serve] models {names} created in {time.perf_counter() - t0:.1f} s")
    bufs = serve.alloc_io(models, mb)
    for m, b in zip(models, bufs):          # both hand-off slots hold real prefixes
        m.prefill(mb, b["pixels"], b["text_ids"], b["kv0"], state=b.get("state"))
        m.prefill(mb, b["pixels"], b["text_ids"], b["kv1"], state=b.get("state"))
    torch.cuda.synchronize()
    js = vla.nonblocking_stream(0)
    t0 = time.perf_counter()
    prof = serve.profile_locksteps(models, bufs, mb, cus, reps=3, log=log, join_stream=js)
    prof_dj = serve.profile_locksteps(models, bufs, mb, cus, reps=3, log=log, join_stream=js, disjoint=True)
    log(f"[serve] profiled guarded and disjoint tables in {time.perf_counter() - t0:.1f} s")
    cu_table, dur_lut = serve.best_cu_table(prof, cus)
    cu_dj, dur_dj = serve.best_cu_table(prof_dj, cus)
    dur_static = {cu: prof[i] for i, cu in enumerate(cus)}
    val = GpuValidator(models, cfgs, slo, f0, args.validate_seconds, js, RM + 2, log_prefix="[serve]")

    def arm(label, dur, sim_kw, gpu_kw, rate=f0, slo_=None, traffic="poisson", r_max=RM):
        s = slo if slo_ is None else slo_
        r_sim, rows = serve.max_robots(dur, s, mb, rate, T, E, traffic=traffic, r_max=r_max, **sim_kw)
        v = val if rate == f0 else GpuValidator(models, cfgs, s, rate, args.validate_seconds, js, r_max + 2,
                                                log_prefix="[serve]")
        best, checks = v.search(r_sim, r_max, mb=mb, traffic=traffic, slo=s, **gpu_kw)
        log(f"[serve] {label}: {best} robots at >= 98 % on the GPU (simulated {r_sim})")
        return {"robots_at_98": best, "chunks_per_s": best * rate, "robots_at_98_sim": r_sim,
                "gpu_validation": checks,
                "attainment_by_robots_sim": {str(x["robots"]): round(x["attainment"], 4) for x in rows}}

    studies = {}
    t0 = time.perf_counter()
    # execution-mode ablation
    studies["guarded_cu_table"] = arm("guarded (VLM restricted by the table, action stage on all CUs)", dur_lut, {},
                                      {"cu_table": cu_table})
    studies["disjoint_cu_table"] = arm("disjoint (VLM on k CUs, action stage on the other 256 - k)", dur_dj, {},
                                       {"cu_table": cu_dj, "disjoint": True})
    studies["stage_disaggregation_only"] = arm("stage disaggregation only (no restriction)", dur_static[256], {},
                                               {"default_cu": 256})
    studies["monolithic"] = arm("Monolithic", dur_static[256], {"mode": "monolithic"}, {"mode": "monolithic"})
    # queue policies
    for pol in ("rr", "lqf"):
        studies[f"guarded_{pol}"] = arm(f"guarded, {pol.upper()}", dur_lut, {"policy": pol},
                                        {"cu_table": cu_table, "policy": pol})
    # the paper's traffic shape: periodic, random phase per robot, 2 Hz, per-model SLOs
    paper_slo = [{"pi0": 156.0, "smolvla": 50.0, "gr00t": 53.0}.get(n, args.slo_ms) for n in names]
    studies["periodic_2hz_paper_slo_guarded"] = arm("periodic 2 Hz, paper SLOs, guarded", dur_lut, {},
                                                    {"cu_table": cu_table}, rate=2.0, slo_=paper_slo,
                                                    traffic="periodic", r_max=4 * RM)
    studies["periodic_2hz_paper_slo_monolithic"] = arm("periodic 2 Hz, paper SLOs, Monolithic", dur_static[256],
                                                       {"mode": "monolithic"}, {"mode": "monolithic"}, rate=2.0,
                                                       slo_=paper_slo, traffic="periodic", r_max=4 * RM)
    log(f"[serve] studies validated in {time.perf_counter() - t0:.1f} s")
    # per-model GPU robot limits (simulated, each model alone) and the
    # traffic controller's assignment they imply for a two-GPU server
    limits = []
    for i, n in enumerate(names):
        c, _ = serve.robot_limit(dur_lut, i, slo[i], mb, f0, T, E)
        limits.append(max(c, 1))
    pops = [max(1, int(1.5 * limits[0]))] + [max(1, int(0.5 * c / max(1, len(names) - 1))) for c in limits[1:]]
    r, obj, opt = serve.traffic_assign(np.ones((len(names), 2), dtype=int), pops, limits)
    studies["robot_limits_alone_sim"] = {n: c for n, c in zip(names, limits)}
    studies["traffic_controller_2gpu_example"] = {"populations": dict(zip(names, pops)), "assignment": r.tolist(),
                                                  "objective": obj, "optimal": opt}
    # fine-tuned variants: nv variants of each architecture (different weights,
    # same shapes) co-located, robot i -> model i mod (nv * architectures); the
    # variants reuse their architecture's profile
    nv = args.serve_variants
    if nv > 1:
        arch_of = [i % len(names) for i in range(nv * len(names))]
        vdur, vcu = serve.expand_tables(dur_lut, cu_table, arch_of)
        vslo = [args.slo_ms] * len(arch_of)
        vcfgs = [cfgs[a].with_(seed=cfgs[a].seed + 17 * (i // len(names))) for i, a in enumerate(arch_of)]
        vmodels = [models[a] if i < len(names) else vla.Model(c, synth.make_weights(c), device=0)
                   for i, (a, c) in enumerate(zip(arch_of, vcfgs))]
        r_sim, rows = serve.max_robots(vdur, vslo, mb, f0, T, E)
        vv = GpuValidator(vmodels, vcfgs, vslo, f0, args.validate_seconds, js, RM + 4, log_prefix="[serve]")
        best, checks = vv.search(r_sim, RM, mb=mb, cu_table=vcu)
        studies["fine_tuned_variants"] = {"models": [f"{names[a]}-v{i // len(names)}" for i, a in enumerate(arch_of)],
                                          "robots_at_98": best, "chunks_per_s": best * f0, "robots_at_98_sim": r_sim,
                                          "gpu_validation": checks}
        log(f"[serve] {len(arch_of)} co-located variants: {best} robots at >= 98 % on the GPU (simulated {r_sim})")
        for m in vmodels[len(names):]:
            m.close()
    g = studies["guarded_cu_table"]
    result = {"metric": METRIC, "value": float(g["chunks_per_s"]), "unit": "action chunks/s", "n_gpus": 1,
              "dtype": "bf16", "data": "synthetic robot traffic, seeded (Poisson 6000 + epoch, periodic 7000 + epoch)",
              "config": {"workload": "co-located " + " + ".join(f"{n}-shaped" for n in names),
                         "max_batch": mb, "slo_ms": args.slo_ms, "rate_hz": f0, "cu_candidates": cus,
                         "validate_s": args.validate_seconds, "sim_epochs": E, "sim_trace_s": T},
              "cu_table": cu_table.tolist(), "cu_table_disjoint": cu_dj.tolist(),
              "lockstep_ms_lut": (dur_lut / 1e6).round(3).tolist(), "studies": studies}
    for m in models:
        m.close()
    print(json.dumps(result), flush=True)


def counters_main(args):
    """For hardware counter passes (rocprofv3 --pmc): launch only the roofline
    kernel (`--which` projection of the benchmark workload, eagerly, with the
    stage's real buffers) and a 256 MiB device copy of known size."""
    import torch
    from paper_2609_12075_amd import synth, vla
    cfg = synth.CONFIGS[args.config]
    B = args.batch or cfg.max_batch
    m = vla.Model(cfg, synth.make_weights(cfg), device=0)
    m.set_graphs(False)
    inp = synth.make_inputs(cfg, B)
    d = {k: torch.from_numpy(v).to("cuda:0") for k, v in inp.items()}
    kv = m.alloc_kv(B)
    act = torch.empty_like(d["noise"])
    m.prefill(B, d["pixels"], d["text_ids"], kv, state=d.get("state"))
    m.denoise(B, kv, d["noise"], 1, act)
    torch.cuda.synchronize()
    flops, plan = m.replay_gemm(args.which, B, args.roofline_iters)
    src = torch.empty(64 << 20, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    kname = vla.Model.kernel_symbol(plan)
    print(json.dumps({"kernel_symbol": kname, "plan": plan, "flops_per_launch": flops, "launches": args.roofline_iters,
                      "copy_probe_bytes": int(src.numel() * 4), "config": cfg.name, "batch": B}), flush=True)
    m.close()


def sync_costs_main(args):
    """What a hand-off between dependent phases costs: a kernel boundary inside
    a replayed graph (empty kernels, and kernels whose blocks each write 4 or
    16 KiB) against a grid-wide barrier inside one kernel (release add /
    acquire polls at agent scope), with the same writes before and a read of
    another block's slice after each barrier. Median of 5 timings of 200
    boundaries or barriers; one JSON line."""
    import torch
    from paper_2609_12075_amd import vla
    dev = torch.device("cuda:0")
    ts = vla.nonblocking_stream(0)
    s = ts
    n = 200
    buf = torch.zeros(2 * 256 * 4096, dtype=torch.float32, device=dev)
    sink = torch.zeros(256 * 256, dtype=torch.float32, device=dev)
    ctr = torch.zeros(1, dtype=torch.int32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def timed(fn, reps=5):
        out = []
        for _ in range(reps):
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(ts)
            fn()
            b.record(ts)
            torch.cuda.synchronize()
            out.append(a.elapsed_time(b) * 1e3)
        return sorted(out)[len(out) // 2]

    res = {"metric": "hand-off cost between dependent phases", "unit": "us", "count": n}
    for grid in (128, 256):
        for kind, words in ((0, 0), (1, 1024), (1, 4096)):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.stream(ts):
                vla.debug_sync_probe(kind, grid, n, words, buf=buf, sink=sink, stream=s)
                torch.cuda.synchronize()
                g.capture_begin()
                vla.debug_sync_probe(kind, grid, n, words, buf=buf, sink=sink, stream=s)
                g.capture_end()
            torch.cuda.synchronize()
            key = f"kernel_boundary_grid{grid}_{words * 4 // 1024}KiB"
            with torch.cuda.stream(ts):
                res[key] = round(timed(g.replay) / n, 3)
            del g
        for words in (0, 1024, 4096):
            def run():
                ctr.zero_()
                vla.debug_sync_probe(2, grid, n, words, buf=buf, ctr=ctr, err=err, sink=sink, stream=s)
            err.zero_()
            with torch.cuda.stream(ts):
                t = timed(run)
            res[f"grid_barrier_grid{grid}_{words * 4 // 1024}KiB"] = round(t / n, 3)
            res[f"grid_barrier_grid{grid}_{words * 4 // 1024}KiB_overruns"] = int(err.item())
            if int(ctr.item()) != n * grid:
                raise RuntimeError(f"barrier counter ended at {int(ctr.item())}, expected {n * grid}")
        log(f"[sync] grid {grid}: " + ", ".join(f"{k}={v}" for k, v in res.items() if f"grid{grid}_" in k))
    print(json.dumps(res), flush=True)


def stage_flops(c) -> tuple:
    """Algorithmic flops per request of the two stages as the library computes
    them (2 M N K per projection, 4 n_q hd Lq Lk per attention; the joint
    expert's last LLM layer only projects K and V; the patch embedding and the
    batch-independent time conditioning are left out). Returns (prefill,
    action step)."""
    from paper_2609_12075_amd import synth
    hd, D, Hq, Hk = c.head_dim, c.llm_d, c.n_q * c.head_dim, c.n_kv * c.head_dim
    T, P, F = c.tokens_per_img, c.prefix_len, c.llm_mlp
    joint = c.head_kind == synth.HEAD_JOINT
    pre = 0.0
    if c.vit_layers > 0:
        Tv = c.patch_tokens                      # the encoder's sequence per image
        d, f, Ti = c.vit_d, c.vit_mlp, c.n_img * Tv
        pre += c.vit_layers * (2 * Ti * d * 3 * d + 4 * c.n_img * d * Tv * Tv + 2 * Ti * d * d + 2 * 2 * Ti * d * f)
        pre += 2 * (c.n_img * T) * (d * c.pix_shuffle ** 2) * D
    full = c.llm_layers - (1 if joint else 0)
    pre += full * (2 * P * D * (Hq + 2 * Hk) + 4 * c.n_q * hd * P * P + 2 * P * Hq * D + 2 * P * D * 2 * F + 2 * P * F * D)
    if joint:
        pre += 2 * P * D * 2 * Hk
    else:
        Da = c.act_d
        pre += 2 * P * D * Da + 2 * P * Da * c.act_layers * 2 * Da
    Da, Fa, H, A = c.act_d, c.act_mlp, c.horizon, c.action_dim
    if joint:
        step = 2 * H * A * Da + 2 * 2 * H * Da * Da + 2 * H * Da * A
        step += c.act_layers * (2 * H * Da * (Hq + 2 * Hk) + 4 * c.n_q * hd * H * (P + H) + 2 * H * Hq * Da
                                + 2 * H * Da * 2 * Fa + 2 * H * Fa * Da)
    else:
        L = H + 1
        step = 2 * H * A * Da + 2 * H * Da * A
        step += c.act_layers * (2 * L * Da * 3 * Da + 4 * Da * L * L + 2 * L * Da * Da + 2 * L * Da * Da
                                + 4 * Da * L * P + 2 * L * Da * Da + 2 * 2 * L * Da * Fa)
    return float(pre), float(step)


def stages_main(args):
    """Stage times per (config, batch): graph replays of prefill and of the
    whole denoise (N Euler steps) on one stream, median of --stage-reps
    replays after warm-ups, and the algorithmic TFLOP/s and share of the bf16
    MFMA peak they imply."""
    import numpy as np
    import torch
    from paper_2609_12075_amd import synth, vla
    out = {}
    for name in args.stage_configs.split(","):
        base = synth.CONFIGS[name]
        Bs = [int(b) for b in args.stage_batches.split(",") if int(b) <= max(base.max_batch, 1)]
        cfg = base.with_(max_batch=max(Bs))
        m = vla.Model(cfg, synth.make_weights(cfg), device=0)
        torch.cuda.synchronize()
        stream = vla.nonblocking_stream(0)
        pre_f, step_f = stage_flops(cfg)
        peak = PEAK["f32" if cfg.dtype == synth.DTYPE_F32 else "bf16"]
        for B in Bs:
            inp = synth.make_inputs(cfg, B)
            d = {k: torch.from_numpy(v).to("cuda:0") for k, v in inp.items()}
            kv = m.alloc_kv(B)
            act = torch.empty_like(d["noise"])
            torch.cuda.synchronize()

            def med(fn):
                for _ in range(args.stage_warmup):
                    fn()
                torch.cuda.synchronize()
                evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.stage_reps + 1)]
                evs[0].record(stream)
                for i in range(args.stage_reps):
                    fn()
                    evs[i + 1].record(stream)
                torch.cuda.synchronize()
                return float(np.median([evs[i].elapsed_time(evs[i + 1]) for i in range(args.stage_reps)]))
            pre = med(lambda: m.prefill(B, d["pixels"], d["text_ids"], kv, state=d.get("state"), stream=stream))
            den = med(lambda: m.denoise(B, kv, d["noise"], cfg.steps, act, stream=stream))
            step = den / cfg.steps
            rec = {"prefill_ms": round(pre, 4), "adit_step_ms": round(step, 4), "denoise_ms": round(den, 4),
                   "prefill_tflops": round(B * pre_f / pre / 1e9, 2), "adit_tflops": round(B * step_f / step / 1e9, 2)}
            rec["prefill_mfma_frac"] = round(rec["prefill_tflops"] / peak, 4)
            rec["adit_mfma_frac"] = round(rec["adit_tflops"] / peak, 4)
            out[f"{name}:B{B}"] = rec
            log(f"[stages] {name} B={B}: prefill {pre:.3f} ms ({rec['prefill_tflops']} TFLOP/s, "
                f"{100 * rec['prefill_mfma_frac']:.1f} %), ADiT step {step:.4f} ms ({rec['adit_tflops']} TFLOP/s, "
                f"{100 * rec['adit_mfma_frac']:.1f} %)")
            del kv, act, d
        m.close()
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "stage times per config and batch", "reps": args.stage_reps, "warmup": args.stage_warmup,
                      "flops_per_request": {n: stage_flops(synth.CONFIGS[n]) for n in args.stage_configs.split(",")},
                      "stages": out}), flush=True)


def _layer_params(cfg, flat, dtype, prefixes):
    """Oracle parameters (bf16-rounded for bf16 models) of the tensors whose
    names start with one of `prefixes`, in `dtype`."""
    import numpy as np
    from oracle import vla as O
    from paper_2609_12075_amd import synth
    W = {}
    for k, v in synth.weight_views(cfg, flat).items():
        if k.startswith(prefixes):
            src = O.bf16_round(v) if cfg.dtype == synth.DTYPE_BF16 else np.asarray(v, np.float32)
            W[k] = src.astype(dtype)
    return W


def oracle_request_seconds(cfg, flat, dtype):
    """Seconds the CPU oracle needs for one request of `cfg` (batch 1):
    prefill and denoise, each from timed samples scaled by layer counts (one
    ViT block per image, one full LLM block, one action-stage layer per Euler
    step), so a pi0-shaped request costs a few seconds of CPU instead of a
    minute. Inputs are seeded; the oracle's arithmetic does not depend on
    their values."""
    import numpy as np
    from oracle import vla as O
    from paper_2609_12075_amd import synth
    rng = np.random.default_rng(0)
    joint = cfg.head_kind == synth.HEAD_JOINT
    pre_s = 0.0
    if cfg.vit_layers > 0:
        W = _layer_params(cfg, flat, dtype, ("vit.0.",))
        x = rng.standard_normal((cfg.tokens_per_img, cfg.vit_d)).astype(dtype)
        t = time.perf_counter()
        O.vit_layer(cfg, W, 0, x)
        pre_s += cfg.n_img * cfg.vit_layers * (time.perf_counter() - t)
    W = _layer_params(cfg, flat, dtype, ("llm.0.",))
    h = rng.standard_normal((cfg.prefix_len, cfg.llm_d)).astype(dtype)
    t = time.perf_counter()
    O.llm_layer(cfg, W, 0, h, np.arange(cfg.prefix_len))
    pre_s += cfg.llm_layers * (time.perf_counter() - t)
    one = cfg.with_(act_layers=1, llm_layers=1)
    if joint:
        W = _layer_params(cfg, flat, dtype, ("act.0.", "act.in", "act.t1", "act.t2", "act.lnf", "act.out"))
        pre = {"k": [rng.standard_normal((cfg.n_kv, cfg.prefix_len, cfg.head_dim)).astype(dtype)],
               "v": [rng.standard_normal((cfg.n_kv, cfg.prefix_len, cfg.head_dim)).astype(dtype)]}
        fn = O.joint_velocity
    else:
        W = _layer_params(cfg, flat, dtype, ("dit.0.", "dit.t", "dit.ain", "dit.pos", "dit.modf", "dit.out"))
        pre = {"kc": [rng.standard_normal((cfg.prefix_len, cfg.act_d)).astype(dtype)],
               "vc": [rng.standard_normal((cfg.prefix_len, cfg.act_d)).astype(dtype)],
               "state": rng.standard_normal(cfg.act_d).astype(dtype)}
        fn = O.dit_velocity
    x = rng.standard_normal((cfg.horizon, cfg.action_dim)).astype(dtype)
    fn(one, W, pre, x, 1.0)
    t = time.perf_counter()
    fn(one, W, pre, x, 0.5)
    den_s = cfg.steps * cfg.act_layers * (time.perf_counter() - t)
    return pre_s, den_s


def cpu_baseline_colocated(cfgs, flats, budget_s):
    """The CPU oracle on the co-located workload: per model, seconds per
    request (prefill, denoise) in fp64 (the parity precision) and fp32 with
    all BLAS threads, and in fp64 on one core for the SmolVLA-shaped model;
    plus one whole SmolVLA-shaped request end to end as a check of the
    layer-scaled estimate. CPU chunks/s = 2 / (s_pi0 + s_smolvla) (robots
    alternate between the two models)."""
    import numpy as np
    from oracle import vla as O
    from paper_2609_12075_amd import synth
    blas, threads = "unknown", os.cpu_count() or 1
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            blas = f"{info[0].get('internal_api')} {info[0].get('version')} ({info[0].get('threading_layer', '')})"
            threads = int(info[0].get("num_threads", threads))
    except Exception:
        threadpool_limits = None
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    t0 = time.perf_counter()
    # repeat the sampled timings (median of each) until about budget_s of CPU work
    samples = {(c.name, d): [] for c in cfgs for d in ("f64", "f32")}
    reps = 0
    while reps < 1 or (time.perf_counter() - t0 < 0.7 * budget_s and reps < 9):
        for c, f in zip(cfgs, flats):
            for dname, dt in (("f64", np.float64), ("f32", np.float32)):
                samples[(c.name, dname)].append(oracle_request_seconds(c, f, dt))
        reps += 1
    per = {}
    for c in cfgs:
        e = {}
        for dname in ("f64", "f32"):
            pre_s = float(np.median([x[0] for x in samples[(c.name, dname)]]))
            den_s = float(np.median([x[1] for x in samples[(c.name, dname)]]))
            e[dname] = {"prefill_s": round(pre_s, 3), "denoise_s": round(den_s, 3), "request_s": round(pre_s + den_s, 3)}
        per[c.name] = e
    single = None
    smol = [(c, f) for c, f in zip(cfgs, flats) if c.name == "smolvla"]
    if smol and threadpool_limits is not None:
        c, f = smol[0]
        with threadpool_limits(limits=1, user_api="blas"):
            pre_s, den_s = oracle_request_seconds(c, f, np.float64)
        single = {"model": c.name, "request_s": round(pre_s + den_s, 3), "cores": 1}
    check = None
    if smol:
        c, f = smol[0]
        W = O.params(c, f)
        t = time.perf_counter()
        O.run(c, W, synth.make_inputs(c, 1))
        check = {"model": c.name, "measured_request_s": round(time.perf_counter() - t, 3),
                 "estimated_request_s": per[c.name]["f64"]["request_s"]}
        del W
    el = time.perf_counter() - t0
    tot = {d: sum(per[c.name][d]["request_s"] for c in cfgs) for d in ("f64", "f32")}
    n = len(cfgs)
    return {"value": round(n / tot["f64"], 5), "unit": "action chunks/s", "cores": threads, "kind": "oracle",
            "sample": (f"co-located {' + '.join(c.name for c in cfgs)} at batch 1, numpy fp64 on {threads} BLAS "
                       f"threads: one ViT block per image, one LLM block and one action-stage layer per model timed "
                       f"(median of {reps}) and scaled by layer and Euler-step counts, plus one whole "
                       f"SmolVLA-shaped request as a check; {el:.1f} s of CPU"),
            "f32_value": round(n / tot["f32"], 5), "per_model_s": per,
            "single_core": single, "whole_request_check": check, "cpu_model": cpu_model, "blas": blas,
            "host_cpus": os.cpu_count()}


def flops_per_request(c):
    """(prefill, all Euler steps) algorithmic flops of one request."""
    pre, step = stage_flops(c)
    return pre, step * c.steps


def colocated_main(args):
    """The metric: action chunks/s at >= 98 % SLO attainment for the
    co-located pi0-shaped + SmolVLA-shaped workload (see the module
    docstring). Prints one JSON line."""
    import numpy as np
    import torch
    from paper_2609_12075_amd import serve, synth, vla

    names = args.serve_models.split(",")
    f, K = args.rate, args.steps
    mbs = sorted(int(x) for x in args.serve_batches.split(","))
    mb_prof = mbs[-1]
    cfgs = [synth.CONFIGS[n].with_(max_batch=mb_prof) for n in names]
    slo = [args.slo_ms] * len(cfgs)
    cus = [int(x) for x in args.serve_cus.split(",")]
    t_all = time.perf_counter()
    flats = [synth.make_weights(c) for c in cfgs]
    models = [vla.Model(c, w, device=0) for c, w in zip(cfgs, flats)]
    log(f"[bench] models {names} (max_batch {mb_prof}) created in {time.perf_counter() - t_all:.1f} s")
    bufs = serve.alloc_io(models, mb_prof)
    for m, b in zip(models, bufs):          # both hand-off slots hold real prefixes
        m.prefill(mb_prof, b["pixels"], b["text_ids"], b["kv0"], state=b.get("state"))
        m.prefill(mb_prof, b["pixels"], b["text_ids"], b["kv1"], state=b.get("state"))
    torch.cuda.synchronize()
    js = vla.nonblocking_stream(0)          # join stream of every lockstep

    # ---- 1. lockstep table under each VLM CU restriction, profiled once at the
    # largest batch cap; a smaller cap's table is the leading buckets of it
    # (and, per combination, when its action half ends: chunks are delivered
    # then with --delivery adit)
    t0 = time.perf_counter()
    prof_all, adit_all = serve.profile_locksteps(models, bufs, mb_prof, cus, reps=3, log=log, join_stream=js,
                                                 with_adit=True)
    log(f"[bench] profiled {prof_all.size} lockstep entries in {time.perf_counter() - t0:.1f} s")
    if args.dump_profile:
        np.savez(args.dump_profile, prof=prof_all, adit=adit_all, cus=np.asarray(cus), models=np.asarray(names))

    # ---- 2. simulated sweep per batch cap (max_batch of the scheduler)
    robots = list(range(1, args.serve_max_robots + 1))
    early = args.delivery == "adit"
    by_mb = {}
    for mbx in mbs:
        nbx = serve.n_buckets(mbx)
        sub = np.ascontiguousarray(prof_all[:, :, :nbx, :, :nbx])
        ct, dl, al = serve.best_cu_table(sub, cus, np.ascontiguousarray(adit_all[:, :, :nbx, :, :nbx]))
        rows_x, r_x = serve.sweep_robots(dl, slo, mbx, robots, f, args.serve_seconds, args.serve_epochs,
                                         adit_ns=al if early else None)
        by_mb[mbx] = {"robots_at_98_sim": r_x, "cu_table": ct, "dur": dl, "adit": al, "sub": sub, "sweep": rows_x}
        log(f"[bench] max_batch {mbx}: simulated {r_x} robots at >= 98 % "
            f"({args.serve_epochs} x {args.serve_seconds:.0f} s traces, delivery {args.delivery})")
    mb = max(mbs, key=lambda x: (by_mb[x]["robots_at_98_sim"], -x))
    prof, cu_table, dur_lut = by_mb[mb]["sub"], by_mb[mb]["cu_table"], by_mb[mb]["dur"]
    adit_lut = by_mb[mb]["adit"]
    rows, r_sim = by_mb[mb]["sweep"], by_mb[mb]["robots_at_98_sim"]
    # the other delivery point at the chosen cap, simulated, for comparison
    _, r_other = serve.sweep_robots(dur_lut, slo, mb, robots, f, args.serve_seconds, args.serve_epochs,
                                    adit_ns=None if early else adit_lut)
    log(f"[bench] serving with max_batch {mb} (simulated with the other delivery point: {r_other} robots)")
    nb = serve.n_buckets(mb)
    full = nb - 1                            # bucket of the serving batch

    # ---- timed steps: saturated locksteps cycling through the model pairings
    # (model k mod n's VLM stage beside model k + 1 mod n's action stage)
    n_models = len(models)

    def lockstep(k):
        mv, ma = k % n_models, (k + 1) % n_models
        xv, xa = bufs[mv], bufs[ma]
        vla.step(models[mv], mb, xv["pixels"], xv["text_ids"], xv["kv0"], models[ma], mb, xa["kv1"], xa["noise"],
                 cfgs[ma].steps, xa["act1"], vlm_cu_count=int(cu_table[mv, full, ma, full]), state=xv.get("state"),
                 join_stream=js)
    for k in range(args.warmup):
        lockstep(k)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    t_wall = time.perf_counter()
    evs[0].record(js)
    for i in range(K):
        lockstep(args.warmup + i)
        evs[i + 1].record(js)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_per_step = evs[0].elapsed_time(evs[K]) / K
    log(f"[bench] {K} saturated locksteps: {ms_per_step:.3f} ms/step (wall {wall * 1e3 / K:.3f}), "
        f"{mb * 1e3 / ms_per_step:.1f} chunks/s")

    # ---- 3. real-time validation on the GPU (online executor, per-robot inputs)
    t0 = time.perf_counter()
    val = GpuValidator(models, cfgs, slo, f, args.validate_seconds, js, args.serve_max_robots + 2)
    best, checks = val.search(r_sim, args.serve_max_robots, mb=mb, cu_table=cu_table, delivery=args.delivery)
    value = best * f
    log(f"[bench] GPU-validated: {best} robots at >= 98 % -> {value} action chunks/s "
        f"({time.perf_counter() - t0:.1f} s of validation)")

    # ---- stage times alone at the serving batch (table entries with one half empty, unrestricted)
    ki = cus.index(256) if 256 in cus else len(cus) - 1
    stages = {}
    for i, c in enumerate(cfgs):
        pre_ms = prof[ki, i, full, 0, 0] / 1e6
        den_ms = prof[ki, 0, 0, i, full] / 1e6
        pf, df = flops_per_request(c)
        stages[c.name] = {"batch": mb, "prefill_ms": round(pre_ms, 3), "denoise_ms": round(den_ms, 3),
                          "adit_step_ms": round(den_ms / c.steps, 4),
                          "prefill_mfma_frac": round(mb * pf / (pre_ms * 1e-3) / 1e12 / PEAK["bf16"], 4),
                          "adit_mfma_frac": round(mb * df / (den_ms * 1e-3) / 1e12 / PEAK["bf16"], 4)}

    # ---- roofline: the replayable projection with the most time per served pair of batches
    kern = {}
    for i, (c, m) in enumerate(zip(cfgs, models)):
        for which in (0, 1, 2, 3, 4):
            if which == 4 and c.vit_layers == 0:
                continue
            m.replay_gemm(which, mb, 3, stream=js)
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(js)
            flops, plan = m.replay_gemm(which, mb, args.roofline_iters, stream=js)
            b.record(js)
            torch.cuda.synchronize()
            us = a.elapsed_time(b) * 1e3 / args.roofline_iters
            joint = c.head_kind == synth.HEAD_JOINT
            n_launch = {0: c.llm_layers - (1 if joint else 0), 1: c.llm_layers - (1 if joint else 0),
                        2: c.act_layers * c.steps, 3: c.act_layers * c.steps, 4: c.vit_layers}[which]
            kern[(c.name, which)] = {"flops": flops, "us": us, "plan": plan, "launches": n_launch,
                                     "symbol": vla.Model.kernel_symbol(plan)}
            log(f"[bench] kernel {c.name} {GEMM_NAMES[which]}: {us:.2f} us/launch, {flops / us / 1e6:.1f} TFLOP/s, "
                f"{n_launch} launches per batch, plan {plan}")
    dom = max(kern, key=lambda k: kern[k]["us"] * kern[k]["launches"])
    kd = kern[dom]
    achieved = kd["flops"] / kd["us"] / 1e6
    traffic = None
    tf = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tf):
        from paper_2609_12075_amd import profsum
        trec = json.load(open(tf)).get(f"{dom[0]}:B{mb}:{kd['symbol']}")
        if trec and trec.get("source_hash") == profsum.source_hash():
            traffic = trec["traffic_bytes"]
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK["bf16"], "unit": "TFLOP/s",
                "frac": round(achieved / PEAK["bf16"], 4), "traffic": traffic,
                "kernel": f"{dom[0]}-shaped {GEMM_NAMES[dom[1]]}", "kernel_symbol": kd["symbol"],
                "flops_per_launch": kd["flops"], "us_per_launch": round(kd["us"], 3),
                "launches_per_batch": kd["launches"], "batch": mb}

    out = {
        "metric": METRIC, "value": float(value), "unit": "action chunks/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": ("synthetic: seeded Poisson robot traffic, per-robot U[0,1) pixels, U[0,1000) text ids, N(0,1) "
                 "noise; random-init N(0,0.02) weights"),
        "config": {"workload": "co-located " + " + ".join(f"{n}-shaped" for n in names) +
                               f", Poisson {f:g} Hz per robot, {args.slo_ms:g} ms SLO, robots at >= 98 % attainment",
                   "models": names, "rate_hz": f, "slo_ms": args.slo_ms, "max_batch": mb, "policy": "esf",
                   "chunk_delivery": ("when the request's action stage ends" if early else
                                      "at the end of the lockstep that ran its action stage"),
                   "vlm_cu_candidates": cus, "parallelism": "single GPU, two streams (VLM CU-restricted)"},
        "robots_at_98": best, "gpu_validation": checks,
        "robots_at_98_sim": r_sim, "sim": {"epochs": args.serve_epochs, "trace_s": args.serve_seconds,
                                           "sweep": rows},
        "robots_at_98_sim_by_max_batch": {str(x): by_mb[x]["robots_at_98_sim"] for x in mbs},
        "robots_at_98_sim_other_delivery": {"delivery": "lockstep" if early else "adit", "robots": r_other},
        "saturated_lockstep_chunks_per_s": round(mb * 1e3 / ms_per_step, 2),
        "stages": stages,
        "adit_step_ms": {n: stages[n]["adit_step_ms"] for n in stages},
        "cu_table": cu_table.tolist(), "lockstep_ms_lut": (dur_lut / 1e6).round(3).tolist(),
        "adit_end_ms_lut": (adit_lut / 1e6).round(3).tolist(),
        "roofline": roofline,
        "kernels": {f"{k[0]}:{GEMM_NAMES[k[1]]}": {"us": round(v["us"], 3), "launches_per_batch": v["launches"],
                                                    "tflops": round(v["flops"] / v["us"] / 1e6, 2),
                                                    "mfma_frac": round(v["flops"] / v["us"] / 1e6 / PEAK["bf16"], 4),
                                                    "symbol": v["symbol"]}
                    for k, v in kern.items()},
    }
    for m in models:
        m.close()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline_colocated(cfgs, flats, args.cpu_seconds)
    out["bench_wall_s"] = round(time.perf_counter() - t_all, 1)
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="smolvla")
    ap.add_argument("--batch", type=int, default=0, help="requests per stage batch (default: max_batch)")
    ap.add_argument("--cu", type=int, default=0,
                    help="compute units the VLM stream may use (multiple of 8); 0: the fastest of --cu-candidates, "
                         "profiled before the timed steps")
    ap.add_argument("--cu-candidates", default="256,192,128,64",
                    help="VLM CU counts to profile (multiples of 32 keep every shader engine equally populated)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--roofline-iters", type=int, default=50)
    ap.add_argument("--copy-probe", action="store_true", help="also run a 256 MiB device copy (counter scaling)")
    ap.add_argument("--counters", action="store_true", help="launch only the roofline kernel and a copy (PMC passes)")
    ap.add_argument("--which", type=int, default=2, help="projection for --counters (see vla_debug.h)")
    ap.add_argument("--lockstep", action="store_true",
                    help="one model's saturated locksteps (--config, --batch, --cu) instead of the serving metric")
    ap.add_argument("--rate", type=float, default=10.0, help="requests per second per robot (default workload)")
    ap.add_argument("--serve", action="store_true", help="co-located serving studies (controls, policies, traffic)")
    ap.add_argument("--serve-models", default="pi0,smolvla")
    ap.add_argument("--serve-batch", type=int, default=4, help="batch cap of the --serve studies")
    ap.add_argument("--serve-batches", default="2,4,8",
                    help="batch caps the default workload tries (simulated); the best is validated on the GPU")
    ap.add_argument("--serve-cus", default="64,128,192,256")
    ap.add_argument("--serve-rates", default="10,20,30")
    ap.add_argument("--serve-max-robots", type=int, default=32)
    ap.add_argument("--serve-seconds", type=float, default=30.0)
    ap.add_argument("--serve-epochs", type=int, default=5)
    ap.add_argument("--serve-no-validate", action="store_true")
    ap.add_argument("--serve-variants", type=int, default=2, help="fine-tuned variants per architecture in the co-location study")
    ap.add_argument("--validate-seconds", type=float, default=20.0,
                    help="seconds of real-time traffic per GPU validation run")
    ap.add_argument("--slo-ms", type=float, default=100.0)
    ap.add_argument("--delivery", choices=("adit", "lockstep"), default="lockstep",
                    help="when a request completes: at the end of the lockstep that ran its action stage "
                         "(default) or when that action stage ends")
    ap.add_argument("--dump-profile", default="",
                    help="write the lockstep profile (durations and action-half ends per CU count) to this .npz")
    ap.add_argument("--sync-costs", action="store_true",
                    help="kernel-boundary vs in-kernel grid-barrier cost (what fusing dependent phases would trade)")
    ap.add_argument("--stages", action="store_true", help="stage times per config and batch instead of the lockstep bench")
    ap.add_argument("--stage-configs", default="tiny,smolvla,smolvla_vit,pi0,gr00t")
    ap.add_argument("--stage-batches", default="1,4,16")
    ap.add_argument("--stage-reps", type=int, default=200)
    ap.add_argument("--stage-warmup", type=int, default=20)
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the serving hot path here is a single-GPU build "
              "(replicas on more GPUs would share nothing on the hot path). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.serve:
        serve_main(args)
        return
    if args.counters:
        counters_main(args)
        return
    if args.stages:
        stages_main(args)
        return
    if args.sync_costs:
        sync_costs_main(args)
        return
    if not args.lockstep:
        colocated_main(args)
        return

    import numpy as np
    import torch
    from paper_2609_12075_amd import synth, vla

    cfg = synth.CONFIGS[args.config]
    B = args.batch or cfg.max_batch
    N = cfg.steps
    dtype = "bf16" if cfg.dtype == synth.DTYPE_BF16 else "f32"
    dev = torch.device("cuda:0")
    log(f"[bench] config {cfg.name} B={B} steps/chunk={N} vlm_cu={args.cu or 'auto'}")
    t0 = time.perf_counter()
    weights = synth.make_weights(cfg)
    m = vla.Model(cfg, weights, device=0)
    log(f"[bench] model created in {time.perf_counter() - t0:.1f} s")
    inp = synth.make_inputs(cfg, B)
    d = {k: torch.from_numpy(v).to(dev) for k, v in inp.items()}
    kv = [m.alloc_kv(B), m.alloc_kv(B)]
    act = [torch.empty_like(d["noise"]), torch.empty_like(d["noise"])]
    # every timed launch goes to one non-blocking stream: vla_step runs the
    # action half on it directly (no cross-queue wait pending during the graph)
    torch.cuda.synchronize()
    stream = vla.nonblocking_stream(0)

    def lockstep(k):
        # VLM stage of batch k into kv[k % 2] alongside the action stage of batch k - 1
        adit_b = B if k > 0 else 0
        vla.step(m, B, d["pixels"], d["text_ids"], kv[k % 2], m, adit_b, kv[(k - 1) % 2], d["noise"], N,
                 act[(k - 1) % 2], vlm_cu_count=args.cu, state=d.get("state"), join_stream=stream)

    auto_cu = args.cu == 0
    if auto_cu:
        args.cu = 256
    t0 = time.perf_counter()
    for k in range(args.warmup):
        lockstep(k)
    torch.cuda.synchronize()
    log(f"[bench] warmup ({args.warmup} locksteps incl. graph capture) {time.perf_counter() - t0:.1f} s")

    # The VLM stream's CU restriction for this (VLM batch, action batch)
    # combination: the fastest candidate in a short profile (the paper's
    # offline restriction table, for the one combination the benchmark runs).
    # Two passes over the candidates, 6 timed locksteps each, averaged, so a
    # momentary slowdown does not decide the choice.
    cu_profile = None
    if auto_cu:
        cands = [int(x) for x in args.cu_candidates.split(",")]
        sums = {cu: 0.0 for cu in cands}
        for _ in range(2):
            for cu in cands:
                args.cu = cu
                for k in range(1, 3):
                    lockstep(k)
                torch.cuda.synchronize()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                for k in range(1, 7):
                    lockstep(k)
                b.record(stream)
                torch.cuda.synchronize()
                sums[cu] += a.elapsed_time(b) / 6
        cu_profile = {cu: round(sums[cu] / 2, 4) for cu in cands}
        args.cu = min(cu_profile, key=cu_profile.get)
        log(f"[bench] lockstep ms by VLM CU count {cu_profile}: using {args.cu}")

    K = args.steps
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(K + 2)]
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    evs[0].record(stream)
    for i in range(K):
        lockstep(args.warmup + i)
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    # one more lockstep drains the last timed batch (for its latency only)
    lockstep(args.warmup + K)
    evs[K + 1].record(stream)
    torch.cuda.synchronize()
    elapsed_ms = evs[0].elapsed_time(evs[K])
    ms_per_step = elapsed_ms / K
    value = B * K / (elapsed_ms / 1e3)
    steps_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(K + 1)]
    # a batch admitted at lockstep i finishes at the end of lockstep i + 1
    lat = [steps_ms[i] + steps_ms[i + 1] for i in range(K)]
    slo = SLO_MS.get(cfg.name, 100.0)
    attain = float(np.mean([x <= slo for x in lat]))
    log(f"[bench] {K} locksteps: {ms_per_step:.3f} ms/step, {value:.1f} chunks/s (wall {wall * 1e3 / K:.3f} ms/step)")

    # ---- stages alone (graph replays on the same stream)
    def time_alone(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    pre_ms = time_alone(lambda: m.prefill(B, d["pixels"], d["text_ids"], kv[0], state=d.get("state"), stream=stream))
    den_ms = time_alone(lambda: m.denoise(B, kv[0], d["noise"], N, act[0], stream=stream))
    log(f"[bench] alone: prefill {pre_ms:.3f} ms, denoise {den_ms:.3f} ms ({den_ms / N:.3f} ms/step)")

    # ---- roofline of the projection kernels (HIP events around back-to-back launches)
    kern = {}
    for which in (0, 1, 2, 3):
        m.replay_gemm(which, B, 3, stream=stream)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        flops, plan = m.replay_gemm(which, B, args.roofline_iters, stream=stream)
        b.record(stream)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / args.roofline_iters
        kern[which] = (flops, us, plan)
        log(f"[bench] kernel {GEMM_NAMES[which]}: {us:.2f} us/launch, {flops / us / 1e6:.1f} TFLOP/s, plan {plan}")
    # The roofline entry: of the gate/up projections that run as one kernel
    # (no K split) whose instantiation (tile, epilogue) no other projection of
    # this workload uses, so rocprof's per-kernel average is this launch's
    # duration: the one with the most time per lockstep (launches x duration).
    per_step = {w: n for w, n in ((0, cfg.llm_layers - 1), (2, cfg.act_layers * N)) if kern[w][2]["splits"] == 1}
    dom = max(per_step, key=lambda w: kern[w][1] * per_step[w])
    flops, us, plan = kern[dom]
    kname = vla.Model.kernel_symbol(plan)
    achieved = flops / us / 1e6
    traffic = None
    tf = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tf):
        # HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs, valid
        # only while the kernel source is the one the counters were taken on
        from paper_2609_12075_amd import profsum
        rec = json.load(open(tf)).get(f"{cfg.name}:B{B}:{kname}")
        if rec and rec.get("source_hash") == profsum.source_hash():
            traffic = rec["traffic_bytes"]
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK[dtype], "unit": "TFLOP/s",
                "frac": round(achieved / PEAK[dtype], 4), "traffic": traffic,
                "kernel": GEMM_NAMES[dom], "kernel_symbol": kname, "flops_per_launch": flops,
                "us_per_launch": round(us, 3), "launches_per_step": per_step[dom]}

    out = {
        "metric": "saturated lockstep throughput of one model (not the serving metric)", "value": round(value, 2),
        "unit": "action chunks/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype,
        "data": "synthetic (seeded U[0,1) pixels, U[0,1000) text ids, N(0,1) noise; random-init N(0,0.02) weights)",
        "config": {"workload": f"{cfg.name}-shaped VLA, one lockstep = prefill(batch k) || denoise(batch k-1)",
                   "batch": B, "euler_steps": N, "prefix_tokens": cfg.prefix_len, "horizon": cfg.horizon,
                   "vlm_cu_count": args.cu, "parallelism": "single GPU, two streams"},
        "lockstep_ms_by_vlm_cu": cu_profile,
        "adit_step_ms": round(den_ms / N, 4), "prefill_ms": round(pre_ms, 4), "denoise_ms": round(den_ms, 4),
        "chunk_latency_ms_max": round(max(lat), 3), "slo_ms": slo, "slo_attainment_closed_loop": attain,
        "roofline": roofline,
        "kernels": {GEMM_NAMES[w]: {"us": round(kern[w][1], 3), "tflops": round(kern[w][0] / kern[w][1] / 1e6, 2),
                                    "mfma_frac": round(kern[w][0] / kern[w][1] / 1e6 / PEAK[dtype], 4),
                                    "k_ranges": kern[w][2]["splits"]}
                    for w in kern},
    }
    if args.copy_probe:
        # a plain device copy of known size, to scale hardware byte counters
        src = torch.empty(64 << 20, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        out["copy_probe_bytes"] = int(src.numel() * 4)
    if not args.no_cpu_baseline:
        log(f"[bench] CPU oracle baseline (~{args.cpu_seconds:.0f} s)")
        out["cpu_baseline"] = cpu_baseline(cfg, weights, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    m.close()


if __name__ == "__main__":
    main()
