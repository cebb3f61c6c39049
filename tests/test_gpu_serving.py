"""The scheduler driving the GPU (vla_step on CU-masked streams, wall clock):
two co-located models, every request served, records consistent with the
serving rules, and the served actions identical to standalone runs."""
import numpy as np
import pytest

from paper_2609_12075_amd import synth
from tests.gpu_util import log, model, rel_l2, run

pytestmark = pytest.mark.gpu

A = synth.CONFIGS["tiny"]
B = synth.reduced(synth.CONFIGS["smolvla"], max_batch=4)


def test_scheduler_on_gpu_two_models():
    import torch
    from paper_2609_12075_amd import serve
    ma, mb = model(A), model(B)
    mbatch = 4
    bufs = serve.alloc_io([ma, mb], mbatch)
    s = serve.Scheduler([100.0, 100.0], mbatch, "esf")
    s.set_gpu([ma, mb], bufs)
    s.set_cu(192)
    arr = synth.poisson_arrivals(6, 20.0, 1.0, epoch=0, n_models=2)
    log(f"[serving] {len(arr)} requests over 1 s, 6 robots at 20 Hz")
    req, ls = s.run(arr, drain_ns=int(2e9))
    torch.cuda.synchronize()
    s.close()
    assert (req["t_done_ns"] > 0).all(), "every request served"
    assert (req["t_done_ns"] > req["t_vlm_start_ns"]).all()
    assert (req["t_vlm_start_ns"] >= req["t_arrival_ns"]).all()
    assert int(ls["vlm_batch"].sum()) == len(arr) == int(ls["adit_batch"].sum())
    for x in ls:
        assert x["vlm_batch"] in (0, 1, 2, 4) and x["cu_count"] == 192
    log(f"[serving] {len(ls)} locksteps, attainment {serve.attainment(req):.3f}, p99 {serve.p99_ms(req):.2f} ms")
    # the last action batch of each model equals a standalone run on the same rows
    for m, cfg in ((0, A), (1, B)):
        last = [x for x in ls if x["adit_model"] == m][-1]
        b = int(last["adit_batch"])
        slot = 1 - int(last["slot"])      # the action half reads the previous lockstep's slot
        got = bufs[m]["act%d" % slot][:b].cpu().numpy()
        ref, _ = run(cfg, synth.make_inputs(cfg, b))
        np.testing.assert_array_equal(got, ref)


def test_monolithic_on_gpu():
    """The Monolithic control on the GPU: each batch runs the VLM stage and then
    the action stage back to back; every request is served and the last
    batch's actions equal a standalone run."""
    import torch
    from paper_2609_12075_amd import serve
    ma, mb = model(A), model(B)
    mbatch = 4
    bufs = serve.alloc_io([ma, mb], mbatch)
    s = serve.Scheduler([100.0, 100.0], mbatch, "esf", "monolithic")
    s.set_gpu([ma, mb], bufs)
    arr = synth.poisson_arrivals(4, 20.0, 0.5, epoch=1, n_models=2)
    log(f"[serving] monolithic: {len(arr)} requests over 0.5 s")
    req, ls = s.run(arr, drain_ns=int(2e9))
    torch.cuda.synchronize()
    s.close()
    assert (req["t_done_ns"] > 0).all()
    assert (ls["vlm_model"] == ls["adit_model"]).all() and (ls["vlm_batch"] == ls["adit_batch"]).all()
    assert int(ls["vlm_batch"].sum()) == len(arr)
    for m, cfg in ((0, A), (1, B)):
        last = [x for x in ls if x["vlm_model"] == m][-1]
        b = int(last["vlm_batch"])
        got = bufs[m]["act0"][:b].cpu().numpy()
        ref, _ = run(cfg, synth.make_inputs(cfg, b))
        np.testing.assert_array_equal(got, ref)


C = synth.reduced(synth.CONFIGS["gr00t"], vit_layers=1, max_batch=2)


def _served_batches(arr, ls, n_models):
    """Request indices of every VLM batch, in lockstep order: each model's
    FIFO admits its requests in arrival order."""
    fifo = [[i for i in range(len(arr)) if int(arr["model"][i]) == m] for m in range(n_models)]
    out = []
    for x in ls:
        b, m = int(x["vlm_batch"]), int(x["vlm_model"])
        if b:
            out.append((m, fifo[m][:b]))
            fifo[m] = fifo[m][b:]
    return out


@pytest.mark.parametrize("disjoint,delivery", [(False, "lockstep"), (True, "lockstep"), (False, "adit")],
                         ids=["guarded", "disjoint", "guarded-early-delivery"])
def test_online_executor_gathers_and_scatters_per_request(disjoint, delivery):
    """Requests bring their own seeded inputs (row i of the generators for
    request i) and their own output buffers; the library gathers them into
    its stage rows and scatters each chunk back. Every chunk equals a
    standalone run of the batch it was served in (same rows, same order),
    so a wrong gather or scatter row fails; DiT requests alternate between a
    given state and none (zeros). Both CU partitions: the guarded one (only
    the VLM half restricted) and the disjoint one; and chunks delivered as
    soon as their action half ends (copied out on the delivery stream while
    the VLM half may still run), timed inside their lockstep."""
    import torch
    from paper_2609_12075_amd import serve
    cfgs = [A, B, C]
    ms = [model(c) for c in cfgs]
    mbatch = 2
    s = serve.Scheduler([100.0, 100.0, 100.0], mbatch, "esf")
    s.set_gpu_online(ms)
    s.set_cu(128)
    s.set_disjoint(disjoint)      # disjoint: the action half on the other 128 CUs
    s.set_delivery(delivery)
    arr = synth.poisson_arrivals(6, 15.0, 0.8, epoch=3, n_models=3)
    log(f"[serving] online: {len(arr)} requests, 3 models")
    ins, outs, ios, keep = [], [], [], []
    for i in range(len(arr)):
        cfg = cfgs[int(arr["model"][i])]
        inp = synth.make_inputs(cfg, 1, first_row=i)
        if "state" in inp and i % 2:
            inp["state"] = None                      # no state: the library gathers zeros
        d = {k: torch.from_numpy(v[0]).cuda() for k, v in inp.items() if v is not None}
        o = torch.full((cfg.horizon, cfg.action_dim), float("nan"), device="cuda")
        ins.append(inp); outs.append(o); keep.append(d)
        ios.append(serve.Scheduler.request_io(d["pixels"], d["text_ids"], d["noise"], o, d.get("state")))
    req, ls = s.run(arr, drain_ns=int(3e9), ios=ios)
    torch.cuda.synchronize()
    s.close()
    assert (req["t_done_ns"] > 0).all(), "every request served"
    log(f"[serving] online: {len(ls)} locksteps, attainment {serve.attainment(req):.3f}")
    assert ((ls["t_start_ns"] <= ls["t_chunks_ns"]) & (ls["t_chunks_ns"] <= ls["t_end_ns"])).all()
    if delivery == "lockstep":
        assert (ls["t_chunks_ns"] == ls["t_end_ns"]).all()
    # every request completes at its action lockstep's delivery time
    chunk_times = sorted(int(x["t_chunks_ns"]) for x in ls if x["adit_batch"] > 0)
    assert set(int(t) for t in req["t_done_ns"]) <= set(chunk_times)
    for m, idx in _served_batches(arr, ls, 3):
        cfg = cfgs[m]
        batch = {k: np.concatenate([ins[i][k] for i in idx]) for k in ("pixels", "text_ids", "noise")}
        if cfg.head_kind == synth.HEAD_DIT:
            batch["state"] = np.stack([ins[i]["state"][0] if ins[i]["state"] is not None
                                       else np.zeros(cfg.state_dim, np.float32) for i in idx])
        ref, _ = run(cfg, batch)
        for j, i in enumerate(idx):
            np.testing.assert_array_equal(outs[i].cpu().numpy(), ref[j], err_msg=f"request {i} model {m}")


def test_online_calls_on_gpu_with_cu_table():
    """submit / run_lockstep / poll driven from the host on the GPU, with a
    CU restriction table per (VLM model, batch, action model, batch): every
    lockstep record carries the table's entry for its combination and every
    completion's chunk matches its own batch-1 run to the batch-invariance
    bound."""
    import torch
    from paper_2609_12075_amd import serve
    cfgs = [A, B]
    ms = [model(c) for c in cfgs]
    mbatch = 2
    s = serve.Scheduler([100.0, 100.0], mbatch, "esf")
    s.set_gpu_online(ms)
    nb = serve.n_buckets(mbatch)
    table = np.zeros((2, nb, 2, nb), np.int32)
    for mv in range(2):
        for bv in range(nb):
            for ma in range(2):
                for ba in range(nb):
                    table[mv, bv, ma, ba] = [64, 128, 192, 256][(mv + bv + ma + ba) % 4]
    s.set_cu(256, table)
    outs, keep, ids = {}, [], []
    for i in range(8):
        m = i % 2
        cfg = cfgs[m]
        inp = synth.make_inputs(cfg, 1, first_row=20 + i)
        d = {k: torch.from_numpy(v[0]).cuda() for k, v in inp.items()}
        o = torch.full((cfg.horizon, cfg.action_dim), float("nan"), device="cuda")
        keep.append(d)
        outs[100 + i] = (m, o, inp)
        s.submit(100 + i, m, s.clock_ns(), serve.Scheduler.request_io(d["pixels"], d["text_ids"], d["noise"], o))
    recs, comps = [], []
    while s.pending():
        r = s.run_lockstep()
        recs.append(r)
        comps.extend(s.poll())
    torch.cuda.synchronize()
    s.close()
    assert sorted(int(c["id"]) for c in comps) == sorted(outs)
    for r in recs:
        mv, bv, ma, ba = int(r["vlm_model"]), int(r["vlm_batch"]), int(r["adit_model"]), int(r["adit_batch"])
        exp = table[max(mv, 0), serve.bucket(bv), max(ma, 0), serve.bucket(ba)]
        assert int(r["cu_count"]) == exp, (mv, bv, ma, ba)
    for c in comps:
        m, o, inp = outs[int(c["id"])]
        ref, _ = run(cfgs[m], inp)
        got = o.cpu().numpy()
        assert np.isfinite(got).all()
        assert rel_l2(got, ref[0].astype(np.float64)) <= (1e-5 if cfgs[m].dtype == synth.DTYPE_F32 else 2e-3)
