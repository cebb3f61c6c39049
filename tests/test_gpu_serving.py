"""The scheduler driving the GPU (vla_step on CU-masked streams, wall clock):
two co-located models, every request served, records consistent with the
serving rules, and the served actions identical to standalone runs."""
import numpy as np
import pytest

from paper_2609_12075_amd import synth
from tests.gpu_util import log, model, run

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
