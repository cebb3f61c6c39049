"""End-to-end parity of the HIP path (through the C ABI) against the CPU
oracle on seeded inputs, plus the bit-exact bookkeeping properties:
determinism, row permutation, batch-size invariance, prefix KV untouched by
the action stage, graphs vs direct launches, and lockstep co-execution.

Tolerances (final actions, rel-L2 over [B, H, A]): 1e-4 for the fp32 model,
2e-2 for bf16 models."""
import numpy as np
import pytest

from paper_2609_12075_amd import synth
from tests.gpu_util import check_chunk, drop_model, kv_arrays, log, model, oracle_run, rel_l2, run, to_dev

pytestmark = pytest.mark.gpu

TINY = synth.CONFIGS["tiny"]
SMOL_R = synth.reduced(synth.CONFIGS["smolvla"], max_batch=4)
PI0_R = synth.reduced(synth.CONFIGS["pi0"], vit_layers=2, max_batch=3)
GR00T_R = synth.reduced(synth.CONFIGS["gr00t"], vit_layers=2, max_batch=3)

SMOLVIT_R = synth.reduced(synth.CONFIGS["smolvla_vit"], vit_layers=2, max_batch=3)

TOL = {synth.DTYPE_F32: 1e-4, synth.DTYPE_BF16: 2e-2}


def check_parity(cfg, B, steps=None, with_state=True):
    inp = synth.make_inputs(cfg, B)
    if not with_state and "state" in inp:
        inp = {k: v for k, v in inp.items() if k != "state"}
    act, kv = run(cfg, inp, steps=steps)
    ref, pre = oracle_run(cfg, inp, steps=steps)
    check_chunk(act, ref, inp["noise"], TOL[cfg.dtype], f"{cfg.name} B={B}")
    # prefix hand-off
    if cfg.head_kind == synth.HEAD_JOINT:
        K = kv_arrays(cfg, kv, B)
        for l in range(cfg.llm_layers):
            rk = rel_l2(K[l, 0], np.stack([p["k"][l] for p in pre]))
            rv = rel_l2(K[l, 1], np.stack([p["v"][l] for p in pre]))
            assert rk <= TOL[cfg.dtype] and rv <= TOL[cfg.dtype], (l, rk, rv)
    else:
        xkv, st = kv_arrays(cfg, kv, B)
        for l in range(cfg.act_layers):
            rk = rel_l2(xkv[:, :, l, 0], np.stack([p["kc"][l] for p in pre]))
            rv = rel_l2(xkv[:, :, l, 1], np.stack([p["vc"][l] for p in pre]))
            assert rk <= TOL[cfg.dtype] and rv <= TOL[cfg.dtype], (l, rk, rv)
        assert rel_l2(st, np.stack([p["state"] for p in pre])) <= TOL[cfg.dtype]
    return act


@pytest.mark.parametrize("B", [1, 3])
def test_tiny_fp32(B):
    check_parity(TINY, B)


@pytest.mark.parametrize("B", [1, 3])
def test_smolvla_reduced(B):
    check_parity(SMOL_R, B)


@pytest.mark.parametrize("B", [1, 2])
def test_pi0_reduced(B):
    check_parity(PI0_R, B)


@pytest.mark.parametrize("B,with_state", [(1, True), (2, True), (2, False)])
def test_gr00t_reduced(B, with_state):
    check_parity(GR00T_R, B, with_state=with_state)


@pytest.mark.parametrize("B", [1, 3])
def test_smolvla_vision_encoder_reduced(B):
    """SmolVLA-shaped model with its vision encoder (512 x 512 images, patch
    16, 4 x 4 token merge), two ViT layers."""
    check_parity(SMOLVIT_R, B)


def test_smolvla_vision_encoder_full_size_sampled_rows():
    """The whole 12-layer vision encoder with the 16-layer LLM and action
    expert at batch 16; the oracle evaluates rows 0 and 15."""
    cfg = synth.CONFIGS["smolvla_vit"]
    B = cfg.max_batch
    inp = synth.make_inputs(cfg, B)
    act, _ = run(cfg, inp)
    rows = [0, B - 1]
    ref, _ = oracle_run(cfg, inp, rows=rows)
    check_chunk(act[rows], ref, inp["noise"][rows], 2e-2, f"smolvla_vit full B={B} rows {rows}")
    drop_model(cfg)


def test_steps_one_and_max_batch():
    check_parity(SMOL_R, SMOL_R.max_batch, steps=1)


def test_smolvla_full_size_sampled_rows():
    """Full SmolVLA-shaped model at its largest batch; the oracle evaluates two
    rows (rows are independent, so a sample suffices)."""
    cfg = synth.CONFIGS["smolvla"]
    B = cfg.max_batch
    inp = synth.make_inputs(cfg, B)
    act, _ = run(cfg, inp)
    rows = [0, B - 1]
    ref, _ = oracle_run(cfg, inp, rows=rows)
    check_chunk(act[rows], ref, inp["noise"][rows], 2e-2, f"smolvla full B={B} rows {rows}")


# Two-layer variants at the largest batch: the projection, attention and
# split plans depend on the row count B * tokens, so these reach the plans
# the full models use at large batch (e.g. the large-tile kernel for the
# LLM's QKV and MLP products and the ViT's MLP down projection).
PI0_R32 = synth.reduced(synth.CONFIGS["pi0"], vit_layers=2, max_batch=32)
GR00T_R32 = synth.reduced(synth.CONFIGS["gr00t"], vit_layers=2, max_batch=32)


@pytest.mark.parametrize("cfg", [PI0_R32, GR00T_R32], ids=lambda c: c.name)
def test_reduced_depth_max_batch_sampled_rows(cfg):
    B = cfg.max_batch
    inp = synth.make_inputs(cfg, B)
    act, _ = run(cfg, inp)
    rows = [0, B // 2, B - 1]
    ref, _ = oracle_run(cfg, inp, rows=rows)
    check_chunk(act[rows], ref, inp["noise"][rows], 2e-2, f"{cfg.name} B={B} rows {rows}")
    drop_model(cfg)


# ---------------------------------------------------------------- bookkeeping (bit-exact)
@pytest.mark.parametrize("cfg", [TINY, SMOL_R, GR00T_R], ids=lambda c: c.name)
def test_determinism_permutation_and_batch_invariance(cfg):
    B = 3
    inp = synth.make_inputs(cfg, B)
    a1, _ = run(cfg, inp)
    a2, _ = run(cfg, inp)
    np.testing.assert_array_equal(a1, a2)
    perm = [2, 0, 1]
    ap, _ = run(cfg, {k: v[perm] for k, v in inp.items()})
    np.testing.assert_array_equal(ap, a1[perm])
    # batch-size invariance: the same request alone. Split-K / split-KV choose
    # their ranges from the launch's block count, so the reduction order (not
    # the data flow) may differ between batch sizes: equal to within rounding.
    one, _ = run(cfg, synth.make_inputs(cfg, 1, first_row=1))
    assert rel_l2(one[0], a1[1].astype(np.float64)) <= TOL[cfg.dtype] / 10


@pytest.mark.parametrize("cfg", [TINY, SMOL_R], ids=lambda c: c.name)
def test_graphs_match_direct_launches(cfg):
    inp = synth.make_inputs(cfg, 2)
    a_graph, kv_g = run(cfg, inp, graphs=True)
    a_direct, kv_d = run(cfg, inp, graphs=False)
    np.testing.assert_array_equal(a_graph, a_direct)
    assert bool((kv_g == kv_d).all())
    model(cfg).set_graphs(True)


def test_graph_replays_stay_exact():
    """Replaying the same captured graphs several times, with other work and
    synchronisations in between, gives the eager result every time."""
    import torch
    cfg = SMOL_R
    m = model(cfg)
    inp = synth.make_inputs(cfg, 2)
    ref, _ = run(cfg, inp, graphs=False)
    m.set_graphs(True)
    d = to_dev(inp)
    kv = m.alloc_kv(2)
    act = torch.empty_like(d["noise"])
    for i in range(4):
        m.prefill(2, d["pixels"], d["text_ids"], kv)
        m.denoise(2, kv, d["noise"], cfg.steps, act)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(act.cpu().numpy(), ref)
        _ = (torch.ones(1000, device="cuda") * i).sum().item()


def test_prefix_kv_untouched_by_action_stage():
    import torch
    cfg = SMOL_R
    m = model(cfg)
    d = to_dev(synth.make_inputs(cfg, 2))
    kv = m.alloc_kv(2)
    m.prefill(2, d["pixels"], d["text_ids"], kv)
    torch.cuda.synchronize()
    before = kv.clone()
    act = torch.empty_like(d["noise"])
    m.denoise(2, kv, d["noise"], cfg.steps, act)
    torch.cuda.synchronize()
    assert bool((kv == before).all())
    # and the noise input is read-only
    np.testing.assert_array_equal(d["noise"].cpu().numpy(), synth.make_noise(cfg, 2))


@pytest.mark.parametrize("cu,join", [(256, "default"), (128, "default"), (64, "default"), (256, "nonblocking"),
                                     (64, "nonblocking")])
def test_lockstep_matches_separate_stages(cu, join):
    """vla_step(prefill of batch k on a CU-restricted stream, denoise of batch
    k-1 on the action stream) gives the same bits as running them alone; with
    a non-blocking join stream the action half runs on that stream itself."""
    import torch
    from paper_2609_12075_amd import vla
    cfg = SMOL_R
    m = model(cfg)
    m.set_graphs(True)
    prev = synth.make_inputs(cfg, 2, first_row=0)
    cur = synth.make_inputs(cfg, 3, first_row=5)
    ref_prev, _ = run(cfg, prev)
    ref_cur, _ = run(cfg, cur)
    dp, dc = to_dev(prev), to_dev(cur)
    kv_prev, kv_cur = m.alloc_kv(2), m.alloc_kv(3)
    m.prefill(2, dp["pixels"], dp["text_ids"], kv_prev)
    act_prev = torch.empty_like(dp["noise"])
    act_cur = torch.empty_like(dc["noise"])
    js = None
    if join == "nonblocking":
        torch.cuda.synchronize()        # a non-blocking stream does not wait for the default stream
        js = vla.nonblocking_stream(0)
    vla.step(m, 3, dc["pixels"], dc["text_ids"], kv_cur, m, 2, kv_prev, dp["noise"], cfg.steps, act_prev,
             vlm_cu_count=cu, join_stream=js)
    vla.step(None, 0, None, None, None, m, 3, kv_cur, dc["noise"], cfg.steps, act_cur, vlm_cu_count=cu,
             join_stream=js)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(act_prev.cpu().numpy(), ref_prev)
    np.testing.assert_array_equal(act_cur.cpu().numpy(), ref_cur)


def test_lockstep_many_cu_counts():
    """More distinct CU restrictions than the library keeps streams for (it
    retires the least recently used masked stream): every lockstep still gives
    the bits of the stages run alone, on both the VLM and the action side."""
    import torch
    from paper_2609_12075_amd import vla
    cfg = SMOL_R
    m = model(cfg)
    m.set_graphs(True)
    inp = synth.make_inputs(cfg, 2, first_row=3)
    ref_act, ref_kv = run(cfg, inp)
    ref_kv = ref_kv.cpu()
    d = to_dev(inp)
    kv_in, kv_out = m.alloc_kv(2), m.alloc_kv(2)
    m.prefill(2, d["pixels"], d["text_ids"], kv_in)
    act = torch.empty_like(d["noise"])
    plan = [(32, 0), (48, 0), (64, 0), (96, 0), (128, 0), (160, 0), (192, 0), (224, 0), (32, 0), (96, 0),
            (64, 192), (128, 128), (96, 64), (256, 0)]
    for vcu, acu in plan:
        kv_out.zero_()
        act.zero_()
        vla.step(m, 2, d["pixels"], d["text_ids"], kv_out, m, 2, kv_in, d["noise"], cfg.steps, act,
                 vlm_cu_count=vcu, adit_cu_count=acu)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(act.cpu().numpy(), ref_act, err_msg=f"vlm {vcu} adit {acu}")
        assert bool((kv_out.cpu() == ref_kv).all()), f"vlm {vcu} adit {acu}"


def test_two_models_colocated_lockstep():
    """Two different models share the VLM and action streams (one lockstep
    runs model A's prefill with model B's denoise)."""
    import torch
    from paper_2609_12075_amd import vla
    a, b = TINY, SMOL_R
    ma, mb = model(a), model(b)
    ia, ib = synth.make_inputs(a, 1), synth.make_inputs(b, 2)
    ref_a, _ = run(a, ia)
    ref_b, _ = run(b, ib)
    da, db = to_dev(ia), to_dev(ib)
    kv_a, kv_b = ma.alloc_kv(1), mb.alloc_kv(2)
    mb.prefill(2, db["pixels"], db["text_ids"], kv_b)
    act_b = torch.empty_like(db["noise"])
    vla.step(ma, 1, da["pixels"], da["text_ids"], kv_a, mb, 2, kv_b, db["noise"], b.steps, act_b, vlm_cu_count=192)
    act_a = torch.empty_like(da["noise"])
    vla.step(None, 0, None, None, None, ma, 1, kv_a, da["noise"], a.steps, act_a)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(act_a.cpu().numpy(), ref_a)
    np.testing.assert_array_equal(act_b.cpu().numpy(), ref_b)


def test_pi0_and_smolvla_colocated_lockstep():
    """The co-located serving pair: a pi0-shaped prefill beside a
    SmolVLA-shaped denoise in one lockstep, and the reverse, give the bits of
    each stage run alone."""
    import torch
    from paper_2609_12075_amd import vla
    a, b = PI0_R, SMOL_R
    ma, mb = model(a), model(b)
    ia, ib = synth.make_inputs(a, 2, first_row=4), synth.make_inputs(b, 2, first_row=6)
    ref_a, ref_kv_a = run(a, ia)
    ref_b, ref_kv_b = run(b, ib)
    da, db = to_dev(ia), to_dev(ib)
    kv_a, kv_b = ma.alloc_kv(2), mb.alloc_kv(2)
    mb.prefill(2, db["pixels"], db["text_ids"], kv_b)
    act_a, act_b = torch.empty_like(da["noise"]), torch.empty_like(db["noise"])
    vla.step(ma, 2, da["pixels"], da["text_ids"], kv_a, mb, 2, kv_b, db["noise"], b.steps, act_b, vlm_cu_count=128)
    vla.step(None, 0, None, None, None, ma, 2, kv_a, da["noise"], a.steps, act_a, vlm_cu_count=128)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(act_a.cpu().numpy(), ref_a)
    np.testing.assert_array_equal(act_b.cpu().numpy(), ref_b)
    assert bool((kv_a.cpu() == ref_kv_a.cpu()).all())


def test_argument_errors_enqueue_nothing():
    import torch
    from paper_2609_12075_amd import vla
    cfg = TINY
    m = model(cfg)
    d = to_dev(synth.make_inputs(cfg, 1))
    kv = m.alloc_kv(1)
    act = torch.empty_like(d["noise"])
    with pytest.raises(vla.VlaError):
        m.prefill(0, d["pixels"], d["text_ids"], kv)
    with pytest.raises(vla.VlaError):
        m.prefill(cfg.max_batch + 1, d["pixels"], d["text_ids"], kv)
    with pytest.raises(vla.VlaError):
        m.denoise(1, kv, d["noise"], 0, act)
    with pytest.raises(vla.VlaError):
        m.denoise(1, kv, d["noise"], 4, d["noise"])
    with pytest.raises(vla.VlaError):
        vla.step(m, 1, d["pixels"], d["text_ids"], kv, None, 0, None, None, 4, None, vlm_cu_count=100)
    torch.cuda.synchronize()
