"""Host scheduler (C++, through the C ABI, simulated executor) against the
serving rules and against the plain-Python reference scheduler; no GPU."""
import numpy as np
import pytest

from oracle import sched as REF
from paper_2609_12075_amd import serve, synth, vla

MS = 1_000_000


def arr(items):
    a = np.zeros(len(items), dtype=[("t_ns", np.int64), ("model", np.int32)])
    for i, (t, m) in enumerate(items):
        a[i] = (t, m)
    return a


def const_table(n_models, max_batch, ns):
    nb = serve.n_buckets(max_batch)
    t = np.full((n_models, nb, n_models, nb), ns, dtype=np.int64)
    return t


def run(items, slo, max_batch, table, policy="esf", drain=10 ** 9, overhead=0, mode="lockstep"):
    s = serve.Scheduler(slo, max_batch, policy, mode)
    s.set_sim(table, overhead)
    req, ls = s.run(arr(items), drain)
    s.close()
    return req, ls


def test_power_of_two_admission():
    # 3 pending with max_batch 4 -> 2 then 1; 5 pending -> 4 then 1
    for pending, mb, expect in ((3, 4, [2, 1]), (5, 4, [4, 1]), (1, 2, [1]), (2, 2, [2]), (7, 8, [4, 2, 1]),
                                (9, 2, [2, 2, 2, 2, 1])):
        req, ls = run([(0, 0)] * pending, [100.0], mb, const_table(1, mb, 5 * MS))
        batches = [int(x["vlm_batch"]) for x in ls if x["vlm_batch"] > 0]
        assert batches == expect, (pending, mb, batches)


def test_lockstep_pairing_and_slots():
    items = [(0, 0), (0, 0), (0, 1), (1 * MS, 0), (1 * MS, 1), (2 * MS, 1)]
    req, ls = run(items, [50.0, 50.0], 2, const_table(2, 2, 3 * MS))
    prev = (-1, 0)
    for k, x in enumerate(ls):
        # the action half of lockstep k is exactly the VLM half of lockstep k - 1
        assert (int(x["adit_model"]), int(x["adit_batch"])) == prev
        assert x["slot"] == k % 2
        assert x["t_end_ns"] - x["t_start_ns"] == 3 * MS
        prev = (int(x["vlm_model"]), int(x["vlm_batch"])) if x["vlm_batch"] > 0 else (-1, 0)
    assert (req["t_done_ns"] >= 0).all()
    # every request is done one lockstep after its VLM lockstep
    for r in req:
        assert r["t_done_ns"] - r["t_vlm_start_ns"] == 6 * MS


def test_earliest_slo_first_choice():
    # lockstep 0 serves a blocker; at lockstep 1 (t = 5 ms) both queues hold a
    # head: model 1's (arrived later) has less time left (10-3 < 100-4 ms)
    items = [(0, 0), (1 * MS, 0), (2 * MS, 1)]
    req, ls = run(items, [100.0, 10.0], 1, const_table(2, 1, 5 * MS))
    assert ls[1]["vlm_model"] == 1
    # equal SLOs: the older head wins; ties go to the lowest model index
    req, ls = run([(0, 1), (0, 0)], [20.0, 20.0], 1, const_table(2, 1, 1 * MS))
    assert ls[0]["vlm_model"] == 0
    req, ls = run([(0, 0), (1 * MS, 1), (2 * MS, 0)], [20.0, 20.0], 1, const_table(2, 1, 5 * MS))
    assert ls[1]["vlm_model"] == 1


def test_policies_differ_on_a_backlog():
    items = [(0, 0)] * 6 + [(0, 1)]
    _, ls_lqf = run(items, [100.0, 100.0], 2, const_table(2, 2, MS), policy="lqf")
    assert [int(x["vlm_model"]) for x in ls_lqf[:3]] == [0, 0, 0]
    _, ls_rr = run(items, [100.0, 100.0], 2, const_table(2, 2, MS), policy="rr")
    assert [int(x["vlm_model"]) for x in ls_rr[:2]] == [0, 1]


def test_slo_accounting_boundary():
    # latency = 2 locksteps of 5 ms = 10 ms: met at SLO 10 ms, missed at 9.999
    req, _ = run([(0, 0)], [10.0], 1, const_table(1, 1, 5 * MS))
    assert req["met_slo"][0] == 1
    req, _ = run([(0, 0)], [9.999], 1, const_table(1, 1, 5 * MS))
    assert req["met_slo"][0] == 0
    assert serve.attainment(req) == 0.0


def test_unfinished_requests_count_as_misses():
    req, ls = run([(0, 0)] * 4, [1000.0], 1, const_table(1, 1, 10 * MS), drain=15 * MS)
    assert (req["t_done_ns"] < 0).any()
    assert serve.attainment(req) < 1.0
    req, ls = run([], [10.0], 1, const_table(1, 1, MS))
    assert len(req) == 0 and len(ls) == 0


def test_lookup_table_cardinality():
    # power-of-two batches up to max_batch: (log2(max_batch) + 1)^2 non-empty pairs per model pair
    for mb in (1, 2, 4, 8, 16):
        nb = serve.n_buckets(mb)
        assert (nb - 1) ** 2 == (int(np.log2(mb)) + 1) ** 2


def test_cu_table_applied_per_combination():
    mb = 2
    cu = np.zeros((1, 3, 1, 3), dtype=np.int32)
    cu[0, serve.bucket(2), 0, serve.bucket(2)] = 168
    s = serve.Scheduler([100.0], mb)
    s.set_sim(const_table(1, mb, MS))
    s.set_cu(192, cu)
    _, ls = s.run(arr([(0, 0)] * 6), 10 ** 9)
    got = [(int(x["vlm_batch"]), int(x["adit_batch"]), int(x["cu_count"])) for x in ls]
    assert (2, 2, 168) in got and (2, 0, 192) in got


def _random_case(seed):
    rng = np.random.default_rng(seed)
    nm = int(rng.integers(1, 4))
    mb = int(2 ** rng.integers(0, 4))
    nb = serve.n_buckets(mb)
    table = rng.integers(1 * MS, 20 * MS, size=(nm, nb, nm, nb)).astype(np.int64)
    slo = [float(x) for x in rng.uniform(10, 120, nm)]
    n = int(rng.integers(0, 80))
    t = np.sort(rng.integers(0, 300 * MS, n))
    if n > 5:
        t[3:6] = t[3]                     # a burst of simultaneous arrivals
    items = [(int(a), int(rng.integers(0, nm))) for a in t]
    policy = ["esf", "rr", "lqf"][seed % 3]
    overhead = int(rng.integers(0, 200_000))
    return items, slo, mb, table, policy, overhead


@pytest.mark.parametrize("seed", range(40))
def test_matches_reference_scheduler(seed):
    items, slo, mb, table, policy, overhead = _random_case(seed)
    drain = 50 * MS if seed % 4 == 0 else 10 ** 9
    req, ls = run(items, slo, mb, table, policy=policy, drain=drain, overhead=overhead)
    rreq, rls = REF.simulate(items, slo, mb, table.tolist(), policy=policy, drain_ns=drain, overhead_ns=overhead)
    assert len(ls) == len(rls)
    for a, b in zip(ls, rls):
        assert tuple(int(v) for v in a) == tuple(int(v) for v in b)
    for a, b in zip(req, rreq):
        assert (int(a["t_arrival_ns"]), int(a["t_vlm_start_ns"]), int(a["t_done_ns"]), int(a["model"]),
                int(a["met_slo"])) == (b["t_arrival"], b["t_vlm_start"], b["t_done"], b["model"], b["met"])


@pytest.mark.parametrize("seed", range(24))
def test_delivery_at_action_end_matches_reference(seed):
    """Chunks delivered when their action half ends (a second table, entries
    below and above the lockstep's duration): requests and lockstep records
    equal to the reference, field by field."""
    items, slo, mb, table, policy, overhead = _random_case(seed + 300)
    rng = np.random.default_rng(seed)
    adit = (table * rng.uniform(0.2, 1.3, table.shape)).astype(np.int64)
    s = serve.Scheduler(slo, mb, policy)
    s.set_sim(table, overhead)
    s.set_delivery("adit", adit)
    req, ls = s.run(arr(items), 10 ** 9)
    s.close()
    rreq, rls = REF.simulate(items, slo, mb, table.tolist(), policy=policy, overhead_ns=overhead,
                             delivery="adit", adit_ns=adit.tolist())
    assert [tuple(int(v) for v in a) for a in ls] == [tuple(b) for b in rls]
    for a, b in zip(req, rreq):
        assert (int(a["t_vlm_start_ns"]), int(a["t_done_ns"]), int(a["met_slo"])) == \
            (b["t_vlm_start"], b["t_done"], b["met"])
    for x in ls:
        assert x["t_start_ns"] <= x["t_chunks_ns"] <= x["t_end_ns"]


def test_delivery_at_action_end_closed_form():
    """One model, batch 1: lockstep 0 runs the VLM half of request A (7 ms);
    lockstep 1 the VLM half of B beside A's action half (9 ms in all, the
    action half ends after 4 ms); lockstep 2 B's action half (5 ms alone).
    Delivery at the lockstep end: A at 16 ms, B at 21 ms; at the action
    half's end: A at 7 + 4 = 11 ms, B at 16 + 5 = 21 ms (its action half is
    the whole lockstep). An SLO of 12 ms separates the two readings for A."""
    mb = 1
    nb = serve.n_buckets(mb)
    table = np.zeros((1, nb, 1, nb), dtype=np.int64)
    table[0, 1, 0, 0] = 7 * MS
    table[0, 0, 0, 1] = 5 * MS
    table[0, 1, 0, 1] = 9 * MS
    adit = table.copy()
    adit[0, 1, 0, 1] = 4 * MS
    req, ls = run([(0, 0), (0, 0)], [12.0], mb, table)
    assert req["t_done_ns"].tolist() == [16 * MS, 21 * MS] and req["met_slo"].tolist() == [0, 0]
    s = serve.Scheduler([12.0], mb)
    s.set_sim(table, 0)
    s.set_delivery("adit", adit)
    req, ls = s.run(arr([(0, 0), (0, 0)]), 10 ** 9)
    s.close()
    assert req["t_done_ns"].tolist() == [11 * MS, 21 * MS] and req["met_slo"].tolist() == [1, 0]
    assert ls["t_chunks_ns"].tolist() == [7 * MS, 11 * MS, 21 * MS]


def test_delivery_at_action_end_needs_its_table():
    s = serve.Scheduler([50.0], 1)
    s.set_sim(const_table(1, 1, MS), 0)
    with pytest.raises(vla.VlaError, match="time table"):
        s.set_delivery("adit")
        s.run(arr([(0, 0)]), 10 ** 9)
    with pytest.raises(vla.VlaError, match="unknown delivery"):
        vla._check(serve._lib().vla_sched_set_delivery(s.handle, 7, None))
    s.close()


@pytest.mark.parametrize("seed", range(12))
def test_monolithic_matches_reference(seed):
    items, slo, mb, table, policy, overhead = _random_case(seed + 100)
    req, ls = run(items, slo, mb, table, policy=policy, overhead=overhead, mode="monolithic")
    rreq, rls = REF.simulate(items, slo, mb, table.tolist(), policy=policy, overhead_ns=overhead, mode="monolithic")
    assert [tuple(int(v) for v in a) for a in ls] == [tuple(b) for b in rls]
    for a, b in zip(req, rreq):
        assert (int(a["t_vlm_start_ns"]), int(a["t_done_ns"]), int(a["met_slo"])) == \
            (b["t_vlm_start"], b["t_done"], b["met"])


def test_monolithic_serialises_stages():
    """Monolithic: a batch's latency is VLM-alone + action-alone, with no
    overlap across batches; the lockstep pipeline finishes the same single
    batch after two locksteps."""
    mb = 1
    nb = serve.n_buckets(mb)
    table = np.zeros((1, nb, 1, nb), dtype=np.int64)
    table[0, 1, 0, 0] = 7 * MS        # VLM alone
    table[0, 0, 0, 1] = 5 * MS        # action stage alone
    table[0, 1, 0, 1] = 9 * MS        # co-executed
    req, ls = run([(0, 0), (0, 0)], [100.0], mb, table, mode="monolithic")
    assert req["t_done_ns"].tolist() == [12 * MS, 24 * MS]
    req, ls = run([(0, 0), (0, 0)], [100.0], mb, table)
    assert req["t_done_ns"].tolist() == [16 * MS, 21 * MS]     # 7 | 9 | 5


def test_overrun_and_starvation_injection():
    # a lockstep that overruns (one combination 100x slower) shows up as misses
    mb = 2
    table = const_table(2, mb, 2 * MS)
    table[1, serve.bucket(2), :, :] = 200 * MS
    items = [(i * MS, i % 2) for i in range(40)]
    req, _ = run(items, [50.0, 50.0], mb, table)
    assert serve.attainment(req) < 0.9
    # a model with a slack SLO waits behind a flood of the tight one under ESF
    items = [(i * MS // 2, 0) for i in range(60)] + [(0, 1)]
    items.sort()
    req, ls = run(items, [5.0, 1000.0], 1, const_table(2, 1, MS))
    first_m1 = next(i for i, x in enumerate(ls) if x["vlm_model"] == 1)
    assert first_m1 > 0
    assert req["t_done_ns"][[i for i, (_, m) in enumerate(items) if m == 1][0]] > 0


def test_traffic_generators():
    a = synth.poisson_arrivals(8, 20.0, 5.0, 0)
    assert (np.diff(a["t_ns"]) >= 0).all()
    assert set(np.unique(a["model"])) <= {0, 1}
    # rate: about 8 robots x 20 Hz x 5 s
    assert 600 < len(a) < 1000
    p = synth.periodic_arrivals(4, 2.0, 3.0, 0)
    for r in range(4):
        t = np.sort(p["t_ns"][p["robot"] == r])
        assert np.allclose(np.diff(t), 0.5e9, atol=2)
        assert 0 <= t[0] < 0.5e9


def test_sweep_finds_capacity_knee():
    """With a fixed 10 ms lockstep at batch <= 4, capacity is bounded: the
    sweep's answer must be monotone-consistent (attainment falls with load)."""
    mb = 4
    nb = serve.n_buckets(mb)
    table = np.zeros((2, nb, 2, nb), dtype=np.int64)
    for iv in range(nb):
        for ia in range(nb):
            table[:, iv, :, ia] = (2 + 2 * iv + ia) * MS
    rows, best = serve.sweep_robots(table, [100.0, 100.0], mb, [2, 8, 32, 128], 20.0, 3.0, 2)
    att = [r["attainment"] for r in rows]
    assert att[0] >= 0.98 and att[-1] < 0.5
    assert best in (2, 8, 32)


def test_variant_tables_reuse_the_architecture_profile():
    """Fine-tuned variants share their architecture's lockstep entries."""
    mb = 2
    nb = serve.n_buckets(mb)
    rng = np.random.default_rng(3)
    dur = rng.integers(1, 100, size=(2, nb, 2, nb)).astype(np.int64)
    cu = rng.integers(1, 32, size=(2, nb, 2, nb)).astype(np.int32) * 8
    arch = [0, 1, 0, 1]
    vd, vc = serve.expand_tables(dur, cu, arch)
    assert vd.shape == (4, nb, 4, nb) and vc.shape == (4, nb, 4, nb)
    for i in range(4):
        for j in range(4):
            assert (vd[i, :, j, :] == dur[arch[i], :, arch[j], :]).all()
            assert (vc[i, :, j, :] == cu[arch[i], :, arch[j], :]).all()
    # four models run through the scheduler with the expanded table
    items = [(k * MS, k % 4) for k in range(40)]
    req, ls = run(items, [100.0] * 4, mb, vd * (MS // 20), drain=10 ** 10)
    assert (req["t_done_ns"] > 0).all()
    assert {int(x["vlm_model"]) for x in ls if x["vlm_batch"] > 0} == {0, 1, 2, 3}


@pytest.mark.parametrize("seed", range(16))
def test_online_calls_match_reference(seed):
    """The online calls (submit as the clock passes each arrival, one
    run_lockstep at a time, wait_until when idle, poll for completions)
    reproduce the reference scheduler's locksteps and per-request times, with
    completions identified by the ids given at submission."""
    items, slo, mb, table, policy, overhead = _random_case(seed + 200)
    mode = "monolithic" if seed % 5 == 4 else "lockstep"
    rreq, rls = REF.simulate(items, slo, mb, table.tolist(), policy=policy, overhead_ns=overhead, mode=mode)
    s = serve.Scheduler(slo, mb, policy, mode)
    s.set_sim(table, overhead)
    ids = [1000 + 7 * i for i in range(len(items))]
    nxt, recs, comps = 0, [], []
    while True:
        now = s.clock_ns()
        while nxt < len(items) and items[nxt][0] <= now:
            s.submit(ids[nxt], items[nxt][1], items[nxt][0])
            nxt += 1
        if s.pending() == 0:
            if nxt >= len(items):
                break
            s.wait_until(items[nxt][0])
            continue
        r = s.run_lockstep()
        assert r is not None
        recs.append(tuple(int(v) for v in r))
        comps.extend(s.poll(3))          # small cap: the rest stays queued for the next poll
    comps.extend(s.poll())
    assert s.run_lockstep() is None and s.pending() == 0
    assert recs == [tuple(b) for b in rls]
    assert len(comps) == len(items)
    by_id = {int(c["id"]): c for c in comps}
    for i, b in enumerate(rreq):
        c = by_id[ids[i]]
        assert (int(c["t_arrival_ns"]), int(c["t_vlm_start_ns"]), int(c["t_done_ns"]), int(c["model"]),
                int(c["met_slo"])) == (b["t_arrival"], b["t_vlm_start"], b["t_done"], b["model"], b["met"])
    s.close()


def test_online_submit_rejects_bad_requests():
    s = serve.Scheduler([50.0, 80.0], 4)
    s.set_sim(const_table(2, 4, MS), 0)
    with pytest.raises(vla.VlaError):
        s.submit(1, 2, 0)               # model index out of range
    with pytest.raises(vla.VlaError):
        s.submit(1, 0, -5)              # negative arrival
    s.submit(1, 0, 0)
    assert s.pending() == 1
    s.reset()
    assert s.pending() == 0 and s.clock_ns() == 0 and s.run_lockstep() is None
    s.close()
