"""The coordinator across instances (Sections 4.1-4.3): the library's decisions
(hxf_queue_cost, hxf_request_cost, hxf_submit_shared, hxf_wb_select,
hxf_ttest_greater) and the host event loop above them, against the oracle
coordinator driving oracle schedulers.  Everything integer must match exactly
(placements, budgets, finish times, tuning decisions); floating-point test
statistics within 1e-10."""
import numpy as np
import pytest

import synth
from oracle import cluster as K
from oracle import sched as S
from paper_2505_05286_amd import hxf
from paper_2505_05286_amd.cluster import Cluster, InstanceSpec, TunerCfg, calibrate_beta, tune_alpha
from paper_2505_05286_amd.workflows import Req, Workflow

from ._lib import ensure_built

COST = (6_000 * S.PS, 110 * S.PS, 8_000, 30_000 * S.PS)
ITER = (28_000 * S.PS, 100 * S.PS, 48_000, 2_800)
SHAPE = dict(s1_out=64, n_cand=8, cand_out=256, n_corr=4, corr_in=512, corr_out=256, eval_in=1024, eval_out=128)


def scaled(c, k):
    return tuple(int(v * k) for v in c)


# a heterogeneous cluster: two reference instances, one 1.5x and one 2.5x slower
SPEEDS = (1.0, 1.0, 1.5, 2.5)


def specs(policy=S.POLICY_PQ, speeds=SPEEDS, n_blocks=3000, max_seqs=48, chunk=256):
    lib = [InstanceSpec(scaled(COST, k), scaled(ITER, k), n_blocks, max_seqs, chunk, policy) for k in speeds]
    ora = [dict(cost=scaled(COST, k), iter=scaled(ITER, k), n_blocks=n_blocks, max_seqs=max_seqs, chunk=chunk,
                policy=policy) for k in speeds]
    return lib, ora


def mcfg():
    ensure_built()
    return hxf.model_cfg(synth.ModelShape("sched", 1, 64, 1, 1, 64, 64, 2048, 0), 1 << 20)


def workflows(n, scale=8, rate=1.0, first=0):
    """Workload-5 streams with every length divided by `scale` (keeps the oracle fast) and
    arrivals compressed by `rate`; returned for the library driver and for the oracle."""
    s = SHAPE
    lib, ora = [], []
    for w in synth.workloads.cfg5(vocab=2048, n_wf=first + n)[first:]:
        l1 = max(16, w.schema_len // scale)
        reqs = [[(w.schema[:l1], s["s1_out"] // scale, None, True)],
                [(np.zeros(0, np.int32), s["cand_out"] // scale, (0, 0), b % 2 == 0) for b in range(s["n_cand"])],
                [(w.corrections[k][: s["corr_in"] // scale], s["corr_out"] // scale, (1, 2 * k), False)
                 for k in range(s["n_corr"])],
                [(w.eval_prompt[: s["eval_in"] // scale], s["eval_out"] // scale, None, False)]]
        shapes = [(l1, s["s1_out"] // scale), (16, s["cand_out"] // scale),
                  (16 + s["corr_in"] // scale, s["corr_out"] // scale), (s["eval_in"] // scale, s["eval_out"] // scale)]
        arrival, slo = int(w.arrival_us / 4 / rate), int(w.slo_us // 20)
        lib.append(Workflow(w.workflow, arrival, slo,
                            [[Req(p, m, parent=par, retain=r) for p, m, par, r in st] for st in reqs], shapes))
        ora.append(dict(wid=w.workflow, arrival=arrival, slo=slo, shapes=shapes,
                        stages=[[dict(prompt=[int(t) for t in p], max_new=m, parent=par, retain=r)
                                 for p, m, par, r in st] for st in reqs]))
    return lib, ora


# ---------------------------------------------------------------- single decisions
def test_wb_select_matches_oracle():
    ensure_built()
    rng = np.random.default_rng(7)
    for _ in range(2000):
        n = int(rng.integers(1, 9))
        comp = [int(v) for v in rng.integers(0, 10**7, n)]
        queue = [int(v) for v in rng.integers(0, 10**8, n)]
        if rng.random() < 0.3:
            queue[int(rng.integers(0, n))] = 0
        if rng.random() < 0.2:
            comp = [comp[0]] * n
        alpha = float(rng.integers(0, 11)) / 10 if rng.random() < 0.5 else float(rng.random())
        beta = float(rng.uniform(0, 1e13))
        assert hxf.wb_select(comp, queue, alpha, beta) == K.wb_select(comp, queue, alpha, beta)


def test_wb_select_rejects_bad_arguments():
    ensure_built()
    for args in (([1], [1], -0.1, 1.0), ([1], [1], 1.5, 1.0), ([1], [1], 0.5, -1.0), ([1], [1], 0.5, float("inf")),
                 ([], [], 0.5, 1.0)):
        with pytest.raises(hxf.HxfError):
            hxf.wb_select(*args)


def test_ttest_matches_oracle():
    ensure_built()
    rng = np.random.default_rng(11)
    cases = [([10.0, 14.0], [7.0, 11.0]), ([5.0, 9.0], [3.0, 3.0, 3.0]), ([5.0, 5.0], [5.0, 5.0]),
             ([6.0, 6.0], [5.0, 5.0]), ([4.0, 4.0], [5.0, 5.0])]
    for _ in range(300):
        a = rng.lognormal(17.0, float(rng.uniform(0.05, 1.0)), size=int(rng.integers(2, 60)))
        b = rng.lognormal(17.0 + float(rng.normal(0, 0.3)), float(rng.uniform(0.05, 1.0)), size=int(rng.integers(2, 60)))
        cases.append((list(np.rint(a)), list(np.rint(b))))
    for a, b in cases:
        t1, d1, p1 = hxf.ttest_greater(a, b)
        t2, d2, p2 = K.welch_t_greater(a, b)
        if np.isinf(t2):
            assert t1 == t2
        else:
            assert t1 == pytest.approx(t2, rel=1e-12, abs=1e-12)
        assert d1 == pytest.approx(d2, rel=1e-12)
        assert p1 == pytest.approx(p2, rel=1e-10, abs=1e-14)
        assert (p1 < 0.01) == (p2 < 0.01)


def test_ttest_rejects_short_or_non_finite_samples():
    ensure_built()
    for a, b in (([1.0], [1.0, 2.0]), ([1.0, 2.0], [3.0]), ([1.0, float("nan")], [1.0, 2.0])):
        with pytest.raises(hxf.HxfError):
            hxf.ttest_greater(a, b)


def test_queue_cost_and_shared_budget_match_oracle():
    m = mcfg()
    lib_spec, _ = specs()
    csum = tuple(sum(s.cost_ps[i] for s in lib_spec) for i in range(4))
    b = S.Scheduler(400, 6, 64, COST, ITER, vocab=2048)
    now = 0
    a = hxf.Instance(m, hxf.sched_cfg(400, 6, 64, COST, ITER, executor=hxf.EXEC_NULL))
    rng = np.random.default_rng(5)
    for k in range(60):
        n, out = int(rng.integers(1, 120)), int(rng.integers(1, 30))
        rest = [(int(rng.integers(1, 200)), int(rng.integers(1, 50))) for _ in range(int(rng.integers(0, 3)))]
        p = rng.integers(0, 2048, n).astype(np.int32)
        arr = now - int(rng.integers(0, 10**6))
        ia = a.submit(now, k, 0, arr, 5 * 10**6, p, out, rest=rest, cost_sum=csum, n_instances=len(lib_spec))
        ib = b.submit(now, k, 0, arr, 5 * 10**6, list(p), out, rest=rest, budget_cost_sum=csum, n_inst=len(lib_spec))
        assert ia == ib
        sa, rb = a.request_state(ia), b.reqs[ib]
        assert (sa["t_slo_us"], sa["t_comp_us"], sa["key_us"]) == (rb.t_slo, rb.t_comp, rb.key)
        assert a.request_cost(n, out) == S.t_comp(COST, n, out)
        if k % 3 == 2:
            for _ in range(int(rng.integers(1, 4))):
                st, info = a.step(now)
                st2, info2 = b.step(now)
                assert (st == hxf.IDLE) == (st2 == S.IDLE)
                if st == hxf.IDLE:
                    break
                now += info["t_iter_us"]
                a.drain(), b.drain()
        assert a.queue_cost() == b.queue_cost()
    a.close()


def test_shared_submit_with_own_costs_equals_plain_submit():
    m = mcfg()
    a = hxf.Instance(m, hxf.sched_cfg(400, 6, 64, COST, ITER, executor=hxf.EXEC_NULL))
    b = hxf.Instance(m, hxf.sched_cfg(400, 6, 64, COST, ITER, executor=hxf.EXEC_NULL))
    for k in range(10):
        p = np.arange(5 + 7 * k, dtype=np.int32) % 2048
        ia = a.submit(100 * k, k, 1, 0, 10**6, p, 3 + k, rest=[(40, 9), (10, 2)])
        ib = b.submit(100 * k, k, 1, 0, 10**6, p, 3 + k, rest=[(40, 9), (10, 2)], cost_sum=COST, n_instances=1)
        assert a.request_state(ia) == b.request_state(ib)
    with pytest.raises(hxf.HxfError):
        b.submit(0, 0, 0, 0, 10, np.ones(3, np.int32), 1, cost_sum=COST, n_instances=0)
    a.close()
    b.close()


# ---------------------------------------------------------------- whole replays
def _both(dispatch, alpha, beta, n_wf=24, policy=S.POLICY_PQ, rate=1.6, tuner=None):
    lib_spec, ora_spec = specs(policy)
    wl, wo = workflows(n_wf, rate=rate)
    c = Cluster(mcfg(), lib_spec, dispatch, alpha, beta,
                tuner=None if tuner is None else TunerCfg(tuner["n_min"], tuner["t_min_us"], tuner["p"],
                                                          tuner["grid"]))
    fa = c.run(wl)
    o = K.Coordinator(ora_spec, dispatch, alpha, beta, tuner=tuner)
    fo = o.simulate(wo)
    return c, fa, o, fo


@pytest.mark.parametrize("dispatch,alpha", [("rr", 0.0), ("wb", 0.0), ("wb", 0.3), ("wb", 1.0)])
def test_replay_matches_oracle(dispatch, alpha):
    c, fa, o, fo = _both(dispatch, alpha, 4e9)
    assert fa == fo
    assert all(f > 0 for f in fa)
    assert [e[:5] for e in c.log] == [e[:5] for e in o.placements]
    assert c.deadlocked == o.deadlocked is False
    used = {e[4] for e in c.log}
    assert len(used) > 1 or dispatch == "wb" and alpha == 1.0
    c.close()


def test_replay_with_fcfs_instances_matches_oracle():
    c, fa, o, fo = _both("wb", 0.5, 4e9, policy=S.POLICY_FCFS)
    assert fa == fo
    c.close()


def test_beta_calibration_and_grid_match_oracle():
    lib_spec, ora_spec = specs()
    wl, wo = workflows(10, rate=1.6)
    m = mcfg()
    b1 = calibrate_beta(m, lib_spec, wl[:6])
    b2 = K.beta_from_warmup(ora_spec, wo[:6])
    assert b1 == b2 and b1 > 1.0
    grid = (0.0, 0.5, 0.9, 1.0)
    a1, v1 = tune_alpha(m, lib_spec, wl, b1, grid)
    a2, v2 = K.grid_search(ora_spec, wo, b2, grid)
    assert (a1, v1) == (a2, v2)


def test_online_tuning_matches_oracle():
    # quiet arrivals, then a burst: the t-test must fire and both sides retune alike
    tuner = dict(n_min=5, t_min_us=0, p=0.01, grid=(0.0, 0.5, 1.0))
    lib_spec, ora_spec = specs()
    wl1, wo1 = workflows(10, rate=0.3)
    wl2, wo2 = workflows(24, rate=4.0, first=10)
    shift = wl1[-1].arrival_us + 1
    for w in wl2:
        w.arrival_us = shift + w.arrival_us - wl2[0].arrival_us
    for w in wo2:
        w["arrival"] = shift + w["arrival"] - wo2[0]["arrival"]
    c = Cluster(mcfg(), lib_spec, "wb", 0.0, 4e9, tuner=TunerCfg(5, 0, 0.01, (0.0, 0.5, 1.0)))
    fa = c.run(wl1 + wl2)
    o = K.Coordinator(ora_spec, "wb", 0.0, 4e9, tuner=tuner)
    fo = o.simulate(wo1 + wo2)
    assert fa == fo
    assert len(c.alpha_log) == len(o.alpha_history) >= 2
    for x, y in zip(c.alpha_log, o.alpha_history):
        assert x[0] == y[0] and x[4] == y[4]
        assert x[3] == pytest.approx(y[3], rel=1e-10, abs=1e-14)
    assert any(x[4] is not None for x in c.alpha_log), c.alpha_log
    c.close()
