"""Pins of the coordinator oracle (Sections 4.1-4.3) against closed forms, the
paper's own statements about its score, special cases that reduce to simpler
definitions, and brute force."""
import math

import numpy as np
import pytest
from scipy import stats

from oracle import cluster as K
from oracle import sched as S

ITER = (2_000 * S.PS, 40 * S.PS, 5_000, 1_000)
COST = (2_000 * S.PS, 50 * S.PS, 0, 2_100 * S.PS)


# ---------------------------------------------------------------- dispatch score (Section 4.1)
def test_alpha_one_picks_fastest_and_alpha_zero_shortest_queue():
    comp = [900, 300, 500, 300]
    queue = [10, 4000, 20, 7]
    assert K.wb_select(comp, queue, 1.0, 1e6) == 1          # only execution speed; tie 1/3 -> lower index
    assert K.wb_select(comp, queue, 0.0, 1e6) == 3          # only the queue: smallest t_queue
    assert K.wb_select([5, 5, 5], [0, 0, 0], 0.0, 1e6) == 0  # all tied -> lowest index


def test_reward_equals_c_ref_at_reference_queue():
    # beta = C_ref * Q_ref: at t_queue = Q_ref the queue term is worth C_ref (alpha = 0 part)
    c_ref, q_ref = 12_345.0, 6_789
    beta = c_ref * q_ref
    assert K.wb_score(0, q_ref, 0.0, beta) == pytest.approx(c_ref, rel=1e-15)
    # alpha = 1/2: score = (C_ref - t_comp) / 2 there
    assert K.wb_score(1000, q_ref, 0.5, beta) == pytest.approx((c_ref - 1000) / 2, rel=1e-15)


def test_empty_queue_counts_as_one_microsecond():
    beta = 1e6
    assert K.wb_score(0, 0, 0.0, beta) == K.wb_score(0, 1, 0.0, beta) == beta
    # several empty instances: the compute term decides among them
    assert K.wb_select([800, 200, 400], [0, 0, 5], 0.3, beta) == 1


def test_score_is_monotone_in_both_terms():
    rng = np.random.default_rng(0)
    for _ in range(200):
        a = float(rng.uniform(0, 1))
        beta = float(rng.uniform(1, 1e9))
        c, q = int(rng.integers(0, 10**6)), int(rng.integers(1, 10**6))
        assert K.wb_score(c + 1, q, a, beta) <= K.wb_score(c, q, a, beta)
        assert K.wb_score(c, q + 1, a, beta) <= K.wb_score(c, q, a, beta)


# ---------------------------------------------------------------- instance-average cost (Section 4.2)
def test_mean_cost_of_one_instance_is_its_own_estimate():
    for li, lo in ((0, 1), (17, 3), (4096, 256)):
        assert S.t_comp_mean(COST, 1, li, lo) == S.t_comp(COST, li, lo)


def test_mean_cost_is_the_mean_of_unfloored_estimates():
    a = (1_000_500_000, 333_333, 7, 999_999)
    b = (2_000_000_000, 1_000_001, 0, 3_000_000)
    s = tuple(x + y for x, y in zip(a, b))
    for li, lo in ((1, 1), (100, 7), (5000, 64)):
        ra = a[0] + a[1] * li + a[2] * li * li + a[3] * lo
        rb = b[0] + b[1] * li + b[2] * li * li + b[3] * lo
        assert S.t_comp_mean(s, 2, li, lo) == math.floor((ra + rb) / 2 / S.PS)


def test_shared_budget_uses_average_costs():
    # two instances, the second twice as slow: average cost = 1.5x the first's
    fast = (0, S.PS, 0, 0)                # t_comp = L_in us
    slow = (0, 2 * S.PS, 0, 0)
    s = S.Scheduler(64, 8, 64, fast, ITER)
    csum = tuple(x + y for x, y in zip(fast, slow))
    rid = s.submit(0, 0, 0, 0, 10_000, [1] * 40, 1, rest=[(60, 0)], budget_cost_sum=csum, n_inst=2)
    r = s.reqs[rid]
    # budgets from averages 60 and 90: 10000 * 60 / 150; urgency key from the local cost 40
    assert r.t_slo == 4000 and r.t_comp == 40 and r.key == 4000 - 40


# ---------------------------------------------------------------- queueing cost (Section 4.1)
def test_queue_cost_brute_force():
    s = S.Scheduler(256, 2, 32, COST, ITER)
    ids = [s.submit(0, w, 0, 0, 10**9, [1] * n, m) for w, (n, m) in enumerate([(20, 2), (40, 1), (10, 3)])]
    tc = {i: s.reqs[i].t_comp for i in ids}
    assert s.queue_cost() == sum(tc.values())
    now = 0
    live = set(ids)
    while live:
        st, info = s.step(now)
        now += info["t_iter_us"]
        for d in s.drain():
            live.discard(d["id"])
        assert s.queue_cost() == sum(tc[i] for i in live)


# ---------------------------------------------------------------- t-test (Section 4.3)
def test_welch_two_and_two_with_equal_spread_has_two_dof():
    # equal variances and sizes 2 and 2: dof = 2, and P(T_2 >= t) = 1/2 - t / (2 sqrt(2 + t^2))
    x_new, x_ref = [10.0, 14.0], [7.0, 11.0]
    t, dof, p = K.welch_t_greater(x_new, x_ref)
    # means 12 and 9, each variance 8: t = 3 / sqrt(8/2 + 8/2) = 3 / sqrt(8)
    assert t == pytest.approx(3 / math.sqrt(8), rel=1e-14)
    assert dof == pytest.approx(2.0, rel=1e-14)
    assert p == pytest.approx(0.5 - t / (2 * math.sqrt(2 + t * t)), rel=1e-12)


def test_welch_with_constant_reference_has_one_dof():
    # reference without spread, new window of two: dof = 1 (Cauchy): P = 1/2 - atan(t)/pi
    x_new, x_ref = [5.0, 9.0], [3.0, 3.0, 3.0]
    t, dof, p = K.welch_t_greater(x_new, x_ref)
    assert t == pytest.approx(4 / math.sqrt(8 / 2), rel=1e-14)
    assert dof == pytest.approx(1.0, rel=1e-14)
    assert p == pytest.approx(0.5 - math.atan(t) / math.pi, rel=1e-12)


def test_welch_direction_and_degenerate_cases():
    lo, hi = [1.0, 2.0, 3.0, 4.0], [11.0, 12.0, 13.0, 14.0]
    assert K.welch_t_greater(hi, lo)[2] < 1e-4       # new window slower: significant
    assert K.welch_t_greater(lo, hi)[2] > 1 - 1e-4   # faster: not a regression
    assert K.welch_t_greater([5.0, 5.0], [5.0, 5.0])[2] == 1.0
    assert K.welch_t_greater([6.0, 6.0], [5.0, 5.0])[2] == 0.0


def test_welch_matches_the_library_t_test_routine():
    rng = np.random.default_rng(1)
    for _ in range(50):
        a = rng.lognormal(3.0, 0.4, size=int(rng.integers(2, 40)))
        b = rng.lognormal(3.1, 0.7, size=int(rng.integers(2, 40)))
        t, dof, p = K.welch_t_greater(a, b)
        ref = stats.ttest_ind(a, b, equal_var=False, alternative="greater")
        assert t == pytest.approx(ref.statistic, rel=1e-10)
        assert p == pytest.approx(ref.pvalue, rel=1e-9, abs=1e-15)


def test_percentile_definition():
    # 95 of 1..100 are <= 95; with 20 values the 19th; one value is its own P95
    assert K.percentile95(list(range(100, 0, -1))) == 95
    assert K.percentile95(list(range(1, 21))) == 19
    assert K.percentile95(list(range(1, 22))) == 20    # ceil(0.95 * 21) = 20
    assert K.percentile95([7]) == 7
    assert K.percentile95([3, float("inf"), 1] + [2] * 17) == 3    # 19 of 20 finite ones cover 95%
    assert K.percentile95([3, float("inf"), float("inf")] + [2] * 17) == float("inf")


# ---------------------------------------------------------------- the coordinator loop
def _wf(wid, arrival, slo, stages, shapes):
    return dict(wid=wid, arrival=arrival, slo=slo, stages=stages, shapes=shapes)


def _req(n, max_new, parent=None, retain=False, seed=0):
    return dict(prompt=[(seed * 31 + k) % 2048 for k in range(n)], max_new=max_new, parent=parent, retain=retain)


def _two_stage(wid, arrival):
    # stage 0 retained and forked twice by stage 1, then a fresh stage 2
    return _wf(wid, arrival, 10**9,
               [[_req(40, 4, retain=True, seed=wid)], [_req(3, 5, (0, 0)), _req(3, 5, (0, 0))], [_req(30, 2)]],
               [(40, 4), (19, 5), (30, 2)])


def spec(cost, it=ITER, n_blocks=512, max_seqs=16, chunk=64):
    return dict(cost=cost, iter=it, n_blocks=n_blocks, max_seqs=max_seqs, chunk=chunk)


def test_forks_run_on_their_parents_instance():
    co = K.Coordinator([spec(COST), spec(COST), spec(COST)], "rr")
    co.simulate([_two_stage(w, 1000 * w) for w in range(6)])
    where = {(p[1], p[2], p[3]): p[4] for p in co.placements}
    for w in range(6):
        assert where[(w, 1, 0)] == where[(w, 1, 1)] == where[(w, 0, 0)]
    assert all(st["finish"] > 0 for st in co.states)


def test_one_instance_reduces_to_a_plain_instance_loop():
    wfs = [_two_stage(w, 700 * w) for w in range(5)]
    co = K.Coordinator([spec(COST)], "wb", 0.5, 1e6)
    fin = co.simulate(wfs)
    # the same replay written directly against one scheduler
    s = S.Scheduler(512, 16, 64, COST, ITER)
    placed, left, done_at = {}, {}, {}
    owner = {}

    def start(w, j, now):
        ids = []
        for q in w["stages"][j]:
            par = 0 if q["parent"] is None else placed[(w["wid"], q["parent"][0])][q["parent"][1]]
            rid = s.submit(now, w["wid"], j, w["arrival"], w["slo"], q["prompt"], q["max_new"], parent=par,
                           retain=q["retain"], rest=w["shapes"][j + 1:])
            owner[rid] = (w, j)
            ids.append(rid)
        placed[(w["wid"], j)] = ids
        left[(w["wid"], j)] = len(ids)
        if j == 2:
            s.release(placed[(w["wid"], 0)][0])

    now, k = 0, 0
    while k < len(wfs) or any(v > 0 for v in left.values()):
        while k < len(wfs) and wfs[k]["arrival"] <= now:
            start(wfs[k], 0, now)
            k += 1
        st, info = s.step(now)
        if st == S.IDLE:
            now = wfs[k]["arrival"]
            continue
        now += info["t_iter_us"]
        for d in s.drain():
            w, j = owner[d["id"]]
            left[(w["wid"], j)] -= 1
            if left[(w["wid"], j)] == 0:
                if j < 2:
                    start(w, j + 1, now)
                else:
                    done_at[w["wid"]] = now
    assert fin == [done_at[w["wid"]] for w in wfs]


def test_tuning_prefers_the_fast_instance_when_the_other_is_much_slower():
    fast, slow = COST, tuple(20 * c for c in COST)
    it_fast, it_slow = ITER, tuple(20 * c for c in ITER)
    specs = [spec(fast, it_fast), spec(slow, it_slow)]
    trace = [_two_stage(w, 10_000 * w) for w in range(12)]   # the fast instance is often busy
    beta = K.beta_from_warmup(specs, trace[:4])
    grid = tuple(k / 10 for k in range(11))
    best, vals = K.grid_search(specs, trace, beta, grid)
    # alpha = 0 balances queues onto the slow instance; alpha = 1 never uses it
    assert vals[-1] < vals[0]
    assert vals[grid.index(best)] == min(vals) and best > 0.0
    assert all(v > min(vals) for v in vals[:grid.index(best)])


def test_beta_from_two_warmup_queries_by_hand():
    """beta = C_ref * Q_ref (Section 4.1) over warm-up dispatches at alpha = 0
    (reading: means over the decisions of the instances' mean t_comp and mean
    t_queue).  Two instances with t_comp = L_in and 2 L_in microseconds, 1 ms
    iterations, two one-request queries:
      t = 0:  L_in 100 -> costs (100, 200), queues (0, 0): decision (150, 0); tie -> instance 0
      t = 10: L_in  50 -> costs (50, 100), instance 0 still runs the first (queue 100):
              decision (75, 50); 1/100 < 1/1 -> instance 1
    C_ref = (150 + 75) / 2 = 112.5, Q_ref = (0 + 50) / 2 = 25, beta = 2812.5."""
    it = (1000 * S.PS, 0, 0, 0)
    specs = [spec((0, S.PS, 0, 0), it), spec((0, 2 * S.PS, 0, 0), it)]
    wfs = [_wf(0, 0, 10 ** 7, [[_req(100, 1)]], [(100, 1)]),
           _wf(1, 10, 10 ** 7, [[_req(50, 1, seed=1)]], [(50, 1)])]
    assert K.beta_from_warmup(specs, wfs) == 2812.5
    co = K.Coordinator(specs, "wb", 0.0, 1.0, record=True)
    co.simulate(wfs)
    assert co.decisions == [(150.0, 0.0), (75.0, 50.0)]
    assert [p[4] for p in co.placements] == [0, 1]
    # with the queue mean below 1 us it counts as 1: one query alone gives C_ref * 1
    assert K.beta_from_warmup(specs, wfs[:1]) == 150.0


def test_tuning_is_indifferent_with_one_instance():
    trace = [_two_stage(w, 3_000 * w) for w in range(8)]
    best, vals = K.grid_search([spec(COST)], trace, 1e6, tuple(k / 10 for k in range(11)))
    assert len(set(vals)) == 1 and best == 0.0


def test_regression_triggers_retuning():
    # a burst after a quiet period: latencies of the second window rise sharply
    specs = [spec(COST), spec(tuple(8 * c for c in COST), tuple(8 * c for c in ITER))]
    quiet = [_two_stage(w, 60_000 * w) for w in range(10)]
    burst = [_two_stage(10 + w, 600_000 + 500 * w) for w in range(30)]
    co = K.Coordinator(specs, "wb", 0.0, 1e9, tuner=dict(n_min=5, t_min_us=0, p=0.01, grid=(0.0, 0.5, 1.0)))
    co.simulate(quiet + burst)
    trig = [h for h in co.alpha_history if h[4] is not None]
    assert trig, co.alpha_history
    assert all(h[3] < 0.01 for h in trig)
    assert all(h[3] >= 0.01 for h in co.alpha_history if h[4] is None)
