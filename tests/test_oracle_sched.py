"""Pins of the oracle scheduler against the paper's worked examples and the
mathematics of the local priority queue (Section 4.2)."""
import os

import numpy as np
import pytest

from oracle import sched as S
from oracle import paged as P

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def read_table2():
    rows, exp = [], {}
    for line in open(os.path.join(GOLD, "table2_local_queue.txt")):
        line = line.strip()
        if line.startswith("# expect"):
            k, v = line[2:].split()
            exp[k] = int(v)
        elif line and not line.startswith("#"):
            i, a, u = line.split()
            rows.append((int(i), round(float(a) * 1e6), round(float(u) * 1e6)))
    return rows, exp


def read_kv(name):
    d = {}
    for line in open(os.path.join(GOLD, name)):
        if line.strip() and not line.startswith("#"):
            k, v = line.split()
            d[k] = int(v)
    return d


UNIT_PREFILL = (0, S.PS, 0, 0)     # t_comp = L_in microseconds
UNIT_DECODE = (0, 0, 0, S.PS)      # t_comp = L_out microseconds
ITER = (1000 * S.PS, 0, 0, 0)


def _table2_sched(policy, now):
    """Queue whose urgencies at ``now`` are Table 2's, each request a one-stage
    workflow arriving when it enters the queue (so t_SLO = T_SLO)."""
    rows, _ = read_table2()
    s = S.Scheduler(n_blocks=64, max_seqs=1, chunk_tokens=4096, cost=UNIT_PREFILL, iter_cost=ITER,
                    policy=policy)
    for rid, arr, u in rows:
        t_comp = 100
        # U(now) = t_comp - (T_SLO - (now - arr))  =>  T_SLO = t_comp + now - arr - U
        t_slo = t_comp + now - arr - u
        got = s.submit(arr, rid, 0, arr, t_slo, list(range(100)), 1)
        assert got == rid
    return s, rows


def test_table2_pq_order_and_selection():
    now = 70_000_000
    _, exp = read_table2()
    s, rows = _table2_sched(S.POLICY_PQ, now)
    for rid, arr, u in rows:
        r = s.reqs[rid]
        assert S.urgency(r.t_comp, r.t_slo, now - r.enq) == u
    # highest urgency first; the two 19.0 entries keep arrival order
    assert s.queue_order() == [6, 7, 3, 5, 1, 2, 4]
    st, info = s.step(now)
    assert info["admitted"] == [exp["expect_pq_first"]]


def test_table2_fcfs_selection():
    now = 70_000_000
    _, exp = read_table2()
    s, _ = _table2_sched(S.POLICY_FCFS, now)
    assert s.queue_order() == [1, 2, 3, 4, 5, 6, 7]
    st, info = s.step(now)
    assert info["admitted"] == [exp["expect_fcfs_first"]]


def test_fig3_debit_propagation():
    g = read_kv("fig3_slo_debit.txt")
    s = S.Scheduler(4096, 8, 4096, UNIT_DECODE, ITER)
    c1, c2 = g["cost1_us"], g["cost2_us"]
    r1 = s.submit(0, 0, 0, 0, g["slo_us"], [1], c1, rest=[(1, c2)])
    assert s.reqs[r1].t_comp == c1
    assert s.reqs[r1].t_slo == g["budget1_us"]
    late = s.submit(g["elapsed_after_1_us"], 0, 1, 0, g["slo_us"], [1], c2)
    on_time = s.submit(g["budget1_us"], 0, 1, 0, g["slo_us"], [1], c2)
    assert s.reqs[late].t_slo == g["budget2_us"]
    assert s.reqs[on_time].t_slo == g["budget2_on_time_us"]
    assert g["budget2_on_time_us"] - g["budget2_us"] == g["elapsed_after_1_us"] - g["budget1_us"]


@pytest.mark.parametrize("costs", [(40, 60), (5, 7, 11, 13), (1000, 1, 1, 1000), (3, 0, 9)])
def test_on_schedule_budgets_partition_remaining_time(costs):
    """If every stage takes exactly its budget, the budgets split T_SLO in
    proportion to cost (within one microsecond of floor error per stage)."""
    T = 1_000_003
    elapsed, got = 0, []
    for j, c in enumerate(costs):
        b = S.slo_budget(T, elapsed, c, costs[j + 1:])
        got.append(b)
        elapsed += b
    assert T - len(costs) <= sum(got) <= T
    for b, c in zip(got, costs):
        assert abs(b - T * c / sum(costs)) <= len(costs)


def test_budget_floors_toward_minus_infinity():
    # behind schedule: negative remaining time gives a negative budget, floored
    assert S.slo_budget(100, 107, 1, [2]) == -3      # -7 * 1 / 3 = -2.33 -> -3
    assert S.slo_budget(100, 0, 0, []) == 100         # zero total cost


def test_single_instance_average_cost_is_own_cost():
    # the instance average over one instance is the instance's own estimate
    assert S.t_comp((7 * S.PS, 3 * S.PS, 0, 5 * S.PS), 10, 4) == 7 + 30 + 20


def test_t_comp_hand_values_with_quadratic_term():
    """Section 4.1's t_comp = t_prefill(L_in) + t_decode(L_out) with the quadratic
    prefill term, worked by hand (picosecond coefficients, floored microseconds)."""
    cost = (1_500_000, 2_000_000, 300, 4_000_000)
    # 1.5e6 + 2e6*1000 + 300*1000^2 + 4e6*10 = 2_341_500_000 ps = 2341.5 us -> 2341
    assert S.t_comp(cost, 1000, 10) == 2341
    # quadratic term alone: 806 * 8192^2 = 54_089_744_384 ps -> 54089 us
    assert S.t_comp((0, 0, 806, 0), 8192, 0) == 54089
    # 234 * 3000^2 + 17 * 1e6 * 256 = 2_106_000_000 + 4_352_000_000 = 6_458_000_000 ps -> 6458 us
    assert S.t_comp((0, 0, 234, 17_000_000), 3000, 256) == 6458
    # one picosecond short of a whole microsecond floors down: 999_999 + 1 * 1^2 ... = 999_999 + 0
    assert S.t_comp((999_998, 0, 1, 0), 1, 0) == 0
    assert S.t_comp((999_999, 0, 1, 0), 1, 0) == 1
    # the same costs through a scheduler's submit
    s = S.Scheduler(4096, 8, 2048, cost, ITER)
    rid = s.submit(0, 0, 0, 0, 10 ** 7, [1] * 1000, 10)
    assert s.reqs[rid].t_comp == 2341


def test_llf_key_and_order_differ_from_pq_by_hand():
    """LLF (Section 5.1's least-laxity baseline, reading: key = workflow arrival +
    end-to-end SLO - (own cost + the later stages' costs)) against PQ (key =
    enqueue + budget - own cost), three requests submitted at t = 0 with
    t_comp = L_in microseconds:
        A: arrival    0, SLO 1000, L_in 100, later stage L_in 400
           LLF 0 + 1000 - 500 = 500;   PQ budget 1000*100/500 = 200, key 200 - 100 = 100
        B: arrival    0, SLO  610, L_in 300, no later stage
           LLF 610 - 300 = 310;        PQ budget 610, key 610 - 300 = 310
        C: arrival -150, SLO  900, L_in 200, later stage L_in 100
           LLF -150 + 900 - 300 = 450; PQ budget (900-150)*200/300 = 500, key 300
    PQ order A, C, B; LLF order B, C, A.  Leaving out the later stages' costs in
    LLF would give B (310), C (550), A (900) -> still B first but C keyed 550;
    using the enqueue time instead of the workflow arrival would key C at 600,
    after A."""
    keys = {}
    for pol in (S.POLICY_PQ, S.POLICY_LLF):
        s = S.Scheduler(64, 1, 4096, UNIT_PREFILL, ITER, policy=pol)
        a = s.submit(0, 1, 0, 0, 1000, [1] * 100, 1, rest=[(400, 1)])
        b = s.submit(0, 2, 0, 0, 610, [1] * 300, 1)
        c = s.submit(0, 3, 0, -150, 900, [1] * 200, 1, rest=[(100, 1)])
        keys[pol] = [s.reqs[r].key for r in (a, b, c)]
        order = s.queue_order()
        if pol == S.POLICY_PQ:
            assert order == [a, c, b]
        else:
            assert order == [b, c, a]
        st, info = s.step(0)
        assert info["admitted"] == [order[0]]
    assert keys[S.POLICY_PQ] == [100, 310, 300]
    assert keys[S.POLICY_LLF] == [500, 310, 450]


def test_urgency_is_negative_laxity_and_static_key():
    s = S.Scheduler(64, 8, 512, (0, 2 * S.PS, 0, 3 * S.PS), ITER)
    rid = s.submit(1000, 0, 0, 0, 50_000, list(range(40)), 5, rest=[(100, 10)])
    r = s.reqs[rid]
    for now in (1000, 2500, 99_000):
        u = S.urgency(r.t_comp, r.t_slo, now - r.enq)
        laxity = (r.enq + r.t_slo) - now - r.t_comp
        assert u == -laxity == now - r.key


def test_aging_overtakes_and_time_shift_invariance():
    s = S.Scheduler(64, 8, 512, UNIT_PREFILL, ITER)
    old = s.submit(0, 0, 0, 0, 10_000 + 100, list(range(100)), 1)      # slack 10000
    new = s.submit(3000, 1, 0, 3000, 7_500 + 100, list(range(100)), 1)  # slack 7500, 3000 us younger
    assert s.queue_order() == [old, new]     # older by 3000 > slack difference 2500
    s2 = S.Scheduler(64, 8, 512, UNIT_PREFILL, ITER)
    d = 123_456_789
    s2.submit(d, 0, 0, d, 10_100, list(range(100)), 1)
    s2.submit(3000 + d, 1, 0, 3000 + d, 7_600, list(range(100)), 1)
    assert s2.queue_order() == s.queue_order()
    assert [s2.reqs[i].t_slo for i in (1, 2)] == [s.reqs[i].t_slo for i in (1, 2)]


def test_stage_position_breaks_ties():
    s = S.Scheduler(64, 8, 512, UNIT_PREFILL, ITER)
    a = s.submit(0, 0, 1, 0, 1000 + 10, list(range(10)), 1)
    b = s.submit(0, 1, 3, 0, 1000 + 10, list(range(10)), 1)
    assert s.queue_order() == [b, a]


def _run(s, max_steps=10000):
    now, steps = 0, []
    for _ in range(max_steps):
        st, info = s.step(now)
        if st == S.IDLE:
            break
        steps.append(info)
        now += info["t_iter_us"]
    return steps


def test_continuous_batching_invariants():
    rng = np.random.default_rng(0)
    s = S.Scheduler(n_blocks=40, max_seqs=3, chunk_tokens=64, cost=(0, S.PS, 0, 20 * S.PS),
                    iter_cost=(500 * S.PS, S.PS, 0, 0))
    lens = [50, 130, 16, 17, 200, 1]
    ids = [s.submit(0, i, 0, 0, 10 ** 7, rng.integers(0, 2048, n), int(rng.integers(1, 9)))
           for i, n in enumerate(lens)]
    steps = _run(s)
    for info in steps:
        assert info["n_prefill_tokens"] <= 64
        assert len(info["batch_ids"]) <= 3
    for rid in ids:
        r = s.reqs[rid]
        assert r.state == S.DONE and len(r.generated) == r.max_new
        assert len(r.bt) == P.pages_for(len(r.context) + r.max_new - 1)
    assert s.alloc.n_free() == 40
    done = s.drain()
    assert sorted(d["id"] for d in done) == ids


def test_strict_head_of_line_admission():
    s = S.Scheduler(n_blocks=10, max_seqs=8, chunk_tokens=1000, cost=UNIT_PREFILL, iter_cost=ITER)
    big = s.submit(0, 0, 0, 0, 100, list(range(150)), 2)        # 10 pages, most urgent
    small = s.submit(0, 1, 0, 0, 10 ** 6, list(range(10)), 2)   # 1 page
    s.alloc.alloc(1)                                             # pool one short for `big`
    st, info = s.step(0)
    assert st == S.IDLE and s.queue_order() == [big, small]


def test_fork_shares_full_pages_and_reprefills_tail():
    s = S.Scheduler(n_blocks=64, max_seqs=8, chunk_tokens=256, cost=UNIT_PREFILL, iter_cost=ITER)
    par = s.submit(0, 0, 0, 0, 10 ** 6, list(range(40)), 3, retain=True)   # 42 tokens of KV
    _run(s)
    p = s.reqs[par]
    n = len(p.context) + len(p.generated)                  # 43 tokens, last one without KV
    assert n == 43 and len(p.bt) == 3
    kid = s.submit(100, 0, 1, 0, 10 ** 6, [5, 6], 4, parent=par)
    k = s.reqs[kid]
    shared = (n - 1) // 16
    assert k.bt == p.bt[:shared] and k.pf_pos0 == 16 * shared
    assert k.pf_tokens == (p.context + p.generated)[16 * shared:] + [5, 6]
    assert [s.alloc.ref[b] for b in p.bt] == [2, 2, 1]
    _run(s)
    assert len(k.bt) == P.pages_for(n + 2 + 3) and k.bt[:shared] == p.bt[:shared]
    assert [s.alloc.ref[b] for b in p.bt] == [1, 1, 1]
    s.release(par)
    assert s.alloc.n_free() == 64


def test_errors():
    s = S.Scheduler(n_blocks=4, max_seqs=8, chunk_tokens=64, cost=UNIT_PREFILL, iter_cost=ITER)
    with pytest.raises(S.SchedError) as e:
        s.submit(0, 0, 0, 0, 1, list(range(100)), 1)
    assert e.value.code == S.ENOMEM
    with pytest.raises(S.SchedError) as e:
        s.submit(0, 0, 0, 0, 1, [1], 0)
    assert e.value.code == S.EINVAL
    with pytest.raises(S.SchedError) as e:
        s.submit(0, 0, 0, 0, 1, [1], 1, parent=99)
    assert e.value.code == S.ENOTFOUND
    a = s.submit(0, 0, 0, 0, 1, [1], 1)
    with pytest.raises(S.SchedError) as e:
        s.submit(0, 0, 0, 0, 1, [1], 1, parent=a)
    assert e.value.code == S.ESTATE
    s.cancel(a)
    assert s.alloc.n_free() == 4 and s.queue_order() == []


def _engine_run(policy, weights, prompts, max_new, chunk=64):
    from oracle.engine import DecoderExecutor
    s = S.Scheduler(n_blocks=64, max_seqs=3, chunk_tokens=chunk, cost=(0, S.PS, 0, 30 * S.PS),
                    iter_cost=(500 * S.PS, S.PS, 0, 0), policy=policy, vocab=weights.shape.vocab)
    ex = DecoderExecutor(weights, keep_logits=False)
    slos = [10 ** 6, 3000, 10 ** 5, 2000]
    ids = [s.submit(0, i, 0, 0, slos[i], p, m) for i, (p, m) in enumerate(zip(prompts, max_new))]
    now = 0
    while True:
        st, info = s.step(now, executor=ex)
        if st == S.IDLE:
            break
        now += info["t_iter_us"]
    return {i: s.tokens(rid) for i, rid in enumerate(ids)}, s


def test_tokens_do_not_depend_on_policy():
    """Scheduling does not change model inputs (Section 4, problem formulation):
    PQ, FCFS and LLF give every request the same greedy tokens, equal to
    decoding each prompt on its own."""
    import synth
    from oracle import model as M
    w = M.Weights(synth.model_shape("tiny"))
    rng = np.random.default_rng(5)
    prompts = [rng.integers(0, 2048, n) for n in (40, 90, 17, 65)]
    max_new = [3, 5, 2, 4]
    runs = [_engine_run(p, w, prompts, max_new)[0] for p in (S.POLICY_PQ, S.POLICY_FCFS, S.POLICY_LLF)]
    assert runs[0] == runs[1] == runs[2]
    ref, _ = M.generate(w, prompts, max_new, keep_logits=False)
    assert [list(map(int, t)) for t in ref] == [runs[0][i] for i in range(4)]


def test_fork_tokens_equal_decoding_the_full_context():
    import synth
    from oracle import model as M
    from oracle.engine import DecoderExecutor
    w = M.Weights(synth.model_shape("tiny"))
    rng = np.random.default_rng(6)
    s = S.Scheduler(64, 4, 32, (0, S.PS, 0, S.PS), (S.PS, 0, 0, 0), vocab=2048)
    ex = DecoderExecutor(w, keep_logits=False)
    prompt = rng.integers(0, 2048, 37)
    par = s.submit(0, 0, 0, 0, 10 ** 6, prompt, 4, retain=True)
    _run_exec(s, ex)
    app = rng.integers(0, 2048, 5)
    kid = s.submit(0, 0, 1, 0, 10 ** 6, app, 3, parent=par)
    _run_exec(s, ex)
    full = list(prompt) + s.tokens(par) + list(app)
    ref, _ = M.generate(w, [np.asarray(full)], [3], keep_logits=False)
    assert s.tokens(kid) == list(map(int, ref[0]))


def _run_exec(s, ex):
    now = 0
    while True:
        st, info = s.step(now, executor=ex)
        if st == S.IDLE:
            return
        now += info["t_iter_us"]


def test_iteration_cost_terms():
    # hand value: 1 ms fixed, 2 us per prefill token, 3 ns per decode context token,
    # 5 ps per attention pair, 0.5 us per decode row
    it = (1000 * S.PS, 2 * S.PS, 3000, 5, S.PS // 2)
    assert S.t_iter(it, 100, 8, 40_000, 1_000_000) == 1000 + 200 + 120 + 5 + 4
    # four coefficients: a decode row costs what a prefill token does
    it4 = it[:4]
    for n_pf, n_dec in ((0, 64), (2048, 32), (17, 0)):
        assert S.t_iter(it4, n_pf, n_dec, 12345, 678) == S.t_iter(it4 + (it4[1],), n_pf, n_dec, 12345, 678)
    # floor toward minus infinity of the picosecond sum
    assert S.t_iter((S.PS - 1, 0, 0, 0, 0), 0, 0, 0, 0) == 0
