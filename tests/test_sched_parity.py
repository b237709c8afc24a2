"""The library's host scheduler (scheduler-only executor, no GPU) against the
oracle scheduler: queue order, per-iteration batches and admissions, block
tables, timestamps, budgets and tokens must be bit-identical."""
import numpy as np
import pytest

import synth
from oracle import sched as S
from paper_2505_05286_amd import hxf

from ._lib import ensure_built


@pytest.fixture(scope="module", autouse=True)
def _built():
    ensure_built()


class Pair:
    """The same action stream applied to the oracle and to the library."""

    def __init__(self, n_blocks, max_seqs, chunk, cost, it, policy=S.POLICY_PQ, vocab=2048, max_context=1 << 20):
        self.o = S.Scheduler(n_blocks, max_seqs, chunk, cost, it, policy=policy, vocab=vocab)
        shape = synth.ModelShape("sched", 1, 64, 1, 1, 64, 64, vocab, 0)
        mcfg = hxf.model_cfg(shape, max_context)
        scfg = hxf.sched_cfg(n_blocks, max_seqs, chunk, cost, it, policy=policy, executor=hxf.EXEC_NULL)
        self.g = hxf.Instance(mcfg, scfg)
        self.ids = []

    def submit(self, now, wf, stage, arr, slo, prompt, max_new, parent=0, retain=False, rest=()):
        err_o = err_g = None
        try:
            a = self.o.submit(now, wf, stage, arr, slo, list(prompt), max_new, parent=parent, retain=retain,
                              rest=rest)
        except S.SchedError as e:
            err_o, a = e.code, None
        try:
            b = self.g.submit(now, wf, stage, arr, slo, prompt, max_new, parent=parent, retain=retain, rest=rest)
        except hxf.HxfError as e:
            err_g, b = e.code, None
        assert err_o == err_g and a == b
        if a is not None:
            ra, rb = self.o.reqs[a], self.g.request_state(a)
            assert (ra.t_comp, ra.t_slo, ra.key, ra.enq) == (rb["t_comp_us"], rb["t_slo_us"], rb["key_us"],
                                                             rb["t_submit_us"])
            self.ids.append(a)
        assert self.o.queue_order() == self.g.queue_order()
        return a

    def step(self, now):
        so, io = self.o.step(now)
        sg, ig = self.g.step(now)
        assert so == sg
        if so == S.IDLE:
            return so, None
        ids, adm = self.g.last_batch()
        assert ids == io["batch_ids"] and adm == io["admitted"]
        for k in ("n_tokens", "n_decode", "n_prefill_tokens", "n_logit_rows", "t_iter_us", "n_admitted",
                  "n_finished", "free_blocks", "sum_decode_ctx", "prefill_attn"):
            assert ig[k] == io[k], k
        assert self.o.queue_order() == self.g.queue_order()
        return so, io

    def check_all(self):
        for rid in self.ids:
            assert self.o.tokens(rid) == self.g.tokens(rid)
            assert self.o.block_table(rid) == self.g.block_table(rid)
            assert self.o.reqs[rid].state == self.g.request_state(rid)["state"]
        do = self.o.drain()
        dg = self.g.drain()
        assert len(do) == len(dg)
        for a, b in zip(do, dg):
            for k in ("id", "workflow", "stage", "t_submit", "t_first_sched", "t_first_token", "t_finish", "t_slo",
                      "t_comp", "n_generated", "met_slo"):
                kb = {"workflow": "workflow_id", "stage": "stage_index"}.get(k, k)
                kb = kb if kb in b else kb + "_us"
                assert a[k] == b[kb], k

    def run(self, now=0, max_steps=100000):
        for _ in range(max_steps):
            st, info = self.step(now)
            if st == S.IDLE:
                return now
            now += info["t_iter_us"]
        raise AssertionError("did not drain")


COST = (300 * S.PS, 2 * S.PS, 1, 40 * S.PS)
ITER = (800 * S.PS, 3 * S.PS, S.PS // 50, 1)
ITER5 = (800 * S.PS, 3 * S.PS, S.PS // 50, 1, S.PS // 7)     # decode rows priced apart


@pytest.mark.parametrize("it", [ITER, ITER5])
@pytest.mark.parametrize("policy", [S.POLICY_PQ, S.POLICY_FCFS, S.POLICY_LLF])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_streams_match(policy, seed, it):
    rng = np.random.default_rng(100 + seed)
    p = Pair(n_blocks=int(rng.integers(40, 120)), max_seqs=int(rng.integers(2, 9)), chunk=int(rng.integers(16, 200)),
             cost=COST, it=it, policy=policy)
    now = 0
    retained = []
    for k in range(60):
        r = rng.random()
        if r < 0.45:
            n = int(rng.integers(1, 300))
            nst = int(rng.integers(0, 4))
            rest = [(int(rng.integers(1, 500)), int(rng.integers(1, 50))) for _ in range(nst)]
            rid = p.submit(now, k, int(rng.integers(0, 4)), now - int(rng.integers(0, 5000)),
                           int(rng.integers(1000, 200000)), rng.integers(0, 2048, n), int(rng.integers(0, 12)),
                           retain=bool(rng.random() < 0.3), rest=rest)
            if rid is not None and p.o.reqs[rid].retain:
                retained.append(rid)
        elif r < 0.55 and retained:
            par = retained[int(rng.integers(0, len(retained)))]
            p.submit(now, 999, 2, 0, 50000, rng.integers(0, 2048, int(rng.integers(0, 40))),
                     int(rng.integers(1, 10)), parent=par)
        elif r < 0.6 and retained:
            rid = retained.pop(int(rng.integers(0, len(retained))))
            eo = eg = None
            try:
                p.o.release(rid)
            except S.SchedError as e:
                eo = e.code
            try:
                p.g.release(rid)
            except hxf.HxfError as e:
                eg = e.code
            assert eo == eg
            if eo is not None:
                retained.append(rid)
        elif r < 0.63 and p.ids:
            rid = p.ids[int(rng.integers(0, len(p.ids)))]
            eo = eg = None
            try:
                p.o.cancel(rid)
            except S.SchedError as e:
                eo = e.code
            try:
                p.g.cancel(rid)
            except hxf.HxfError as e:
                eg = e.code
            assert eo == eg
        else:
            st, info = p.step(now)
            now += info["t_iter_us"] if info else int(rng.integers(1, 3000))
    p.run(now)
    p.check_all()


def test_table2_selection_matches():
    now = 70_000_000
    rows = [(1, 22.4, 14.5), (2, 46.3, 13.2), (3, 52.3, 19.0), (4, 62.4, 13.1), (5, 62.8, 19.0), (6, 64.4, 26.9),
            (7, 65.0, 21.9)]
    p = Pair(64, 1, 4096, (0, S.PS, 0, 0), (1000 * S.PS, 0, 0, 0))
    for rid, a, u in rows:
        a, u = round(a * 1e6), round(u * 1e6)
        p.submit(a, rid, 0, a, 100 + now - a - u, list(range(100)), 1)
    assert p.g.queue_order() == [6, 7, 3, 5, 1, 2, 4]
    st, info = p.step(now)
    assert info["admitted"] == [6]


def test_forks_and_cfg4_shape_match():
    """Prefix-shared forks (4096-token parents, 8 branches, corrections on even branches), small scale."""
    p = Pair(n_blocks=2000, max_seqs=64, chunk=512, cost=COST, it=ITER)
    rng = np.random.default_rng(3)
    parents = [p.submit(0, w, 0, 0, 10 ** 9, rng.integers(0, 2048, 300), 0, retain=True) for w in range(4)]
    now = p.run(0)
    forks = {}
    for w, par in enumerate(parents):
        for b in range(8):
            forks[(w, b)] = p.submit(now, w, 1, 0, 10 ** 9, [], 20, parent=par, retain=(b % 2 == 0))
    now = p.run(now)
    for w in range(4):
        for b in range(0, 8, 2):
            p.submit(now, w, 2, 0, 10 ** 9, rng.integers(0, 2048, 40), 1, parent=forks[(w, b)])
    p.run(now)
    p.check_all()
    # all siblings of one parent share its first (n-1)//16 pages
    for w, par in enumerate(parents):
        s = (300 - 1) // 16
        for b in range(8):
            assert p.g.block_table(forks[(w, b)])[:s] == p.g.block_table(par)[:s]


def test_errors_match():
    p = Pair(n_blocks=4, max_seqs=2, chunk=64, cost=COST, it=ITER, max_context=1 << 20)
    p.submit(0, 0, 0, 0, 1, list(range(100)), 1)       # ENOMEM
    p.submit(0, 0, 0, 0, 1, [1], 0)                    # EINVAL
    p.submit(0, 0, 0, 0, 1, [1], 1, parent=77)         # ENOTFOUND
    a = p.submit(0, 0, 0, 0, 1, [1], 1)
    p.submit(0, 0, 0, 0, 1, [1], 1, parent=a)          # ESTATE
    p.submit(0, 0, 0, 0, 1, [5000], 1)                 # token out of range


def test_budget_int64_extremes_match():
    p = Pair(64, 4, 64, (0, 10 ** 12, 10 ** 9, 10 ** 12), ITER)
    p.submit(-(10 ** 15), 0, 0, -(10 ** 15) - 7, 4 * 10 ** 15, list(range(40)), 3, rest=[(1000, 500)] * 7)
    p.submit(10 ** 12, 1, 1, 0, -(10 ** 9), list(range(20)), 2, rest=[(3, 4)])
    p.run(0)
    p.check_all()
