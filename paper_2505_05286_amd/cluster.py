"""Several serving instances under one global coordinator, on one virtual clock.

The paper schedules at two levels (Section 3.2): a global coordinator assigns
each LLM request of a workflow to a model instance, and every instance orders
its own queue by urgency (Section 4.2).  This module is the coordinator's
event loop over N library instances in scheduler-only mode (no device work:
each iteration lasts what the instance's calibrated cost model says), so a
heterogeneous cluster can be studied on the CPU.  It provides

* workload-balanced dispatch (Section 4.1): t_comp and t_queue per instance and
  the score (1 - alpha) * beta / t_queue - alpha * t_comp, all computed by the
  library (hxf_request_cost, hxf_queue_cost, hxf_wb_select), with round-robin as
  the load-agnostic baseline;
* per-request SLO budgets from the instance-average costs (Section 4.2,
  hxf_submit_shared);
* online alpha tuning (Section 4.3): alpha starts at 0; a sliding window of
  completed queries; a one-sided t-test (hxf_ttest_greater) of the new window's
  latencies against the previous window's; on p < 0.01 the recent trace is
  replayed for alpha in {0, 0.1, ..., 1} and the alpha with the lowest simulated
  95th-percentile latency is taken;
* the once-per-deployment calibration of beta = C_ref * Q_ref from warm-up
  queries.

Rules the paper leaves open (each is a stated reading, also followed by the
host reference):

* A request that continues a retained parent's KV (a fork) goes to the parent's
  instance: KV is not moved between instances.  Every other request is
  dispatched by the coordinator.
* Event order at one instant: first the completions of iterations ending then
  (instances in index order, completions in finishing order, each possibly
  dispatching the next stage), then workflow arrivals, then every idle instance
  with work starts its next iteration (index order).
* Window: it closes at the first query completion at which it holds at least
  ``n_min`` completed queries and spans at least ``t_min_us``; the next window
  opens there.  The t-test compares the end-to-end latencies of the queries
  completed in the two most recent windows.
* Replayed trace: every query that arrived from the earliest arrival among the
  two windows' queries up to the trigger (the compared queries and the load
  around them), replayed from empty instances with the same configurations and
  relative arrival times.  T_0.95 is the ceil(0.95 n)-th smallest latency; ties
  go to the smaller alpha.
* beta: C_ref is the mean over the warm-up dispatches of the instances' mean
  t_comp for the request, Q_ref the mean over the same dispatches of the
  instances' mean t_queue (at least 1 us); the warm-up dispatches with alpha = 0.
"""
import time
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

from . import hxf

ALPHA_GRID = tuple(k / 10.0 for k in range(11))


@dataclass
class InstanceSpec:
    """One instance of the cluster: its cost models (ps coefficients, as in
    hxf_sched_cfg) and capacity."""
    cost_ps: tuple
    iter_ps: tuple
    n_blocks: int
    max_seqs: int
    chunk_tokens: int
    policy: int = hxf.POLICY_PQ


@dataclass
class TunerCfg:
    n_min: int = 5               # completed queries per window, at least (the paper's example)
    t_min_us: int = 0            # window span, at least
    p_threshold: float = 0.01
    grid: tuple = ALPHA_GRID


@dataclass
class _Flow:
    wf: object                   # workflows.Workflow (read only)
    stage: int = -1
    done: List[int] = field(default_factory=list)
    reqs: List[list] = field(default_factory=list)   # per stage: [(instance, id) or None]
    finish_us: int = -1


def completion_p95(latencies):
    """The time within which 95% of the queries completed (Section 4.3's T_0.95): the
    ceil(0.95 n)-th smallest latency; a query that never completed counts as infinite."""
    v = sorted(latencies)
    return v[(95 * len(v) + 99) // 100 - 1]


class Cluster:
    """N scheduler-only instances and the coordinator.  ``dispatch`` is "wb"
    (workload-balanced, Section 4.1) or "rr" (round-robin)."""

    def __init__(self, mcfg, specs, dispatch="wb", alpha=0.0, beta=1.0, tuner: Optional[TunerCfg] = None,
                 record_dispatch=False):
        if dispatch not in ("wb", "rr"):
            raise ValueError("dispatch must be 'wb' or 'rr'")
        self.mcfg, self.specs = mcfg, list(specs)
        self.n = len(self.specs)
        self.dispatch, self.alpha, self.beta, self.tuner = dispatch, float(alpha), float(beta), tuner
        self.record_dispatch = record_dispatch
        self.inst = [hxf.Instance(mcfg, hxf.sched_cfg(s.n_blocks, s.max_seqs, s.chunk_tokens, s.cost_ps, s.iter_ps,
                                                      policy=s.policy, executor=hxf.EXEC_NULL))
                     for s in self.specs]
        self.cost_sum = tuple(sum(int(s.cost_ps[i]) for s in self.specs) for i in range(4))
        self.rr = 0
        self.log = []                # (time, workflow, stage, index, instance, id) per request
        self.dispatch_log = []       # (mean t_comp, mean t_queue) per coordinator decision
        self.alpha_log = []          # (time, t, dof, p, alpha chosen or None)
        self.tune_seconds = []       # host time of each alpha grid search
        self.deadlocked = False
        self.iterations = 0

    # ------------------------------------------------------------ coordinator
    def _choose(self, prompt_len, max_new):
        if self.dispatch == "rr":
            m = self.rr % self.n
            self.rr += 1
            return m
        comp = [i.request_cost(prompt_len, max_new) for i in self.inst]
        # an instance's iteration is run when it starts; the requests it finishes are
        # still unfinished until its end, so they are added back
        queue = [i.queue_cost() + sum(c["t_comp_us"] for c in p) for i, p in zip(self.inst, self.pending)]
        if self.record_dispatch:
            self.dispatch_log.append((sum(comp) / self.n, sum(queue) / self.n))
        return hxf.wb_select(comp, queue, self.alpha, self.beta)

    def _submit_stage(self, f, now):
        w = f.wf
        f.stage += 1
        j = f.stage
        rest = w.shapes[j + 1:]
        placed = []
        for k, r in enumerate(w.stages[j]):
            if r.parent is not None:
                m, pid = f.reqs[r.parent[0]][r.parent[1]]
            else:
                m, pid = self._choose(len(r.prompt), r.max_new), 0
            rid = self.inst[m].submit(now, w.wid, j, w.arrival_us, w.slo_us, r.prompt, r.max_new, parent=pid,
                                      retain=r.retain, rest=rest, cost_sum=self.cost_sum, n_instances=self.n)
            placed.append((m, rid))
            self.by_req[(m, rid)] = f
            self.log.append((now, w.wid, j, k, m, rid))
        f.reqs.append(placed)
        f.done.append(0)
        # retained requests that no later stage forks from are released
        for s in range(j):
            if any(q.parent is not None and q.parent[0] == s for st in w.stages[j + 1:] for q in st):
                continue
            for k, q in enumerate(w.stages[s]):
                if q.retain and f.reqs[s][k] is not None:
                    m, rid = f.reqs[s][k]
                    self.inst[m].release(rid)
                    f.reqs[s][k] = None

    # ------------------------------------------------------------ event loop
    def run(self, workflows, max_iterations=10 ** 8):
        """Replay the workflows (workflows.Workflow records, not modified); returns
        the per-workflow finish times (-1: never finished) in the input order."""
        flows = self.flows = [_Flow(w) for w in workflows]
        order = sorted(range(len(flows)), key=lambda i: (flows[i].wf.arrival_us, i))
        self.by_req = {}
        busy: List[Optional[int]] = [None] * self.n
        pending = self.pending = [[] for _ in range(self.n)]
        nxt, active = 0, 0
        win, win_start, ref = [], None, None     # queries completed in the open / previous window
        t = flows[order[0]].wf.arrival_us if flows else 0
        while True:
            ended = []
            for m in range(self.n):
                if busy[m] == t:
                    busy[m] = None
                    ended.extend((m, c) for c in pending[m])
                    pending[m] = []
            for m, c in ended:
                f = self.by_req[(m, c["id"])]
                j = c["stage_index"]
                f.done[j] += 1
                if f.done[j] < len(f.wf.stages[j]):
                    continue
                if j + 1 < len(f.wf.stages):
                    self._submit_stage(f, t)
                    continue
                f.finish_us = t
                active -= 1
                if self.tuner is not None:
                    if win_start is None:
                        win_start = t
                    win.append(f)
                    if len(win) >= self.tuner.n_min and t - win_start >= self.tuner.t_min_us:
                        if ref is not None:
                            self._check_regression(win, ref, t)
                        ref = win
                        win, win_start = [], t
            while nxt < len(order) and flows[order[nxt]].wf.arrival_us <= t:
                self._submit_stage(flows[order[nxt]], t)
                nxt += 1
                active += 1
            for m in range(self.n):
                if busy[m] is not None:
                    continue
                st, info = self.inst[m].step(t)
                if st == hxf.IDLE:
                    continue
                self.iterations += 1
                busy[m] = t + info["t_iter_us"]
                pending[m] = self.inst[m].drain()
            cand = [b for b in busy if b is not None]
            if nxt < len(order):
                cand.append(flows[order[nxt]].wf.arrival_us)
            if not cand:
                # nothing runs and nothing arrives: unfinished workflows are stuck (their
                # queued requests can never be admitted)
                self.deadlocked = active > 0
                break
            t = min(cand)
            if self.iterations >= max_iterations:
                raise RuntimeError("iteration limit")
        self.flows = flows
        return [f.finish_us for f in flows]

    # ------------------------------------------------------------ alpha tuning
    def _check_regression(self, new, ref, now):
        tstat, dof, p = hxf.ttest_greater([f.finish_us - f.wf.arrival_us for f in new],
                                          [f.finish_us - f.wf.arrival_us for f in ref])
        chosen = None
        if p < self.tuner.p_threshold:
            t0 = min(f.wf.arrival_us for f in ref + new)
            trace = [f.wf for f in self.flows if t0 <= f.wf.arrival_us <= now]
            c0 = time.perf_counter()
            chosen, _ = tune_alpha(self.mcfg, self.specs, trace, self.beta, self.tuner.grid)
            self.tune_seconds.append(time.perf_counter() - c0)
            self.alpha = chosen
        self.alpha_log.append((now, tstat, dof, p, chosen))

    def stats(self):
        lat = np.array([f.finish_us - f.wf.arrival_us if f.finish_us >= 0 else np.inf for f in self.flows])
        slo = np.array([f.wf.slo_us for f in self.flows], dtype=np.float64)
        pp = float(completion_p95(list(lat)))
        return {"workflows": len(self.flows), "finished": int(np.sum(np.isfinite(lat))),
                "deadlocked": self.deadlocked, "slo_attainment": float(np.mean(lat <= slo)),
                "p95_latency_s": pp / 1e6 if np.isfinite(pp) else None,
                "mean_latency_s": float(np.mean(lat[np.isfinite(lat)]) / 1e6) if np.isfinite(lat).any() else None,
                "iterations": self.iterations,
                "per_instance_requests": [sum(1 for e in self.log if e[4] == m) for m in range(self.n)]}

    def close(self):
        for i in self.inst:
            i.close()


def _shifted(trace):
    """The trace with arrivals relative to its first arrival."""
    from dataclasses import replace
    t0 = min(w.arrival_us for w in trace)
    return [replace(w, arrival_us=w.arrival_us - t0) for w in trace]


def simulated_p95(mcfg, specs, trace, alpha, beta):
    """T_0.95(alpha) of Section 4.3 on the trace replayed on a fresh cluster with fixed
    alpha (a query that never finishes, e.g. when its instance's KV pool fills with
    retained pages, counts as infinite)."""
    c = Cluster(mcfg, specs, "wb", alpha, beta)
    wfs = _shifted(trace)
    fin = c.run(wfs)
    c.close()
    return completion_p95([f - w.arrival_us if f >= 0 else float("inf") for f, w in zip(fin, wfs)])


def tune_alpha(mcfg, specs, trace, beta, grid=ALPHA_GRID):
    """alpha* = argmin over the grid of the simulated P95 (Section 4.3); ties go to the
    smaller alpha.  Returns (alpha*, [P95 per grid value])."""
    vals = [simulated_p95(mcfg, specs, trace, a, beta) for a in grid]
    best = 0
    for k in range(1, len(vals)):
        if vals[k] < vals[best]:
            best = k
    return grid[best], vals


def calibrate_beta(mcfg, specs, warmup):
    """beta = C_ref * Q_ref (Section 4.1) from the warm-up queries, dispatched with
    alpha = 0: C_ref = mean over the coordinator's decisions of the instances' mean
    t_comp, Q_ref = the same mean of their t_queue (at least 1 us)."""
    c = Cluster(mcfg, specs, "wb", 0.0, 1.0, record_dispatch=True)
    c.run(_shifted(warmup))
    c.close()
    if not c.dispatch_log:
        return 1.0
    c_ref = sum(d[0] for d in c.dispatch_log) / len(c.dispatch_log)
    q_ref = sum(d[1] for d in c.dispatch_log) / len(c.dispatch_log)
    return c_ref * max(q_ref, 1.0)
