"""Oracle of the global coordinator over several instances -- TEST INFRASTRUCTURE ONLY.

Plain restatement of the paper's coordinator-level rules, driving oracle
schedulers (``oracle.sched.Scheduler``) on one virtual clock:

* Section 4.1, compute cost: t_comp of the request on each instance (its own
  cost model); queueing cost: the sum of t_comp over the instance's unfinished
  requests (``Scheduler.queue_cost``);
* Section 4.1, dispatch score ``(1 - alpha) * beta / t_queue - alpha * t_comp``,
  highest score wins; beta = C_ref * Q_ref;
* Section 4.2, SLO budget from the instance-average costs (``budget_cost_sum``
  of ``Scheduler.submit``);
* Section 4.3, alpha tuning: alpha = 0 at cold start; windows of completed
  queries; a one-sided two-sample t-test of the latest window's latencies
  against the previous window's; if p < 0.01, every alpha of {0, 0.1, ..., 1}
  is simulated on the recent trace and the one with the lowest 95th-percentile
  latency is kept.

Readings where the paper is silent (shared with the library's coordinator as
documented behaviour, not code): a fork runs on its parent's instance; a queue
cost of 0 counts as 1 us; score ties go to the lowest instance index; events at
one instant are taken as iteration ends (instance order), then arrivals, then
iteration starts (instance order); the t-test is Welch's (unequal variances); a
window closes at the first completion that gives it ``n_min`` queries and a span
of ``t_min_us``; the replayed trace is every query that arrived between the
earliest arrival among the compared windows' queries and the trigger; P95 ties go to the smaller alpha; beta's references
are means over the warm-up dispatches (alpha = 0) of the instances' mean t_comp
and mean t_queue (at least 1 us).

Workflows are plain dicts: ``wid``, ``arrival``, ``slo``, ``shapes`` (later
stages' (L_in, L_out)), ``stages``: lists of requests, each a dict with
``prompt``, ``max_new``, ``parent`` ((stage, index) or None) and ``retain``.
"""
import heapq
import math

from scipy import special

from . import sched as S


def wb_score(t_comp_us, t_queue_us, alpha, beta):
    """Dispatch score of Section 4.1 (an empty queue counts as 1 us)."""
    q = float(max(t_queue_us, 1))
    return (1.0 - alpha) * (beta / q) - alpha * float(t_comp_us)


def wb_select(t_comp_us, t_queue_us, alpha, beta):
    scores = [wb_score(c, q, alpha, beta) for c, q in zip(t_comp_us, t_queue_us)]
    best = max(scores)
    return scores.index(best)


def welch_t_greater(x_new, x_ref):
    """One-sided two-sample t-test (Section 4.3), H1: mean(x_new) > mean(x_ref),
    unequal variances: returns (t, dof, p)."""
    n1, n2 = len(x_new), len(x_ref)
    m1 = sum(float(v) for v in x_new) / n1
    m2 = sum(float(v) for v in x_ref) / n2
    v1 = sum((float(v) - m1) ** 2 for v in x_new) / (n1 - 1)
    v2 = sum((float(v) - m2) ** 2 for v in x_ref) / (n2 - 1)
    a, b = v1 / n1, v2 / n2
    if a + b == 0.0:
        if m1 > m2:
            return math.inf, float(n1 + n2 - 2), 0.0
        return (0.0 if m1 == m2 else -math.inf), float(n1 + n2 - 2), 1.0
    t = (m1 - m2) / math.sqrt(a + b)
    dof = (a + b) ** 2 / (a * a / (n1 - 1) + b * b / (n2 - 1))
    p = float(special.stdtr(dof, -t))     # P(T >= t) = P(T <= -t)
    return t, dof, p


def percentile95(values):
    """T_0.95 of Section 4.3, the time by which 95% of the queries have completed:
    the smallest value with at least 95% of the values at or below it."""
    ordered = sorted(values)
    for v in ordered:
        if 100 * sum(1 for u in ordered if u <= v) >= 95 * len(ordered):
            return v
    return ordered[-1]


class Coordinator:
    """specs: list of dicts with cost, iter, n_blocks, max_seqs, chunk, policy."""

    def __init__(self, specs, dispatch="wb", alpha=0.0, beta=1.0, tuner=None, vocab=2048, record=False):
        self.specs = specs
        self.n = len(specs)
        self.scheds = [S.Scheduler(s["n_blocks"], s["max_seqs"], s["chunk"], s["cost"], s["iter"],
                                   policy=s.get("policy", S.POLICY_PQ), vocab=vocab) for s in specs]
        self.cost_sum = tuple(sum(s["cost"][i] for s in specs) for i in range(4))
        self.dispatch, self.alpha, self.beta, self.tuner = dispatch, alpha, beta, tuner
        self.vocab = vocab
        self.next_rr = 0
        self.record = record
        self.decisions = []          # (mean t_comp, mean t_queue) per dispatch decision
        self.placements = []         # (time, wid, stage, index, instance, id)
        self.alpha_history = []      # (time, t, dof, p, new alpha or None)
        self.deadlocked = False

    def pick(self, prompt_len, max_new):
        if self.dispatch == "rr":
            m = self.next_rr % self.n
            self.next_rr += 1
            return m
        costs = [S.t_comp(s["cost"], prompt_len, max_new) for s in self.specs]
        # unfinished = queued or running, or finishing in an iteration still in flight
        queues = [sc.queue_cost() + sum(c["t_comp"] for c in fl) for sc, fl in zip(self.scheds, self.in_flight)]
        if self.record:
            self.decisions.append((sum(costs) / self.n, sum(queues) / self.n))
        return wb_select(costs, queues, self.alpha, self.beta)

    def start_stage(self, st, now):
        w = st["wf"]
        j = len(st["placed"])
        later = w["shapes"][j + 1:]
        row = []
        for k, q in enumerate(w["stages"][j]):
            if q["parent"] is None:
                m, par = self.pick(len(q["prompt"]), q["max_new"]), 0
            else:
                m, par = st["placed"][q["parent"][0]][q["parent"][1]]
            rid = self.scheds[m].submit(now, w["wid"], j, w["arrival"], w["slo"], q["prompt"], q["max_new"],
                                        parent=par, retain=q["retain"], rest=later,
                                        budget_cost_sum=self.cost_sum, n_inst=self.n)
            row.append((m, rid))
            self.owner[(m, rid)] = st
            self.placements.append((now, w["wid"], j, k, m, rid))
        st["placed"].append(row)
        st["finished"].append(0)
        for s_prev in range(j):
            forked_later = False
            for stage in w["stages"][j + 1:]:
                for q in stage:
                    if q["parent"] is not None and q["parent"][0] == s_prev:
                        forked_later = True
            if forked_later:
                continue
            for k, q in enumerate(w["stages"][s_prev]):
                if q["retain"] and st["placed"][s_prev][k] is not None:
                    m, rid = st["placed"][s_prev][k]
                    self.scheds[m].release(rid)
                    st["placed"][s_prev][k] = None

    def simulate(self, workflows):
        states = [dict(wf=w, placed=[], finished=[], finish=-1) for w in workflows]
        self.states_by_wf = states
        self.owner = {}
        events = []                  # (time, kind, key): kind 0 = iteration end of instance key, 1 = arrival
        for i, st in enumerate(states):
            heapq.heappush(events, (st["wf"]["arrival"], 1, i))
        running = [False] * self.n
        self.in_flight = [[] for _ in range(self.n)]   # completions of each instance's running iteration
        open_wf = 0
        window, window_t0, ref = [], None, None     # workflows completed in the open / previous window
        while events:
            now = events[0][0]
            batch = []
            while events and events[0][0] == now:
                batch.append(heapq.heappop(events))
            finished_now = []
            for _, kind, key in batch:       # iteration ends come first (kind 0), by instance
                if kind == 0:
                    running[key] = False
                    finished_now += [(key, c) for c in self.in_flight[key]]
                    self.in_flight[key] = []
            for key, c in finished_now:
                st = self.owner[(key, c["id"])]
                j = c["stage"]
                st["finished"][j] += 1
                if st["finished"][j] != len(st["wf"]["stages"][j]):
                    continue
                if j + 1 < len(st["wf"]["stages"]):
                    self.start_stage(st, now)
                    continue
                st["finish"] = now
                open_wf -= 1
                if self.tuner is not None:
                    if window_t0 is None:
                        window_t0 = now
                    window.append(st["wf"])
                    if len(window) >= self.tuner["n_min"] and now - window_t0 >= self.tuner["t_min_us"]:
                        if ref is not None:
                            self.regression_check(window, ref, now)
                        ref = window
                        window, window_t0 = [], now
            for _, kind, key in batch:
                if kind == 1:
                    self.start_stage(states[key], now)
                    open_wf += 1
            for m in range(self.n):
                if running[m]:
                    continue
                code, info = self.scheds[m].step(now)
                if code == S.IDLE:
                    continue
                running[m] = True
                self.in_flight[m] = self.scheds[m].drain()
                heapq.heappush(events, (now + info["t_iter_us"], 0, m))
        self.deadlocked = open_wf > 0
        self.states = states
        return [st["finish"] for st in states]

    def regression_check(self, new, ref, now):
        lat = {id(st["wf"]): st["finish"] - st["wf"]["arrival"] for st in self.states_by_wf}
        t, dof, p = welch_t_greater([lat[id(w)] for w in new], [lat[id(w)] for w in ref])
        alpha = None
        if p < self.tuner["p"]:
            since = min(w["arrival"] for w in ref + new)
            trace = [st["wf"] for st in self.states_by_wf if since <= st["wf"]["arrival"] <= now]
            alpha, _ = grid_search(self.specs, trace, self.beta, self.tuner["grid"], self.vocab)
            self.alpha = alpha
        self.alpha_history.append((now, t, dof, p, alpha))


def rebase(trace):
    t0 = min(w["arrival"] for w in trace)
    return [dict(w, arrival=w["arrival"] - t0) for w in trace]


def replay_p95(specs, trace, alpha, beta, vocab=2048):
    """T_0.95(alpha): P95 end-to-end latency of the trace on fresh instances."""
    co = Coordinator(specs, "wb", alpha, beta, vocab=vocab)
    wfs = rebase(trace)
    fin = co.simulate(wfs)
    return percentile95([f - w["arrival"] if f >= 0 else math.inf for f, w in zip(fin, wfs)])


def grid_search(specs, trace, beta, grid, vocab=2048):
    """alpha* = argmin of the simulated P95 over the grid (first minimum)."""
    vals = [replay_p95(specs, trace, a, beta, vocab) for a in grid]
    k = vals.index(min(vals))
    return grid[k], vals


def beta_from_warmup(specs, warmup, vocab=2048):
    """beta = C_ref * Q_ref from the warm-up queries dispatched with alpha = 0."""
    co = Coordinator(specs, "wb", 0.0, 1.0, vocab=vocab, record=True)
    co.simulate(rebase(warmup))
    if not co.decisions:
        return 1.0
    c_ref = sum(d[0] for d in co.decisions) / len(co.decisions)
    q_ref = sum(d[1] for d in co.decisions) / len(co.decisions)
    return c_ref * max(q_ref, 1.0)
