"""Host-side workflow driver for one instance.

Plays the role the paper gives its coordinator for one instance (Section 3.3,
"Multi-stage dependency management"): a query is a chain of stages; a stage
may fan out into parallel requests (candidates) and may fork from a retained
earlier request; stage j+1 is submitted when every request of stage j has
finished, with the remaining stages' shapes passed for the SLO budget.  All
scheduling arithmetic stays in the library; this module only sequences
submissions, releases retained KV that no later stage needs, and records
per-workflow latency against the end-to-end SLO.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

from . import hxf


@dataclass
class Req:
    prompt: np.ndarray               # token ids (appended tokens for a fork)
    max_new: int
    parent: Optional[Tuple[int, int]] = None   # (stage, request index) whose retained KV is continued
    retain: bool = False


@dataclass
class Workflow:
    wid: int
    arrival_us: int
    slo_us: int
    stages: List[List[Req]]
    shapes: List[Tuple[int, int]]    # representative (L_in, L_out) per stage, for later-stage budgets
    ids: List[List[int]] = field(default_factory=list)
    done: List[int] = field(default_factory=list)
    stage: int = -1
    finish_us: int = -1


class Driver:
    def __init__(self, inst, workflows, measured=False):
        self.inst = inst
        self.wf = sorted(workflows, key=lambda w: w.arrival_us)
        self.measured = measured
        self.deadlocked = False
        self.by_id = {}
        self.iterations = 0
        self.tokens = 0
        self.prefill_tokens = 0
        self.decode_tokens = 0
        self.stage_waits = {}        # stage index -> queueing delays (first scheduled - submitted), us

    def _submit_stage(self, w, now):
        w.stage += 1
        j = w.stage
        rest = w.shapes[j + 1:]
        ids = []
        for r in w.stages[j]:
            parent = 0 if r.parent is None else w.ids[r.parent[0]][r.parent[1]]
            rid = self.inst.submit(now, w.wid, j, w.arrival_us, w.slo_us, r.prompt, r.max_new, parent=parent,
                                   retain=r.retain, rest=rest)
            ids.append(rid)
            self.by_id[rid] = w
        w.ids.append(ids)
        w.done.append(0)
        # retained requests of earlier stages that no later stage forks from can go
        for s in range(j):
            needed = any(q.parent is not None and q.parent[0] == s for st in w.stages[j + 1:] for q in st)
            if needed:
                continue
            for k, q in enumerate(w.stages[s]):
                if q.retain and w.ids[s][k] is not None:
                    self.inst.release(w.ids[s][k])
                    w.ids[s][k] = None

    def run(self, max_iterations=10 ** 7, report=None, report_every=500):
        """Replay the workflows to completion; report(iterations, now_us, finished) is
        called every `report_every` iterations when given."""
        now, nxt = 0, 0
        active = 0
        while nxt < len(self.wf) or active:
            while nxt < len(self.wf) and self.wf[nxt].arrival_us <= now:
                self._submit_stage(self.wf[nxt], self.wf[nxt].arrival_us if not self.measured else now)
                nxt += 1
                active += 1
            st, info = self.inst.step(now)
            if st == hxf.IDLE:
                if nxt < len(self.wf):
                    now = max(now, self.wf[nxt].arrival_us)
                    continue
                if active:
                    # Nothing is runnable, nothing else arrives, and workflows are unfinished:
                    # the KV that finished stages retain for their forks fills the pool and the
                    # queued requests cannot be admitted (no preemption).  Stop; the unfinished
                    # workflows count as SLO misses.
                    self.deadlocked = True
                break
            self.iterations += 1
            self.tokens += info["n_tokens"]
            self.prefill_tokens += info["n_prefill_tokens"]
            self.decode_tokens += info["n_logit_rows"]
            now += info["t_iter_us"]
            for c in self.inst.drain():
                w = self.by_id[c["id"]]
                j = c["stage_index"]
                if "t_first_sched_us" in c:
                    self.stage_waits.setdefault(j, []).append(c["t_first_sched_us"] - c["t_submit_us"])
                w.done[j] += 1
                if w.done[j] == len(w.stages[j]):
                    if j + 1 < len(w.stages):
                        self._submit_stage(w, c["t_finish_us"])
                    else:
                        w.finish_us = c["t_finish_us"]
                        active -= 1
            if report is not None and self.iterations % report_every == 0:
                report(self.iterations, now, sum(1 for w in self.wf if w.finish_us >= 0))
            if self.iterations >= max_iterations:
                raise RuntimeError("iteration limit")
        return now

    def stats(self):
        """Latency and SLO attainment per workflow; a workflow that never finished (a
        deadlocked run) has infinite latency and misses its SLO."""
        done = [w for w in self.wf if w.finish_us >= 0]
        lat = np.array([w.finish_us - w.arrival_us if w.finish_us >= 0 else np.inf for w in self.wf], dtype=np.float64)
        slo = np.array([w.slo_us for w in self.wf], dtype=np.float64)
        makespan = max(w.finish_us for w in done) - min(w.arrival_us for w in self.wf) if done else 0
        p95 = float(np.percentile(lat, 95))
        waits = [np.asarray(self.stage_waits.get(j, [0]), dtype=np.float64) / 1e6
                 for j in range(max(self.stage_waits, default=-1) + 1)]
        return {
            "workflows": len(self.wf),
            "finished": len(done),
            "deadlocked": self.deadlocked,
            "slo_attainment": float(np.mean(lat <= slo)),
            "p95_latency_s": p95 / 1e6 if np.isfinite(p95) else None,
            "mean_latency_s": float(np.mean([w.finish_us - w.arrival_us for w in done]) / 1e6) if done else None,
            "p95_slo_scale": float(np.percentile(lat / (slo / 10.0), 95)) if np.isfinite(p95) else None,
            "throughput_wf_per_s": len(done) / (makespan / 1e6) if makespan > 0 else 0.0,
            # workflows in flight, averaged over the run (Little's law: total latency / makespan)
            "mean_in_flight": float(sum(w.finish_us - w.arrival_us for w in done) / makespan) if makespan > 0 else 0.0,
            # per stage index: mean and P95 of the requests' queueing delay (submission to first batch)
            "stage_wait_mean_s": [round(float(np.mean(x)), 3) for x in waits],
            "stage_wait_p95_s": [round(float(np.percentile(x, 95)), 3) for x in waits],
            "iterations": self.iterations,
            "prefill_tokens": self.prefill_tokens,
            "decode_tokens": self.decode_tokens,
        }
