"""Workload-5 replay (four-stage workflows with forks, Poisson arrivals) on the
virtual clock: the library's scheduler (scheduler-only executor) and the
oracle scheduler, driven by the same workflow driver, must finish every
workflow at the same virtual time; the local-queue policies are compared."""
import numpy as np
import pytest

import synth
from oracle import sched as S
from paper_2505_05286_amd import hxf
from paper_2505_05286_amd.workflows import Driver, Req, Workflow

from ._lib import ensure_built

COST = (6_000 * S.PS, 110 * S.PS, 8_000, 30_000 * S.PS)
ITER = (28_000 * S.PS, 100 * S.PS, 48_000, 2_800)
SHAPE = dict(s1_out=64, n_cand=8, cand_out=256, n_corr=4, corr_in=512, corr_out=256, eval_in=1024, eval_out=128)


def workflows(n, scale=8):
    """Workload-5 streams with every length divided by `scale` (keeps the oracle fast)."""
    out = []
    s = SHAPE
    for w in synth.workloads.cfg5(vocab=2048, n_wf=n):
        l1 = max(16, w.schema_len // scale)
        stages = [[Req(w.schema[:l1], s["s1_out"] // scale, retain=True)],
                  [Req(np.zeros(0, np.int32), s["cand_out"] // scale, parent=(0, 0), retain=(b % 2 == 0))
                   for b in range(s["n_cand"])],
                  [Req(w.corrections[k][: s["corr_in"] // scale], s["corr_out"] // scale, parent=(1, 2 * k))
                   for k in range(s["n_corr"])],
                  [Req(w.eval_prompt[: s["eval_in"] // scale], s["eval_out"] // scale)]]
        shapes = [(l1, s["s1_out"] // scale), (16, s["cand_out"] // scale),
                  (16 + s["corr_in"] // scale, s["corr_out"] // scale), (s["eval_in"] // scale, s["eval_out"] // scale)]
        slo = int(w.slo_us // 20)
        out.append(Workflow(w.workflow, w.arrival_us // 4, slo, stages, shapes))
    return out


class OracleInstance:
    """The oracle scheduler behind the binding's Instance interface."""

    def __init__(self, n_blocks, max_seqs, chunk, policy):
        self.s = S.Scheduler(n_blocks, max_seqs, chunk, COST, ITER, policy=policy, vocab=2048)

    def submit(self, now, wf, stage, arr, slo, prompt, max_new, parent=0, retain=False, rest=()):
        return self.s.submit(now, wf, stage, arr, slo, list(map(int, prompt)), max_new, parent=parent, retain=retain,
                             rest=rest)

    def step(self, now):
        st, info = self.s.step(now)
        return (hxf.IDLE if st == S.IDLE else hxf.OK), info

    def drain(self):
        return [dict(id=d["id"], stage_index=d["stage"], t_finish_us=d["t_finish"], t_submit_us=d["t_submit"],
                     t_first_sched_us=d["t_first_sched"]) for d in self.s.drain()]

    def release(self, rid):
        self.s.release(rid)


def library_instance(n_blocks, max_seqs, chunk, policy):
    ensure_built()
    shape = synth.ModelShape("sched", 1, 64, 1, 1, 64, 64, 2048, 0)
    return hxf.Instance(hxf.model_cfg(shape, 1 << 20),
                        hxf.sched_cfg(n_blocks, max_seqs, chunk, COST, ITER, policy=policy, executor=hxf.EXEC_NULL))


@pytest.mark.parametrize("policy", [S.POLICY_PQ, S.POLICY_FCFS])
def test_workflow_replay_matches_oracle(policy):
    wf_a, wf_b = workflows(24), workflows(24)
    a = Driver(library_instance(3000, 48, 256, policy), wf_a)
    b = Driver(OracleInstance(3000, 48, 256, policy), wf_b)
    a.run()
    b.run()
    assert [w.finish_us for w in wf_a] == [w.finish_us for w in wf_b]
    assert a.stats() == b.stats()
    assert all(w.finish_us > w.arrival_us for w in wf_a)


def test_policies_on_workload5_shape():
    """Local-queue ablation on one instance (Section 5.3 compares PQ with FCFS):
    all policies serve every workflow; the numbers are reported, not asserted."""
    res = {}
    for name, pol in (("pq", hxf.POLICY_PQ), ("fcfs", hxf.POLICY_FCFS), ("llf", hxf.POLICY_LLF)):
        wf = workflows(120)
        d = Driver(library_instance(6000, 64, 512, pol), wf)
        d.run()
        res[name] = d.stats()
        assert res[name]["workflows"] == 120
    print({k: (round(v["slo_attainment"], 3), round(v["p95_latency_s"], 2)) for k, v in res.items()})
