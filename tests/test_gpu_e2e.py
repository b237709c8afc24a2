"""End-to-end parity of the serving instance on the GPU (hxf_submit / hxf_step /
hxf_drain through the C ABI) against the CPU oracle.

Bit-exact: queue order, per-iteration batches and admissions, block tables
(the oracle scheduler decides them from lengths alone), greedy token ids.
Floating point: fp32 logits of every sampled row within 2e-2 of the oracle's
float64 logits, measured as max|diff| / max|ref| per row.  Argmax decisions
are compared under teacher forcing (both sides fed the oracle's tokens); a
differing id is accepted only as a near-tie: the oracle's logit of the GPU's
id is within 2e-2 * max|ref| of the oracle's maximum.
"""
import numpy as np
import pytest

import synth
from oracle import model as M
from oracle import sched as S
from paper_2505_05286_amd import hxf
from paper_2505_05286_amd.device import DeviceModel, Engine

from .gpu_util import log, rel_max_err

pytestmark = pytest.mark.gpu

TOL = 2e-2
COST = (200 * S.PS, 50_000, 10, 150 * S.PS)
ITER = (500 * S.PS, 1000, 20, 1)

_models = {}


def device_model(name, n_layers=None):
    key = (name, n_layers)
    if key not in _models:
        _models.clear()
        shape = synth.model_shape(name, n_layers)
        log(f"uploading {shape.name}")
        gains = synth.gen_norm_gains(shape)       # a distinct gain per norm: miswired norms fail
        _models[key] = (shape, DeviceModel(shape, lambda l: synth.gen_layer(shape, l), synth.gen_embed(shape),
                                           synth.gen_lm_head(shape), gains, device="cuda:0"),
                        M.Weights(shape, norm_gains=gains))
    return _models[key]


def run_engine(eng, reqs, forced=None, now=0, keep_logits=True):
    """Submit (wf, stage, prompt, max_new, slo, kwargs) records, step to idle.
    Returns ids, per-id list of logits rows, per-step (batch ids, admitted)."""
    ids = []
    for i, (wf, stage, prompt, mx, slo, kw) in enumerate(reqs):
        ids.append(eng.inst.submit(now, wf, stage, now, slo, prompt, mx,
                                   forced=None if forced is None else forced[i], **kw))
    logits = {r: [] for r in ids}
    steps = []
    while True:
        st, info = eng.inst.step(now)
        if st == hxf.IDLE:
            break
        steps.append(eng.inst.last_batch())
        if keep_logits:
            for r in ids:
                try:
                    logits[r].append(eng.inst.last_logits(r))
                except hxf.HxfError:
                    pass
        now += info["t_iter_us"]
    return ids, logits, steps, now


def oracle_schedule(reqs, n_blocks, max_seqs, chunk, vocab):
    s = S.Scheduler(n_blocks, max_seqs, chunk, COST, ITER, vocab=vocab)
    ids = [s.submit(0, wf, st, 0, slo, list(p), mx, **kw) for wf, st, p, mx, slo, kw in reqs]
    order = s.queue_order()
    steps, now = [], 0
    while True:
        st, info = s.step(now)
        if st == S.IDLE:
            break
        steps.append((info["batch_ids"], info["admitted"]))
        now += info["t_iter_us"]
    return ids, order, steps, {r: s.block_table(r) for r in ids}


def compare_free_running(name, gpu_tok, ref_tok, ref_lg):
    """Free-running greedy ids must equal the oracle's up to the first near tie (the
    oracle's logit of the GPU's choice within TOL * max|logit| of its own top logit);
    the contexts differ after that, so the rest is left to the teacher-forced run."""
    ref_tok = list(map(int, ref_tok))
    assert len(gpu_tok) == len(ref_tok), (name, gpu_tok, ref_tok)
    for j, (g, r) in enumerate(zip(gpu_tok, ref_tok)):
        if g == r:
            continue
        lg = np.asarray(ref_lg[j], np.float64)
        gap = (lg[r] - lg[g]) / np.max(np.abs(lg))
        assert gap <= TOL, f"{name}: step {j} gpu {g} oracle {r}, oracle logit gap {gap:.3e} is no near tie"
        log(f"{name}: near tie at step {j} (gap {gap:.2e}): gpu {g}, oracle {r}; comparison stops there")
        return j
    return len(ref_tok)


def compare_forced(name, gpu_tok, gpu_logits, ref_lg):
    worst, ties = 0.0, 0
    assert len(gpu_logits) == len(ref_lg), (len(gpu_logits), len(ref_lg))
    for j, (g, r) in enumerate(zip(gpu_logits, ref_lg)):
        worst = max(worst, rel_max_err(g, r))
        a = int(np.argmax(r))
        if gpu_tok[j] != a:
            margin = r[a] - r[gpu_tok[j]]
            assert margin <= TOL * np.max(np.abs(r)), f"{name} step {j}: id {gpu_tok[j]} vs {a}, margin {margin}"
            ties += 1
    assert worst <= TOL, f"{name}: logits rel err {worst}"
    return worst, ties


def test_cfg1_tiny_full():
    """Workload 1: tiny decoder, prompts 64/128/192/256, 8 greedy tokens, chunk 128, 64 pages."""
    shape, dm, w = device_model("tiny")
    stages = synth.workloads.cfg1()
    reqs = [(s.workflow, 0, s.prompt, s.max_new_tokens, s.wf_slo_us, {}) for s in stages]
    o_ids, o_order, o_steps, o_bt = oracle_schedule(reqs, 64, 4, 128, shape.vocab)
    ref_tok, ref_lg = M.generate(w, [s.prompt for s in stages], [8] * 4)
    # free running
    eng = Engine(dm, max_context=512, n_blocks=64, max_seqs=4, chunk_tokens=128, cost_ps=COST, iter_ps=ITER)
    for wf, st, p, mx, slo, kw in reqs:
        eng.inst.submit(0, wf, st, 0, slo, p, mx, **kw)
    assert eng.inst.queue_order() == o_order
    steps, now = [], 0
    while True:
        st, info = eng.inst.step(now)
        if st == hxf.IDLE:
            break
        steps.append(eng.inst.last_batch())
        now += info["t_iter_us"]
    assert [tuple(map(list, s)) for s in steps] == [(a, b) for a, b in o_steps]
    for k, rid in enumerate(o_ids):
        assert eng.inst.block_table(rid) == o_bt[rid]
        toks = eng.inst.tokens(rid)
        log(f"cfg1 req {rid}: gpu {toks} oracle {list(ref_tok[k])}")
        compare_free_running(f"cfg1 req {rid}", toks, ref_tok[k], ref_lg[k])
    done = eng.inst.drain()
    assert sorted(d["id"] for d in done) == o_ids
    # teacher forced, logits of every sampled row
    eng2 = Engine(dm, max_context=512, n_blocks=64, max_seqs=4, chunk_tokens=128, cost_ps=COST, iter_ps=ITER)
    ids, lg, _, _ = run_engine(eng2, reqs, forced=ref_tok)
    for k, rid in enumerate(ids):
        worst, ties = compare_forced(f"cfg1 req {rid}", eng2.inst.tokens(rid), lg[rid], ref_lg[k])
        log(f"cfg1 forced req {rid}: logits rel err {worst:.2e}, near ties {ties}")


@pytest.mark.parametrize("name,layers,lens,chunk", [("llama8b", 2, (100, 300, 700), 256),
                                                    ("llama8b", 1, (600, 1500), 1024),
                                                    ("qwen32b", 1, (90, 400), 128),
                                                    ("llama70b", 1, (90, 500), 256)])
def test_full_width_layer_truncated(name, layers, lens, chunk):
    """Full-width 8B, 32B and 70B shapes (vocab 128256 / 152064, GQA 4 / 5 / 8), few layers,
    chunked prefill co-batched with decode, teacher forced."""
    shape, dm, w = device_model(name, layers)
    rng = np.random.default_rng(len(lens))
    prompts = [rng.integers(0, shape.vocab, n) for n in lens]
    mx = [4] * len(lens)
    ref_tok, ref_lg = M.generate(w, prompts, mx)
    reqs = [(i, 0, p, 4, 10 ** 7, {}) for i, p in enumerate(prompts)]
    eng = Engine(dm, max_context=2048, n_blocks=400, max_seqs=8, chunk_tokens=chunk, cost_ps=COST, iter_ps=ITER)
    ids, lg, steps, _ = run_engine(eng, reqs, forced=ref_tok)
    o_ids, _, o_steps, o_bt = oracle_schedule(reqs, 400, 8, chunk, shape.vocab)
    assert [tuple(map(list, s)) for s in steps] == [(a, b) for a, b in o_steps]
    for k, rid in enumerate(ids):
        assert eng.inst.block_table(rid) == o_bt[rid]
        worst, ties = compare_forced(f"{name} req {rid}", eng.inst.tokens(rid), lg[rid], ref_lg[k])
        log(f"{name}-L{layers} req {rid} (prompt {lens[k]}): logits rel err {worst:.2e}, near ties {ties}")


def test_forks_share_prefix_pages():
    """A retained parent forked into branches (shared full pages, re-prefilled tail)
    gives each child the tokens of decoding its full context from scratch."""
    shape, dm, w = device_model("tiny")
    rng = np.random.default_rng(21)
    eng = Engine(dm, max_context=512, n_blocks=80, max_seqs=8, chunk_tokens=64, cost_ps=COST, iter_ps=ITER)
    prompt = rng.integers(0, shape.vocab, 45)
    par = eng.inst.submit(0, 0, 0, 0, 10 ** 7, prompt, 3, retain=True)
    now = 0
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    ptoks = eng.inst.tokens(par)
    ref_par, _ = M.generate(w, [prompt], [3])
    assert ptoks == list(map(int, ref_par[0]))
    apps = [rng.integers(0, shape.vocab, n) for n in (0, 1, 16, 33)]
    kids = [eng.inst.submit(now, 0, 1, 0, 10 ** 7, a, 5, parent=par) for a in apps]
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    full = [np.concatenate([prompt, ptoks, a]).astype(np.int64) for a in apps]
    ref, _ = M.generate(w, full, [5] * len(full))
    shared = (len(prompt) + 3 - 1) // 16
    for k, rid in enumerate(kids):
        assert eng.inst.block_table(rid)[:shared] == eng.inst.block_table(par)[:shared]
        assert eng.inst.tokens(rid) == list(map(int, ref[k])), f"fork {k}"


def test_fork_of_a_teacher_forced_parent_continues_from_the_forced_tokens():
    """A parent fed forced tokens holds them in its sequence: a fork continues from
    prompt + forced tokens (not from the parent's own argmax)."""
    shape, dm, w = device_model("tiny")
    rng = np.random.default_rng(22)
    eng = Engine(dm, max_context=512, n_blocks=80, max_seqs=8, chunk_tokens=64, cost_ps=COST, iter_ps=ITER)
    prompt = rng.integers(0, shape.vocab, 38)
    own, _ = M.generate(w, [prompt], [3])
    forced = [int(t + 1) % shape.vocab for t in own[0]]          # never the argmax
    par = eng.inst.submit(0, 0, 0, 0, 10 ** 7, prompt, 3, retain=True, forced=forced)
    now = 0
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    app = rng.integers(0, shape.vocab, 5)
    kid = eng.inst.submit(now, 0, 1, 0, 10 ** 7, app, 4, parent=par)
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    ref, ref_lg = M.generate(w, [np.concatenate([prompt, forced, app]).astype(np.int64)], [4])
    compare_free_running("fork of a forced parent", eng.inst.tokens(kid), ref[0], ref_lg[0])


def test_policy_does_not_change_tokens_and_runs_are_deterministic():
    shape, dm, w = device_model("tiny")
    rng = np.random.default_rng(8)
    prompts = [rng.integers(0, shape.vocab, n) for n in (33, 120, 7, 64, 90)]
    out = []
    for policy in (hxf.POLICY_PQ, hxf.POLICY_FCFS, hxf.POLICY_PQ):
        eng = Engine(dm, max_context=512, n_blocks=64, max_seqs=3, chunk_tokens=48, cost_ps=COST, iter_ps=ITER,
                     policy=policy)
        reqs = [(i, i % 3, p, 6, [10 ** 6, 2000, 40000, 900, 10 ** 5][i], {}) for i, p in enumerate(prompts)]
        ids, lg, _, _ = run_engine(eng, reqs)
        out.append(([eng.inst.tokens(r) for r in ids], [np.stack(lg[r]) for r in ids]))
    assert out[0][0] == out[1][0] == out[2][0]
    for a, b in zip(out[0][1], out[2][1]):
        np.testing.assert_array_equal(a, b)          # same policy twice: bit-identical logits


@pytest.mark.parametrize("name,layers", [("tiny", None), ("llama8b", 2)])
def test_graph_replays_match_eager_steps(name, layers, monkeypatch):
    """Decode-only iterations replay a captured graph of the forward.  Two engines run
    the same requests step by step, one replaying graphs and one launching eagerly,
    interleaved (eager work and synchronisations between the replays); every step's
    sampled ids and logits rows must be bit-identical, with the graph replayed many
    times and re-captured when the block tables outgrow their padding."""
    shape, dm, w = device_model(name, layers)
    rng = np.random.default_rng(31)
    prompts = [rng.integers(0, shape.vocab, n) for n in (40, 1000, 7, 300)]
    engines = []
    for env in (None, "1"):
        if env is None:
            monkeypatch.delenv("HXF_NO_GRAPHS", raising=False)
        else:
            monkeypatch.setenv("HXF_NO_GRAPHS", env)
        eng = Engine(dm, max_context=4096, n_blocks=600, max_seqs=8, chunk_tokens=256, cost_ps=COST, iter_ps=ITER)
        ids = [eng.inst.submit(0, i, 0, 0, 10 ** 7, p, 1100) for i, p in enumerate(prompts)]
        engines.append((eng, ids))
    monkeypatch.delenv("HXF_NO_GRAPHS", raising=False)
    (ga, ia), (gb, ib) = engines
    now, n_decode_steps = 0, 0
    while True:
        sa, infa = ga.inst.step(now)
        sb, infb = gb.inst.step(now)
        assert sa == sb
        if sa == hxf.IDLE:
            break
        assert infa["n_tokens"] == infb["n_tokens"] and infa["n_decode"] == infb["n_decode"]
        if infa["n_prefill_tokens"] == 0:
            n_decode_steps += 1
        for ra, rb in zip(ia, ib):
            try:
                la = ga.inst.last_logits(ra)
            except hxf.HxfError:
                continue
            np.testing.assert_array_equal(la, gb.inst.last_logits(rb))
        now += 1000
    assert n_decode_steps > 1000
    for ra, rb in zip(ia, ib):
        assert ga.inst.tokens(ra) == gb.inst.tokens(rb)
    log(f"{name}: {n_decode_steps} decode-only steps, graph replays bit-identical to eager launches")


def test_prefill_only_iteration_after_two_tile_fork_decode():
    """Regression: six forks of one parent (Hq/Hkv = 4, so their shared pages go to
    two-tile items) decode together, then a new request's prompt runs in an iteration
    with no decoding sequence.  The decode work list of that iteration must be empty
    (the executor reuses one plan object across iterations), and the new request's
    tokens are the oracle's."""
    shape, dm, w = device_model("llama8b", 2)
    rng = np.random.default_rng(43)
    eng = Engine(dm, max_context=1024, n_blocks=200, max_seqs=8, chunk_tokens=256, cost_ps=COST, iter_ps=ITER)
    prompt = rng.integers(0, shape.vocab, 100)
    par = eng.inst.submit(0, 0, 0, 0, 10 ** 7, prompt, 1, retain=True)
    now = 0
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    kids = [eng.inst.submit(now, 0, 1, 0, 10 ** 7, np.zeros(0, np.int64), 3, parent=par) for _ in range(6)]
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    fresh = rng.integers(0, shape.vocab, 40)
    rid = eng.inst.submit(now, 1, 0, 0, 10 ** 7, fresh, 3)
    st, _ = eng.inst.step(now)
    assert st != hxf.IDLE and eng.inst.last_batch()[0] == [rid]     # the prompt alone: no decode rows
    while eng.inst.step(now)[0] != hxf.IDLE:
        now += 1000
    ref, ref_lg = M.generate(w, [fresh.astype(np.int64)], [3])
    compare_free_running("prefill after two-tile decode", eng.inst.tokens(rid), ref[0], ref_lg[0])
    full = np.concatenate([prompt, eng.inst.tokens(par)]).astype(np.int64)
    kref, kref_lg = M.generate(w, [full], [3])
    for k in kids:
        compare_free_running("fork", eng.inst.tokens(k), kref[0], kref_lg[0])


def test_graph_replays_match_eager_steps_with_forks(monkeypatch):
    """The same comparison for forks of one retained parent decoding together (their
    shared full pages attended by multi-row work items)."""
    shape, dm, w = device_model("llama8b", 2)
    rng = np.random.default_rng(41)
    prompt = rng.integers(0, shape.vocab, 700)
    apps = [rng.integers(0, shape.vocab, n) for n in (0, 3, 20, 40, 5)]
    engines = []
    for env in (None, "1"):
        if env is None:
            monkeypatch.delenv("HXF_NO_GRAPHS", raising=False)
        else:
            monkeypatch.setenv("HXF_NO_GRAPHS", env)
        eng = Engine(dm, max_context=2048, n_blocks=300, max_seqs=8, chunk_tokens=256, cost_ps=COST, iter_ps=ITER)
        par = eng.inst.submit(0, 0, 0, 0, 10 ** 7, prompt, 2, retain=True)
        now = 0
        while eng.inst.step(now)[0] != hxf.IDLE:
            now += 1000
        kids = [eng.inst.submit(now, 0, 1, 0, 10 ** 7, a, 400, parent=par) for a in apps]
        engines.append((eng, kids, now))
    monkeypatch.delenv("HXF_NO_GRAPHS", raising=False)
    (ga, ka, now), (gb, kb, _) = engines
    steps = 0
    while True:
        sa, _ = ga.inst.step(now)
        sb, _ = gb.inst.step(now)
        assert sa == sb
        if sa == hxf.IDLE:
            break
        steps += 1
        for ra, rb in zip(ka, kb):
            try:
                la = ga.inst.last_logits(ra)
            except hxf.HxfError:
                continue
            np.testing.assert_array_equal(la, gb.inst.last_logits(rb))
        now += 1000
    assert steps > 390
    for ra, rb in zip(ka, kb):
        assert ga.inst.tokens(ra) == gb.inst.tokens(rb)


def test_checked_mode_runs_clean(monkeypatch):
    """HXF_CHECK=1 validates every index the kernels follow (tokens, positions, KV slots,
    block tables, attention work items) on the host before each launch: a run with forks
    (shared-prefix decode items), chunked prefill and plain decode raises nothing and gives
    the tokens of an unchecked run."""
    shape, dm, w = device_model("tiny")
    rng = np.random.default_rng(31)
    prompt = rng.integers(0, shape.vocab, 70)
    others = [rng.integers(0, shape.vocab, n) for n in (20, 130)]
    apps = [rng.integers(0, shape.vocab, n) for n in (0, 5, 17)]

    def run():
        eng = Engine(dm, max_context=512, n_blocks=96, max_seqs=8, chunk_tokens=64, cost_ps=COST, iter_ps=ITER)
        par = eng.inst.submit(0, 0, 0, 0, 10 ** 7, prompt, 3, retain=True)
        now = 0
        while eng.inst.step(now)[0] != hxf.IDLE:
            now += 1000
        ids = [eng.inst.submit(now, 0, 1, 0, 10 ** 7, a, 6, parent=par) for a in apps]
        ids += [eng.inst.submit(now, 1 + k, 0, 0, 10 ** 7, p, 6) for k, p in enumerate(others)]
        while eng.inst.step(now)[0] != hxf.IDLE:
            now += 1000
        return [eng.inst.tokens(r) for r in ids]

    plain = run()
    monkeypatch.setenv("HXF_CHECK", "1")
    checked = run()
    assert checked == plain
