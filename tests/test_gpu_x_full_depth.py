"""Full-depth oracle parity on the GPU: the 32-layer 8B model on samples of
workloads 2, 3 and 4, each run through hxf_submit / hxf_step in the workload's
own batch setting and compared with the float64 oracle run over every layer
(the 64-layer 32B shape of workload 5 is in test_gpu_y_full_depth_32b.py).

Sampling (sequences are independent, so the oracle recomputes only a few):
* workload 2: all 64 sequences run on the GPU (decode batch of 64); the two with
  the shortest contexts (1024 and 1167 tokens) are compared: the prompt's last
  row and two decode steps;
* workload 3: the 32 decodes run while the 16 prompts are prefilled in
  2048-token chunks; the shortest prompt (2386 tokens, prefilled over two
  iterations co-batched with the 32 decode rows) is compared;
* workload 4: a prefill-only retained parent (the first 1024 tokens of the
  workload's first shared prompt) forked into 8 branches that decode through the
  shared-prefix work items; every branch's 2 rows are compared.  Branches append
  0, 0, 1, 2, 3, 5, 8 and 13 tokens, so rows mapped to the wrong branch differ,
  and the two with nothing appended must agree bit for bit.

Every RMSNorm gets its own random gain on both sides, so a miswired norm pointer
fails.  Logits: per row max|diff| / max|ref| <= 2e-2; greedy ids under teacher
forcing with the oracle's tokens, a differing id accepted only as a near tie (the
oracle's logit gap within 2e-2 of max|ref|), and the near ties counted.
Block tables and per-iteration batches equal the oracle scheduler's.
"""
import time

import numpy as np
import pytest

import synth
from oracle import model as M
from oracle import sched as S
from paper_2505_05286_amd import hxf
from paper_2505_05286_amd.device import DeviceModel, Engine

from . import bf16_emulation as E
from .gpu_util import log, rel_max_err

pytestmark = pytest.mark.gpu

TOL = 2e-2
# A row's bound is max(TOL, DRIFT x the error of the bf16-rounding forward on the same
# inputs): bf16 arithmetic alone drifts past TOL after a few layers of these random
# weights, by an amount that adds up with depth.
DRIFT = 2.0
COST = (200 * S.PS, 50_000, 10, 150 * S.PS)
ITER = (500 * S.PS, 1000, 20, 1)
APPEND4 = (0, 0, 1, 2, 3, 5, 8, 13)
PARENT4 = 1024


def pages(n):
    return -(-n // 16)


def load(name):
    t0 = time.time()
    shape = synth.model_shape(name)
    gains = synth.gen_norm_gains(shape)
    bits = {}

    def layer(l):
        bits[l] = synth.gen_layer(shape, l)
        return bits[l]

    embed, lm = synth.gen_embed(shape), synth.gen_lm_head(shape)
    log(f"full depth: generating and uploading {shape.name} ({shape.n_layers} layers)")
    dm = DeviceModel(shape, layer, embed, lm, gains, device="cuda:0")
    log(f"full depth: {shape.name} on the GPU after {time.time() - t0:.0f} s")
    return shape, dm, gains, bits, embed, lm


def tick(layer):
    """Oracle progress: a line every 8 layers, so a long float64 pass shows it is alive."""
    if layer % 8 == 7:
        log(f"  oracle layer {layer + 1}")


def compare_rows(name, gpu_tok, gpu_rows, ref_rows, emul_rows):
    """Every row's logits within its bound, max(TOL, DRIFT x the drift of the bf16-rounding
    forward on the same inputs); ids equal, or a near tie within that bound.
    Returns (worst error, worst error / bound, near ties)."""
    assert len(gpu_rows) == len(ref_rows) == len(emul_rows), (name, len(gpu_rows), len(ref_rows))
    worst, worst_frac, ties, drift = 0.0, 0.0, 0, 0.0
    for j, (g, r, e) in enumerate(zip(gpu_rows, ref_rows, emul_rows)):
        d = rel_max_err(e, r)
        bound = max(TOL, DRIFT * d)
        err = rel_max_err(g, r)
        worst, drift = max(worst, err), max(drift, d)
        worst_frac = max(worst_frac, err / bound)
        assert err <= bound, f"{name} row {j}: logits rel err {err:.3e} > bound {bound:.3e} (bf16 drift {d:.3e})"
        a = int(np.argmax(r))
        if gpu_tok[j] != a:
            gap = (r[a] - r[gpu_tok[j]]) / np.max(np.abs(r))
            assert gap <= bound, f"{name} row {j}: gpu id {gpu_tok[j]} vs oracle {a}, gap {gap:.3e} is no near tie"
            ties += 1
    log(f"{name}: {len(ref_rows)} rows, logits rel err {worst:.2e} (bf16-rounding forward: {drift:.2e}), "
        f"{worst_frac:.2f} of the bound, near ties {ties}")
    return worst, worst_frac, ties


def collect(inst, ids, rows):
    for r in ids:
        try:
            rows[r].append(inst.last_logits(r))
        except hxf.HxfError:
            pass


def oracle_replay(reqs, n_blocks, max_seqs, chunk, vocab, n_steps):
    """Batches and block tables the oracle scheduler decides for these submissions."""
    s = S.Scheduler(n_blocks, max_seqs, chunk, COST, ITER, vocab=vocab)
    ids = [s.submit(now, wf, st, arr, slo, list(p), mx) for now, wf, st, arr, slo, p, mx in reqs]
    steps, now = [], 0
    for _ in range(n_steps):
        st, info = s.step(now)
        assert st == S.OK
        steps.append((info["batch_ids"], info["admitted"]))
        now += info["t_iter_us"]
    return ids, steps, s


# ------------------------------------------------------------------ 8B, 32 layers
@pytest.fixture(scope="module")
def m8b():
    shape, dm, gains, bits, embed, lm = load("llama8b")
    w = M.Weights(shape, keep_layers=True, norm_gains=gains, layer_bits=lambda l: bits.pop(l), embed_bits=embed,
                  lm_head_bits=lm)
    yield shape, dm, w
    del dm, w


@pytest.fixture(scope="module")
def ref8b(m8b):
    """The oracle over all 32 layers for every 8B sample, in three passes, and the
    bf16-rounding forward on the same inputs (fed the oracle's tokens)."""
    shape, _, w = m8b
    V, L = shape.vocab, shape.n_layers
    t0 = time.time()
    cfg2 = synth.workloads.cfg2(V)
    s2 = [int(i) for i in np.argsort([len(s.prompt) for s in cfg2], kind="stable")[:2]]
    _, prompts3 = synth.workloads.cfg3(V)
    p3 = int(np.argmin([len(s.prompt) for s in prompts3]))
    parents4, _, _ = synth.workloads.cfg4(V)
    parent = parents4[0].prompt[:PARENT4].astype(np.int64)
    rng = np.random.default_rng(404)
    apps = [rng.integers(0, V, n) for n in APPEND4]
    apps[1] = apps[0].copy()
    shared = (PARENT4 - 1) // 16 * 16
    prompts = [cfg2[i].prompt.astype(np.int64) for i in s2] + [prompts3[p3].prompt.astype(np.int64), parent]
    rows1 = [[len(p) - 1] for p in prompts[:3]] + [[]]
    out = {}
    tok2, tok4, tok3 = [[], []], [[] for _ in APPEND4], None
    for kind, fwd in (("ref", M.forward), ("emul", E.forward)):
        lg2, lg4 = [[], []], [[] for _ in APPEND4]
        seqs = [M.Sequence(L) for _ in range(4)]
        log(f"full depth {kind} pass 1: prefill of {sum(len(p) for p in prompts)} tokens ({time.time() - t0:.0f} s)")
        o = fwd(w, seqs, prompts, logit_rows=rows1, progress=tick)
        for k in range(2):
            lg2[k].append(o[k][0])
        lg3 = o[2][0]
        if kind == "ref":
            tok2 = [[int(np.argmax(o[k][0]))] for k in range(2)]
            tok3 = int(np.argmax(lg3))
        forks = [seqs[3].fork(shared) for _ in APPEND4]
        for step in (1, 2):
            log(f"full depth {kind} pass {step + 1} ({time.time() - t0:.0f} s)")
            if step == 1:
                chunks = [np.array([t[0]]) for t in tok2] + [np.concatenate([parent[shared:], a]) for a in apps]
            else:
                chunks = [np.array([t[1]]) for t in tok2] + [np.array([t[0]]) for t in tok4]
            o = fwd(w, seqs[:2] + forks, chunks, progress=tick)
            for k in range(2):
                lg2[k].append(o[k][0])
                if kind == "ref":
                    tok2[k].append(int(np.argmax(o[k][0])))
            for b in range(len(APPEND4)):
                lg4[b].append(o[2 + b][0])
                if kind == "ref":
                    tok4[b].append(int(np.argmax(o[2 + b][0])))
        out[kind] = dict(lg2=lg2, lg3=lg3, lg4=lg4)
    log(f"full depth oracle and bf16-rounding forward (8B) done in {time.time() - t0:.0f} s")
    return dict(s2=s2, tok2=tok2, p3=p3, tok3=tok3, parent=parent, apps=apps, tok4=tok4,
                lg2=out["ref"]["lg2"], lg3=out["ref"]["lg3"], lg4=out["ref"]["lg4"],
                em2=out["emul"]["lg2"], em3=out["emul"]["lg3"], em4=out["emul"]["lg4"])


def test_cfg2_full_depth(m8b, ref8b):
    """Workload 2 on the GPU (64 sequences, 2048-token chunks, then a decode batch of
    64); the two shortest contexts against the oracle over all 32 layers."""
    shape, dm, _ = m8b
    cfg2 = synth.workloads.cfg2(shape.vocab)
    s2, other_new = ref8b["s2"], 200
    mx = [3 if i in s2 else other_new for i in range(len(cfg2))]
    n_blocks = sum(pages(len(s.prompt) + m - 1) for s, m in zip(cfg2, mx)) + 64
    eng = Engine(dm, max_context=8192 + other_new + 16, n_blocks=n_blocks, max_seqs=64, chunk_tokens=2048,
                 cost_ps=COST, iter_ps=ITER)
    ids = []
    for i, s in enumerate(cfg2):
        forced = ref8b["tok2"][s2.index(i)] if i in s2 else None
        ids.append(eng.inst.submit(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, mx[i], forced=forced))
    samp = [ids[i] for i in s2]
    rows = {r: [] for r in samp}
    batches, n_dec, now = [], [], 0
    while any(eng.inst.request_state(r)["state"] != 3 for r in samp):
        st, info = eng.inst.step(now)
        assert st == hxf.OK
        batches.append(eng.inst.last_batch())
        before = {r: len(rows[r]) for r in samp}
        collect(eng.inst, samp, rows)
        if any(len(rows[r]) > before[r] for r in samp) and info["n_prefill_tokens"] == 0:
            n_dec.append(info["n_decode"])
        now += info["t_iter_us"]
    log(f"cfg2 full depth: {len(batches)} iterations; decode batch sizes of the sampled steps {n_dec}")
    assert n_dec and all(n == 64 for n in n_dec)
    reqs = [(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, m) for s, m in zip(cfg2, mx)]
    o_ids, o_steps, o_s = oracle_replay(reqs, n_blocks, 64, 2048, shape.vocab, len(batches))
    assert o_ids == ids
    assert [tuple(map(list, b)) for b in batches] == [(a, b) for a, b in o_steps]
    for k, i in enumerate(s2):
        rid = ids[i]
        assert eng.inst.block_table(rid) == o_s.block_table(rid)
        compare_rows(f"cfg2 ctx {len(cfg2[i].prompt)}", eng.inst.tokens(rid), rows[rid], ref8b["lg2"][k],
                     ref8b["em2"][k])
    del eng


def test_cfg3_full_depth(m8b, ref8b):
    """Workload 3 on the GPU: 32 running decodes, then the 16 prompts in 2048-token
    chunks co-batched with them; the shortest prompt against the oracle."""
    shape, dm, _ = m8b
    decodes, prompts = synth.workloads.cfg3(shape.vocab)
    p3 = ref8b["p3"]
    dec_new = 256
    n_blocks = sum(pages(len(s.prompt) + dec_new) for s in decodes) + sum(pages(len(s.prompt)) for s in prompts) + 64
    eng = Engine(dm, max_context=8192 + 16, n_blocks=n_blocks, max_seqs=64, chunk_tokens=2048, cost_ps=COST,
                 iter_ps=ITER)
    inst = eng.inst
    for s in decodes:
        inst.submit(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, dec_new)
    now = 0
    while True:
        st, info = inst.step(now)
        assert st == hxf.OK
        now += info["t_iter_us"]
        if info["n_prefill_tokens"] == 0:
            break
    ids = [inst.submit(now, s.workflow, 0, now, s.wf_slo_us, s.prompt, 1,
                       forced=[ref8b["tok3"]] if k == p3 else None) for k, s in enumerate(prompts)]
    rid = ids[p3]
    rows = {rid: []}
    chunks_with = []
    while inst.request_state(rid)["state"] != 3:
        st, info = inst.step(now)
        assert st == hxf.OK
        b, _ = inst.last_batch()
        if rid in b:
            chunks_with.append((info["n_prefill_tokens"], info["n_decode"]))
        collect(inst, [rid], rows)
        now += info["t_iter_us"]
    log(f"cfg3 full depth: prompt of {len(prompts[p3].prompt)} tokens over iterations (prefill, decode rows) "
        f"{chunks_with}")
    assert len(chunks_with) >= 2 and all(d == 32 for _, d in chunks_with)
    compare_rows(f"cfg3 prompt {len(prompts[p3].prompt)}", inst.tokens(rid), rows[rid], [ref8b["lg3"]],
                 [ref8b["em3"]])
    del eng


def test_cfg4_full_depth(m8b, ref8b):
    """Workload 4's candidate stage: a retained prefill-only parent forked into 8
    branches decoding through the shared-prefix items."""
    shape, dm, _ = m8b
    parent, apps = ref8b["parent"], ref8b["apps"]
    n_blocks = pages(PARENT4) + sum(pages(16 + len(a) + 1) for a in apps) + 32
    eng = Engine(dm, max_context=PARENT4 + 64, n_blocks=n_blocks, max_seqs=16, chunk_tokens=2048, cost_ps=COST,
                 iter_ps=ITER)
    inst = eng.inst
    par = inst.submit(0, 0, 0, 0, 10 ** 12, parent, 0, retain=True)
    now = 0
    while inst.step(now)[0] != hxf.IDLE:
        now += 1000
    kids = [inst.submit(now, 0, 1, 0, 10 ** 12, a, 2, parent=par, forced=ref8b["tok4"][b])
            for b, a in enumerate(apps)]
    rows = {r: [] for r in kids}
    while True:
        st, info = inst.step(now)
        if st == hxf.IDLE:
            break
        collect(inst, kids, rows)
        now += 1000
    shared = (PARENT4 - 1) // 16
    bts = [inst.block_table(r) for r in kids]
    for bt in bts:
        assert bt[:shared] == inst.block_table(par)[:shared]
    # the decode step's work list groups the branches on their shared pages
    ctx = [PARENT4 + len(a) + 1 for a in apps]
    width = max(len(b) for b in bts)
    tab = np.zeros((len(kids), width), np.int32)
    for i, b in enumerate(bts):
        tab[i, :len(b)] = b
    items, _ = hxf.op_decode_plan(len(kids), shape.n_q_heads, shape.n_kv_heads, ctx, tab, width)
    log(f"cfg4 full depth: decode plan rows per item {sorted(set(int(x) for x in items[:, 3]))}")
    assert (items[:, 3] > 1).any()
    for b, r in enumerate(kids):
        compare_rows(f"cfg4 branch {b} (+{len(apps[b])})", inst.tokens(r), rows[r], ref8b["lg4"][b],
                     ref8b["em4"][b])
    for a, b in ((0, 1),):
        for x, y in zip(rows[kids[a]], rows[kids[b]]):
            np.testing.assert_array_equal(x, y)
    del eng
