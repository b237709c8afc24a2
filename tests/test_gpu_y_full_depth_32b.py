"""Full-depth oracle parity on the GPU for the workload-5 shape: the 64-layer
32B model on one workflow of workload 5 (a stage-1 request on the first 256
tokens of the first workflow's prompt, retained, then two forks of it: nothing
appended, as a candidate; 24 tokens of its first correction prompt appended),
through hxf_submit / hxf_step, against the float64 oracle over every layer (run
layer by layer from the same bf16 bits).  The prompt is a prefix: the oracle's
float64 cost at the workload's 2048-8192-token prompts would be minutes per
request.  Decode steps at full depth are covered by the 8B tests; here every
request produces one token.  Bounds as in test_gpu_x_full_depth.py (the
bf16-rounding forward runs on the same inputs).
"""
import time

import numpy as np
import pytest

import synth
from oracle import model as M
from paper_2505_05286_amd import hxf
from paper_2505_05286_amd.device import Engine

from . import bf16_emulation as E
from .gpu_util import log
from .test_gpu_x_full_depth import COST, ITER, collect, compare_rows, load, tick

pytestmark = pytest.mark.gpu


# ------------------------------------------------------------------ 32B, 64 layers
def test_cfg5_full_depth_32b():
    """Workload 5's shape: a stage-1 request (first 256 tokens of the first workflow's
    prompt, retained) and two forks of it, over all 64 layers of the 32B model."""
    shape, dm, gains, bits, embed, lm = load("qwen32b")
    V, L = shape.vocab, shape.n_layers
    w = M.Weights(shape, keep_layers=False, norm_gains=gains, layer_bits=lambda l: bits[l], embed_bits=embed,
                  lm_head_bits=lm)
    wf = synth.workloads.cfg5(vocab=V, n_wf=1)[0]
    prompt = wf.schema[:256].astype(np.int64)
    apps = [np.zeros(0, np.int64), wf.corrections[0][:24].astype(np.int64)]
    n = len(prompt) + 1                     # the parent's sequence: prompt + its one token
    shared = (n - 1) // 16 * 16
    t0 = time.time()
    res, tokp, tokf = {}, None, None
    for kind, fwd in (("ref", M.forward), ("emul", E.forward)):
        par = M.Sequence(L)
        lgp = fwd(w, [par], [prompt], progress=tick)[0][0]
        if kind == "ref":
            tokp = int(np.argmax(lgp))
        log(f"cfg5 32B {kind}: prompt pass after {time.time() - t0:.0f} s")
        S_ = np.concatenate([prompt, [tokp]])
        forks = [par.fork(shared) for _ in apps]
        outs = fwd(w, forks, [np.concatenate([S_[shared:], a]) for a in apps], progress=tick)
        if kind == "ref":
            tokf = [int(np.argmax(o[0])) for o in outs]
        res[kind] = ([lgp], [[o[0]] for o in outs])
        log(f"cfg5 32B {kind}: fork pass after {time.time() - t0:.0f} s")
    bits.clear()
    eng = Engine(dm, max_context=512, n_blocks=64, max_seqs=8, chunk_tokens=2048, cost_ps=COST, iter_ps=ITER)
    inst = eng.inst
    rest = [(16, 256), (16 + 512, 256), (1024, 128)]
    pid = inst.submit(0, 0, 0, 0, wf.slo_us, prompt, 1, retain=True, rest=rest, forced=[tokp])
    rows = {pid: []}
    now = 0
    while True:
        st, info = inst.step(now)
        if st == hxf.IDLE:
            break
        collect(inst, [pid], rows)
        now += info["t_iter_us"]
    compare_rows("cfg5 32B stage 1", inst.tokens(pid), rows[pid], res["ref"][0], res["emul"][0])
    kids = [inst.submit(now, 0, 1 + k, 0, wf.slo_us, a, 1, parent=pid, rest=rest[1 + k:], forced=[tokf[k]])
            for k, a in enumerate(apps)]
    rows = {r: [] for r in kids}
    while True:
        st, info = inst.step(now)
        if st == hxf.IDLE:
            break
        collect(inst, kids, rows)
        now += info["t_iter_us"]
    for k, r in enumerate(kids):
        assert inst.block_table(r)[:shared // 16] == inst.block_table(pid)[:shared // 16]
        compare_rows(f"cfg5 32B fork +{len(apps[k])}", inst.tokens(r), rows[r], res["ref"][1][k],
                     res["emul"][1][k])
    del eng, dm
