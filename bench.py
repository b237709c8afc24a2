#!/usr/bin/env python3
"""Throughput of one MI355X serving instance on the decode workload.

Workload (synthetic, seeded): Llama-3-8B-shaped decoder (32 layers, d 4096,
32 query / 8 KV heads of 128, SwiGLU 14336, vocab 128256, bf16 weights
N(0, 0.02)); 64 sequences whose contexts are lognormal (median 3000, sigma
0.5, clipped to [1024, 8192]) with uniform random token ids, KV pages of 16.
The prompts are prefilled (untimed, chunks of 2048 tokens co-batched with the
decodes that start as prompts finish), then every step is one continuous-
batching iteration with all 64 sequences decoding: scheduler, metadata
upload, 32 layers of GEMMs / RoPE / paged attention, LM head, argmax, and the
sampled ids back on the host.

Prints one JSON line.  `value` is decode tokens/s over the K timed steps.
`roofline` is the paged decode attention (the largest single item of the
step): its split-K kernel plus the log-sum-exp merge that follows it, the
algorithmic K+V bytes per layer over their summed average duration, timed with
HIP events that each launch itself stamps with the kernel's start and end
(hipExtLaunchKernel) on the instance's stream; `attention_only` is the split-K
kernel alone.  `gemm_roofline` is the MFMA roofline of the prefill projections
(2080 rows: workload 3's 2048-token chunk plus 32 decodes), timed the same way
over profiled mixed iterations.  `cpu_baseline` times the CPU oracle on a
bounded sample of the decode step.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "prefill+decode tokens/s per MI355X at 8B shape; decode-attn HBM % of peak"
HBM_PEAK_GBS = 8000.0
# HBM bytes per launch pair of decode_attn_kernel<128> + decode_merge_kernel<128> from
# hardware counters (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE, over
# `bench.py --attn-kernel-probe`, each scaled by what the counter reads for a 1 GiB
# copy: 2.000 and 1.000); valid for the kernels as they stand, to be re-measured
# whenever they change.
DECODE_ATTN_TRAFFIC = {"bytes_per_launch": 842_801_290, "algorithmic_bytes_per_launch": 829_956_096,
                       "attention_bytes": 838_459_399, "merge_bytes": 4_341_892,
                       "sample": "attention probe, 64 contexts of the benchmark, 202626 tokens"}
BATCH = 64
MAX_NEW = 1000


def progress(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(shape, ctxs, n_layers_sample=4, iters=3):
    """Oracle (float64 numpy) on consecutive decode iterations of the same batch
    through the first `n_layers_sample` layers plus the LM head, scaled to the
    full depth."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import model as M

    part = shape.with_layers(n_layers_sample)
    w = M.Weights(part)
    for l in range(n_layers_sample):
        w.layer(l)
    w.lm_head_f32()
    w.embed_rows(np.zeros(1, np.int64))
    rng = np.random.default_rng(0)
    seqs = []
    for c in ctxs:
        s = M.Sequence(n_layers_sample)
        for l in range(n_layers_sample):
            s.k[l] = rng.standard_normal((int(c), shape.n_kv_heads, shape.head_dim))
            s.v[l] = rng.standard_normal((int(c), shape.n_kv_heads, shape.head_dim))
        s.n = int(c)
        seqs.append(s)
    t_fwd = t_lm = 0.0
    h = rng.standard_normal((len(ctxs), shape.d_model))
    for _ in range(iters):
        feed = [np.array([int(rng.integers(0, shape.vocab))]) for _ in ctxs]
        t0 = time.perf_counter()
        M.forward(w, seqs, feed)
        t_fwd += time.perf_counter() - t0
        t0 = time.perf_counter()
        w.logits(h)
        t_lm += time.perf_counter() - t0
    t_fwd /= iters
    t_lm /= iters
    t_layers = max(t_fwd - t_lm, 1e-9)          # forward = layers + LM head
    t_step = t_layers * shape.n_layers / n_layers_sample + t_lm
    blas = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
    cores = max(blas) if blas else (os.cpu_count() or 1)
    return {"value": round(len(ctxs) / t_step, 3), "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"{iters} consecutive decode iterations of the {len(ctxs)} sequences through "
                       f"{n_layers_sample} of {shape.n_layers} layers ({t_layers:.2f} s each) plus the LM head "
                       f"({t_lm:.2f} s), float64 numpy, scaled to {shape.n_layers} layers"),
            "measured_s": round(iters * (t_fwd + t_lm), 2)}


def _blas_cores():
    from threadpoolctl import threadpool_info
    blas = [i.get("num_threads", 0) for i in threadpool_info() if i.get("user_api") == "blas"]
    return int(max(blas) if blas else (os.cpu_count() or 1))


def _oracle_iteration(shape, prefill, decodes, n_layers_sample, seed=0):
    """Time one oracle forward (float64 numpy) of a batch through the first
    `n_layers_sample` layers: `prefill` = list of (position, chunk length), `decodes` =
    list of context lengths; earlier KV is random.  Returns (seconds for the sampled
    layers, seconds for the final norm + LM head on the batch's logit rows)."""
    import numpy as np

    from oracle import model as M

    part = shape.with_layers(n_layers_sample)
    w = M.Weights(part)
    for l in range(n_layers_sample):
        w.layer(l)
    w.lm_head_f32()
    rng = np.random.default_rng(seed)
    seqs, chunks = [], []
    for pos, n in list(prefill) + [(c - 1, 1) for c in decodes]:
        s = M.Sequence(n_layers_sample)
        if pos > 0:
            for l in range(n_layers_sample):
                s.k[l] = rng.standard_normal((int(pos), shape.n_kv_heads, shape.head_dim))
                s.v[l] = rng.standard_normal((int(pos), shape.n_kv_heads, shape.head_dim))
        s.n = int(pos)
        seqs.append(s)
        chunks.append(rng.integers(0, shape.vocab, int(n)))
    w.embed_rows(np.zeros(1, np.int64))
    t0 = time.perf_counter()
    M.forward(w, seqs, chunks)
    t_all = time.perf_counter() - t0
    h = rng.standard_normal((len(seqs), shape.d_model))
    t0 = time.perf_counter()
    w.logits(h)
    t_lm = time.perf_counter() - t0
    return max(t_all - t_lm, 1e-9), t_lm


def cpu_baselines():
    """The CPU oracle timed on each workload (a baseline only, never a target): the tiny
    configuration in full; one representative iteration of workloads 3-5 through a
    sample of layers, scaled to the full depth (decode cost of workload 4 scaled from
    32 of its 256 sequences)."""
    import numpy as np

    import synth
    from oracle import model as M

    out = {"kind": "oracle", "cores": _blas_cores(), "workloads": []}
    # 1: tiny, full run
    shape = synth.model_shape("tiny")
    reqs = synth.workloads.cfg1(shape.vocab)
    w = M.Weights(shape)
    t0 = time.perf_counter()
    M.generate(w, [r.prompt for r in reqs], [r.max_new_tokens for r in reqs], keep_logits=False)
    t = time.perf_counter() - t0
    out["workloads"].append({"workload": 1, "value": round((640 + 32) / t, 1), "unit": "tokens/s",
                             "sample": f"full run: 640 prompt + 32 generated tokens in {t:.2f} s"})
    progress(f"oracle baseline 1: {t:.2f} s")
    # 3: one mixed iteration (2048-token chunk at position 4096 + 32 decodes at 2560), 1 of 32 layers
    shape = synth.model_shape("llama8b")
    tl, tm = _oracle_iteration(shape, [(4096, 2048)], [2560] * 32, 1)
    t_it = tl * shape.n_layers + tm
    out["workloads"].append({"workload": 3, "value": round(2080 / t_it, 2), "unit": "tokens/s",
                             "sample": (f"one mixed iteration (2048-token chunk at position 4096 + 32 decodes at "
                                        f"context 2560) through 1 of 32 layers ({tl:.2f} s) plus the LM head "
                                        f"({tm:.2f} s), scaled to 32 layers")})
    progress(f"oracle baseline 3: {t_it:.1f} s per iteration")
    # 4: one branch decode iteration, 32 of the 256 sequences at context 4352 (dense per sequence), 1 layer
    tl, tm = _oracle_iteration(shape, [], [4352] * 32, 1)
    t_it = (tl * shape.n_layers + tm) * 256 / 32
    out["workloads"].append({"workload": 4, "value": round(256 / t_it, 2), "unit": "tokens/s",
                             "sample": (f"one branch decode iteration of 32 of the 256 sequences (context 4352, "
                                        f"per-sequence KV) through 1 of 32 layers ({tl:.2f} s) plus the LM head "
                                        f"({tm:.2f} s), scaled to 32 layers and 256 sequences")})
    progress(f"oracle baseline 4: {t_it:.1f} s per iteration")
    # 5: 32B shape, one mixed iteration (2048-token chunk at 2048 + 64 decodes at 5000), 1 of 64 layers
    shape = synth.model_shape("qwen32b")
    tl, tm = _oracle_iteration(shape, [(2048, 2048)], [5000] * 64, 1)
    t_it = tl * shape.n_layers + tm
    out["workloads"].append({"workload": 5, "value": round(2112 / t_it, 2), "unit": "tokens/s",
                             "sample": (f"one mixed iteration of the 32B shape (2048-token chunk at position 2048 + "
                                        f"64 decodes at context 5000) through 1 of 64 layers ({tl:.2f} s) plus the "
                                        f"LM head ({tm:.2f} s), scaled to 64 layers")})
    progress(f"oracle baseline 5: {t_it:.1f} s per iteration")
    return out


# Calibrated cost-model coefficients in picoseconds (data, measured on one MI355X):
# t_comp = (c0 + c1*L_in + c2*L_in^2 + d1*L_out) / 1e6 us  (Section 4.1's t_prefill + t_decode)
# t_iter = (i0 + i1*T + i2*sum_decode_ctx + i3*prefill_attention_pairs) / 1e6 us
COST_PS = {
    # (c0, c1, c2, d1) of t_comp and (i0, i1, i2, i3) of the virtual iteration, picoseconds:
    # fitted to measured iterations on one MI355X by `bench.py --calibrate <model>` (five-term
    # iteration model, decode rows priced apart)
    "llama8b": ((4_383_794_963, 16_710_429, 234, 4_470_257_482), (4_383_794_963, 14_089_711, 20_149, 469, 3_934_053)),
    "qwen32b": ((13_843_718_843, 69_707_878, 806, 14_035_778_677),
                (13_843_718_843, 61_297_098, 38_500, 1_612, 34_363_125)),
    "llama70b": ((25_849_666_649, 154_627_611, 572, 26_181_289_978), (25_849_666_649, 140_833_739, 80_963, 1_144, 0)),
}


def load_model(name, n_layers=None):
    import synth
    from paper_2505_05286_amd.device import DeviceModel
    shape = synth.model_shape(name, n_layers)
    t0 = time.time()
    progress(f"generating and uploading {shape.name}-shaped bf16 weights")
    dm = DeviceModel(shape, lambda l: synth.gen_layer(shape, l), synth.gen_embed(shape), synth.gen_lm_head(shape),
                     synth.norm_weight(shape), device="cuda:0")
    progress(f"weights ready in {time.time() - t0:.1f} s")
    return shape, dm


def step_until(inst, now, cond, timed=None, per_step=None):
    """Step until cond(info) is true; return (now, iterations, prefill tokens, decode rows, seconds).
    per_step(info) is called after every iteration."""
    import torch
    from paper_2505_05286_amd import hxf
    it = pf = dec = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while True:
        st, info = inst.step(now)
        if st == hxf.IDLE:
            break
        now += info["t_iter_us"]
        it += 1
        pf += info["n_prefill_tokens"]
        dec += info["n_logit_rows"]
        if per_step is not None:
            per_step(info)
        if cond(info):
            break
    torch.cuda.synchronize()
    return now, it, pf, dec, time.perf_counter() - t0


def workload1(reps=20):
    """The tiny parity configuration end to end (4 requests, prompts 64-256, chunk 128,
    8 greedy tokens each), repeated; timing is informational (launch-bound)."""
    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    shape, dm = load_model("tiny")
    reqs = synth.workloads.cfg1(shape.vocab)
    cost, it = (200_000_000, 50_000, 0, 150_000_000), (150_000_000, 1_000_000, 0, 0)
    times, iters = [], 0
    for _ in range(reps):
        eng = Engine(dm, max_context=512, n_blocks=64, max_seqs=8, chunk_tokens=128, cost_ps=cost, iter_ps=it,
                     clock=hxf.CLOCK_MEASURED)
        for r in reqs:
            eng.inst.submit(0, r.workflow, 0, 0, r.wf_slo_us, r.prompt, r.max_new_tokens)
        now, n, pf, dec, dt = step_until(eng.inst, 0, lambda i: False)
        times.append(dt)
        iters = n
        del eng
    t = sorted(times)[len(times) // 2]
    return {"workload": "1: tiny decoder, 4 requests (prompts 64/128/192/256, chunk 128, 8 tokens each)",
            "iterations": iters, "ms_per_run_median": round(t * 1e3, 3), "ms_per_iteration": round(t / iters * 1e3, 3),
            "tokens_per_s": round((640 + 32) / t, 1)}


MODEL_NAMES = {"llama8b": "Llama-3-8B", "qwen32b": "Qwen2.5-32B", "llama70b": "Llama-3.1-70B"}


def describe(shape):
    return (f"{MODEL_NAMES.get(shape.name, shape.name)} shape ({shape.n_layers} layers, d {shape.d_model}, "
            f"{shape.n_q_heads}q/{shape.n_kv_heads}kv heads of {shape.head_dim}, SwiGLU {shape.ffn_dim}, "
            f"vocab {shape.vocab})")


def kv_pages_that_fit(shape, reserve_gb=8.0, frac=0.9):
    """KV pages that fit the device memory left after the weights (a margin for the
    workspace and torch's allocator kept aside)."""
    import torch
    free, _ = torch.cuda.mem_get_info()
    page = 2 * shape.n_kv_heads * shape.head_dim * 2 * 16 * shape.n_layers
    return int(max(free - reserve_gb * 1e9, 0) * frac // page)


MFMA_BF16_PEAK_TFLOPS = 2500.0


def mixed_iteration_profile(dm, shape, n_profiled=3, n_warm=2, n_timed=8):
    """Timing of workload-3 mixed iterations (a 2048-token prefill chunk co-batched with
    32 decode rows: 2080-row projections).  The 32 decodes are prefilled first (untimed),
    the 16 prompts submitted; `n_warm` mixed iterations warm up, `n_timed` are timed by the
    host clock around them (their prefill tokens per second are the bench line's prefill
    rate), then `n_profiled` run with profiling on (eager launches, HIP events stamped by
    every GEMM and prefill-attention launch).  Returns the MFMA roofline of each projection
    and of a whole layer's four, 2*M*N*K / kernel time / 2.5 PFLOP/s, the prefill attention's,
    and the timed prefill rate."""
    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    decodes, prompts = synth.workloads.cfg3(shape.vocab)
    cost, it = COST_PS.get(shape.name, COST_PS["llama8b"])
    total = sum(-(-(len(s.prompt) + 4096) // 16) for s in decodes) + sum(-(-len(s.prompt) // 16) for s in prompts)
    eng = Engine(dm, max_context=8192 + 4096, n_blocks=total + 256, max_seqs=64, chunk_tokens=2048, cost_ps=cost,
                 iter_ps=it, clock=hxf.CLOCK_MEASURED)
    inst = eng.inst
    for s in decodes:
        inst.submit(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, s.max_new_tokens)
    now, *_ = step_until(inst, 0, lambda i: i["n_prefill_tokens"] == 0)
    for s in prompts:
        inst.submit(now, s.workflow, 0, now, s.wf_slo_us, s.prompt, s.max_new_tokens)
    def after(k):
        """A step_until condition true on its k-th call."""
        calls = [0]

        def cond(_info):
            calls[0] += 1
            return calls[0] >= k
        return cond

    now, *_ = step_until(inst, now, after(n_warm))
    now, t_it, t_pf, t_dec, t_dt = step_until(inst, now, after(n_timed))
    prefill = {"tokens_per_s": round(t_pf / t_dt, 1), "prefill_tokens": t_pf, "decode_rows": t_dec,
               "iterations": t_it, "ms_per_iteration": round(t_dt / t_it * 1e3, 3),
               "workload": "3: mixed iterations, 2048-token prefill chunk + 32 decode rows, after "
                           f"{n_warm} untimed ones; host clock around the {t_it} iterations"}
    inst.profile_enable(True)
    rows = []
    now, iters, pf, dec, dt = step_until(inst, now, lambda i: len(rows) >= n_profiled,
                                         per_step=lambda i: rows.append(i["n_tokens"]))
    prof = inst.profile()
    inst.profile_enable(False)
    del eng, inst
    peak = MFMA_BF16_PEAK_TFLOPS
    per = {}
    for k in ("qkv", "o", "gate_up", "down"):
        ms, fl, n = prof["gemm_ms"][k], prof["gemm_flops"][k], prof["gemm_launches"][k]
        ach = fl / (ms * 1e-3) / 1e12
        per[k] = {"launches": n, "avg_us": round(ms / n * 1e3, 1), "tflops": round(ach, 1),
                  "frac": round(ach / peak, 4)}
    fl = sum(prof["gemm_flops"][k] for k in per)
    ms = sum(prof["gemm_ms"][k] for k in per)
    layer = fl / (ms * 1e-3) / 1e12
    pa = prof["prefill_attn_flops"] / (prof["prefill_attn_ms"] * 1e-3) / 1e12
    return {"bound": "mfma", "achieved": round(layer, 1), "peak": peak, "unit": "TFLOP/s",
            "frac": round(layer / peak, 4), "traffic": None,
            "kernels": "gemm_big_kernel (QKV, O, gate/up + SwiGLU, down) of every layer",
            "workload": "3: mixed iterations, 2048-token prefill chunk + 32 decode rows",
            "rows_per_iteration": rows, "iterations_profiled": iters,
            "ms_per_iteration_profiled": round(dt / iters * 1e3, 2),
            "timing": "kernel-stamped HIP events, 2*M*N*K per launch over its duration",
            "per_projection": per,
            "prefill_timed": prefill,
            "prefill_attention": {"launches": prof["prefill_attn_launches"], "tflops": round(pa, 1),
                                  "frac": round(pa / peak, 4),
                                  "avg_us": round(prof["prefill_attn_ms"] / max(prof["prefill_attn_launches"], 1)
                                                  * 1e3, 1)}}


def workload3(model="llama8b"):
    """Mixed iterations: 32 running decodes (context U[1024, 4096]) co-batched with chunked
    prefill (2048 tokens per iteration) of 16 prompts of length U[2048, 8192]."""
    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    shape, dm = load_model(model)
    decodes, prompts = synth.workloads.cfg3(shape.vocab)
    cost, it = COST_PS[model]
    total = sum(-(-(len(s.prompt) + 4096) // 16) for s in decodes) + sum(-(-len(s.prompt) // 16) for s in prompts)
    eng = Engine(dm, max_context=8192 + 4096, n_blocks=total + 256, max_seqs=64, chunk_tokens=2048, cost_ps=cost,
                 iter_ps=it, clock=hxf.CLOCK_MEASURED)
    inst = eng.inst
    for s in decodes:
        inst.submit(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, s.max_new_tokens)
    progress("prefilling the 32 decode sequences (untimed)")
    now, *_ = step_until(inst, 0, lambda i: i["n_prefill_tokens"] == 0)
    for s in prompts:
        inst.submit(now, s.workflow, 0, now, s.wf_slo_us, s.prompt, s.max_new_tokens)
    progress("timed: mixed chunked-prefill + decode iterations")
    now, iters, pf, dec, dt = step_until(inst, now, lambda i: i["n_prefill_tokens"] == 0)
    return {"workload": f"3: {describe(shape)}, 16 prompts U[2048,8192] chunked 2048 + 32 decodes ctx U[1024,4096]",
            "iterations": iters, "ms_per_iteration": round(dt / iters * 1e3, 3), "prefill_tokens": pf,
            "prefill_tokens_per_s": round(pf / dt, 1), "decode_tokens_per_s": round(dec / dt, 1),
            "tokens_per_s": round((pf + dec) / dt, 1)}


def workload4():
    """Shared-prefix candidates: 32 prefill-only 4096-token parents, 8 forks each decoding
    256 tokens (256 sequences), then a 512-token correction prefill on the even branches."""
    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    shape, dm = load_model("llama8b")
    parents, forks, corr = synth.workloads.cfg4(shape.vocab)
    cost, it = COST_PS["llama8b"]
    n_blocks = 32 * 256 + 256 * 18 + 128 * 34 + 512
    eng = Engine(dm, max_context=4096 + 256 + 512 + 16, n_blocks=n_blocks, max_seqs=256, chunk_tokens=2048,
                 cost_ps=cost, iter_ps=it, clock=hxf.CLOCK_MEASURED)
    inst = eng.inst
    pid = [inst.submit(0, p.workflow, 0, 0, p.wf_slo_us, p.prompt, 0, retain=True) for p in parents]
    progress("timed: prefill of 32 x 4096-token parents")
    now, it1, pf1, _, dt1 = step_until(inst, 0, lambda i: False)
    fid = {}
    for f in forks:
        fid[(f.workflow, f.branch)] = inst.submit(now, f.workflow, 1, 0, f.wf_slo_us, f.prompt, f.max_new_tokens,
                                                  parent=pid[f.workflow], retain=f.retain_kv)
    for p in pid:
        inst.release(p)
    progress("timed: 256 forked branches decoding 256 tokens each")
    shared = (len(parents[0].prompt) - 1) // 16 * 16         # tokens of the parents' shared full pages
    kv = {"logical": 0, "unique": 0}

    n_prof = [0]

    def it_p_count():
        n_prof[0] += 1
        return n_prof[0] >= 8

    def count(info):
        # (token, kv-head) pairs of context attended this iteration, per sequence and once per page
        kv["logical"] += info["sum_decode_ctx"]
        kv["unique"] += info["sum_decode_ctx"] - (info["n_decode"] - len(parents)) * shared
    # the forks' first iterations re-prefill the parents' partial last pages; once every
    # fork decodes, 8 iterations are profiled (eager launches, kernel-stamped events) and
    # the rest, which replay a captured graph, are timed
    now, it0, _, _, _ = step_until(inst, now, lambda i: i["n_prefill_tokens"] == 0, per_step=count)
    inst.profile_enable(True)
    now, it_p, _, _, _ = step_until(inst, now, lambda i: it_p_count(), per_step=count)
    prof = inst.profile()
    inst.profile_enable(False)
    dec_p = max(prof["decode_attn_launches"] / shape.n_layers, 1)   # profiled iterations with decode rows
    now, it2, pf2, dec2, dt2 = step_until(inst, now, lambda i: False, per_step=count)
    per_tok = 2 * shape.n_kv_heads * shape.head_dim * 2 * shape.n_layers     # K+V bytes per token, all layers
    for c in corr:
        inst.submit(now, c.workflow, 2, 0, c.wf_slo_us, c.prompt, c.max_new_tokens, parent=fid[(c.workflow, c.branch)])
    for (w, b), f in fid.items():
        if b % 2 == 0:
            inst.release(f)
    progress("timed: 512-token correction prefill on 128 branches")
    now, it3, pf3, _, dt3 = step_until(inst, now, lambda i: False)
    return {"workload": "4: 8B, 32 shared 4096-token prompts x 8 branches x 256 tokens, 512-token corrections",
            "parent_prefill_tokens_per_s": round(pf1 / dt1, 1),
            "branch_decode_tokens_per_s": round(dec2 / dt2, 1), "branch_iterations_timed": it2,
            "branch_iterations_profiled": it_p, "branch_iterations_untimed_tail_prefill": it0,
            "branch_ms_per_iteration": round(dt2 / it2 * 1e3, 3),
            "branch_kv_gb_per_iteration": {"logical": round(kv["logical"] * per_tok / (it0 + it2 + it_p) / 1e9, 2),
                                           "unique": round(kv["unique"] * per_tok / (it0 + it2 + it_p) / 1e9, 2),
                                           "read": round(prof["decode_attn_bytes"] / dec_p / 1e9, 2)},
            "branch_attention_ms_per_iteration": round(prof["decode_attn_ms"] / dec_p, 3),
            "branch_attention_read_tb_per_s": round(prof["decode_attn_bytes"] / (prof["decode_attn_ms"] * 1e-3) / 1e12,
                                                    3),
            "branch_gemm_ms_per_iteration": {k: round(prof["gemm_ms"][k] / it_p, 3) for k in prof["gemm_ms"]},
            "branch_gemm_tflops": {k: round(prof["gemm_flops"][k] / max(prof["gemm_ms"][k], 1e-9) / 1e9, 1)
                                   for k in prof["gemm_ms"]},
            "correction_prefill_tokens_per_s": round(pf3 / dt3, 1)}


def cfg5_workflows(n, vocab, model="qwen32b"):
    import numpy as np
    import synth
    from paper_2505_05286_amd.workflows import Req, Workflow
    s = synth.workloads.CFG5_SHAPE
    out = []
    for w in synth.workloads.cfg5(vocab=vocab, n_wf=n, model=model):
        stages = [[Req(w.schema, s["s1_out"], retain=True)],
                  [Req(np.zeros(0, np.int32), s["cand_out"], parent=(0, 0), retain=(b % 2 == 0))
                   for b in range(s["n_cand"])],
                  [Req(w.corrections[k], s["corr_out"], parent=(1, 2 * k)) for k in range(s["n_corr"])],
                  [Req(w.eval_prompt, s["eval_out"])]]
        shapes = [(w.schema_len, s["s1_out"]), (16, s["cand_out"]), (16 + s["corr_in"], s["corr_out"]),
                  (s["eval_in"], s["eval_out"])]
        out.append(Workflow(w.workflow, w.arrival_us, w.slo_us, stages, shapes))
    return out


def workload5(n_wf, policy, model="qwen32b", rate=0.5):
    """Replay of four-stage workflows (Poisson arrivals, `rate` per second; configured:
    the Qwen2.5-32B shape at 0.5/s) driven by the local priority queue; scheduling runs on
    the virtual clock, the forward on the GPU."""
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    from paper_2505_05286_amd.workflows import Driver
    import torch
    shape, dm = load_model(model)
    wfs = cfg5_workflows(n_wf, shape.vocab, model)
    for w in wfs:
        w.arrival_us = int(w.arrival_us * 0.5 / rate)    # generated at 0.5 workflows/s
    cost, it = COST_PS[model]
    pol = {"pq": hxf.POLICY_PQ, "fcfs": hxf.POLICY_FCFS, "llf": hxf.POLICY_LLF}[policy]
    n_blocks = min(40_000, kv_pages_that_fit(shape))
    eng = Engine(dm, max_context=8192 + 64 + 256 + 512 + 256 + 16, n_blocks=n_blocks, max_seqs=128,
                 chunk_tokens=2048, cost_ps=cost, iter_ps=it, policy=pol)
    d = Driver(eng.inst, wfs)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    d.run(report=lambda it, now, fin: progress(f"{it} iterations, virtual {now / 1e6:.0f} s, {fin}/{n_wf} "
                                                f"workflows done, {time.perf_counter() - t0:.0f} s"))
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = d.stats()
    st.update({"workload": f"5: {describe(shape)}, {n_wf} four-stage workflows, Poisson {rate}/s, policy {policy}",
               "kv_pages": n_blocks,
               "gpu_seconds": round(dt, 2), "prefill_tokens_per_s": round(st["prefill_tokens"] / dt, 1),
               "decode_tokens_per_s": round(st["decode_tokens"] / dt, 1)})
    return st


def calibrate(model, rows_out=None):
    """Fit the virtual-clock iteration model, t = i0 + i1*T_prefill + i2*sum_decode_ctx +
    i3*prefill_attn + i4*n_decode, to iterations measured on this GPU (measured clock):
    batches of 1-128 sequences at two contexts, prefilled in 2048-token chunks and then
    decoding together for ten decode-only iterations (the rest of their output budget is
    cancelled), lone prefills of 512-8192 tokens, and chunked prefill co-batched with 32
    decodes.  The first two decode-only iterations of a batch shape (eager, then the HIP
    graph capture) are left out.  From the fit it also derives the request cost model
    (c0, c1, c2, d1 of t_comp, Section 4.1: a lone request's chunked prefill and batch-1
    decode steps) and the isolated-latency reference per prompt and output token that the
    workflow SLOs are scaled from."""
    import numpy as np
    from scipy.optimize import nnls

    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    import torch

    shape, dm = load_model(model)
    cost, it = COST_PS[model]
    chunk = 2048
    n_blocks = min(128 * (4096 + 16) // 16 + 1024, kv_pages_that_fit(shape))
    eng = Engine(dm, max_context=8192 + 512, n_blocks=n_blocks, max_seqs=128, chunk_tokens=chunk, cost_ps=cost,
                 iter_ps=it, clock=hxf.CLOCK_MEASURED)
    inst = eng.inst
    rng = np.random.default_rng(11)
    rows = []
    skipped = [0]

    def run(reqs, label, decode_iters=None):
        now = 0
        ids = [inst.submit(now, 0, 0, 0, 10 ** 12, rng.integers(0, shape.vocab, L).astype(np.int32), n_new)
               for L, n_new in reqs]
        n, prev, run_len, n_dec_only = 0, None, 0, 0
        while True:
            st, info = inst.step(now)
            if st == hxf.IDLE:
                break
            now += info["t_iter_us"]
            n += 1
            key = (info["n_decode"], info["n_prefill_tokens"])
            run_len = run_len + 1 if key == prev else 1
            prev = key
            if info["n_prefill_tokens"] == 0:
                n_dec_only += 1
                if run_len <= 2:
                    skipped[0] += 1
                    continue
            rows.append((info["n_prefill_tokens"], info["n_decode"], info["sum_decode_ctx"], info["prefill_attn"],
                         info["t_iter_us"], label))
            if decode_iters is not None and n_dec_only >= decode_iters + 2:
                break
        for r in ids:
            if inst.request_state(r)["state"] in (0, 1, 2):
                inst.cancel(r)
        inst.drain()
        progress(f"calibration: {label}: {n} iterations")

    run([(256, 4)], "warmup")
    rows.clear()
    skipped[0] = 0
    for ctx in (1000, 4000):      # ten decode steps stay within one 64-page block-table width
        for B in (1, 8, 32, 64, 128):
            n_new = -(-B * ctx // chunk) + 16      # still decoding when the last prompt is prefilled
            run([(ctx, n_new)] * B, f"decode B={B} ctx={ctx}", decode_iters=10)
    for L in (512, 2048, 4096, 8192):
        run([(L, 1)], f"lone prefill {L}")
    run([(2048, 40)] * 32 + [(8192, 1)] * 2, "mixed: 32 decodes + chunked prefill")
    torch.cuda.synchronize()
    X = np.array([[1.0, r[0], r[2], r[3], r[1]] for r in rows])
    y = np.array([r[4] for r in rows], dtype=np.float64)
    coef, _ = nnls(X, y)                      # us per unit, non-negative
    pred = X @ coef
    rel = np.abs(pred - y) / y
    i_ps = [int(round(c * 1e6)) for c in coef]
    i0, i1, i2, i3, i4 = coef
    # request cost model from the fit (a lone request, chunks of `chunk`, decode at ~4096 context)
    c_ps = [int(round(i0 * 1e6)), int(round((i1 + i0 / chunk + i3 * chunk / 2) * 1e6)), int(round(i3 / 2 * 1e6)),
            int(round((i0 + i4 + i2 * 4096) * 1e6))]
    ref = {"base_us": round(i0, 1), "per_prompt_token_us": round(i1 + i0 / chunk + i3 * (chunk / 2 + 2048), 3),
           "per_output_token_us": round(i0 + i4 + i2 * 4096, 1)}
    dec = np.array([r[0] == 0 for r in rows])
    if rows_out:
        with open(rows_out, "w") as f:
            json.dump([list(r) + [float(pv)] for r, pv in zip(rows, pred)], f)
    return {"calibration": model, "iterations": len(rows), "left_out": skipped[0], "iter_ps": i_ps, "cost_ps": c_ps,
            "decode_only_median_rel_err": round(float(np.median(rel[dec])), 4) if dec.any() else None,
            "isolated_reference": ref, "median_rel_err": round(float(np.median(rel)), 4),
            "p90_rel_err": round(float(np.percentile(rel, 90)), 4)}


ABLATION_SCENARIOS = [
    # (name, arrival-rate multiple of 0.5 workflows/s, SLO multiple of the isolated latency, tenant mix)
    ("configured: 0.5 wf/s, SLO 10x", 1.0, 10, None),
    ("0.6 wf/s, SLO 10x", 1.2, 10, None),
    ("0.7 wf/s, SLO 10x", 1.4, 10, None),
    ("0.8 wf/s, SLO 10x", 1.6, 10, None),
    ("tight SLO: 0.6 wf/s, SLO 5x", 1.2, 5, None),
    ("two tenants at 0.6 wf/s: SLO 5x (even) / 20x (odd)", 1.2, None, (5, 20)),
]


def policy_ablation(n_wf=300):
    """Local-queue policy ablation (PQ vs FCFS vs LLF) on config-5 workflows, run by
    the scheduler-only executor on the virtual clock: the iteration time is the
    calibrated cost model's, so no GPU is needed and every run is deterministic.
    Reports SLO attainment and P95 latency per scenario and policy."""
    import numpy as np

    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.workflows import Driver

    shape = synth.model_shape("qwen32b")
    cost, it = COST_PS["qwen32b"]
    pols = [("pq", hxf.POLICY_PQ), ("fcfs", hxf.POLICY_FCFS), ("llf", hxf.POLICY_LLF)]
    out = []
    for name, rate, slo, mix in ABLATION_SCENARIOS:
        row = {"scenario": name}
        for pname, pol in pols:
            wfs = cfg5_workflows(n_wf, shape.vocab)
            for w in wfs:
                w.arrival_us = int(w.arrival_us / rate)
                scale = slo if mix is None else mix[w.wid % 2]
                w.slo_us = w.slo_us * scale // 10   # generated at 10x the isolated latency
            mcfg = hxf.model_cfg(shape, 8192 + 64 + 256 + 512 + 256 + 16)
            scfg = hxf.sched_cfg(40_000, 128, 2048, cost, it, policy=pol, executor=hxf.EXEC_NULL)
            inst = hxf.Instance(mcfg, scfg)
            d = Driver(inst, wfs)
            d.run()
            st = d.stats()
            rnd = lambda v: None if v is None else round(v, 2)
            res = {"slo_attainment": round(st["slo_attainment"], 4), "p95_latency_s": rnd(st["p95_latency_s"]),
                   "mean_latency_s": rnd(st["mean_latency_s"]), "finished": st["finished"],
                   "mean_in_flight": rnd(st["mean_in_flight"]), "stage_wait_mean_s": st["stage_wait_mean_s"],
                   "stage_wait_p95_s": st["stage_wait_p95_s"]}
            if mix is not None:
                for t, sc in enumerate(mix):
                    sel = [w for w in d.wf if w.wid % 2 == t]
                    res[f"slo_attainment_{sc}x"] = round(float(np.mean([0 <= w.finish_us - w.arrival_us <= w.slo_us
                                                                        for w in sel])), 4)
            row[pname] = res
            del inst
            progress(f"{name}: {pname} {res}")
        out.append(row)
    return {"ablation": "local queue policy, config 5 (32B shape), virtual clock", "workflows": n_wf,
            "scenarios": out}


def measured_ablation(n_wf, rate, policies=("pq", "fcfs", "llf"), slo_scale=10, model="qwen32b", tenants=None):
    """The local-queue policy ablation on the GPU with the measured clock: the same
    workload-5 workflows (arrivals rescaled to `rate` per second, SLO = slo_scale x the
    isolated latency) replayed through the HIP instance once per policy; every
    iteration's duration is its measured wall time (idle gaps are skipped to the next
    arrival), so latencies and SLO attainment are served times, not cost-model times.
    tenants=(a, b): even workflows get SLO a x, odd ones b x (two tenants)."""
    import torch

    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import Engine
    from paper_2505_05286_amd.workflows import Driver
    shape, dm = load_model(model)
    cost, it = COST_PS[model]
    pols = {"pq": hxf.POLICY_PQ, "fcfs": hxf.POLICY_FCFS, "llf": hxf.POLICY_LLF}
    n_blocks = min(40_000, kv_pages_that_fit(shape))
    out = []
    for name in policies:
        wfs = cfg5_workflows(n_wf, shape.vocab, model)
        for w in wfs:
            w.arrival_us = int(w.arrival_us * 0.5 / rate)
            w.slo_us = w.slo_us * (slo_scale if tenants is None else tenants[w.wid % 2]) // 10
        eng = Engine(dm, max_context=8192 + 64 + 256 + 512 + 256 + 16, n_blocks=n_blocks, max_seqs=128,
                     chunk_tokens=2048, cost_ps=cost, iter_ps=it, policy=pols[name], clock=hxf.CLOCK_MEASURED)
        d = Driver(eng.inst, wfs, measured=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        d.run(report=lambda i, now, fin: progress(f"{name}: {i} iterations, clock {now / 1e6:.0f} s, {fin}/{n_wf} "
                                                  f"workflows done, {time.perf_counter() - t0:.0f} s"),
              report_every=1000)
        torch.cuda.synchronize()
        st = d.stats()
        rnd = lambda v: None if v is None else round(v, 2)
        res = {"policy": name, "slo_attainment": round(st["slo_attainment"], 4),
               "p95_latency_s": rnd(st["p95_latency_s"]), "mean_latency_s": rnd(st["mean_latency_s"]),
               "finished": st["finished"], "iterations": st["iterations"],
               "gpu_seconds": round(time.perf_counter() - t0, 1), "mean_in_flight": rnd(st["mean_in_flight"]),
               "stage_wait_mean_s": st["stage_wait_mean_s"], "stage_wait_p95_s": st["stage_wait_p95_s"]}
        if tenants is not None:
            for t, sc in enumerate(tenants):
                sel = [w for w in d.wf if w.wid % 2 == t]
                res[f"slo_attainment_{sc}x"] = round(sum(0 <= w.finish_us - w.arrival_us <= w.slo_us
                                                         for w in sel) / max(len(sel), 1), 4)
        progress(json.dumps(res))
        out.append(res)
        del d, eng
    return {"ablation": f"local queue policy on the GPU, measured clock, {MODEL_NAMES[model]} shape",
            "workflows": n_wf, "rate_wf_per_s": rate, "slo_scale": slo_scale if tenants is None else list(tenants),
            "kv_pages": n_blocks,
            "results": out}


CLUSTER_SPEEDS = (1.0, 1.0, 2.0, 2.0)
CLUSTER_SCENARIOS = [
    # (name, [(workflows, arrival rate in workflows/s), ...] in sequence)
    ("steady 1.0 wf/s", [(300, 1.0)]),
    ("steady 1.2 wf/s", [(300, 1.2)]),
    ("shift 0.8 -> 1.6 wf/s", [(150, 0.8), (150, 1.6)]),
]


def cluster_sim():
    """Coordinator across four scheduler-only instances (Sections 4.1-4.3) on config-5
    workflows: two instances with this GPU's calibrated 32B cost models and two with
    every coefficient doubled (an older GPU), on one virtual clock.  Round-robin vs
    workload-balanced dispatch (fixed alpha, and online alpha tuning from alpha = 0),
    with PQ or FCFS local queues.  CPU only; deterministic."""
    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.cluster import Cluster, InstanceSpec, TunerCfg, calibrate_beta

    shape = synth.model_shape("qwen32b")
    cost, it = COST_PS["qwen32b"]
    mcfg = hxf.model_cfg(shape, 8192 + 64 + 256 + 512 + 256 + 16)

    def specs(policy):
        return [InstanceSpec(tuple(int(c * k) for c in cost), tuple(int(c * k) for c in it), 40_000, 128, 2048,
                             policy) for k in CLUSTER_SPEEDS]

    runs = [("rr+pq", "rr", 0.0, hxf.POLICY_PQ, None), ("wb+fcfs tuned", "wb", 0.0, hxf.POLICY_FCFS, TunerCfg()),
            ("wb+pq alpha 0", "wb", 0.0, hxf.POLICY_PQ, None), ("wb+pq alpha 0.5", "wb", 0.5, hxf.POLICY_PQ, None),
            ("wb+pq alpha 0.9", "wb", 0.9, hxf.POLICY_PQ, None), ("wb+pq tuned", "wb", 0.0, hxf.POLICY_PQ, TunerCfg())]
    out = []
    for name, phases in CLUSTER_SCENARIOS:
        n_total = sum(n for n, _ in phases)
        wfs = cfg5_workflows(n_total, shape.vocab)
        base = [w.arrival_us for w in wfs]     # generated at 0.5 workflows/s
        t, k = 0.0, 0
        for n, rate in phases:
            start = base[k]
            for i in range(k, k + n):
                wfs[i].arrival_us = int(t + (base[i] - start) * 0.5 / rate)
            t = wfs[k + n - 1].arrival_us + (base[k + n] - base[k + n - 1]) * 0.5 / rate if k + n < n_total else t
            k += n
        beta = calibrate_beta(mcfg, specs(hxf.POLICY_PQ), wfs[:20])
        row = {"scenario": name, "beta_us2": beta}
        for label, disp, alpha, pol, tuner in runs:
            c = Cluster(mcfg, specs(pol), disp, alpha, beta, tuner=tuner)
            t0 = time.perf_counter()
            c.run(wfs)
            dt = time.perf_counter() - t0
            st = c.stats()
            res = {"slo_attainment": round(st["slo_attainment"], 4), "p95_latency_s": st["p95_latency_s"],
                   "mean_latency_s": round(st["mean_latency_s"], 2), "requests_per_instance": st["per_instance_requests"],
                   "host_seconds": round(dt, 2)}
            if tuner is not None:
                res["retunings"] = [(round(x[0] / 1e6, 1), round(x[3], 5), x[4]) for x in c.alpha_log
                                    if x[4] is not None]
                res["windows_tested"] = len(c.alpha_log)
                res["grid_search_s"] = round(sum(c.tune_seconds) / max(len(c.tune_seconds), 1), 2)
            c.close()
            row[label] = res
            progress(f"{name}: {label} {res}")
        out.append(row)
    return {"cluster": "4 instances (2 x calibrated 32B cost model, 2 x half speed), config-5 workflows, "
                       "virtual clock", "scenarios": out}


def hbm_copy_probe(nbytes=4 << 30, reps=5):
    """Achievable HBM bandwidth for context: the library's copy kernel (16-byte loads and
    stores) on a 4 GiB buffer, bytes read plus bytes written per second (best of `reps`)."""
    import torch
    from paper_2505_05286_amd import hxf
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    dst = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    st = torch.cuda.current_stream().cuda_stream
    hxf.op_copy(src.data_ptr(), dst.data_ptr(), nbytes, st)
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        hxf.op_copy(src.data_ptr(), dst.data_ptr(), nbytes, st)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del src, dst
    gbs = 2 * nbytes / (best * 1e-3) / 1e9
    return {"kernel": "copy_kernel (hxf_op_copy)", "bytes_moved": 2 * nbytes, "ms": round(best, 3),
            "gb_per_s": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
            "note": "a copy reads and writes HBM at once; a read-only stream, like the decode attention's, runs faster"}


def hbm_read_probe(nbytes=8 << 30, reps=5):
    """Achievable HBM read bandwidth for context: the library's streaming-read kernel
    (16-byte loads, four in flight per thread, 4096 workgroups) over an 8 GiB buffer,
    bytes read per second (best of `reps`)."""
    import torch
    from paper_2505_05286_amd import hxf
    src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
    sink = torch.empty(hxf.READ_SINK_WORDS, dtype=torch.int32, device="cuda:0")
    st = torch.cuda.current_stream().cuda_stream
    hxf.op_read(src.data_ptr(), nbytes, sink.data_ptr(), st)
    best = None
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        hxf.op_read(src.data_ptr(), nbytes, sink.data_ptr(), st)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        best = ms if best is None else min(best, ms)
    del src, sink
    gbs = nbytes / (best * 1e-3) / 1e9
    return {"kernel": "read_kernel (hxf_op_read)", "bytes_read": nbytes, "ms": round(best, 3),
            "gb_per_s": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}


def gemm_probe(reps=3, M=2080):
    """Only the four prefill projections of the 8B shape at 2080 rows (a 2048-token chunk
    plus 32 decodes), `reps` times each, through the library's GEMM entry point with
    random bf16 operands: the short program the MFMA-counter runs profile."""
    import torch

    from paper_2505_05286_amd import hxf

    hxf.lib()
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    st = torch.cuda.current_stream().cuda_stream
    shapes = [("qkv", 6144, 4096, hxf.EPI_BF16), ("o", 4096, 4096, hxf.EPI_RESID),
              ("gate_up", 2 * 14336, 4096, hxf.EPI_SWIGLU), ("down", 4096, 14336, hxf.EPI_RESID)]
    out = []
    for name, N, K, epi in shapes:
        rows = N // 2 if epi == hxf.EPI_SWIGLU else N
        A = (torch.randn(M, K, device=dev, generator=g) * 0.5).to(torch.bfloat16)
        packed = []
        for _ in range(2 if epi == hxf.EPI_SWIGLU else 1):
            W = (torch.randn(rows, K, device=dev, generator=g) * 0.02).to(torch.bfloat16)
            P = torch.empty(hxf.packed_weight_bytes(rows, K) // 2, dtype=torch.int16, device=dev)
            hxf.op_pack_weight(W.data_ptr(), rows, K, P.data_ptr(), st)
            packed.append(P)
        n_out = rows
        C = torch.zeros(M, n_out, device=dev, dtype=torch.bfloat16 if epi in (hxf.EPI_BF16, hxf.EPI_SWIGLU)
                        else torch.float32)
        wsn = hxf.op_gemm_workspace_bytes(M, N, K)
        ws = torch.empty(max(wsn, 256), dtype=torch.uint8, device=dev)
        for _ in range(reps):
            hxf.op_gemm(A.data_ptr(), K, packed[0].data_ptr(), packed[-1].data_ptr() if len(packed) > 1 else 0,
                        C.data_ptr(), n_out, M, N, K, epi, ws.data_ptr(), ws.numel(), st)
        torch.cuda.synchronize()
        out.append({"gemm": name, "M": M, "N": N, "K": K, "flops": 2 * M * N * K, "launches": reps})
    return {"probe": "prefill GEMMs at 2080 rows", "gemms": out}


PREFILL_PROBE_CHUNKS = ((0, 2048), (2048, 2048), (6144, 2048), (0, 1024), (4352, 512), (4080, 16))


def prefill_attn_probe(reps=11):
    """Only the chunked-prefill attention (plus its merge when items are cut), one chunk
    of one sequence at a time at the 8B head shape, `reps` times per chunk (first position,
    queries) of PREFILL_PROBE_CHUNKS: the short program the kernel-trace run profiles (each
    call uploads its work list and synchronises, so per-kernel times come from the trace)."""
    import numpy as np
    import torch

    import synth
    from paper_2505_05286_amd import hxf

    hxf.lib()
    shape = synth.model_shape("llama8b")
    hq, hkv, dh = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    out = []
    for p0, n in PREFILL_PROBE_CHUNKS:
        pages = -(-(p0 + n) // 16)
        bt = np.arange(pages, dtype=np.int32)[None, :]
        per = hkv * pages * 16 * dh
        kp = (torch.randn(per, device=dev, generator=g) * 0.5).to(torch.bfloat16)
        vp = (torch.randn(per, device=dev, generator=g) * 0.5).to(torch.bfloat16)
        q = (torch.randn(n * hq * dh, device=dev, generator=g) * 0.5).to(torch.bfloat16)
        o = torch.empty_like(q)
        btd = torch.from_numpy(bt).to(dev)
        wsn = hxf.op_prefill_attention_workspace_bytes(1, hq, hkv, [n])
        ws = torch.empty(max(wsn, 256), dtype=torch.uint8, device=dev)
        for _ in range(reps):
            hxf.op_prefill_attention(q.data_ptr(), kp.data_ptr(), vp.data_ptr(), pages, btd.data_ptr(), pages, [0],
                                     [p0], [n], o.data_ptr(), 1, hq, hkv, dh, ws.data_ptr(), ws.numel())
        torch.cuda.synchronize()
        flops = (p0 * n + n * (n + 1) // 2) * 4 * dh * hq
        out.append({"first_position": p0, "queries": n, "launches": reps, "flops": flops})
    return {"probe": "prefill attention, one 8B-shaped chunk per call", "chunks": out}


def attn_kernel_probe(reps=8):
    """Only the paged decode-attention kernel (plus its merge) on the benchmark's
    64 contexts, `reps` times, then one 1 GiB device copy of known size: the short
    program the hardware-counter runs profile (the copy calibrates FETCH_SIZE and
    WRITE_SIZE).  KV pages are contiguous per sequence, contents random bf16."""
    import numpy as np
    import torch

    import synth
    from paper_2505_05286_amd import hxf

    hxf.lib()
    shape = synth.model_shape("llama8b")
    hq, hkv, dh = shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    stages = synth.workloads.cfg2(vocab=shape.vocab, n=BATCH, max_new_tokens=MAX_NEW)
    ctx = np.array([len(s.prompt) + 8 for s in stages], np.int32)
    pages = -(-ctx // 16)
    n_blocks = int(pages.sum())
    bt_w = int(pages.max())
    bt = np.zeros((BATCH, bt_w), np.int32)
    off = 0
    for b, n in enumerate(pages):
        bt[b, :n] = np.arange(off, off + n)
        off += n
    dev = "cuda:0"
    g = torch.Generator(device=dev).manual_seed(0)
    per = hkv * n_blocks * 16 * dh
    kp = (torch.randn(per, device=dev, generator=g) * 0.5).to(torch.bfloat16)
    vp = (torch.randn(per, device=dev, generator=g) * 0.5).to(torch.bfloat16)
    q = (torch.randn(BATCH * hq * dh, device=dev, generator=g) * 0.5).to(torch.bfloat16)
    out = torch.empty_like(q)
    btd = torch.from_numpy(bt).to(dev)
    wsb = hxf.op_decode_attention_workspace_bytes(BATCH, hq, hkv, dh, ctx)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    st = torch.cuda.current_stream().cuda_stream
    for _ in range(reps):
        hxf.op_decode_attention(q.data_ptr(), kp.data_ptr(), vp.data_ptr(), n_blocks, btd.data_ptr(), bt_w, ctx,
                                out.data_ptr(), BATCH, hq, hkv, dh, ws.data_ptr(), wsb, st)
    copy_bytes = 1 << 30
    src = torch.empty(copy_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    hxf.op_copy(src.data_ptr(), dst.data_ptr(), copy_bytes, st)
    torch.cuda.synchronize()
    return {"probe": "decode attention kernel", "launches": reps, "sum_context_tokens": int(ctx.sum()),
            "kv_bytes_per_launch": int(ctx.sum()) * 2 * hkv * dh * 2, "copy_bytes": copy_bytes}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm-roofline", action="store_true",
                    help="skip the profiled workload-3 iterations that give gemm_roofline")
    ap.add_argument("--workload", type=int, default=2, choices=(1, 2, 3, 4, 5),
                    help="2 (default) prints the benchmark line; 1, 3-5 print per-workload measurements")
    ap.add_argument("--n-workflows", type=int, default=16, help="workload 5: workflows replayed")
    ap.add_argument("--policy", default="pq", choices=("pq", "fcfs", "llf"), help="workload 5: local queue policy")
    ap.add_argument("--attn-kernel-probe", action="store_true",
                    help="run only the decode-attention kernel and a calibration copy (for counter runs)")
    ap.add_argument("--cpu-baselines", action="store_true",
                    help="CPU baseline leg for workloads 1, 3, 4 and 5: the oracle timed on the host cores")
    ap.add_argument("--gemm-probe", action="store_true",
                    help="run only the four 2080-row prefill GEMMs (for MFMA counter runs)")
    ap.add_argument("--prefill-attn-probe", action="store_true",
                    help="run only the prefill attention on six chunk shapes (for kernel-trace runs)")
    ap.add_argument("--policy-ablation", action="store_true",
                    help="PQ / FCFS / LLF on config-5 workflows, virtual clock, scheduler only (CPU)")
    ap.add_argument("--measured-ablation", action="store_true",
                    help="PQ / FCFS / LLF on workload-5 workflows on the GPU with the measured clock "
                         "(--n-workflows, --rate, --slo-scale)")
    ap.add_argument("--tenants", help="--measured-ablation: two tenants' SLO multiples, e.g. 5,20 (even / odd "
                                      "workflows)")
    ap.add_argument("--slo-scale", type=int, default=10, help="--measured-ablation: SLO as a multiple of the "
                                                               "isolated latency")
    ap.add_argument("--cluster-sim", action="store_true",
                    help="coordinator across 4 heterogeneous scheduler-only instances: dispatch and alpha tuning (CPU)")
    ap.add_argument("--calibration-rows", help="--calibrate: also write the measured iterations (JSON) here")
    ap.add_argument("--model", choices=("llama8b", "qwen32b", "llama70b"),
                    help="model shape for workloads 2, 3 and 5 (default: 8B for 2 and 3, 32B for 5)")
    ap.add_argument("--rate", type=float, default=0.5, help="workload 5: workflow arrival rate (per second)")
    ap.add_argument("--calibrate", choices=("llama8b", "qwen32b", "llama70b"),
                    help="fit the virtual-clock iteration and request cost models to this GPU")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    if args.attn_kernel_probe:
        print(json.dumps(attn_kernel_probe()), flush=True)
        return

    if args.cpu_baselines:
        print(json.dumps(cpu_baselines()), flush=True)
        return

    if args.gemm_probe:
        print(json.dumps(gemm_probe()), flush=True)
        return

    if args.prefill_attn_probe:
        print(json.dumps(prefill_attn_probe()), flush=True)
        return

    if args.calibrate:
        print(json.dumps(calibrate(args.calibrate, args.calibration_rows)), flush=True)
        return

    if args.measured_ablation:
        tenants = tuple(int(x) for x in args.tenants.split(",")) if args.tenants else None
        print(json.dumps(measured_ablation(args.n_workflows, args.rate, slo_scale=args.slo_scale,
                                           model=args.model or "qwen32b", tenants=tenants)), flush=True)
        return

    if args.cluster_sim:
        print(json.dumps(cluster_sim()), flush=True)
        return

    if args.policy_ablation:
        print(json.dumps(policy_ablation(300 if args.n_workflows == 16 else args.n_workflows)), flush=True)
        return

    if args.workload != 2:
        fn = {1: workload1, 3: lambda: workload3(args.model or "llama8b"), 4: workload4,
              5: lambda: workload5(args.n_workflows, args.policy, args.model or "qwen32b", args.rate)}[args.workload]
        print(json.dumps(fn()), flush=True)
        return

    import numpy as np
    import torch

    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import DeviceModel, Engine

    hxf.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    shape = synth.model_shape(args.model or "llama8b")
    t0 = time.time()
    progress(f"generating and uploading {shape.name}-shaped bf16 weights")
    dm = DeviceModel(shape, lambda l: synth.gen_layer(shape, l), synth.gen_embed(shape), synth.gen_lm_head(shape),
                     synth.norm_weight(shape), device="cuda:0")
    progress(f"weights ready in {time.time() - t0:.1f} s")
    stages = synth.workloads.cfg2(vocab=shape.vocab, n=BATCH, max_new_tokens=MAX_NEW)
    ctxs = [len(s.prompt) for s in stages]
    max_context = 8192 + MAX_NEW
    n_blocks = sum(-(-(c + MAX_NEW - 1) // 16) for c in ctxs) + 256
    # cost model (ps): used only to order the queue; iteration cost irrelevant here
    cost = (2_000 * 10 ** 6, 100_000, 10, 6_000 * 10 ** 6)
    eng = Engine(dm, max_context=max_context, n_blocks=n_blocks, max_seqs=BATCH, chunk_tokens=2048, cost_ps=cost,
                 iter_ps=(10 ** 9, 0, 0, 0), clock=hxf.CLOCK_MEASURED)
    inst = eng.inst
    ids = [inst.submit(0, s.workflow, 0, 0, s.wf_slo_us, s.prompt, s.max_new_tokens) for s in stages]
    progress(f"prefilling {sum(ctxs)} prompt tokens of {BATCH} sequences (chunk 2048)")
    now, pf_tokens, pf_iters = 0, 0, 0
    torch.cuda.synchronize()
    tp0 = time.perf_counter()
    while True:
        st, info = inst.step(now)
        now += info["t_iter_us"]
        pf_tokens += info["n_prefill_tokens"]
        pf_iters += 1
        if info["n_prefill_tokens"] == 0:
            break
    torch.cuda.synchronize()
    t_pf = time.perf_counter() - tp0
    progress(f"prefill: {pf_tokens} tokens in {pf_iters} iterations, {t_pf:.2f} s")
    for _ in range(args.warmup):
        st, info = inst.step(now)
        now += info["t_iter_us"]
        assert info["n_decode"] == BATCH and info["n_prefill_tokens"] == 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st, info = inst.step(now)
        now += info["t_iter_us"]
        assert info["n_decode"] == BATCH and info["n_prefill_tokens"] == 0
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    progress(f"decode: {args.steps} steps in {dt:.3f} s")
    # The timed steps replay a captured graph of the forward, whose kernels HIP events
    # cannot time one by one; the roofline pass repeats the same decode step (eager
    # launches, kernel-stamped events on every decode-attention and merge launch).
    roof_steps = min(args.steps, 16)
    inst.profile_enable(True)
    for _ in range(roof_steps):
        st, info = inst.step(now)
        now += info["t_iter_us"]
        assert info["n_decode"] == BATCH and info["n_prefill_tokens"] == 0
    torch.cuda.synchronize()
    prof = inst.profile()
    inst.profile_enable(False)
    value = BATCH * args.steps / dt
    launches = max(prof["decode_attn_launches"], 1)
    avg_ms = prof["decode_attn_ms"] / launches
    merge_ms = prof["decode_merge_ms"] / launches
    bytes_per_launch = prof["decode_attn_bytes"] / launches
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    achieved_merged = bytes_per_launch / ((avg_ms + merge_ms) * 1e-3) / 1e9
    sum_ctx_now = sum(inst.request_state(r)["n_kv"] for r in ids)
    default_shape = shape.name == "llama8b"
    out = {
        "metric": METRIC if default_shape else METRIC.replace("8B shape", f"{MODEL_NAMES[shape.name]} shape"),
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": (f"decode iteration, {describe(shape)}, 64 sequences, contexts lognormal(median "
                                "3000, sigma 0.5) clipped to [1024, 8192], 16-token KV pages"),
                   "value_is": "decode tokens/s of the timed steps (64 sequences x steps / seconds)",
                   "batch": BATCH, "layers": shape.n_layers, "sum_context_tokens": int(sum_ctx_now)},
        "prefill_tokens_per_s": None,
        "prefill_tokens_per_s_source": None,
        "cfg2_prefill_untimed_tokens_per_s": round(pf_tokens / t_pf, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved_merged, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved_merged / HBM_PEAK_GBS, 4),
                     "traffic": DECODE_ATTN_TRAFFIC["bytes_per_launch"] if default_shape else None,
                     "traffic_sample": DECODE_ATTN_TRAFFIC if default_shape else None,
                     "kernel": "decode_attn_kernel<128> + decode_merge_kernel<128> (split-K attention and its "
                               "log-sum-exp merge, one layer per launch pair)",
                     "avg_launch_us": round((avg_ms + merge_ms) * 1e3, 2),
                     "timing": (f"kernel-stamped HIP events on the {int(launches)} decode-attention and merge launch "
                                f"pairs of {roof_steps} eager decode steps run right after the timed (graph-replayed) "
                                "steps"),
                     "bytes_per_launch": int(bytes_per_launch),
                     "attention_only": {"kernel": "decode_attn_kernel<128>", "avg_us": round(avg_ms * 1e3, 2),
                                        "achieved": round(achieved, 1),
                                        "frac": round(achieved / HBM_PEAK_GBS, 4)}},
    }
    # weight-streaming GEMMs of the same profiled steps: weight bytes per launch / duration
    wbytes = {"qkv": shape.qkv_dim * shape.d_model, "o": shape.d_model * shape.q_dim,
              "gate_up": 2 * shape.ffn_dim * shape.d_model, "down": shape.d_model * shape.ffn_dim,
              "lm_head": shape.vocab * shape.d_model}
    out["decode_gemms"] = {}
    for k, nbytes in wbytes.items():
        n = max(prof["gemm_launches"][k], 1)
        us = prof["gemm_ms"][k] / n * 1e3
        out["decode_gemms"][k] = {"avg_us": round(us, 2), "weight_tb_s": round(2 * nbytes / (us * 1e-6) / 1e12, 3)}
    out["hbm_copy_probe"] = hbm_copy_probe()
    out["hbm_read_probe"] = hbm_read_probe()
    del eng, inst
    if not args.no_gemm_roofline:
        progress("workload-3 mixed iterations, profiled: MFMA roofline of the 2080-row projections")
        out["gemm_roofline"] = mixed_iteration_profile(dm, shape)
        out["prefill_tokens_per_s"] = out["gemm_roofline"]["prefill_timed"]["tokens_per_s"]
        out["prefill_tokens_per_s_source"] = ("workload 3, timed mixed iterations (gemm_roofline.prefill_timed): "
                                              "prefill tokens / host-clock seconds")
    if not args.no_cpu_baseline:
        progress("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(shape, ctxs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
