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
`roofline` is the paged decode-attention kernel (the largest single kernel of
the step): algorithmic K+V bytes per launch over its average duration, timed
with HIP events on the instance's stream.  `cpu_baseline` times the CPU
oracle on a bounded sample of the same step.
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


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import synth
    from paper_2505_05286_amd import hxf
    from paper_2505_05286_amd.device import DeviceModel, Engine

    hxf.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    shape = synth.model_shape("llama8b")
    t0 = time.time()
    progress("generating and uploading 8B-shaped bf16 weights")
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
    inst.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st, info = inst.step(now)
        now += info["t_iter_us"]
        assert info["n_decode"] == BATCH and info["n_prefill_tokens"] == 0
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    prof = inst.profile()
    progress(f"decode: {args.steps} steps in {dt:.3f} s")
    value = BATCH * args.steps / dt
    launches = max(prof["decode_attn_launches"], 1)
    avg_ms = prof["decode_attn_ms"] / launches
    bytes_per_launch = prof["decode_attn_bytes"] / launches
    achieved = bytes_per_launch / (avg_ms * 1e-3) / 1e9
    sum_ctx_now = sum(inst.request_state(r)["n_kv"] for r in ids)
    out = {
        "metric": METRIC,
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
        "config": {"workload": ("decode iteration, Llama-3-8B shape (32 layers, d 4096, 32q/8kv heads of 128, "
                                "SwiGLU 14336, vocab 128256), 64 sequences, contexts lognormal(median 3000, "
                                "sigma 0.5) clipped to [1024, 8192], 16-token KV pages"),
                   "batch": BATCH, "layers": shape.n_layers, "sum_context_tokens": int(sum_ctx_now)},
        "prefill_tokens_per_s": round(pf_tokens / t_pf, 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "decode_attn_kernel<128>", "avg_launch_us": round(avg_ms * 1e3, 2),
                     "bytes_per_launch": int(bytes_per_launch)},
    }
    del eng, inst
    if not args.no_cpu_baseline:
        progress("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(shape, ctxs)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
