"""Seeded request streams for the five synthetic workloads.

Only lengths, token ids, arrival times and end-to-end SLOs are drawn here.
Scheduling and model arithmetic live elsewhere.  Every stream is a list of
``Stage`` records; ``parent`` names the stage (in the same workflow) whose
retained KV a forked request continues from.

Token ids are uniform in [0, vocab).  Times are integer microseconds.

End-to-end SLOs are ``slo_scale`` times a reference isolated latency
``REF_US(L_in, L_out)`` summed over the workflow's critical path.  The
reference figures below are fixed data: a lone request's latency on one MI355X
(chunked prefill, batch-1 decode at ~4k context), as measured for each 8B/32B/70B
shape by ``bench.py --calibrate``; the tiny shape's are nominal.
"""
from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

# Reference isolated latency per shape: base + per-prompt-token + per-output-token (us).
REF_LATENCY = {
    "tiny": (200, 0.05, 150),
    "llama8b": (4384, 17.7, 4470),
    "qwen32b": (13844, 73.0, 14036),
    "llama70b": (25850, 157.0, 26181),
}


def ref_isolated_us(model, l_in, l_out):
    b, p, d = REF_LATENCY[model]
    return int(b + p * l_in + d * l_out)


@dataclass
class Stage:
    workflow: int
    stage_index: int
    prompt: np.ndarray               # int32 token ids (appended tokens for a fork)
    max_new_tokens: int
    parent: Optional[Tuple[int, int]] = None   # (stage_index, branch) of the parent
    branch: int = 0
    retain_kv: bool = False
    rest: List[Tuple[int, int]] = field(default_factory=list)  # (L_in, L_out) of later stages
    wf_arrival_us: int = 0
    wf_slo_us: int = 0


def _ids(rng, vocab, n):
    return rng.integers(0, vocab, size=int(n), dtype=np.int64).astype(np.int32)


def cfg1(vocab=2048, slo_scale=10):
    """Tiny decoder: 4 one-stage workflows, prompts 64/128/192/256, 8 tokens each, all at t=0."""
    rng = np.random.default_rng(0)
    out = []
    for w, n in enumerate((64, 128, 192, 256)):
        p = _ids(rng, vocab, n)
        slo = slo_scale * ref_isolated_us("tiny", n, 8)
        out.append(Stage(w, 0, p, 8, wf_arrival_us=0, wf_slo_us=slo))
    return out


def cfg2_contexts(n=64, seed=1):
    """Decode contexts ~ lognormal(median 3000, sigma 0.5), rounded, clipped to [1024, 8192]."""
    rng = np.random.default_rng(seed)
    c = np.rint(rng.lognormal(np.log(3000.0), 0.5, size=n)).astype(np.int64)
    return np.clip(c, 1024, 8192).astype(np.int32), rng


def cfg2(vocab=128256, n=64, max_new_tokens=80):
    ctx, rng = cfg2_contexts(n)
    return [Stage(i, 0, _ids(rng, vocab, c), max_new_tokens, wf_slo_us=10**12) for i, c in enumerate(ctx)]


def cfg3(vocab=128256):
    """16 prompts U[2048, 8192] for chunked prefill + 32 running decodes with context U[1024, 4096]."""
    rng = np.random.default_rng(2)
    pl = rng.integers(2048, 8193, size=16)
    dl = rng.integers(1024, 4097, size=32)
    decodes = [Stage(100 + i, 0, _ids(rng, vocab, c), 4096, wf_slo_us=10**12) for i, c in enumerate(dl)]
    prompts = [Stage(i, 0, _ids(rng, vocab, c), 1,
                     wf_slo_us=10 * ref_isolated_us("llama8b", int(c), 1)) for i, c in enumerate(pl)]
    return decodes, prompts


def cfg4(vocab=128256, n_wf=32, prompt_len=4096, branches=8, new_tokens=256, corr_len=512):
    """Shared 4096-token prompts, 8 forks each decoding 256 tokens, 512-token correction on even branches."""
    rng = np.random.default_rng(3)
    parents, forks, corrections = [], [], []
    for w in range(n_wf):
        parents.append(Stage(w, 0, _ids(rng, vocab, prompt_len), 0, retain_kv=True, wf_slo_us=10**12))
    for w in range(n_wf):
        for b in range(branches):
            forks.append(Stage(w, 1, np.zeros(0, np.int32), new_tokens, parent=(0, 0), branch=b,
                               retain_kv=(b % 2 == 0), wf_slo_us=10**12))
    for w in range(n_wf):
        for b in range(0, branches, 2):
            corrections.append(Stage(w, 2, _ids(rng, vocab, corr_len), 1, parent=(1, b), branch=b,
                                     wf_slo_us=10**12))
    return parents, forks, corrections


@dataclass
class Workflow:
    workflow: int
    arrival_us: int
    slo_us: int
    schema_len: int
    schema: np.ndarray
    corrections: List[np.ndarray]
    eval_prompt: np.ndarray


CFG5_SHAPE = dict(s1_out=64, n_cand=8, cand_out=256, n_corr=4, corr_in=512, corr_out=256,
                  eval_in=1024, eval_out=128)


def cfg5(vocab=152064, n_wf=300, mean_interarrival_s=2.0, slo_scale=10, model="qwen32b"):
    """300 four-stage workflows with Poisson arrivals (0.5 workflows/s)."""
    rng = np.random.default_rng(4)
    s = CFG5_SHAPE
    gaps = rng.exponential(mean_interarrival_s * 1e6, size=n_wf)
    arrivals = np.floor(np.cumsum(gaps)).astype(np.int64)
    out = []
    for w in range(n_wf):
        l1 = int(rng.integers(2048, 8193))
        schema = _ids(rng, vocab, l1)
        corr = [_ids(rng, vocab, s["corr_in"]) for _ in range(s["n_corr"])]
        ev = _ids(rng, vocab, s["eval_in"])
        # forks re-prefill only the parent's partial last page (at most 16 tokens) plus
        # their appended tokens
        iso = (ref_isolated_us(model, l1, s["s1_out"])
               + ref_isolated_us(model, 16, s["cand_out"])
               + ref_isolated_us(model, 16 + s["corr_in"], s["corr_out"])
               + ref_isolated_us(model, s["eval_in"], s["eval_out"]))
        out.append(Workflow(w, int(arrivals[w]), slo_scale * iso, l1, schema, corr, ev))
    return out
