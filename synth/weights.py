"""Seeded bf16 weights N(0, 0.02) for a Llama-style decoder.

Tensor numbering: 0 = token embedding [V, d]; layer l owns tensors
1 + 7*l + j for j over LAYER_TENSORS; the LM head [V, d] is 1 + 7*L.
Every matrix is stored [out_features, in_features] (row-major, the input
dimension contiguous).  Norm weights are all ones.

A tensor is filled in chunks of CHUNK elements; chunk c of tensor t draws
``standard_normal(float32)`` from ``default_rng(SeedSequence([seed, t, c]))``,
is multiplied by float32(0.02) and rounded to bf16 (nearest even).
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from .bf16 import f32_to_bf16_bits

WEIGHT_STD = 0.02
CHUNK = 1 << 22
LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")
BF16_ONE = 0x3F80


def _threads():
    n = os.environ.get("SYNTH_THREADS")
    if n:
        return max(1, int(n))
    return max(1, min(16, os.cpu_count() or 1))


def tensor_shape(shape, name):
    d, f, v = shape.d_model, shape.ffn_dim, shape.vocab
    return {
        "embed": (v, d),
        "lm_head": (v, d),
        "wq": (shape.q_dim, d),
        "wk": (shape.kv_dim, d),
        "wv": (shape.kv_dim, d),
        "wo": (d, shape.q_dim),
        "w_gate": (f, d),
        "w_up": (f, d),
        "w_down": (d, f),
    }[name]


def tensor_index(shape, name, layer=None):
    if name == "embed":
        return 0
    if name == "lm_head":
        return 1 + 7 * shape.n_layers
    return 1 + 7 * layer + LAYER_TENSORS.index(name)


def _fill_chunk(seed, t, c, out_flat):
    n = out_flat.size
    rng = np.random.default_rng(np.random.SeedSequence([seed, t, c]))
    x = rng.standard_normal(n, dtype=np.float32)
    x *= np.float32(WEIGHT_STD)
    out_flat[:] = f32_to_bf16_bits(x)


def gen_tensor(shape, name, layer=None, seed=None, pool=None):
    """bf16 bits (uint16 ndarray) of one weight tensor."""
    seed = shape.weight_seed if seed is None else seed
    t = tensor_index(shape, name, layer)
    shp = tensor_shape(shape, name)
    out = np.empty(int(np.prod(shp)), dtype=np.uint16)
    n_chunks = (out.size + CHUNK - 1) // CHUNK
    jobs = [(c, out[c * CHUNK:(c + 1) * CHUNK]) for c in range(n_chunks)]
    if pool is not None:
        list(pool.map(lambda j: _fill_chunk(seed, t, j[0], j[1]), jobs))
    elif n_chunks > 1:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(lambda j: _fill_chunk(seed, t, j[0], j[1]), jobs))
    else:
        for c, buf in jobs:
            _fill_chunk(seed, t, c, buf)
    return out.reshape(shp)


def gen_layer(shape, layer, seed=None):
    """dict name -> bf16 bits for every matrix of one decoder layer."""
    with ThreadPoolExecutor(_threads()) as ex:
        return {n: gen_tensor(shape, n, layer, seed, pool=ex) for n in LAYER_TENSORS}


def gen_embed(shape, seed=None):
    return gen_tensor(shape, "embed", seed=seed)


def gen_lm_head(shape, seed=None):
    return gen_tensor(shape, "lm_head", seed=seed)


def norm_weight(shape):
    """RMSNorm gain: all ones, as bf16 bits."""
    return np.full(shape.d_model, BF16_ONE, dtype=np.uint16)


NORM_STREAM = 7_000_001


def gen_norm_gains(shape, seed=None, spread=0.5):
    """Distinct RMSNorm gains for every norm, for tests that must tell the norms
    apart (the workloads themselves use all-ones gains).  Each element is
    1 + spread * U(-1, 1), rounded to bf16; one stream per seed.
    Returns a dict of bf16 bits: attn [L, d], ffn [L, d], final [d]."""
    seed = shape.weight_seed if seed is None else seed
    rng = np.random.default_rng(np.random.SeedSequence([seed, NORM_STREAM]))
    L, d = shape.n_layers, shape.d_model
    g = 1.0 + spread * rng.uniform(-1.0, 1.0, (2 * L + 1, d)).astype(np.float32)
    bits = f32_to_bf16_bits(g.astype(np.float32)).reshape(2 * L + 1, d)
    return {"attn": bits[:L].copy(), "ffn": bits[L:2 * L].copy(), "final": bits[2 * L].copy()}
