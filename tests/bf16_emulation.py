"""The decoder forward with bf16 rounding where the GPU path rounds -- TEST
INFRASTRUCTURE, used to bound what bf16 arithmetic itself costs at depth.

The same definition as oracle.model.forward (float64 throughout), except that a
value is rounded to bf16 (nearest even) wherever the HIP path stores one:
the RMSNorm outputs that feed the QKV, gate/up and LM-head GEMMs, the q/k/v
projections, q and k after RoPE, the attention probabilities before the PV
product (the normaliser keeps the unrounded sum) and the attention output, and
the SwiGLU activation that feeds the down projection.  The residual stream and
every accumulation stay float64 (the GPU keeps them in fp32).  It shares no code
with the HIP path; with rounding switched off it is the oracle's forward
(tests/test_bf16_drift.py).

A bf16 forward drifts from the exact one by a per-layer amount that adds up over
depth, so the full-depth GPU tests bound the GPU's logits error by the drift this
forward shows on the same inputs.
"""
import numpy as np

import synth
from oracle import model as M

F = np.float64


def bf16(x):
    """Round to the nearest bf16 (ties to even), returned as float64."""
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.asarray(x, np.float32))).astype(F)


def _attention(q, k, v, q_pos, k_pos, rnd):
    n, hq, dh = q.shape
    grp = hq // k.shape[1]
    mask = np.asarray(k_pos)[None, :] > np.asarray(q_pos)[:, None]
    out = np.empty_like(q)
    for h in range(hq):
        g = h // grp
        s = (q[:, h, :] @ k[:, g, :].T) / np.sqrt(F(dh))
        s = np.where(mask, -np.inf, s)
        p = np.exp(s - np.max(s, axis=-1, keepdims=True))
        out[:, h, :] = (rnd(p) @ v[:, g, :]) / np.sum(p, axis=-1, keepdims=True)
    return rnd(out)


def forward(weights, seqs, chunks, logit_rows=None, progress=None, rounding=True):
    """oracle.model.forward with the GPU path's bf16 roundings (none if rounding=False)."""
    rnd = bf16 if rounding else (lambda x: x)
    sh = weights.shape
    dh, hq, hkv = sh.head_dim, sh.n_q_heads, sh.n_kv_heads
    lens = [len(c) for c in chunks]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    pos = [np.arange(s.n, s.n + len(c)) for s, c in zip(seqs, chunks)]
    x = weights.embed_rows(np.concatenate([np.asarray(c) for c in chunks]))
    for l in range(sh.n_layers):
        w = weights.layer(l)
        h = rnd(M.rmsnorm(x, weights.attn_norm[l], sh.rms_eps))
        q = rnd(h @ w["wq"].T).reshape(-1, hq, dh)
        k = rnd(h @ w["wk"].T).reshape(-1, hkv, dh)
        v = rnd(h @ w["wv"].T).reshape(-1, hkv, dh)
        att = np.empty_like(q)
        for i, s in enumerate(seqs):
            a, b = offs[i], offs[i + 1]
            qi = rnd(M.apply_rope(q[a:b], pos[i], sh.rope_base))
            ki = rnd(M.apply_rope(k[a:b], pos[i], sh.rope_base))
            s.append(l, ki, v[a:b])
            att[a:b] = _attention(qi, s.k[l], s.v[l], pos[i], np.arange(s.k[l].shape[0]), rnd)
        x = x + att.reshape(-1, hq * dh) @ w["wo"].T
        h = rnd(M.rmsnorm(x, weights.ffn_norm[l], sh.rms_eps))
        x = x + rnd(M.silu(h @ w["w_gate"].T) * (h @ w["w_up"].T)) @ w["w_down"].T
        if progress is not None:
            progress(l)
    for s, c in zip(seqs, chunks):
        s.n += len(c)
    rows = []
    for i in range(len(seqs)):
        sel = [lens[i] - 1] if logit_rows is None else logit_rows[i]
        rows.append(offs[i] + np.asarray(sel, dtype=int))
    flat = np.concatenate(rows) if rows else np.zeros(0, int)
    hf = rnd(M.rmsnorm(x[flat], weights.final_norm, sh.rms_eps))
    lg = weights.logits(hf) if len(flat) else np.zeros((0, sh.vocab))
    out, o = [], 0
    for r in rows:
        out.append(lg[o:o + len(r)])
        o += len(r)
    return out
