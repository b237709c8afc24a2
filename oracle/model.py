"""Oracle decoder forward (float64) -- TEST INFRASTRUCTURE ONLY.

The paper serves its models through a continuous-batching engine and treats
the model itself as a black box (Section 5.1, "Runtime"); it defines no model
arithmetic.  What is computed here is the standard Llama-style decoder that
the synthetic workloads name:

    x   = E[ids]
    per layer:
        h       = rmsnorm(x) * g_attn              rmsnorm(v) = v / sqrt(mean(v^2) + eps)
        q, k, v = h Wq^T, h Wk^T, h Wv^T           (W stored [out, in])
        q, k    = rope(q, pos), rope(k, pos)       rotate-half, theta_i = base^(-2i/dh)
        o_hq    = softmax(q_hq K_g^T / sqrt(dh) + causal mask) V_g,   g = hq // (Hq/Hkv)
        x       = x + concat(o) Wo^T
        h       = rmsnorm(x) * g_ffn
        x       = x + (silu(h Wgate^T) * (h Wup^T)) Wdown^T,  silu(z) = z / (1 + e^-z)
    logits = (rmsnorm(x) * g_final) Wlm^T ;  token = argmax (lowest index on ties)

Weights are the bf16 values from ``synth`` upcast exactly to float64, so the
comparison with the bf16 GPU path measures arithmetic error only.

Parity pins (tests/test_oracle_model.py): brute-force triple-loop attention,
softmax row sums, causal-mask perturbation, RoPE relative-position identity,
RMSNorm closed form, GQA -> MHA reduction, chunk invariance, decode == prefill.
"""
import numpy as np

import synth

F = np.float64


# ---------------------------------------------------------------- primitives
def rmsnorm(x, g, eps):
    x = np.asarray(x, F)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, F)


def rope_angles(positions, head_dim, base):
    """angle[p, i] = pos_p * base^(-2i/dh) for i < dh/2, in float64."""
    i = np.arange(head_dim // 2, dtype=F)
    theta = np.power(F(base), -2.0 * i / head_dim)
    return np.asarray(positions, F)[:, None] * theta[None, :]


def apply_rope(x, positions, base):
    """Rotate-half RoPE on x [n, H, dh] at positions [n]."""
    x = np.asarray(x, F)
    dh = x.shape[-1]
    ang = rope_angles(positions, dh, base)          # [n, dh/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., : dh // 2], x[..., dh // 2:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s, axis=-1):
    s = np.asarray(s, F)
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q, k, v, q_pos, k_pos):
    """Causal GQA attention.

    q [n, Hq, dh]; k, v [c, Hkv, dh]; q_pos [n]; k_pos [c].
    Query i attends to key t iff k_pos[t] <= q_pos[i].  Returns [n, Hq, dh].
    """
    q, k, v = np.asarray(q, F), np.asarray(k, F), np.asarray(v, F)
    n, hq, dh = q.shape
    hkv = k.shape[1]
    grp = hq // hkv
    mask = np.asarray(k_pos)[None, :] > np.asarray(q_pos)[:, None]     # [n, c]
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(F(dh))
    for h in range(hq):
        g = h // grp
        s = (q[:, h, :] @ k[:, g, :].T) * scale
        s = np.where(mask, -np.inf, s)
        out[:, h, :] = softmax(s) @ v[:, g, :]
    return out


def silu(z):
    z = np.asarray(z, F)
    return z / (1.0 + np.exp(-z))


def argmax_lowest(x):
    """Row argmax; the lowest index wins ties (numpy's argmax already does)."""
    return np.argmax(np.asarray(x), axis=-1)


# ---------------------------------------------------------------- weights
class Weights:
    """float64 view of the synthetic bf16 weights of one model shape.

    Layers are converted on first use and kept (``keep_layers``) or dropped
    after use, so a shape whose float64 weights exceed host memory can still
    be run layer by layer.
    """

    def __init__(self, shape, seed=None, keep_layers=True, norm_gains=None, layer_bits=None, embed_bits=None,
                 lm_head_bits=None):
        """norm_gains: None (every RMSNorm gain is 1, as in the workloads) or a dict of
        bf16 bits with one gain per norm: attn [L, d], ffn [L, d], final [d].
        layer_bits(l), embed_bits, lm_head_bits: the synthetic bf16 bits, when the
        caller already holds them (default: drawn from ``synth`` with the seed)."""
        self.shape = shape
        self.seed = shape.weight_seed if seed is None else seed
        self.keep = keep_layers
        self._layer_bits = layer_bits
        self._layers = {}
        self._embed_bits = embed_bits
        self._lm = None if lm_head_bits is None else synth.bf16_bits_to_f32(lm_head_bits)
        L = shape.n_layers
        if norm_gains is None:
            ones = synth.bf16_bits_to_f32(synth.norm_weight(shape)).astype(F)
            self.attn_norm = [ones] * L
            self.ffn_norm = [ones] * L
            self.final_norm = ones
        else:
            self.attn_norm = [synth.bf16_bits_to_f32(norm_gains["attn"][l]).astype(F) for l in range(L)]
            self.ffn_norm = [synth.bf16_bits_to_f32(norm_gains["ffn"][l]).astype(F) for l in range(L)]
            self.final_norm = synth.bf16_bits_to_f32(norm_gains["final"]).astype(F)

    def layer(self, l):
        if l in self._layers:
            return self._layers[l]
        raw = synth.gen_layer(self.shape, l, self.seed) if self._layer_bits is None else self._layer_bits(l)
        w = {k: synth.bf16_bits_to_f32(v).astype(F) for k, v in raw.items()}
        if self.keep:
            self._layers[l] = w
        return w

    def embed_rows(self, ids):
        if self._embed_bits is None:
            self._embed_bits = synth.gen_embed(self.shape, self.seed)
        return synth.bf16_bits_to_f32(self._embed_bits[np.asarray(ids)]).astype(F)

    def lm_head_f32(self):
        if self._lm is None:
            self._lm = synth.bf16_bits_to_f32(synth.gen_lm_head(self.shape, self.seed))
        return self._lm

    def logits(self, h):
        """h [r, d] float64 -> logits [r, V] float64 (vocabulary processed in slices)."""
        lm = self.lm_head_f32()
        out = np.empty((h.shape[0], lm.shape[0]), F)
        step = 16384
        for v0 in range(0, lm.shape[0], step):
            out[:, v0:v0 + step] = h @ lm[v0:v0 + step].astype(F).T
        return out


# ---------------------------------------------------------------- forward
class Sequence:
    """Dense per-layer KV history of one sequence (the oracle's KV cache)."""

    def __init__(self, n_layers):
        self.k = [None] * n_layers
        self.v = [None] * n_layers
        self.n = 0          # tokens whose KV is stored

    def fork(self, n_keep):
        """A new sequence holding a copy of this one's KV for positions [0, n_keep):
        the context a forked request continues from (KV of earlier positions
        depends only on earlier tokens)."""
        assert 0 <= n_keep <= self.n
        s = Sequence(len(self.k))
        for l in range(len(self.k)):
            if self.k[l] is not None and n_keep > 0:
                s.k[l] = self.k[l][:n_keep].copy()
                s.v[l] = self.v[l][:n_keep].copy()
        s.n = n_keep
        return s

    def append(self, layer, k, v):
        if self.k[layer] is None:
            self.k[layer], self.v[layer] = k, v
        else:
            self.k[layer] = np.concatenate([self.k[layer], k])
            self.v[layer] = np.concatenate([self.v[layer], v])


def forward(weights, seqs, chunks, logit_rows=None, progress=None):
    """Run one forward pass over several independent sequences.

    seqs: list of Sequence; chunks: list of int arrays of new token ids (one per
    sequence), placed at positions seq.n .. seq.n + len - 1.  Appends their KV.
    logit_rows: per sequence, the local row indices whose logits are wanted
    (default: the last row).  progress(layer), if given, is called after each
    layer (long runs report liveness).  Returns a list of float64 logit arrays.
    """
    sh = weights.shape
    dh, hq, hkv = sh.head_dim, sh.n_q_heads, sh.n_kv_heads
    lens = [len(c) for c in chunks]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(int)
    pos = [np.arange(s.n, s.n + len(c)) for s, c in zip(seqs, chunks)]
    x = weights.embed_rows(np.concatenate([np.asarray(c) for c in chunks]))
    for l in range(sh.n_layers):
        w = weights.layer(l)
        h = rmsnorm(x, weights.attn_norm[l], sh.rms_eps)
        q = (h @ w["wq"].T).reshape(-1, hq, dh)
        k = (h @ w["wk"].T).reshape(-1, hkv, dh)
        v = (h @ w["wv"].T).reshape(-1, hkv, dh)
        att = np.empty_like(q)
        for i, s in enumerate(seqs):
            a, b = offs[i], offs[i + 1]
            qi = apply_rope(q[a:b], pos[i], sh.rope_base)
            ki = apply_rope(k[a:b], pos[i], sh.rope_base)
            s.append(l, ki, v[a:b])
            kpos = np.arange(s.k[l].shape[0])
            att[a:b] = attention(qi, s.k[l], s.v[l], pos[i], kpos)
        x = x + att.reshape(-1, hq * dh) @ w["wo"].T
        h = rmsnorm(x, weights.ffn_norm[l], sh.rms_eps)
        x = x + (silu(h @ w["w_gate"].T) * (h @ w["w_up"].T)) @ w["w_down"].T
        if progress is not None:
            progress(l)
    for s, c in zip(seqs, chunks):
        s.n += len(c)
    rows = []
    for i in range(len(seqs)):
        sel = [lens[i] - 1] if logit_rows is None else logit_rows[i]
        rows.append(offs[i] + np.asarray(sel, dtype=int))
    flat = np.concatenate(rows) if rows else np.zeros(0, int)
    hf = rmsnorm(x[flat], weights.final_norm, sh.rms_eps)
    lg = weights.logits(hf) if len(flat) else np.zeros((0, sh.vocab))
    out, o = [], 0
    for r in rows:
        out.append(lg[o:o + len(r)])
        o += len(r)
    return out


def generate(weights, prompts, max_new, forced=None, keep_logits=True):
    """Greedy decoding of several prompts together (independent sequences).

    Generates ``max_new[i]`` tokens for prompt i; the first comes from the
    prompt's last position.  The last generated token is not fed back.
    ``forced[i]`` (optional) replaces the fed-back token at each step
    (teacher forcing); the argmax is still reported.
    Returns (tokens, logits): tokens[i] int array, logits[i] [max_new, V].
    """
    n = len(prompts)
    seqs = [Sequence(weights.shape.n_layers) for _ in range(n)]
    toks = [[] for _ in range(n)]
    lgs = [[] for _ in range(n)]
    active = [i for i in range(n) if max_new[i] > 0]
    if not active:
        return [np.zeros(0, np.int64) for _ in range(n)], [np.zeros((0, weights.shape.vocab)) for _ in range(n)]
    res = forward(weights, [seqs[i] for i in active], [np.asarray(prompts[i]) for i in active])
    for i, lg in zip(active, res):
        toks[i].append(int(argmax_lowest(lg[0])))
        if keep_logits:
            lgs[i].append(lg[0])
    while True:
        active = [i for i in range(n) if len(toks[i]) < max_new[i]]
        if not active:
            break
        feed = []
        for i in active:
            k = len(toks[i]) - 1
            feed.append(np.array([forced[i][k] if forced is not None else toks[i][k]]))
        res = forward(weights, [seqs[i] for i in active], feed)
        for i, lg in zip(active, res):
            toks[i].append(int(argmax_lowest(lg[0])))
            if keep_logits:
                lgs[i].append(lg[0])
    return ([np.asarray(t, np.int64) for t in toks],
            [np.stack(l) if l else np.zeros((0, weights.shape.vocab)) for l in lgs])
