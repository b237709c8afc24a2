"""Pins of the oracle decoder against what the mathematics fixes.

Each test would fail on a plausible slip in oracle/model.py or oracle/paged.py:
a dropped 1/sqrt(dh), a transposed weight, a wrong RoPE pairing or sign, a
causal mask off by one, a wrong GQA head mapping, a wrong slot formula.
"""
import math

import numpy as np
import pytest

import synth
from oracle import model as M
from oracle import paged as P


def brute_attention(q, k, v, q_pos, k_pos):
    """Textbook causal attention with explicit loops (float64)."""
    n, hq, dh = q.shape
    c, hkv, _ = k.shape
    grp = hq // hkv
    out = np.zeros((n, hq, dh))
    for i in range(n):
        for h in range(hq):
            g = h // grp
            s = []
            for t in range(c):
                if k_pos[t] <= q_pos[i]:
                    s.append(sum(float(q[i, h, d]) * float(k[t, g, d]) for d in range(dh)) / math.sqrt(dh))
                else:
                    s.append(None)
            mx = max(x for x in s if x is not None)
            w = [0.0 if x is None else math.exp(x - mx) for x in s]
            z = sum(w)
            for t in range(c):
                if w[t]:
                    out[i, h] += (w[t] / z) * v[t, g]
    return out


@pytest.mark.parametrize("n,c,hq,hkv,dh", [(3, 5, 4, 2, 8), (1, 7, 2, 2, 16), (4, 4, 6, 3, 8)])
def test_attention_matches_brute_force(n, c, hq, hkv, dh):
    rng = np.random.default_rng(11)
    q = rng.standard_normal((n, hq, dh))
    k = rng.standard_normal((c, hkv, dh))
    v = rng.standard_normal((c, hkv, dh))
    k_pos = np.arange(c)
    q_pos = np.arange(c - n, c)
    ref = brute_attention(q, k, v, q_pos, k_pos)
    np.testing.assert_allclose(M.attention(q, k, v, q_pos, k_pos), ref, rtol=1e-10, atol=1e-12)


def test_softmax_rows_sum_to_one_and_shift_invariant():
    rng = np.random.default_rng(1)
    s = rng.standard_normal((7, 33)) * 20
    p = M.softmax(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-12)
    np.testing.assert_allclose(M.softmax(s + 1000.0), M.softmax(s), rtol=1e-9, atol=1e-300)  # max subtraction


def test_single_key_attention_returns_value():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 4, 8))
    k = rng.standard_normal((1, 2, 8))
    v = rng.standard_normal((1, 2, 8))
    o = M.attention(q, k, v, np.array([0]), np.array([0]))
    np.testing.assert_allclose(o[0, 0], v[0, 0])
    np.testing.assert_allclose(o[0, 3], v[0, 1])   # head 3 of 4 reads kv-head 1 of 2


def test_gqa_reduces_to_mha_with_replicated_kv():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((5, 4, 8))
    k = rng.standard_normal((6, 2, 8))
    v = rng.standard_normal((6, 2, 8))
    rep_k = np.repeat(k, 2, axis=1)
    rep_v = np.repeat(v, 2, axis=1)
    qp, kp = np.arange(1, 6), np.arange(6)
    np.testing.assert_allclose(M.attention(q, k, v, qp, kp), M.attention(q, rep_k, rep_v, qp, kp), atol=1e-13)


def test_rope_rotate_half_pairing_and_identity():
    dh, base = 16, 10000.0
    x = np.zeros((1, 1, dh))
    x[0, 0, 0] = 1.0
    for p in (0, 1, 7, 1000):
        y = M.apply_rope(x, np.array([p]), base)[0, 0]
        assert y[0] == pytest.approx(math.cos(p)) and y[dh // 2] == pytest.approx(math.sin(p))
        assert np.count_nonzero(np.abs(y) > 1e-15) <= 2
    # frequency of pair i is base^(-2i/dh)
    x = np.zeros((1, 1, dh))
    x[0, 0, 3] = 1.0
    y = M.apply_rope(x, np.array([5]), base)[0, 0]
    assert y[3] == pytest.approx(math.cos(5 * base ** (-6 / dh)))
    rng = np.random.default_rng(4)
    z = rng.standard_normal((3, 2, dh))
    np.testing.assert_array_equal(M.apply_rope(z, np.zeros(3, int), base), z)


def test_rope_relative_position():
    rng = np.random.default_rng(5)
    dh = 32
    q = rng.standard_normal((1, 1, dh))
    k = rng.standard_normal((1, 1, dh))

    def dot(m, n):
        return float(np.sum(M.apply_rope(q, np.array([m]), 1e4) * M.apply_rope(k, np.array([n]), 1e4)))

    for m, n in ((3, 1), (10, 8), (102, 100), (5000, 4998)):
        assert dot(m, n) == pytest.approx(dot(2, 0), rel=1e-9, abs=1e-9)
    assert abs(dot(3, 1) - dot(3, 2)) > 1e-6


def test_rmsnorm_closed_form():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((4, 64)) * 3
    eps = 1e-5
    y = M.rmsnorm(x, np.ones(64), eps)
    ms = np.mean(x * x, -1)
    np.testing.assert_allclose(np.mean(y * y, -1), ms / (ms + eps), rtol=1e-12)
    g = rng.standard_normal(64)
    np.testing.assert_allclose(M.rmsnorm(x, g, eps), y * g, rtol=1e-12)


def test_silu_identities():
    z = np.linspace(-30, 30, 61)
    assert M.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(M.silu(z) - M.silu(-z), z, atol=1e-12)
    assert M.silu(np.array([40.0]))[0] == pytest.approx(40.0)


def _odd_shape():
    # every weight non-square, so a transposed operand cannot run
    return synth.ModelShape("odd", 2, 96, 4, 2, 16, 80, 300, weight_seed=9)


@pytest.fixture(scope="module")
def tiny():
    return M.Weights(synth.model_shape("tiny"))


def test_forward_shapes_on_non_square_weights():
    w = M.Weights(_odd_shape())
    seq = M.Sequence(2)
    lg = M.forward(w, [seq], [np.array([1, 2, 3])], logit_rows=[[0, 1, 2]])[0]
    assert lg.shape == (3, 300) and np.all(np.isfinite(lg))


def test_uniform_attention_closed_form():
    """Wq = Wk = 0 gives uniform causal attention; with permutation Wv, Wo, a
    zero FFN and an identity LM head, the logits of position i are
    rmsnorm(x_i + mean_{t<=i} o(t)) with o(t)[j] = rmsnorm(x_t)[perm_v[perm_o[j]]]."""
    sh = synth.ModelShape("perm", 1, 32, 2, 2, 16, 24, 32, weight_seed=0)
    w = M.Weights(sh)
    rng = np.random.default_rng(7)
    perm_v = rng.permutation(32)
    perm_o = rng.permutation(32)
    lay = {k: np.zeros_like(v) for k, v in w.layer(0).items()}
    lay["wv"][np.arange(32), perm_v] = 1.0      # v[i] = h[perm_v[i]]
    lay["wo"][np.arange(32), perm_o] = 1.0      # o[i] = a[perm_o[i]]
    w._layers[0] = lay
    w._lm = np.eye(32, dtype=np.float32)
    ids = np.array([3, 9, 27, 4, 30])
    x = w.embed_rows(ids)
    h = M.rmsnorm(x, np.ones(32), sh.rms_eps)
    lg = M.forward(w, [M.Sequence(1)], [ids], logit_rows=[list(range(5))])[0]
    for i in range(5):
        a = h[: i + 1].mean(0)[perm_v]
        expect = M.rmsnorm(x[i] + a[perm_o], np.ones(32), sh.rms_eps)
        np.testing.assert_allclose(lg[i], expect, rtol=1e-12, atol=1e-14)


def test_ffn_closed_form_with_distinct_norm_gains():
    """Pins the FFN half of a layer and which gain each RMSNorm uses.  Wq = Wk = 0
    (uniform causal attention), Wv and Wo permutations, W_gate and W_up scaled
    row selections (a * e_sel_g[f], b * e_sel_u[f]), W_down a row selection
    (e_sel_d[j]), an identity LM head and a different random gain for the
    attention, FFN and final norms.  Position i then has the closed form
        y = x_i + (mean_{t<=i} n(x_t, g_a)[perm_v])[perm_o]
        u = n(y, g_f)
        z = y + (silu(a u[sel_g]) * (b u[sel_u]))[sel_d]
        logits_i = n(z, g_out),   n(v, g) = v / sqrt(mean(v^2) + eps) * g,
    which a slip such as SiLU on the up projection, the FFN norm fed the layer
    input, a swapped gain or the second residual added to u instead of y breaks."""
    d, F = 32, 48
    sh = synth.ModelShape("ffn", 1, d, 2, 2, 16, F, d, weight_seed=0)
    gains = synth.gen_norm_gains(sh, seed=3)
    w = M.Weights(sh, norm_gains=gains)
    rng = np.random.default_rng(17)
    perm_v, perm_o = rng.permutation(d), rng.permutation(d)
    sel_g, sel_u = rng.integers(0, d, F), rng.integers(0, d, F)
    sel_d = rng.permutation(F)[:d]
    a, b = 1.5, -0.75
    lay = {k: np.zeros_like(v) for k, v in w.layer(0).items()}
    lay["wv"][np.arange(d), perm_v] = 1.0
    lay["wo"][np.arange(d), perm_o] = 1.0
    lay["w_gate"][np.arange(F), sel_g] = a
    lay["w_up"][np.arange(F), sel_u] = b
    lay["w_down"][np.arange(d), sel_d] = 1.0
    w._layers[0] = lay
    w._lm = np.eye(d, dtype=np.float32)
    g_a, g_f, g_o = (synth.bf16_bits_to_f32(x).astype(np.float64)
                     for x in (gains["attn"][0], gains["ffn"][0], gains["final"]))
    assert not np.allclose(g_a, g_f) and not np.allclose(g_f, g_o)
    ids = np.array([5, 11, 30, 2, 19, 7])
    x = w.embed_rows(ids)
    eps = sh.rms_eps

    def n(v, g):
        return v / math.sqrt(float(np.mean(v * v)) + eps) * g

    lg = M.forward(w, [M.Sequence(1)], [ids], logit_rows=[list(range(len(ids)))])[0]
    for i in range(len(ids)):
        att = np.mean([n(x[t], g_a) for t in range(i + 1)], axis=0)[perm_v][perm_o]
        y = x[i] + att
        u = n(y, g_f)
        gate, up = a * u[sel_g], b * u[sel_u]
        f = gate / (1.0 + np.exp(-gate)) * up
        z = y + f[sel_d]
        np.testing.assert_allclose(lg[i], n(z, g_o), rtol=1e-12, atol=1e-14)


def test_fork_copies_the_parents_kv_prefix(tiny):
    """A forked sequence continued from the parent's first n tokens of KV gives the
    logits of processing its whole context at once."""
    rng = np.random.default_rng(23)
    ctx = rng.integers(0, 2048, 57)
    app = rng.integers(0, 2048, 6)
    par = M.Sequence(2)
    M.forward(tiny, [par], [ctx])
    kid = par.fork(48)
    got = M.forward(tiny, [kid], [np.concatenate([ctx[48:], app])])[0]
    ref = M.forward(tiny, [M.Sequence(2)], [np.concatenate([ctx, app])])[0]
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)
    assert par.n == 57 and kid.n == 63


def test_causal_mask_future_tokens_do_not_matter(tiny):
    rng = np.random.default_rng(8)
    ids = rng.integers(0, 2048, 40)
    ids2 = ids.copy()
    ids2[25:] = rng.integers(0, 2048, 15)
    a = M.forward(tiny, [M.Sequence(2)], [ids], logit_rows=[list(range(25))])[0]
    b = M.forward(tiny, [M.Sequence(2)], [ids2], logit_rows=[list(range(25))])[0]
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)
    c = M.forward(tiny, [M.Sequence(2)], [ids2], logit_rows=[[25]])[0]
    assert np.max(np.abs(c - a[-1:])) > 1e-6


@pytest.mark.parametrize("chunk", [16, 64, 100])
def test_chunk_invariance(tiny, chunk):
    rng = np.random.default_rng(9)
    ids = rng.integers(0, 2048, 200)
    full = M.forward(tiny, [M.Sequence(2)], [ids], logit_rows=[[199]])[0]
    seq = M.Sequence(2)
    for a in range(0, 200, chunk):
        out = M.forward(tiny, [seq], [ids[a:a + chunk]])[0]
    np.testing.assert_allclose(out, full, rtol=1e-10, atol=1e-10)


def test_decode_equals_prefill_and_batching_is_independent(tiny):
    rng = np.random.default_rng(10)
    p1, p2 = rng.integers(0, 2048, 30), rng.integers(0, 2048, 17)
    toks, lgs = M.generate(tiny, [p1, p2], [4, 3])
    t1, l1 = M.generate(tiny, [p1], [4])
    np.testing.assert_array_equal(toks[0], t1[0])
    np.testing.assert_allclose(lgs[0], l1[0], rtol=1e-10, atol=1e-10)
    # step k logits equal a prefill of prompt + generated[:k]
    full = np.concatenate([p2, toks[1][:2]])
    lg = M.forward(tiny, [M.Sequence(2)], [full])[0]
    np.testing.assert_allclose(lg[0], lgs[1][2], rtol=1e-10, atol=1e-10)


def test_generate_teacher_forcing_reports_argmax(tiny):
    rng = np.random.default_rng(12)
    p = rng.integers(0, 2048, 20)
    toks, lgs = M.generate(tiny, [p], [5])
    forced = [np.array([7, 8, 9, 10, 11])]
    ft, fl = M.generate(tiny, [p], [5], forced=forced)
    assert ft[0][0] == toks[0][0]
    np.testing.assert_array_equal(ft[0], np.argmax(fl[0], -1))
    lg = M.forward(tiny, [M.Sequence(2)], [np.concatenate([p, [7, 8]])])[0]
    np.testing.assert_allclose(fl[0][2], lg[0], rtol=1e-10, atol=1e-10)


# ------------------------------------------------------------------ paged KV
def test_slot_formula_and_reservation():
    bt = [5, 2, 9]
    assert [P.slot(bt, p) for p in (0, 15, 16, 31, 32, 40)] == [80, 95, 32, 47, 144, 152]
    assert P.reservation(64, 8) == 5          # 64 + 7 tokens of KV
    assert P.reservation(64, 1) == 4
    assert P.reservation(64, 0) == 4
    assert P.reservation(65, 0) == 5
    assert P.fork_shared_pages(64) == 3 and P.fork_shared_pages(65) == 4 and P.fork_shared_pages(1) == 0


def test_page_table_permutation_is_bit_identical():
    rng = np.random.default_rng(13)
    nb, ctx = 12, 70
    k = rng.standard_normal((ctx, 2, 8))
    v = rng.standard_normal((ctx, 2, 8))
    q = rng.standard_normal((3, 4, 8))
    outs = []
    for perm_seed in (0, 1, 2):
        bt = list(np.random.default_rng(perm_seed).permutation(nb)[:5])
        kp = np.zeros((nb, 16, 2, 8))
        vp = np.zeros((nb, 16, 2, 8))
        P.scatter(kp, bt, 0, k)
        P.scatter(vp, bt, 0, v)
        outs.append(P.paged_attention(q, np.array([60, 65, 69]), kp, vp, bt, ctx))
    np.testing.assert_array_equal(outs[0], outs[1])
    np.testing.assert_array_equal(outs[0], outs[2])
    dense = M.attention(q, k, v, np.array([60, 65, 69]), np.arange(ctx))
    np.testing.assert_array_equal(outs[0], dense)


def test_allocator_lowest_first_and_refcounts():
    a = P.BlockAllocator(8)
    assert a.alloc(3) == [0, 1, 2]
    assert a.alloc(2) == [3, 4]
    a.release([1, 3])
    assert a.alloc(3) == [1, 3, 5]
    a.share([0, 1])
    a.release([0, 1])
    assert a.n_free() == 2
    assert a.alloc(3) is None
    assert a.n_free() + sum(1 for r in a.ref if r > 0) == 8
