"""The attention parity bound (per (row, head) max|diff| / max|ref| <= ATTN_TOL)
checked on the CPU against what it must accept and what it must reject, at the
context lengths of the 8B workloads:

* accept: attention computed with the kernels' roundings (probabilities rounded
  to bf16 before the PV product, output rounded to bf16) stays well inside it;
* reject: the same attention reading one 16-token page of another sequence, or
  with the partially filled last page swapped into the middle of the block
  table, falls outside it.

No GPU and no library code: the rounded variant is written here from the
kernels' documented arithmetic, the reference is the oracle."""
import numpy as np
import pytest

import synth
from oracle import model as M
from oracle import paged as P

from .gpu_util import ATTN_TOL, attn_rel_err


def bf16(x):
    return synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(np.asarray(x, np.float32))).astype(np.float64)


def rounded_decode_attention(q, k, v, grp):
    """One query per head over ctx keys: fp32-ish scores, P rounded to bf16 for the
    PV product, normaliser from the unrounded P, output rounded to bf16."""
    hq, dh = q.shape
    out = np.empty((hq, dh))
    for h in range(hq):
        g = h // grp
        s = (k[:, g, :] @ q[h]) / np.sqrt(dh)
        p = np.exp(s - s.max())
        out[h] = bf16((bf16(p) @ v[:, g, :]) / p.sum())
    return out


def _case(ctx, seed, hq=32, hkv=8, dh=128):
    rng = np.random.default_rng(seed)
    q = bf16(rng.standard_normal((hq, dh)))
    k = bf16(rng.standard_normal((ctx, hkv, dh)))
    v = bf16(rng.standard_normal((ctx, hkv, dh)))
    return q, k, v


@pytest.mark.parametrize("ctx", [1024, 3000, 8192])
def test_bound_accepts_the_kernels_rounding(ctx):
    q, k, v = _case(ctx, ctx)
    ref = M.attention(q[None], k, v, np.array([ctx - 1]), np.arange(ctx))[0]
    got = rounded_decode_attention(q, k, v, 4)
    err = attn_rel_err(got[None], ref[None])
    assert err < ATTN_TOL / 2, err


@pytest.mark.parametrize("ctx", [3000, 8192])
def test_bound_rejects_a_misread_page(ctx):
    q, k, v = _case(ctx, ctx + 1)
    n_pages = P.pages_for(ctx)
    rng = np.random.default_rng(ctx)
    # pool: this sequence's pages plus one foreign page
    kp = np.zeros((n_pages + 1, 16, 8, 128))
    vp = np.zeros((n_pages + 1, 16, 8, 128))
    bt = list(range(n_pages))
    P.scatter(kp, bt, 0, k)
    P.scatter(vp, bt, 0, v)
    kp[n_pages] = bf16(rng.standard_normal((16, 8, 128)))
    vp[n_pages] = bf16(rng.standard_normal((16, 8, 128)))
    qp = np.array([ctx - 1])
    ref = P.paged_attention(q[None], qp, kp, vp, bt, ctx)
    foreign = list(bt)
    foreign[n_pages // 2] = n_pages
    cases = [("foreign page", foreign)]
    if ctx % 16:
        # full pages hold RoPE'd keys, so permuting them attends the same set; a swap
        # with the partially filled last page moves the context boundary
        last = list(bt)
        last[n_pages - 1], last[1] = last[1], last[n_pages - 1]
        cases.append(("partial last page swapped", last))
    for name, table in cases:
        bad = P.paged_attention(q[None], qp, kp, vp, table, ctx)
        err = attn_rel_err(bad, ref)
        assert err > 2 * ATTN_TOL, (name, err)
