"""CPU checks of the bf16-rounding forward (tests/bf16_emulation.py) that the
full-depth GPU tests use to bound the error bf16 arithmetic itself makes."""
import numpy as np

import synth
from oracle import model as M

from . import bf16_emulation as E


def test_bf16_rounding_is_nearest_even():
    one = 1.0
    ulp = 2.0 ** -7                              # bf16 spacing in [1, 2)
    assert E.bf16(one + ulp / 2) == one          # tie -> even mantissa (1.0)
    assert E.bf16(one + 3 * ulp / 2) == one + 2 * ulp   # tie -> even (1 + 2 ulp)
    assert E.bf16(one + 0.49 * ulp) == one
    assert E.bf16(one + 0.51 * ulp) == one + ulp
    assert E.bf16(-3.0) == -3.0 and E.bf16(0.0) == 0.0


def test_without_rounding_it_is_the_oracle_forward():
    sh = synth.model_shape("tiny")
    gains = synth.gen_norm_gains(sh)
    w = M.Weights(sh, norm_gains=gains)
    rng = np.random.default_rng(4)
    chunks = [rng.integers(0, sh.vocab, n) for n in (37, 5)]
    a = M.forward(w, [M.Sequence(2), M.Sequence(2)], chunks, logit_rows=[[0, 36], [4]])
    b = E.forward(w, [M.Sequence(2), M.Sequence(2)], chunks, logit_rows=[[0, 36], [4]], rounding=False)
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, rtol=1e-12, atol=1e-12)


def test_bf16_drift_grows_with_depth():
    """The rounded forward drifts from the exact one by an amount that grows with
    depth (per-layer roundings add up)."""
    sh = synth.model_shape("tiny").with_layers(8)
    rng = np.random.default_rng(5)
    ids = rng.integers(0, sh.vocab, 24)
    errs = []
    for L in (1, 8):
        wl = M.Weights(sh.with_layers(L), norm_gains={k: (v[:L] if k != "final" else v)
                                                       for k, v in synth.gen_norm_gains(sh).items()},
                       layer_bits=lambda l: synth.gen_layer(sh, l), lm_head_bits=synth.gen_lm_head(sh))
        ref = M.forward(wl, [M.Sequence(L)], [ids])[0][0]
        got = E.forward(wl, [M.Sequence(L)], [ids])[0][0]
        errs.append(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    assert 0 < errs[0] < errs[1]
    assert errs[0] < 2e-2
