"""The float32 KV-cached CPU decoder (the CPU baseline bench.py times) against the
float64 full-recompute oracle: the same logits within float32 rounding, the same
candidates and accepted counts, step after step, with ragged acceptance, segments
closing inside multi-byte commits, both heads and self-verification."""
import numpy as np
import pytest

import oracle
import synth
from oracle.cached import CachedDecoder

TINY = synth.WORKLOADS["tiny_f32"].model


def _gap(row):
    s = np.sort(row)
    return s[-1] - s[-2]


@pytest.mark.parametrize("model,n,tau", [(TINY, 4, 0.5), (TINY.replace(max_patch=4, n_mb=2), 3, 0.75),
                                         (TINY.replace(head="mlp", n_mb=3), 4, 0.5)])
def test_cached_steps_equal_full_recompute(model, n, tau):
    W = synth.make_weights(model, seed=3, gain_jitter=0.2, logit_gain=30.0)
    W64 = oracle.to_float64(W)
    x = [int(b) for b in synth.make_prompt(4, 90)]
    dec = CachedDecoder(W, model, cap=200)
    dec.prefill(x)
    ks = []
    for step in range(12):
        ref = oracle.step(W64, model, x, n, tau)
        got = dec.step(n, tau)
        np.testing.assert_allclose(got["logits"], ref["logits"], rtol=0, atol=1e-4)
        for m in range(n):
            if _gap(ref["logits"][m]) > 1e-2:
                assert int(got["cand"][m]) == int(ref["cand"][m])
        if all(abs(ref["prob"][m] - tau) > 1e-3 for m in range(1, n)):
            assert got["k"] == ref["k"]
        acc = [int(c) for c in ref["cand"][: ref["k"]]]
        ks.append(ref["k"])
        dec.accept(acc)
        x += acc
    assert max(ks) > 1  # acceptance was ragged
    assert len(dec.q) == len(oracle.boundaries(np.array(x), model.max_patch))


def test_cached_verify_equals_oracle_verify():
    W = synth.make_weights(TINY, seed=4, gain_jitter=0.2, logit_gain=30.0)
    W64 = oracle.to_float64(W)
    x = [int(b) for b in synth.make_prompt(5, 70)]
    dec = CachedDecoder(W, TINY, cap=200)
    dec.prefill(x)
    for _ in range(8):
        ref = oracle.verify_step(W64, TINY, x, 5)
        got = dec.verify_step(5)
        np.testing.assert_allclose(got["logits"], ref["logits"], rtol=0, atol=1e-4)
        assert got["k"] == ref["k"]
        x += [int(c) for c in ref["cand"][: ref["k"]]]
        assert dec.x == x
