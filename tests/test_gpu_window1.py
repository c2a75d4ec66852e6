"""GPU parity of window mode 1 in decode -- the MB layers over the whole sequence under
the full LCA mask, each row keeping the outputs it had when it was computed -- against
the oracle's step with window_mode = 1 (Algorithm 1's window slice replaced by the
training mask of Section 3): tiny float32 with two MB layers (where the two modes
differ) on the per-kernel path, the d=256 float32 model on the engine path, ragged
acceptance across segment ends, self-verification (rows truncated after a rejected
draft), a batch of two rows, and the d=1024 bf16 model.  Tolerances as in the other
GPU tests (1e-5 for float32, 2e-2 for bf16, scaled by the logit gain)."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import SELF_VERIFY, base_tol, forced_run, new_decoder

pytestmark = pytest.mark.gpu

TINY1 = synth.WORKLOADS["tiny_f32"].model.replace(n_mb=2, window_mode=1)
SMALL1 = synth.SMALL_F32.replace(window_mode=1)
D1024_1 = synth.WORKLOADS["lca_d1024_b1"].model.replace(window_mode=1)
GAIN = 50.0


def _raw(model, seed=3, gain=GAIN):
    return synth.make_weights(model, seed=seed, gain_jitter=0.3, logit_gain=gain)


def _modes_differ(W, model, prompt, n):
    """The oracle's MB rows of the prompt's first step differ between the two modes by
    more than the tolerance (so a comparison at mode 1 is not passed by mode 0)."""
    x = [int(b) for b in prompt]
    l1 = oracle.step_logits(W, model, x, n)
    l0 = oracle.step_logits(W, model.replace(window_mode=0), x, n)
    assert np.array_equal(l1[0], l0[0])  # the next-byte row does not involve the MB head
    return float(np.max(np.abs(l1[1:] - l0[1:])))


@pytest.mark.parametrize("n,tau", [(3, 0.75), (5, 0.5)])
def test_tiny_mode1_forced(n, tau):
    raw = _raw(TINY1)
    W = oracle.to_float64(raw)
    prompt = synth.make_prompt(1, 200)
    assert _modes_differ(W, TINY1, prompt, n) > 10 * base_tol(TINY1) * GAIN
    dec = new_decoder(TINY1, raw, 1, 512)
    st = forced_run(dec, W, TINY1, [prompt], 40, n, tau, tol=base_tol(TINY1) * GAIN, label=f"w1 n{n}")
    print(st)
    assert st.accepted > st.steps  # ragged: multi-byte commits, segment ends inside them


def test_small_mode1_engine_path():
    raw = _raw(SMALL1, seed=5)
    W = oracle.to_float64(raw)
    prompt = synth.make_prompt(2, 160)
    assert _modes_differ(W, SMALL1, prompt, 4) > 10 * base_tol(SMALL1) * GAIN
    dec = new_decoder(SMALL1, raw, 1, 400)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL1, [prompt], 24, 4, 0.6, tol=base_tol(SMALL1) * GAIN, label="w1 engine")
    print(st)
    assert dec.read_timing()["engine"][0] > 0  # the passes ran in the persistent engine


def test_tiny_mode1_self_verify_and_batch():
    raw = _raw(TINY1, seed=7)
    W = oracle.to_float64(raw)
    prompts = [synth.make_prompt(3, 150), synth.make_prompt(4, 90)]
    dec = new_decoder(TINY1, raw, 2, 400)
    st = forced_run(dec, W, TINY1, prompts, 20, 5, 0.0, mode=SELF_VERIFY, tol=base_tol(TINY1) * GAIN,
                    label="w1 verify")
    print(st)
    st = forced_run(dec, W, TINY1, prompts, 20, [3, 5, 2], 0.6, tol=base_tol(TINY1) * GAIN, label="w1 b2")
    print(st)


@pytest.mark.timeout(900)
def test_d1024_mode1_bf16():
    raw = synth.make_weights(D1024_1, seed=0, logit_gain=8.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(D1024_1, raw, 1, 600)
    st = forced_run(dec, W, D1024_1, [synth.make_prompt(5, 300)], 6, 3, 0.75, tol=base_tol(D1024_1) * 8.0,
                    label="w1 d1024")
    print(st)
