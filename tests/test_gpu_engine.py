"""GPU parity of the persistent engine (one cooperative launch per transformer stack
for passes of at most 16 token rows).

* float32, d=256 / 4 heads / head size 64 (the engine's smallest shape): against the
  oracle at 1e-5 on logits, single row and batched, threshold and verify modes,
  including MB window rebuilds whose passes exceed 16 rows (per-kernel path) mixed
  with engine passes.
* bfloat16, d=1024: engine against the per-kernel path of the same library.
Every test also checks that engine launches ran (timing class "engine")."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import (SELF_VERIFY, THRESHOLD, base_tol, forced_run, free_run, new_decoder)

pytestmark = pytest.mark.gpu

SMALL = synth.SMALL_F32
D1024 = synth.WORKLOADS["lca_d1024_b1"].model


GAIN = 30.0  # logit gain: probabilities spread enough for ragged acceptance
TOL = base_tol(SMALL) * GAIN  # float32 tolerance on the gained logit scale


@pytest.fixture(scope="module")
def small():
    raw = synth.make_weights(SMALL, seed=3, logit_gain=GAIN)
    return raw, oracle.to_float64(raw)


def engine_launches(dec):
    return dec.read_timing()["engine"][0]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("n,tau", [(3, 0.75), (5, 0.5)])
def test_engine_small_f32_forced(small, n, tau):
    raw, W = small
    dec = new_decoder(SMALL, raw, 1, 700)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL, [synth.make_prompt(3, 300)], 12, n, tau, tol=TOL, label=f"engine f32 n={n}")
    print(st)
    assert engine_launches(dec) > 0


@pytest.mark.timeout(300)
def test_engine_small_f32_varying_n(small):
    """The candidate count changes between steps: a commit prepares the next step's
    window update for the previous n, so steps with another n take the general path
    (and rows computed for a smaller n are extended)."""
    raw, W = small
    dec = new_decoder(SMALL, raw, 1, 700)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL, [synth.make_prompt(5, 260)], 12, [3, 5, 2, 5, 4, 1, 6], 0.5, tol=TOL,
                    label="engine f32 varying n")
    print(st)
    assert engine_launches(dec) > 0


@pytest.mark.timeout(300)
def test_engine_small_f32_batched(small):
    """Three rows of different lengths: passes hold 1..3 rows per batch row."""
    raw, W = small
    prompts = [synth.make_prompt(20 + r, L) for r, L in enumerate([40, 170, 333])]
    dec = new_decoder(SMALL, raw, 3, 700)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL, prompts, 6, 4, 0.6, tol=TOL, label="engine f32 b3")
    print(st)
    assert engine_launches(dec) > 0


@pytest.mark.timeout(300)
def test_engine_small_f32_verify(small):
    raw, W = small
    dec = new_decoder(SMALL, raw, 1, 700)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL, [synth.make_prompt(5, 260)], 6, 5, 0.75, mode=SELF_VERIFY, tol=TOL,
                    label="engine verify")
    print(st)
    assert engine_launches(dec) > 0


@pytest.mark.timeout(300)
def test_engine_small_f32_long_groups(small):
    """Space rule only with a wide window: window rebuilds exceed 16 rows and take the
    per-kernel path, the incremental updates between them take the engine."""
    raw, W = small
    model = SMALL.replace(max_patch=0)
    dec = new_decoder(model, raw, 1, 700, max_window=200)
    dec.set_timing(True)
    st = forced_run(dec, W, model, [synth.make_prompt(7, 200)], 10, 4, 0.6, tol=TOL, label="engine long groups")
    print(st)
    assert engine_launches(dec) > 0


@pytest.mark.timeout(300)
def test_engine_matches_per_kernel_path_d1024():
    """Same weights and prompt through both paths: logits within the bf16 tolerance and
    identical bytes over a free-running generation."""
    raw = synth.make_weights(D1024, seed=0, logit_gain=8.0)
    prompt = [synth.make_prompt(4, 600)]
    outs, logits = [], []
    for engine in (True, False):
        dec = new_decoder(D1024, raw, 1, 800, engine=engine)
        dec.set_timing(True)
        dec.prefill(prompt)
        ls = []
        for _ in range(6):
            dec.decode_step(4, 0.75, THRESHOLD)
            ls.append(dec.logits().double().cpu().numpy())
            dec.accept()
        logits.append(np.stack(ls))
        assert (engine_launches(dec) > 0) == engine
        gen, _ = free_run(dec, prompt, 24, 4, 0.75)
        outs.append(gen[0])
        del dec
    err = float(np.max(np.abs(logits[0] - logits[1])))
    print("engine vs per-kernel max logit difference", err)
    assert err < 2e-2 * 8.0
    assert np.array_equal(outs[0], outs[1])
