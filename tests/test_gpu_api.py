"""GPU checks of the C ABI's state machine and error paths, and run-to-run
determinism."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import THRESHOLD, new_decoder
from paper_2608_15454_amd import ECAPACITY, EINVAL, ESTATE, MbpError

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny_f32"].model


@pytest.fixture(scope="module")
def raw():
    return synth.make_weights(TINY, seed=1, gain_jitter=0.2, logit_gain=10.0)


def _code(fn):
    with pytest.raises(MbpError) as e:
        fn()
    return e.value.code


def test_errors_leave_state_usable(raw):
    W = oracle.to_float64(raw)
    dec = new_decoder(TINY, raw, 2, 200, max_n=4)
    assert _code(lambda: dec.prefill([synth.make_prompt(0, 201)])) == ECAPACITY
    assert _code(lambda: dec.prefill([np.zeros(0, np.uint8)])) == EINVAL
    assert _code(lambda: dec.decode_step(3, 0.5)) == ESTATE  # no prefill yet
    p = synth.make_prompt(0, 150)
    dec.prefill([p])
    assert _code(lambda: dec.accept()) == ESTATE  # nothing pending
    assert _code(lambda: dec.decode_step(5, 0.5)) == EINVAL  # n > max_n
    assert _code(lambda: dec.decode_step(3, 1.5)) == EINVAL
    dec.decode_step(3, 0.5)
    assert _code(lambda: dec.decode_step(3, 0.5)) == ESTATE  # previous step not accepted
    want = oracle.step(W, TINY, p, 3, 0.5)
    got = dec.logits()[0].double().cpu().numpy()
    assert np.max(np.abs(got - want["logits"])) < 1e-5
    # an override that would overflow max_ctx is rejected, state unchanged
    assert _code(lambda: dec.accept([np.full(5, 65, np.uint8)])) == EINVAL  # longer than max_n
    dec.accept()
    assert dec.row_length(0) == 150 + int(want["k"])
    big = [np.full(4, 65, np.uint8)]
    for _ in range(12):
        dec.decode_step(3, 0.5)
        dec.accept(big)
    assert dec.row_length(0) == 150 + int(want["k"]) + 48
    dec.decode_step(3, 0.5)
    assert _code(lambda: dec.accept(big)) == ECAPACITY  # 202+ bytes > max_ctx 200
    assert dec.row_length(0) == 150 + int(want["k"]) + 48
    dec.accept([np.zeros(0, np.uint8)])  # commit nothing
    x = list(p) + list(want["cand"][: want["k"]]) + [65] * 48
    dec.decode_step(3, 0.5)
    ref = oracle.step(W, TINY, x, 3, 0.5)
    assert np.max(np.abs(dec.logits()[0].double().cpu().numpy() - ref["logits"])) < 1e-5


def test_reset_and_reprefill_is_deterministic(raw):
    dec = new_decoder(TINY, raw, 1, 300)
    p = synth.make_prompt(3, 120)

    def run():
        dec.prefill([p])
        rows = []
        for _ in range(6):
            dec.decode_step(4, 0.6)
            rows.append(dec.logits().cpu().numpy().copy())
            dec.accept()
        return np.stack(rows)

    a = run()
    dec.reset()
    b = run()
    np.testing.assert_array_equal(a, b)


def test_teacher_forcing_rolls_back_a_verify_step(raw):
    W = oracle.to_float64(raw)
    dec = new_decoder(TINY, raw, 1, 300)
    p = synth.make_prompt(4, 100)
    dec.prefill([p])
    from paper_2608_15454_amd import SELF_VERIFY

    dec.decode_step(5, 0.0, SELF_VERIFY)
    forced = np.array([65, 32, 66], np.uint8)
    dec.accept([forced])
    assert dec.row_length(0) == 103
    dec.decode_step(3, 0.5)
    ref = oracle.step(W, TINY, list(p) + [65, 32, 66], 3, 0.5)
    assert np.max(np.abs(dec.logits()[0].double().cpu().numpy() - ref["logits"])) < 1e-5
