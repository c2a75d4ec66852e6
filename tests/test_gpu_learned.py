"""GPU parity of learned segmentation: the boundary predictor on the encoder states
decides where segments end (Section 2.2, encoder module; at inference a byte ends a
segment when its boundary logit is >= 0, or when the segment reaches max_patch bytes).

* tiny float32 (d=128): teacher-forced steps against the oracle at 1e-5 on logits,
  and the library's segment ends equal to the oracle's (index work, exact): one row,
  ragged rows with a chunked prefill, self-verify, free-running generation;
* float32 d=256 through the persistent engine, same bar;
* bfloat16 d=1024 at the full 4096-byte prompt: every segment end the library took
  is valid for the oracle's boundary logits, where a logit within the bfloat16 margin
  of 0 may go either way.
The float32 tests first check that no oracle boundary logit of the compared
sequences lies within 1e-4 of 0, so that float32 rounding cannot flip a decision."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import (SELF_VERIFY, base_tol, divergence_is_exempt, first_divergence, forced_run, free_run,
                         new_decoder)

pytestmark = pytest.mark.gpu

LEARNED = synth.WORKLOADS["tiny_f32"].model.replace(boundary="learned")
SMALL = synth.SMALL_F32.replace(boundary="learned")
WL = synth.WORKLOADS["learned_d1024_b1"]
BAND = 1e-4  # float32 decisions compared exactly only outside this band


def encoder_logits(W, model, x):
    """Oracle encoder states of the whole sequence, then the boundary logits."""
    x = np.asarray(x, np.int64)
    T = len(x)
    E = np.asarray(W["emb"], np.float64)[x]
    h_e = oracle.stack(E, W, "enc", model.n_enc, oracle.causal_mask(T), np.arange(T), model)
    return oracle.boundary_logits(h_e, W, model.rms_eps), oracle.learned_boundaries(h_e, W, model.max_patch,
                                                                                   model.rms_eps)


def check_segments(dec, W, model, seqs):
    """The library's segment ends equal the oracle's on each committed sequence
    (a segment end at byte i depends on bytes 0..i only)."""
    for b, x in enumerate(seqs):
        z, q = encoder_logits(W, model, x)
        assert np.min(np.abs(z)) > BAND, f"row {b}: a boundary logit lies within {BAND} of 0"
        got = dec.row_boundaries(b)
        assert list(got) == list(q), f"row {b}: segment ends differ"
        assert 0 < len(q) < len(x)


@pytest.fixture(scope="module")
def tiny():
    raw = synth.make_weights(LEARNED, seed=3, gain_jitter=0.3, logit_gain=50.0)
    return raw, oracle.to_float64(raw)


def test_learned_tiny_forced(tiny):
    raw, W = tiny
    dec = new_decoder(LEARNED, raw, 1, 512)
    st = forced_run(dec, W, LEARNED, [synth.make_prompt(1, 200)], 40, 5, 0.5, tol=base_tol(LEARNED) * 50,
                    label="learned")
    print(st)
    assert st.accepted > st.steps
    check_segments(dec, W, LEARNED, st.seqs)


def test_learned_tiny_batched_chunked(tiny):
    """Ragged rows and a prefill split into 64-token passes: each pass decides its
    bytes' segments after its own encoder pass."""
    raw, W = tiny
    prompts = [synth.make_prompt(r, L) for r, L in enumerate([1, 70, 260])]
    dec = new_decoder(LEARNED, raw, 3, 512, max_chunk=64)
    st = forced_run(dec, W, LEARNED, prompts, 8, 4, 0.6, tol=base_tol(LEARNED) * 50, label="learned b3")
    print(st)
    check_segments(dec, W, LEARNED, st.seqs)


def test_learned_tiny_verify(tiny):
    """Self-verify commits the drafts tentatively (segmenting them) and rolls back."""
    raw, W = tiny
    dec = new_decoder(LEARNED, raw, 2, 512)
    prompts = [synth.make_prompt(9, 90), synth.make_prompt(10, 60)]
    st = forced_run(dec, W, LEARNED, prompts, 8, 5, 0.75, mode=SELF_VERIFY, tol=base_tol(LEARNED) * 50,
                    label="learned verify")
    print(st)


def test_learned_tiny_free_running(tiny):
    raw, W = tiny
    prompt = synth.make_prompt(1, 200)
    dec = new_decoder(LEARNED, raw, 1, 512)
    got, ks = free_run(dec, [prompt], 64, 5, 0.5)
    want, steps = oracle.generate(W, LEARNED, prompt, 64, 5, 0.5)
    i = first_divergence(got[0], want)
    if i is not None:
        assert divergence_is_exempt(W, LEARNED, prompt, want, steps, i, 5, 0.5, base_tol(LEARNED) * 50), i
    assert max(int(k[0]) for k in ks) > 1


@pytest.mark.timeout(300)
def test_learned_engine_small_f32():
    gain = 30.0
    raw = synth.make_weights(SMALL, seed=3, logit_gain=gain)
    W = oracle.to_float64(raw)
    dec = new_decoder(SMALL, raw, 1, 700)
    dec.set_timing(True)
    st = forced_run(dec, W, SMALL, [synth.make_prompt(3, 300)], 10, 4, 0.6, tol=base_tol(SMALL) * gain,
                    label="learned engine")
    print(st)
    assert dec.read_timing()["engine"][0] > 0
    check_segments(dec, W, SMALL, st.seqs)


@pytest.mark.timeout(300)
def test_learned_d1024_full_prompt_segments_valid():
    """The d=1024 workload: 4096-byte prompt, then 8 free-running steps (n=3, tau
    0.75).  Each library decision is checked against the oracle's logit with the
    library's own previous segment end (so max_patch closes are checked too), and
    about one byte in three near the end of the sequence ends a segment."""
    model = WL.model
    raw = synth.make_weights(model, seed=0)
    W = oracle.to_float64(raw)
    prompt = synth.make_prompt(0, WL.prompt_len)
    dec = new_decoder(model, raw, 1, WL.prompt_len + 64)
    dec.prefill([prompt])
    x = [int(v) for v in prompt]
    for _ in range(8):
        dec.decode_step(WL.n, WL.tau)
        acc, lens = dec.last_accepted()
        dec.accept()
        x += [int(c) for c in acc[0, : lens[0]]]
    assert dec.row_length(0) == len(x)
    z, _ = encoder_logits(W, model, x)
    q = set(int(v) for v in dec.row_boundaries(0))
    margin = 0.05  # bfloat16 weights, float16 KV caches: boundary logits within a few 1e-3
    prev, band = -1, 0
    for i in range(len(x)):
        forced = model.max_patch > 0 and i - prev >= model.max_patch
        if abs(z[i]) < margin and not forced:
            band += 1
        elif forced or z[i] >= margin:
            assert i in q, f"byte {i}: logit {z[i]:.4f} (segment from {prev + 1}) should end a segment"
        else:
            assert i not in q, f"byte {i}: logit {z[i]:.4f} should not end a segment"
        if i in q:
            prev = i
    tail = sum(1 for i in q if i >= len(x) - 1024) / 1024
    print(f"segments {len(q)} of {len(x)} bytes, {tail:.3f} of the last 1024, {band} decisions inside the margin")
    assert 0.27 < tail < 0.42  # the workload's compression where decoding runs
