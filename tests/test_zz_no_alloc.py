"""The allocation-free forward (mbp_forward_static) against mbp_forward: the same
sequence gives the same per-position NLLs and losses, on two calls in a row (the
second with a shorter sequence, which must not see the first call's scratch
contents), for the float32 tiny model and the d=1024 bfloat16 model; a sequence
beyond the fixed scratch is rejected before any device work."""
import ctypes

import numpy as np
import pytest

import synth
from paper_2608_15454_amd import ECAPACITY, Decoder, MbpError, lib, make_config

pytestmark = pytest.mark.gpu


def _compare(dec, T_list, seed, tol):
    for T in T_list:
        seq = synth.make_prompt(seed, T)
        nll_a, loss_a = dec.forward(seq)
        a_n, a_l = nll_a.double().cpu().numpy(), loss_a.double().cpu().numpy()
        nll_b, loss_b = dec.forward_static(seq)
        b_n, b_l = nll_b.double().cpu().numpy(), loss_b.double().cpu().numpy()
        err = max(float(np.max(np.abs(a_n - b_n))), float(np.max(np.abs(a_l - b_l)) / max(1.0, abs(a_l[4]))))
        print(f"T={T}: max difference {err:.3g}")
        assert err <= tol, f"T={T}: static-scratch forward differs by {err}"
        assert np.all(np.isfinite(b_n)) and np.all(np.isfinite(b_l))


def test_forward_static_tiny_f32_two_calls():
    model = synth.WORKLOADS["tiny_f32"].model
    W = synth.make_weights(model, seed=0, gain_jitter=0.2, logit_gain=4.0)
    dec = Decoder(make_config(model, max_batch=1, max_ctx=400, max_n=8), W)
    _compare(dec, [300, 77], seed=5, tol=1e-5)


def test_forward_static_d1024_bf16_two_calls():
    model = synth.WORKLOADS["lca_d1024_b1"].model
    W = synth.make_weights(model, seed=0)
    dec = Decoder(make_config(model, max_batch=1, max_ctx=1200, max_n=8), W)
    _compare(dec, [1024, 200], seed=6, tol=2e-2)


def test_forward_static_rejects_a_sequence_beyond_its_scratch():
    model = synth.WORKLOADS["lca_d1024_b1"].model
    W = synth.make_weights(model, seed=0)
    T = 6000  # d=1024 with two MB layers: about 13 KiB of scratch per byte, beyond 64 MiB
    cfg = make_config(model, max_batch=1, max_ctx=T + 8, max_n=8)
    assert lib().mbp_forward_workspace_bytes(ctypes.byref(cfg), T) > lib().mbp_forward_static_max_bytes()
    dec = Decoder(cfg, W)
    with pytest.raises(MbpError) as e:
        dec.forward_static(synth.make_prompt(0, T))
    assert e.value.code == ECAPACITY and "static scratch" in str(e.value)
    # the handle stays usable
    _compare(dec, [64], seed=7, tol=2e-2)
