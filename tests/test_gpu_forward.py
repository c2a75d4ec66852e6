"""GPU parity of the full-sequence forward (training form of Section 3: the MB layers
over every position under the full LCA mask, both heads at every position, the
training objective with L_BP) against ``oracle.forward_losses``.

Per-position NLLs within 2 x the logit tolerance (an NLL moves by at most twice the
largest logit error); sums within that times the number of positions; k exact."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import base_tol, forced_run, new_decoder

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny_f32"].model
LP = dict(lam0=0.7, lam1=1.3, lam2=2.0, alpha=0.3, beta=0.1)


def check(dec, W, model, x, tol, **lp):
    lp = {**LP, **lp}
    nll, loss = dec.forward(x, **lp)
    nll, loss = nll.double().cpu().numpy(), loss.double().cpu().numpy()
    ref = oracle.forward_losses(W, model, x, **lp)
    T = len(x)
    e_nt = np.max(np.abs(nll[0, : T - 1] - ref["nll_nt"]), initial=0.0)
    assert e_nt <= 2 * tol, f"next-byte NLL differs by {e_nt:.3g}"
    if len(ref["nll_mb"]):
        e_mb = np.max(np.abs(nll[1, : T - 2] - ref["nll_mb"]))
        assert e_mb <= 2 * tol, f"MB NLL differs by {e_mb:.3g}"
    assert np.all(nll[0, T - 1:] == 0) and np.all(nll[1, max(T - 2, 0):] == 0)
    if not len(ref["nll_mb"]):
        assert np.all(nll[1] == 0)
    st = 2 * tol * T
    np.testing.assert_allclose(loss[:3], [ref["sum_nt"], ref["sum_mb"], ref["l_lm"]], atol=st * 2, rtol=1e-5)
    assert int(loss[5]) == ref["k"]
    np.testing.assert_allclose(loss[3], ref["l_bp"], atol=1e-6)
    np.testing.assert_allclose(loss[4], ref["total"], atol=st * 2, rtol=1e-5)
    return ref


@pytest.mark.parametrize("seed,T", [(3, 200), (4, 37)])
def test_forward_tiny(seed, T):
    raw = synth.make_weights(TINY, seed=seed, gain_jitter=0.3, logit_gain=10.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(TINY, raw, 1, 512)
    ref = check(dec, W, TINY, synth.make_prompt(seed, T), base_tol(TINY) * 10)
    assert ref["l_bp"] > 0 or LP["beta"] <= ref["k"] / T <= LP["alpha"]


def test_forward_two_mb_layers_full_mask():
    """With two MB layers the full-sequence mask differs from the decode window."""
    model = TINY.replace(n_mb=2)
    raw = synth.make_weights(model, seed=5, gain_jitter=0.3, logit_gain=10.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, 512)
    check(dec, W, model, synth.make_prompt(6, 160), base_tol(model) * 10)


def test_forward_chunked_passes():
    """64-token passes: the trunk's commit and the MB layers both span several passes,
    so the LCA mask reaches keys of earlier passes through the forward's cache."""
    model = TINY.replace(n_mb=2)
    raw = synth.make_weights(model, seed=7, gain_jitter=0.3, logit_gain=10.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, 512, max_chunk=64)
    check(dec, W, model, synth.make_prompt(8, 300), base_tol(model) * 10)


def test_forward_learned_boundaries():
    model = TINY.replace(boundary="learned")
    raw = synth.make_weights(model, seed=3, gain_jitter=0.3, logit_gain=10.0)
    W = oracle.to_float64(raw)
    x = synth.make_prompt(1, 200)
    h_e = oracle.trunk(W, model, x)["h_e"]
    assert np.min(np.abs(oracle.boundary_logits(h_e, W, model.rms_eps))) > 1e-4
    dec = new_decoder(model, raw, 1, 512)
    check(dec, W, model, x, base_tol(model) * 10)


@pytest.mark.parametrize("T", [1, 2, 3, 16, 17])
def test_forward_short_sequences(T):
    raw = synth.make_weights(TINY, seed=9, gain_jitter=0.3, logit_gain=10.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(TINY, raw, 1, 64)
    check(dec, W, TINY, synth.make_prompt(9, T), base_tol(TINY) * 10)


def test_forward_without_mb_head():
    model = synth.TINY_FXT
    raw = synth.make_weights(model, seed=10, logit_gain=10.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, 256)
    check(dec, W, model, synth.make_prompt(10, 120), base_tol(model) * 10)


def test_forward_then_decode():
    """The forward forgets the rows; a prefill afterwards decodes as on a new handle."""
    raw = synth.make_weights(TINY, seed=11, gain_jitter=0.3, logit_gain=30.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(TINY, raw, 1, 512)
    check(dec, W, TINY, synth.make_prompt(12, 150), base_tol(TINY) * 30)
    forced_run(dec, W, TINY, [synth.make_prompt(13, 90)], 6, 4, 0.6, tol=base_tol(TINY) * 30, label="after forward")


def test_forward_rejects_mlp_head_and_short_workspace():
    from paper_2608_15454_amd import MbpError
    model = TINY.replace(head="mlp", n_mb=2)
    dec = new_decoder(model, synth.make_weights(model, seed=12), 1, 128)
    with pytest.raises(MbpError):
        dec.forward(synth.make_prompt(14, 20))
    dec = new_decoder(TINY, synth.make_weights(TINY, seed=12), 1, 128)
    import torch
    with pytest.raises(MbpError):
        _short(dec, torch)
    with pytest.raises(MbpError):
        dec.forward(synth.make_prompt(14, 200))  # beyond max_ctx


def _short(dec, torch):
    import ctypes
    from paper_2608_15454_amd import LossParams, MbpError
    x = np.ascontiguousarray(synth.make_prompt(14, 20), dtype=np.uint8)
    need = dec.L.mbp_forward_workspace_bytes(ctypes.byref(dec.cfg), 20)
    work = torch.empty(need - 256, dtype=torch.uint8, device=dec.device)
    nll = torch.zeros((2, 20), device=dec.device)
    loss = torch.zeros(6, device=dec.device)
    lp = LossParams(1, 1, 1, 1, 0)
    rc = dec.L.mbp_forward(dec.h, x.ctypes.data, 20, ctypes.byref(lp), ctypes.c_void_p(work.data_ptr()),
                           work.numel(), ctypes.c_void_p(nll.data_ptr()), ctypes.c_void_p(loss.data_ptr()))
    raise MbpError(rc, "short workspace") if rc else AssertionError("a short workspace was accepted")


@pytest.mark.timeout(300)
def test_forward_d1024_bf16():
    """The d=1024 LCA model (bf16 weights, float16 caches) on 1024 bytes of the
    4096-byte prompt: per-position NLLs within 2 x 2e-2."""
    model = synth.WORKLOADS["lca_d1024_b1"].model
    raw = synth.make_weights(model, seed=0, logit_gain=8.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, 1100)
    x = synth.make_prompt(0, 4096)[:1024]
    ref = check(dec, W, model, x, base_tol(model))
    print("k", ref["k"], "sum_nt", ref["sum_nt"], "sum_mb", ref["sum_mb"])


@pytest.mark.timeout(600)
@pytest.mark.parametrize("T", [24, 48])
def test_forward_d1024_short(T):
    """The d=1024 model on 24 and 48 bytes: every linear layer of the trunk is one pass
    of 17..64 rows with K = 1024 (the one-launch row GEMM, 32- and 64-row tiles)."""
    model = synth.WORKLOADS["lca_d1024_b1"].model
    raw = synth.make_weights(model, seed=0, logit_gain=8.0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, 128)
    ref = check(dec, W, model, synth.make_prompt(3, 256)[:T], base_tol(model))
    print("k", ref["k"], "sum_nt", ref["sum_nt"], "sum_mb", ref["sum_mb"])


@pytest.mark.timeout(600)
@pytest.mark.parametrize("T", [4096, 3900])
def test_forward_d1024_full_sequence(T):
    """The benchmarked configuration: the d=1024 model on the whole 4096-byte sequence,
    the launch shapes the forward bench times (one 4096-row pass per stack), every
    position against the oracle; and 3900 bytes, whose 3900-row passes end in a ragged
    60-row tile of the 256 x 256 GEMM tile (gate / up still has 512 tiles)."""
    wl = synth.WORKLOADS["forward_d1024_t4096"]
    model = wl.model
    raw = synth.make_weights(model, seed=0)
    W = oracle.to_float64(raw)
    dec = new_decoder(model, raw, 1, wl.prompt_len + 8)
    ref = check(dec, W, model, synth.make_prompt(0, wl.prompt_len)[:T], base_tol(model))
    print("k", ref["k"], "sum_nt", ref["sum_nt"], "sum_mb", ref["sum_mb"])
