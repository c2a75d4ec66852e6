"""GPU checks of sampled decoding (temperature / top-p candidates from given uniforms,
threshold acceptance on their probabilities, and speculative sampling of drafts)
against the oracle.  A sampled byte may differ only where the oracle's decision is
inside the logit error: the uniform within that error of a CDF boundary, or a byte's
ranked mass within it of top_p (or, for speculative sampling, the acceptance ratio
within it of its uniform)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_harness import SELF_VERIFY, THRESHOLD, TAU_BAND, base_tol, new_decoder

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny_f32"].model


def _uniforms(rng, B, n):
    u = rng.random((B, 3 * n)).astype(np.float32)
    return u, torch.tensor(u, device="cuda")


def _softmax(l, T):
    z = np.asarray(l, np.float64) / T
    e = np.exp(z - z.max())
    return e / e.sum()


def _dist_near(logits, T, top_p, u, eps):
    """Whether sampling this row with u is within eps of a decision boundary."""
    p = _softmax(logits, T)
    before = np.array([p[(p > p[i]) | ((p == p[i]) & (np.arange(256) < i))].sum() for i in range(256)])
    if np.any(np.abs(before - top_p) < eps):
        return True
    q = oracle.decoding_dist(logits, T, top_p)
    return bool(np.min(np.abs(np.cumsum(q) - u)) < eps)


@pytest.mark.parametrize("T,top_p,n", [(0.7, 0.9, 3), (1.3, 1.0, 5), (1.0, 0.5, 4)])
def test_sampled_threshold_tiny_per_step(T, top_p, n):
    raw = synth.make_weights(TINY, seed=50, logit_gain=5.0)
    W = oracle.to_float64(raw)
    tol = base_tol(TINY) * 5.0
    eps = 20 * tol
    tau = 0.3
    dec = new_decoder(TINY, raw, 1, 400)
    p = synth.make_prompt(12, 100)
    dec.prefill([p])
    x = [int(b) for b in p]
    rng = np.random.default_rng(7)
    exempt = 0
    for step in range(12):
        u, du = _uniforms(rng, 1, n)
        cand, prob, ln = dec.decode_step_sampled(n, tau, THRESHOLD, T, top_p, du)
        ref = oracle.step_sampled(W, TINY, x, n, tau, T, top_p, u[0].astype(np.float64))
        logits = dec.logits()[0].double().cpu().numpy()
        assert np.max(np.abs(logits - ref["logits"])) <= tol
        c, pr, k = cand[0].cpu().numpy(), prob[0].cpu().numpy(), int(ln[0].item())
        ok = True
        for m in range(n):
            if int(c[m]) != int(ref["cand"][m]):
                assert _dist_near(ref["logits"][m], T, top_p, u[0, m], eps), (step, m, c[m], ref["cand"][m])
                ok = False
            else:
                assert abs(float(pr[m]) - ref["prob"][m]) <= 3 * tol
        if ok and k != ref["k"]:
            assert any(abs(ref["prob"][m] - tau) < TAU_BAND for m in range(1, n)), (step, k, ref["k"])
            ok = False
        exempt += 0 if ok else 1
        acc = [int(b) for b in ref["cand"][: ref["k"]]]
        dec.accept([acc])
        x += acc
    print(f"exempt steps {exempt}")
    assert exempt <= 2


@pytest.mark.parametrize("T,top_p,n", [(0.7, 0.9, 3), (1.0, 1.0, 5)])
def test_sampled_verify_tiny_per_step(T, top_p, n):
    raw = synth.make_weights(TINY, seed=51, logit_gain=5.0)
    W = oracle.to_float64(raw)
    tol = base_tol(TINY) * 5.0
    eps = 20 * tol
    dec = new_decoder(TINY, raw, 1, 400)
    p = synth.make_prompt(13, 100)
    dec.prefill([p])
    x = [int(b) for b in p]
    rng = np.random.default_rng(8)
    exempt, ks = 0, []
    for step in range(12):
        u, du = _uniforms(rng, 1, n)
        cand, _, ln = dec.decode_step_sampled(n, 0.5, SELF_VERIFY, T, top_p, du)
        k = int(ln[0].item())
        got = [int(b) for b in cand[0, :k].cpu().numpy()]
        ref = oracle.verify_step_sampled(W, TINY, x, n, T, top_p, u[0].astype(np.float64))
        want = [int(b) for b in ref["bytes"]]
        ks.append(ref["k"])
        if got != want:
            near = any(_dist_near(ref["logits"][m], T, top_p, u[0, m], eps) for m in range(n))
            for m in range(2, n + 1):
                c = int(ref["cand"][m - 1])
                ratio = ref["p"][m - 2][c] / ref["q"][m - 1][c]
                near = near or abs(ratio - u[0, n + m - 1]) < eps * max(1.0, ratio)
                r = np.maximum(ref["p"][m - 2] - ref["q"][m - 1], 0.0)
                if r.sum() > 0:
                    near = near or bool(np.min(np.abs(np.cumsum(r / r.sum()) - u[0, 2 * n + m - 1])) < eps)
            assert near, (step, got, want)
            exempt += 1
            dec.accept([want])  # teacher forcing: roll back and commit the oracle's bytes
        else:
            dec.accept()
        x += want
        assert dec.row_length(0) == len(x)
    print(f"accepted per step {ks}, exempt steps {exempt}")
    assert exempt <= 2


def test_sampled_threshold_engine_path_small_f32():
    model = synth.SMALL_F32
    raw = synth.make_weights(model, seed=52, logit_gain=5.0)
    W = oracle.to_float64(raw)
    tol = base_tol(model) * 5.0
    dec = new_decoder(model, raw, 1, 400)
    p = synth.make_prompt(14, 150)
    dec.prefill([p])
    x = [int(b) for b in p]
    rng = np.random.default_rng(9)
    for step in range(4):
        u, du = _uniforms(rng, 1, 3)
        cand, prob, ln = dec.decode_step_sampled(3, 0.3, THRESHOLD, 0.8, 0.95, du)
        ref = oracle.step_sampled(W, model, x, 3, 0.3, 0.8, 0.95, u[0].astype(np.float64))
        assert np.max(np.abs(dec.logits()[0].double().cpu().numpy() - ref["logits"])) <= tol
        c = cand[0].cpu().numpy()
        for m in range(3):
            if int(c[m]) != int(ref["cand"][m]):
                assert _dist_near(ref["logits"][m], 0.8, 0.95, u[0, m], 20 * tol)
        acc = [int(b) for b in ref["cand"][: ref["k"]]]
        dec.accept([acc])
        x += acc


def test_one_byte_nucleus_is_greedy_d1024():
    wl = synth.WORKLOADS["lca_d1024_b1"]
    raw = synth.make_weights(wl.model, seed=0, logit_gain=30.0)
    dec = new_decoder(wl.model, raw, 1, 700)
    dec.prefill([synth.make_prompt(15, 512)])
    rng = np.random.default_rng(10)
    for step in range(4):
        _, du = _uniforms(rng, 1, 3)
        c1, p1, k1 = dec.decode_step_sampled(3, 0.5, THRESHOLD, 0.7, 1e-6, du)
        c1, p1, k1 = c1.cpu().numpy().copy(), p1.cpu().numpy().copy(), int(k1[0].item())
        assert np.all(p1 == 1.0) and k1 == 3
        dec.accept([[]])  # commit nothing
        c2, _, _ = dec.decode_step(3, 0.5, THRESHOLD)
        np.testing.assert_array_equal(c1, c2.cpu().numpy())
        dec.accept()
