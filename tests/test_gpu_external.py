"""GPU checks of external verification: a next-byte model without MB head (the FxT
baseline) verifies another model's drafts (Section 6, external verification).
Tiny float32 models step by step against the oracle (the verifier's n+1 logit rows
within 1e-5 times the logit gain; kept count and accepted bytes exact, except where
an inspected greedy byte is inside that logit error), free-running equality with the
verifier's greedy decoding, the pending bonus byte before a decode step and under an
override, and the d=1024 bf16 engine path against the verifier's own n = 1 decoding."""
import numpy as np
import pytest

import oracle
import synth
from gpu_harness import THRESHOLD, base_tol, first_divergence, new_decoder, top2_gap

pytestmark = pytest.mark.gpu

TINY = synth.WORKLOADS["tiny_f32"].model
FXT = synth.TINY_FXT


def _pair(seed_d, seed_v, gain, same):
    raw_d = synth.make_weights(TINY, seed=seed_d, logit_gain=gain)
    if same:
        return raw_d, raw_d, TINY
    return raw_d, synth.make_weights(FXT, seed=seed_v, logit_gain=gain), FXT


def _verifier_logits(Wv, cfg_v, x, drafts):
    """The verifier's next-byte logits after x ++ drafts[:m], m = 0..n."""
    rows = []
    for m in range(len(drafts) + 1):
        seq = np.asarray(list(x) + [int(c) for c in drafts[:m]], np.int64)
        tr = oracle.trunk(Wv, cfg_v, seq)
        rows.append(oracle.head_logits(tr["h1"][-1], Wv["nt_norm"], Wv, cfg_v.rms_eps))
    return np.stack(rows)


@pytest.mark.parametrize("same,gain,n", [(False, 1.0, 3), (False, 30.0, 5), (True, 30.0, 4), (True, 30.0, 7)])
def test_external_verify_tiny_per_step(same, gain, n):
    raw_d, raw_v, cfg_v = _pair(40, 41, gain, same)
    Wv = oracle.to_float64(raw_v)
    tol = base_tol(TINY) * max(gain, 1.0)
    D = new_decoder(TINY, raw_d, 1, 400)
    V = new_decoder(cfg_v, raw_v, 1, 400)
    p = synth.make_prompt(6, 120)
    D.prefill([p])
    V.prefill([p])
    x = [int(b) for b in p]
    kept, exempt = 0, 0
    for step in range(10):
        cand, _, _ = D.decode_step(n, 1.0, THRESHOLD)
        drafts = cand[0].cpu().numpy().copy()
        out, ln = V.verify_draft(cand)
        k = int(ln[0].item())
        got = out[0, :k].cpu().numpy()
        ref_l = _verifier_logits(Wv, cfg_v, x, drafts)
        err = float(np.max(np.abs(V.logits()[0].double().cpu().numpy() - ref_l)))
        assert err <= tol, f"step {step}: verifier logits differ by {err:.3g}"
        ref = oracle.verify_external(Wv, cfg_v, x, drafts)
        if k != ref["k"] or not np.array_equal(got, ref["bytes"]):
            span = min(n + 1, max(k, ref["k"]))
            assert any(top2_gap(ref_l[m]) < 2 * tol for m in range(span)), (step, k, ref["k"], got, ref["bytes"])
            exempt += 1
            V.accept([ref["bytes"]])  # teacher forcing: roll back and commit the oracle's bytes
        else:
            V.accept()
        D.accept([ref["bytes"]])
        x += [int(b) for b in ref["bytes"]]
        kept += ref["k"] - 1
        assert D.row_length(0) == V.row_length(0) == len(x)
    print(f"kept drafts {kept}, exempt steps {exempt}")
    if same:  # the drafting model's first draft is its own greedy byte
        assert kept >= 10


@pytest.mark.parametrize("same,gain,n", [(False, 30.0, 3), (True, 30.0, 5)])
def test_external_free_running_equals_verifier_greedy(same, gain, n):
    raw_d, raw_v, cfg_v = _pair(42, 43, gain, same)
    Wv = oracle.to_float64(raw_v)
    tol = base_tol(TINY) * gain
    D = new_decoder(TINY, raw_d, 1, 400)
    V = new_decoder(cfg_v, raw_v, 1, 400)
    p = synth.make_prompt(7, 100)
    D.prefill([p])
    V.prefill([p])
    outb, ks = [], []
    while len(outb) < 24:
        cand, _, _ = D.decode_step(n, 1.0, THRESHOLD)
        out, ln = V.verify_draft(cand)
        acc = out[0, : int(ln[0].item())].cpu().numpy()
        ks.append(len(acc))
        D.accept([acc])
        V.accept()
        outb += [int(b) for b in acc]
    ref = oracle.greedy_generate(Wv, cfg_v, p, 24)
    i = first_divergence(outb[:24], ref)
    if i is not None:  # only at a near-tie of the verifier's greedy byte
        tr = oracle.trunk(Wv, cfg_v, np.asarray(list(p) + [int(b) for b in ref[:i]], np.int64))
        l1 = oracle.head_logits(tr["h1"][-1], Wv["nt_norm"], Wv, cfg_v.rms_eps)
        assert top2_gap(l1) < 2 * tol, f"diverged at byte {i}"
    assert all(1 <= k <= n + 1 for k in ks)
    if same:
        assert max(ks) >= 2


def test_external_pending_bonus_decode_step_and_override():
    raw = synth.make_weights(TINY, seed=44, logit_gain=30.0)
    W = oracle.to_float64(raw)
    D = new_decoder(TINY, raw, 1, 400)
    V = new_decoder(TINY, raw, 1, 400)  # a verifier with an MB head can also decode
    p = synth.make_prompt(8, 90)
    D.prefill([p])
    V.prefill([p])
    x = [int(b) for b in p]
    cand, _, _ = D.decode_step(4, 1.0, THRESHOLD)
    out, ln = V.verify_draft(cand)
    acc = [int(b) for b in out[0, : int(ln[0].item())].cpu().numpy()]
    assert acc == [int(b) for b in oracle.verify_external(W, TINY, x, cand[0].cpu().numpy())["bytes"]]
    V.accept()
    x += acc
    assert V.row_length(0) == len(x)
    # a decode step first commits the pending bonus byte: candidate 1 is the greedy byte after x
    c2, _, _ = V.decode_step(3, 0.5, THRESHOLD)
    ref = oracle.step(W, TINY, x, 3, 0.5)
    assert int(c2[0, 0].item()) == int(ref["cand"][0])
    np.testing.assert_allclose(V.logits()[0].double().cpu().numpy(), ref["logits"], atol=base_tol(TINY) * 30)
    V.accept([[70, 71]])
    x += [70, 71]
    assert V.row_length(0) == len(x)
    # an override after a verification rolls back its drafts and its bonus byte
    D.accept([acc + [70, 71]])
    cand, _, _ = D.decode_step(5, 1.0, THRESHOLD)
    V.verify_draft(cand)
    V.accept([[72, 73, 74]])
    x += [72, 73, 74]
    assert V.row_length(0) == len(x)
    c3, _, _ = V.decode_step(1, 0.5, THRESHOLD)
    assert int(c3[0, 0].item()) == int(oracle.step(W, TINY, x, 1, 0.5)["cand"][0])
    V.accept()
    x += [int(oracle.step(W, TINY, x, 1, 0.5)["cand"][0])]
    # an override after a verification closed with accept(None): the verifier's pending
    # bonus byte was accepted first, so it precedes the override bytes
    D.reset()
    D.prefill([np.array(x, np.uint8)])
    cand, _, _ = D.decode_step(4, 1.0, THRESHOLD)
    out, ln = V.verify_draft(cand)
    acc = [int(b) for b in out[0, : int(ln[0].item())].cpu().numpy()]
    assert acc == [int(b) for b in oracle.verify_external(W, TINY, x, cand[0].cpu().numpy())["bytes"]]
    V.accept()
    V.accept([[75, 76]])
    x += acc + [75, 76]
    assert V.row_length(0) == len(x)
    c4, _, _ = V.decode_step(3, 0.5, THRESHOLD)
    ref = oracle.step(W, TINY, x, 3, 0.5)
    np.testing.assert_allclose(V.logits()[0].double().cpu().numpy(), ref["logits"], atol=base_tol(TINY) * 30)
    V.accept()


def test_external_verify_d1024_engine_equals_verifier_greedy():
    """d=1024 bf16 drafter (2/16/2/2 LCA) and FxT verifier (2/16/4) on the engine path:
    the external loop's bytes equal the verifier's own next-byte decoding (a separate
    handle, n = 1), except at a near-tie of that decoding's greedy byte."""
    wl = synth.WORKLOADS["extverify_d1024_b1"]
    raw_d = synth.make_weights(wl.model, seed=0, logit_gain=30.0)
    raw_v = synth.make_weights(wl.verifier, seed=1, logit_gain=30.0)
    p = synth.make_prompt(9, 512)
    D = new_decoder(wl.model, raw_d, 1, 700)
    V = new_decoder(wl.verifier, raw_v, 1, 700)
    G = new_decoder(wl.verifier, raw_v, 1, 700)
    for dec in (D, V, G):
        dec.prefill([p])
    outb, ks = [], []
    while len(outb) < 40:
        cand, _, _ = D.decode_step(wl.n, 1.0, THRESHOLD)
        out, ln = V.verify_draft(cand)
        acc = out[0, : int(ln[0].item())].cpu().numpy()
        ks.append(len(acc))
        D.accept([acc])
        V.accept()
        outb += [int(b) for b in acc]
    greedy, gaps = [], []
    for _ in range(40):
        c, _, _ = G.decode_step(1, 0.5, THRESHOLD)
        gaps.append(top2_gap(G.logits()[0, 0].double().cpu().numpy()))
        greedy.append(int(c[0, 0].item()))
        G.accept()
    i = first_divergence(outb[:40], greedy)
    print(f"ks {ks}; divergence {i}")
    if i is not None:
        assert gaps[i] < 2 * base_tol(wl.model), f"diverged at byte {i} (gap {gaps[i]:.3g})"
    assert all(1 <= k <= wl.n + 1 for k in ks)


def test_external_verify_tiny_perfect_and_corrupted_drafts():
    """Drafts taken from the verifier's own greedy continuation are all kept (k = n+1,
    the bonus being the next greedy byte); one corrupted draft at m keeps exactly m."""
    import torch
    raw_v = synth.make_weights(FXT, seed=46, logit_gain=30.0)
    Wv = oracle.to_float64(raw_v)
    tol = base_tol(FXT) * 30.0
    V = new_decoder(FXT, raw_v, 1, 400)
    p = synth.make_prompt(10, 80)
    V.prefill([p])
    x = [int(b) for b in p]
    for step, n in enumerate((3, 5, 7, 4, 6, 2)):
        g = oracle.greedy_generate(Wv, FXT, x, n + 1)
        drafts = g[:n].copy()
        bad = step % 2 == 1
        if bad:
            drafts[step % n] = (int(drafts[step % n]) + 1) % 256
        out, ln = V.verify_draft(torch.tensor(drafts[None, :], dtype=torch.uint8, device="cuda"))
        k = int(ln[0].item())
        ref = oracle.verify_external(Wv, FXT, x, drafts)
        assert ref["k"] == ((step % n) + 1 if bad else n + 1)
        if k != ref["k"]:
            ref_l = _verifier_logits(Wv, FXT, x, drafts)
            assert any(top2_gap(ref_l[m]) < 2 * tol for m in range(min(n + 1, max(k, ref["k"])))), (step, k)
            V.accept([ref["bytes"]])
        else:
            np.testing.assert_array_equal(out[0, :k].cpu().numpy(), ref["bytes"])
            V.accept()
        x += [int(b) for b in ref["bytes"]]
        assert V.row_length(0) == len(x)


def test_external_verify_d1024_perfect_drafts():
    """d=1024 FxT verifier, engine path: the verifier's own greedy continuation (from a
    second handle decoding n = 1) as the drafts is kept whole, and the bonus byte is
    the next byte of that continuation (near-ties of the greedy byte excepted)."""
    import torch
    wl = synth.WORKLOADS["extverify_d1024_b1"]
    raw_v = synth.make_weights(wl.verifier, seed=2, logit_gain=30.0)
    p = synth.make_prompt(11, 512)
    V = new_decoder(wl.verifier, raw_v, 1, 700)
    G = new_decoder(wl.verifier, raw_v, 1, 700)
    V.prefill([p])
    G.prefill([p])
    for n in (7, 3, 5):
        greedy, gaps = [], []
        for _ in range(n + 1):
            c, _, _ = G.decode_step(1, 0.5, THRESHOLD)
            gaps.append(top2_gap(G.logits()[0, 0].double().cpu().numpy()))
            greedy.append(int(c[0, 0].item()))
            G.accept()
        if min(gaps) < 2 * base_tol(wl.verifier):
            pytest.skip("near-tie in the greedy continuation")
        out, ln = V.verify_draft(torch.tensor([greedy[:n]], dtype=torch.uint8, device="cuda"))
        assert int(ln[0].item()) == n + 1
        assert [int(b) for b in out[0].cpu().numpy()] == greedy
        V.accept()
        assert V.row_length(0) == G.row_length(0)
