"""GPU parity at the workloads' full sizes, against oracle outputs stored by
``tests/golden/make_large.py`` (the float64 oracle needs minutes per case, so it runs
offline; the stored values come from ``oracle`` and ``synth`` only).

* batch 64, 2048-byte prompts, n = 5, every tau of the workload (0.5, 0.75, 0.9):
  all 64 rows compared element-wise at each step; the commits of more than 16 rows
  run on the matrix-core GEMM path;
* d=2048, batch 16, 8192-byte contexts, n = 7 self-verification: two stored rows
  compared with all 16 running, their accepted bytes equal the oracle's greedy bytes;
* the batch-1 workload at its 4096-byte prompt through a forced segment end, so that
  a commit runs the LM module and the next step's MB window starts a new group.

Comparison rule: the one of ``gpu_harness.compare_step`` (logits within the absolute
tolerance, exempt candidates by their top-1 / top-2 gap, probabilities within 3x the
tolerance), with the accepted count checked twice: it must be the acceptance rule
applied to the library's own probabilities exactly, and equal to the oracle's count
except where an inspected oracle probability lies within max(1e-3, the library's
error on that probability) of tau.
"""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_harness import SELF_VERIFY, THRESHOLD, TAU_BAND, new_decoder, top2_gap

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TOL = 2e-2  # bfloat16 logit tolerance, unscaled by the logit gain


def _load(case):
    p = os.path.join(GOLDEN, f"large_{case}.npz")
    if not os.path.exists(p):
        pytest.skip(f"{p} missing: run tests/golden/make_large.py {case}")
    return np.load(p)


def _check_row(where, g_logits, g_cand, g_prob, g_k, ref_logits, ref_cand, ref_prob, n, tau, counts):
    err = float(np.max(np.abs(g_logits - ref_logits)))
    counts["max_err"] = max(counts["max_err"], err)
    assert err <= TOL, f"{where}: logits differ by {err:.3g}"
    exempt = [top2_gap(ref_logits[m]) < 2 * TOL for m in range(n)]
    for m in range(n):
        if int(g_cand[m]) != int(ref_cand[m]):
            assert exempt[m], f"{where}: candidate {m} = {g_cand[m]} vs oracle {ref_cand[m]}"
            counts["cand_exempt"] += 1
    dp = np.abs(g_prob - ref_prob)
    assert np.all(dp <= 3 * TOL), f"{where}: probabilities differ by {dp.max():.3g}"
    if tau is None:
        return
    # the kernel's decision on its own probabilities is exact
    assert int(g_k) == oracle.threshold_accept(np.asarray(g_prob, np.float64), tau), f"{where}: accept rule"
    ref_k = oracle.threshold_accept(ref_prob, tau)
    counts["accepted"] += ref_k
    if int(g_k) != ref_k:
        span = min(n, max(int(g_k), ref_k) + 1)
        narrow = any(abs(ref_prob[m] - tau) < TAU_BAND for m in range(1, span)) or any(exempt[:span])
        near = narrow or any(abs(ref_prob[m] - tau) < dp[m] for m in range(1, span))
        assert near, f"{where}: accepted {g_k} vs oracle {ref_k} (probs {ref_prob}, tau {tau})"
        counts["k_exempt"] += 1
        counts["k_exempt_wide"] += 0 if narrow else 1


@pytest.mark.timeout(900)
def test_batch64_full_size_every_tau():
    gd = _load("lca_d1024_b64")
    model = synth.WORKLOADS["lca_d1024_b64"].model
    n, B, P = int(gd["n"]), int(gd["batch"]), int(gd["prompt"])
    raw = synth.make_weights(model, seed=0, logit_gain=float(gd["gain"]))
    prompts = [synth.make_prompt(r, P) for r in range(B)]
    dec = new_decoder(model, raw, B, P + 64)
    dec.prefill(prompts)
    counts = dict(max_err=0.0, cand_exempt=0, k_exempt=0, k_exempt_wide=0, accepted=0)
    zero = [np.zeros(0, np.uint8)] * B
    steps = gd["logits"].shape[0]
    for s in range(steps):
        for tau in (0.5, 0.9, 0.75):  # 0.75 last: its bytes are the ones committed
            cand, prob, alen = dec.decode_step(n, tau)
            logits = dec.logits().double().cpu().numpy()
            cand, prob, alen = cand.cpu().numpy(), prob.cpu().numpy(), alen.cpu().numpy()
            for b in range(B):
                _check_row(f"step {s} tau {tau} row {b}", logits[b], cand[b], prob[b], alen[b], gd["logits"][s, b],
                           gd["cand"][s, b], gd["prob"][s, b], n, tau, counts)
            if tau != 0.75:
                dec.accept(zero)  # closes the step, commits nothing
        forced = [gd["forced"][s, b, : gd["forced_len"][s, b]] for b in range(B)]
        if s == 0:
            dec.set_timing(True)
        dec.accept(forced)
        if s == 0:
            t = dec.read_timing()
            dec.set_timing(False)
            # a commit of sum(k) > 16 rows runs the linear layers on the matrix-core GEMM
            assert sum(len(f) for f in forced) > 16
            assert t["gemm"][0] > 0, t
    print(counts)
    assert counts["accepted"] > 3 * steps * B  # acceptance is ragged, not one byte per row


@pytest.mark.timeout(900)
def test_verify_d2048_full_size():
    gd = _load("verify_d2048_b16")
    model = synth.WORKLOADS["verify_d2048_b16"].model
    n, B, P = int(gd["n"]), int(gd["batch"]), int(gd["prompt"])
    rows = [int(r) for r in gd["rows"]]
    raw = synth.make_weights(model, seed=0, logit_gain=float(gd["gain"]))
    prompts = [synth.make_prompt(r, P) for r in range(B)]
    dec = new_decoder(model, raw, B, P + 64)
    dec.prefill(prompts)
    counts = dict(max_err=0.0, cand_exempt=0, k_exempt=0, k_exempt_wide=0, accepted=0)
    for s in range(gd["logits"].shape[0]):
        cand, prob, alen = dec.decode_step(n, 0.0, SELF_VERIFY)
        logits = dec.logits().double().cpu().numpy()
        cand, prob, alen = cand.cpu().numpy(), prob.cpu().numpy(), alen.cpu().numpy()
        acc, lens = dec.last_accepted()
        forced = [acc[b, : lens[b]] for b in range(B)]
        for i, b in enumerate(rows):
            where = f"step {s} row {b}"
            _check_row(where, logits[b], cand[b], prob[b], None, gd["logits"][s, i], gd["cand"][s, i],
                       gd["prob"][s, i], n, None, counts)
            ref_k = int(gd["k"][s, i])
            if int(alen[b]) != ref_k:
                # a verified draft may differ only where a next-byte argmax is inside the error
                span = min(n, max(int(alen[b]), ref_k) + 1)
                near = any(gd["gap"][s, i, m] < 2 * TOL for m in range(span - 1))
                near = near or any(top2_gap(gd["logits"][s, i, m]) < 2 * TOL for m in range(span))
                assert near, f"{where}: accepted {alen[b]} vs oracle {ref_k}"
                counts["k_exempt"] += 1
            # the accepted bytes are the oracle's: c_1 is the next-byte greedy byte and
            # every kept draft equals the greedy byte after the drafts before it
            ref = gd["forced"][s, i, : gd["forced_len"][s, i]]
            greedy = [int(gd["cand"][s, i, 0])] + [int(v) for v in gd["gamma"][s, i] if v >= 0]
            assert [int(v) for v in ref] == greedy[: len(ref)]
            forced[b] = ref
            counts["accepted"] += len(ref)
        dec.accept(forced)
    print(counts)


@pytest.mark.timeout(900)
def test_batch1_prompt4096_lm_pass_and_new_group():
    gd = _load("lca_d1024_b1_lm")
    model = synth.WORKLOADS["lca_d1024_b1"].model
    n, P, tau = int(gd["n"]), int(gd["prompt"]), float(gd["tau"])
    raw = synth.make_weights(model, seed=0, logit_gain=float(gd["gain"]))
    dec = new_decoder(model, raw, 1, P + 64)
    dec.prefill([synth.make_prompt(0, P)])
    counts = dict(max_err=0.0, cand_exempt=0, k_exempt=0, k_exempt_wide=0, accepted=0)
    for s in range(gd["logits"].shape[0]):
        cand, prob, alen = dec.decode_step(n, tau)
        logits = dec.logits().double().cpu().numpy()
        _check_row(f"step {s}", logits[0], cand.cpu().numpy()[0], prob.cpu().numpy()[0], alen.cpu().numpy()[0],
                   gd["logits"][s, 0], gd["cand"][s, 0], gd["prob"][s, 0], n, tau, counts)
        forced = gd["forced"][s, 0, : gd["forced_len"][s, 0]]
        if s == 1:
            assert list(forced) == [0x20]
            before = dec.row_boundaries(0)
            dec.set_timing(True)
            dec.accept([forced])
            t = dec.read_timing()
            dec.set_timing(False)
            q = dec.row_boundaries(0)
            # the space closed a segment at the byte just committed ...
            assert len(q) == len(before) + 1 and q[-1] == dec.row_length(0) - 1
            # ... so the commit ran the LM module: the launches of the commit moved at
            # least the LM module's weights
            d, f = model.d_model, model.d_ff
            lm_weights = model.n_lm * (4 * d * d + 3 * d * f) * 2
            assert sum(v[2] for v in t.values()) >= lm_weights, t
        else:
            dec.accept([forced])
    print(counts)
