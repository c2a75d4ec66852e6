"""Shared helpers of the GPU parity tests: run the HIP library step by step against
the CPU oracle on identical seeded inputs.

Comparison rule (the oracle decides):
  * logits of every candidate row within ``tol`` (absolute);
  * candidate bytes equal, except a row whose oracle top-1 / top-2 logit gap is
    below 2*tol (an argmax inside the allowed logit error);
  * probabilities within 3*tol (absolute; a logit error d moves P by at most ~2dP);
  * accepted counts equal, except at a step where some oracle probability that the
    rule inspects lies within 1e-3 of tau, or a candidate it inspects is exempt.
Teacher forcing: after each step both sides commit the oracle's accepted bytes, so
every step is compared on the same byte sequence.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_15454_amd import SELF_VERIFY, THRESHOLD, Decoder, make_config

TAU_BAND = 1e-3


def base_tol(model) -> float:
    return 1e-5 if model.dtype == "f32" else 2e-2


def top2_gap(row) -> float:
    s = np.sort(np.asarray(row, np.float64))
    return float(s[-1] - s[-2])


def nt_gaps_after(W, model, x, drafts, upto):
    """Top-1/top-2 gaps of the next-byte head after x ++ drafts[:m], m = 1..upto."""
    gaps = []
    for m in range(1, upto + 1):
        seq = np.concatenate([np.asarray(x, np.int64), np.asarray(drafts[:m], np.int64)])
        tr = oracle.trunk(W, model, seq)
        l1 = oracle.head_logits(tr["h1"][-1], W["nt_norm"], W, model.rms_eps)
        gaps.append(top2_gap(l1))
    return gaps


class Stats:
    def __init__(self):
        self.steps = 0
        self.exempt = 0
        self.max_err = 0.0
        self.accepted = 0
        self.timing = None  # kernel classes of the decode steps (forced_run with timing=True)

    def __repr__(self):
        return f"Stats(steps={self.steps}, exempt={self.exempt}, max_err={self.max_err:.3g}, accepted={self.accepted})"


def compare_step(ref, logits, cand, prob, k, n, tau, tol, mode, W=None, model=None, x=None, stats=None, where=""):
    err = float(np.max(np.abs(logits - ref["logits"])))
    if stats is not None:
        stats.max_err = max(stats.max_err, err)
    assert err <= tol, f"{where}: logits differ by {err:.3g} > {tol:.3g}"
    cand_exempt = [top2_gap(ref["logits"][m]) < 2 * tol for m in range(n)]
    for m in range(n):
        if int(cand[m]) != int(ref["cand"][m]):
            assert cand_exempt[m], f"{where}: candidate {m} = {cand[m]} vs oracle {ref['cand'][m]} (gap {top2_gap(ref['logits'][m]):.3g})"
    assert np.all(np.abs(prob - ref["prob"]) <= 3 * tol), f"{where}: probabilities differ"
    if int(k) != int(ref["k"]):
        span = min(n, max(int(k), int(ref["k"])) + 1)
        if mode == THRESHOLD:
            near = any(abs(ref["prob"][m] - tau) < TAU_BAND for m in range(1, span))
        else:
            near = any(g < 2 * tol for g in nt_gaps_after(W, model, x, ref["cand"], span - 1))
        near = near or any(cand_exempt[:span])
        assert near, f"{where}: accepted {k} vs oracle {ref['k']} (probs {ref['prob']}, tau {tau})"
        if stats is not None:
            stats.exempt += 1


def new_decoder(model, W, batch, max_ctx, max_n=8, **kw):
    return Decoder(make_config(model, max_batch=batch, max_ctx=max_ctx, max_n=max_n, **kw), W)


def forced_run(dec, W, model, prompts, steps, n, tau, mode=THRESHOLD, tol=None, label="", timing=False):
    """Teacher-forced comparison over ``steps`` steps; returns Stats.  ``n`` is the
    candidate count of every step, or a list cycled over the steps.  ``timing``: count
    the kernel launches of the compared steps (not the prefill) into Stats.timing."""
    tol = base_tol(model) if tol is None else tol
    dec.prefill(prompts)
    if timing:
        dec.set_timing(True)
    xs = [[int(b) for b in p] for p in prompts]
    st = Stats()
    ns = list(n) if isinstance(n, (list, tuple)) else [n]
    for s in range(steps):
        n = ns[s % len(ns)]
        refs = [oracle.step(W, model, x, n, tau) if mode == THRESHOLD else oracle.verify_step(W, model, x, n)
                for x in xs]
        cand, prob, alen = dec.decode_step(n, tau, mode)
        logits = dec.logits().double().cpu().numpy()
        cand, prob, alen = cand.cpu().numpy(), prob.cpu().numpy(), alen.cpu().numpy()
        for b, r in enumerate(refs):
            compare_step(r, logits[b], cand[b], prob[b], alen[b], n, tau, tol, mode, W, model, xs[b], st,
                         where=f"{label} step {s} row {b}")
        acc = [r["cand"][: r["k"]] for r in refs]
        dec.accept(acc)
        for b, a in enumerate(acc):
            xs[b] += [int(c) for c in a]
            st.accepted += len(a)
        st.steps += 1
    st.seqs = xs  # the committed byte sequences the run ended on
    if timing:
        st.timing = dec.read_timing()
        dec.set_timing(False)
    return st


def free_run(dec, prompts, n_new, n, tau, mode=THRESHOLD):
    """The library generating on its own (accepting its own bytes); per-row outputs."""
    dec.prefill(prompts)
    outs = [[] for _ in prompts]
    ks = []
    while min(len(o) for o in outs) < n_new:
        dec.decode_step(n, tau, mode)
        acc, lens = dec.last_accepted()
        dec.accept()
        ks.append(lens.copy())
        for b in range(len(prompts)):
            outs[b] += [int(c) for c in acc[b, : lens[b]]]
    return [np.array(o[:n_new], dtype=np.uint8) for o in outs], ks


def first_divergence(a, b):
    n = min(len(a), len(b))
    for i in range(n):
        if int(a[i]) != int(b[i]):
            return i
    return None


def divergence_is_exempt(W, model, prompt, ref_out, ref_steps, index, n, tau, tol, mode=THRESHOLD):
    """Whether the oracle step that emitted byte ``index`` is an exempt step."""
    pos = 0
    x = [int(v) for v in prompt]
    for st in ref_steps:
        k = st["k"]
        if pos + k > index:
            if mode == THRESHOLD:
                if any(abs(st["prob"][m] - tau) < TAU_BAND for m in range(1, n)):
                    return True
            logits = oracle.step_logits(W, model, x, n)
            if any(top2_gap(logits[m]) < 2 * tol for m in range(n)):
                return True
            if mode == SELF_VERIFY:
                return any(g < 2 * tol for g in nt_gaps_after(W, model, x, st["cand"], n - 1))
            return False
        x += [int(c) for c in ref_out[pos: pos + k]]
        pos += k
    return False
