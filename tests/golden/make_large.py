"""Expected oracle outputs for the GPU parity tests at the workloads' full sizes.

Writes ``tests/golden/large_<case>.npz``.  Imports only ``oracle`` (the float64 CPU
definition) and ``synth`` (the seeded weights and prompts); nothing here comes from
the HIP library.  The oracle recomputes the whole sequence at every step, so these
take minutes (about 12 for ``lca_d1024_b64``, 10 for ``verify_d2048_b16``, 1 for
``lca_d1024_b1_lm`` on 8 cores); the GPU tests read the files instead of calling the
oracle.

    python tests/golden/make_large.py [case ...]      (default: every case)

Cases (teacher-forced: after every step both sides commit the bytes stored here):

* ``lca_d1024_b64`` -- the batch-64 workload: the d=1024 LCA model (logit gain 8, so
  that acceptance is ragged), 64 rows of 2048-byte prompts, n = 5, three steps.  The
  stored logits serve every tau of the workload (0.5, 0.75, 0.9); the forced bytes
  are the ones accepted at tau = 0.75.
* ``verify_d2048_b16`` -- the verification workload: the d=2048 model (logit gain 8),
  16 rows of 8192-byte contexts, n = 7 self-verification, two steps; rows 0 and 15
  are stored (the oracle's greedy bytes after each kept draft come with them).
* ``lca_d1024_b1_lm`` -- the batch-1 workload as specified (logit gain 1), its
  4096-byte prompt, n = 3, tau = 0.75, four steps; the bytes forced after step 1 are a
  single space, which closes a segment, so the commit runs the LM module and the
  next step's MB window starts a new group.
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

CASES = {
    "lca_d1024_b64": dict(model=synth.WORKLOADS["lca_d1024_b64"].model, gain=8.0, batch=64, prompt=2048, n=5,
                          steps=3, mode="threshold", tau=0.75, rows=list(range(64)), force={}),
    "verify_d2048_b16": dict(model=synth.WORKLOADS["verify_d2048_b16"].model, gain=8.0, batch=16, prompt=8192, n=7,
                             steps=2, mode="verify", tau=0.0, rows=[0, 15], force={}),
    "lca_d1024_b1_lm": dict(model=synth.WORKLOADS["lca_d1024_b1"].model, gain=1.0, batch=1, prompt=4096, n=3,
                            steps=4, mode="threshold", tau=0.75, rows=[0], force={1: [0x20]}),
}


def path(case: str) -> str:
    return os.path.join(HERE, f"large_{case}.npz")


def make(case: str) -> None:
    c = CASES[case]
    model, n, S, rows = c["model"], c["n"], c["steps"], c["rows"]
    t0 = time.time()
    W = oracle.to_float64(synth.make_weights(model, seed=0, logit_gain=c["gain"]))
    R = len(rows)
    logits = np.zeros((S, R, n, 256), np.float32)
    cand = np.zeros((S, R, n), np.uint8)
    prob = np.zeros((S, R, n), np.float64)
    k = np.zeros((S, R), np.int32)
    gamma = np.full((S, R, n), -1, np.int32)  # verify: the greedy bytes seen after each draft prefix
    gap = np.full((S, R, n), np.inf)  # verify: top-1 / top-2 logit gaps of those next-byte rows
    forced = np.zeros((S, R, 8), np.uint8)
    forced_len = np.zeros((S, R), np.int32)
    for i, r in enumerate(rows):
        x = [int(b) for b in synth.make_prompt(r, c["prompt"])]
        for s in range(S):
            if c["mode"] == "threshold":
                ref = oracle.step(W, model, x, n, c["tau"])
            else:
                ref = oracle.verify_step(W, model, x, n)
                gamma[s, i, : len(ref["gamma"])] = ref["gamma"]
                for m, row in enumerate(ref["nt_seen"]):
                    top = np.sort(row)
                    gap[s, i, m] = top[-1] - top[-2]
            logits[s, i] = ref["logits"]
            cand[s, i] = ref["cand"]
            prob[s, i] = ref["prob"]
            k[s, i] = ref["k"]
            acc = c["force"].get(s, [int(b) for b in ref["cand"][: ref["k"]]])
            forced[s, i, : len(acc)] = acc
            forced_len[s, i] = len(acc)
            x += acc
            print(f"[{case}] row {r} step {s}: k={ref['k']} ({time.time() - t0:.0f}s)", flush=True)
    np.savez_compressed(path(case), rows=np.asarray(rows, np.int32), logits=logits, cand=cand, prob=prob, k=k,
                        gamma=gamma, gap=gap, forced=forced, forced_len=forced_len, gain=c["gain"], n=n, tau=c["tau"],
                        prompt=c["prompt"], batch=c["batch"])
    print(f"[{case}] wrote {path(case)} in {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    for name in sys.argv[1:] or list(CASES):
        make(name)
