#!/usr/bin/env python3
"""MBP decode benchmark on one MI355X: accepted bytes/s of the multi-byte-prediction
decode loop (decode step + commit of the accepted bytes), with the roofline of the
dominant kernel and the CPU oracle timed beside it.

Default workload: d=1024 bf16 LCA-MBP model (encoder 2, LM module 16, NT decoder 2,
MB head 2 layers, 16 heads), batch 1, 4096-byte seeded Zipf prompt with space-
delimited patches, n=3, tau=0.75, random N(0, 0.02) weights.

Protocol: prefill + W warm-up steps, reset + prefill again (untimed), then exactly K
timed steps.  A step is one decode_step (NT head, LCA window head, unembedding,
softmax / top-1 / tau acceptance) plus one accept (encoder, segmentation and pooling,
LM module when a segment closes, NT decoder) -- every stage of the hot path.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, vendor figure


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 1024; forward workloads 20)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 16; forward workloads 3)")
    ap.add_argument("--workload", default="lca_d1024_b1")
    ap.add_argument("--n", type=int, default=None)
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--logit-gain", type=float, default=1.0)
    ap.add_argument("--cpu-steps", type=int, default=1,
                    help="float64 full-recompute oracle steps timed beside the cached CPU baseline (0 = skip)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="seconds of float32 KV-cached CPU decoding timed, on all cores and on one (0 = skip)")
    ap.add_argument("--no-batch64", action="store_true", help="default workload only: skip the batch-64 runs")
    ap.add_argument("--no-timing-pass", action="store_true")
    ap.add_argument("--no-engine", action="store_true", help="one kernel launch per layer operation")
    return ap.parse_args()


def cpu_threads():
    try:
        from threadpoolctl import threadpool_info

        info = [i for i in threadpool_info() if i.get("internal_api") in ("openblas", "mkl", "blis")]
        if info:
            return int(info[0]["num_threads"])
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


# A plain device copy of known size launched just before the kernel-timing pass: in a
# profiler trace it marks where that pass starts, and its FETCH_SIZE / WRITE_SIZE
# readings scale the HBM counters of the kernels that follow.
COPY_CAL_BYTES = 256 << 20
# HBM traffic per launch of the dominant kernel class, from counter runs of this
# command (profiles/<class>_<workload>_hbm_counters.md), valid only while the code of
# the source the class is built from is the code that was measured.
CSRC = os.path.join(ROOT, "paper_2608_15454_amd", "csrc")
CLASS_SOURCE = {"engine": "engine.hip", "gemv": "kernels.hip", "gemm": "kernels.hip", "attention": "kernels.hip",
                "other": "kernels.hip"}


def traffic_key(workload, logit_gain=1.0):
    """The name a counter record is filed under: the workload, plus the logit gain when it
    is not the workload's own (acceptance, and so the launches, differ with it)."""
    return workload if logit_gain == 1.0 else f"{workload}_gain{logit_gain:g}"


def code_digest(path):
    """sha256 of a C++ / HIP source with its comments removed and its whitespace
    collapsed: edits to comments or layout leave it, and so a counter record, valid."""
    import hashlib
    import re

    src = open(path).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    src = re.sub(r"\s+", " ", src).strip()
    return hashlib.sha256(src.encode()).hexdigest()


def measured_traffic(kernel_class, workload):
    """Bytes per launch recorded for kernel_class on workload, or None when there is no
    record or the code of the class's source has changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel_class}_{workload}_hbm_counters.md")
    source = CLASS_SOURCE.get(kernel_class)
    if source is None or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get(f"{source} code sha256") != code_digest(os.path.join(CSRC, source)) \
            or fields.get("class") != kernel_class or fields.get("workload") != workload:
        return None
    return int(fields["hbm bytes per launch"])


def run_steps(dec, steps, n, tau, mode, samp=None):
    """samp: (temperature, top_p, uniforms [steps, B, 3n] on the device) for sampled
    decoding."""
    for i in range(steps):
        if samp:
            dec.decode_step_sampled(n, tau, mode, samp[0], samp[1], samp[2][i])
        else:
            dec.decode_step(n, tau, mode)
        dec.accept()


def run_external(dec, ver, steps, n, threshold):
    """External verification: dec drafts n candidates, ver keeps the verified prefix and
    adds its greedy byte; both commit the accepted bytes."""
    for _ in range(steps):
        cand, _, _ = dec.decode_step(n, 1.0, threshold)
        ver.verify_draft(cand)
        acc, lens = ver.last_accepted()
        dec.accept([acc[b, : lens[b]] for b in range(len(lens))])
        ver.accept()


MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 / fp16 matrix cores, vendor figure
VALU_FP32_PEAK_TFLOPS = 157.3   # MI355X fp32 vector


def forward_flops(model, T, q):
    """Algorithmic flops of one full-sequence forward: (linear, attention).  Linear:
    2 per weight per row (encoder, NT and MB layers on T rows, the LM module on the
    K+1 latent rows, the unembedding twice on T rows).  Attention: 4 d per visible
    (query, key) pair (scores and the weighted sum): causal in the encoder, LM module
    and NT decoder; under the LCA mask a position sees its own group up to itself and
    the previous group."""
    d, dff = model.d_model, model.d_ff
    per_layer = 4 * d * d + 3 * d * dff
    K1 = len(q) + 1
    linear = 2.0 * per_layer * (T * (model.n_enc + model.n_nb + model.n_mb) + K1 * model.n_lm) + 2 * 2.0 * T * 256 * d
    starts = [0] + list(q)  # first byte of each group
    lca, g = 0, 0
    for i in range(T):
        while g < len(q) and q[g] <= i:
            g += 1
        lca += i + 1 - (starts[g - 1] if g >= 1 else 0)
    causal = T * (T + 1) / 2
    pairs = (model.n_enc + model.n_nb) * causal + model.n_lm * K1 * (K1 + 1) / 2 + model.n_mb * lca
    return linear, 4.0 * d * pairs


def bench_forward(args, wl):
    """One step = one full-sequence forward of the workload's sequence (both heads at
    every position, the losses); value = bytes of sequence processed per second."""
    import numpy as np
    import torch

    import synth
    from paper_2608_15454_amd import Decoder, make_config

    model, T = wl.model, wl.prompt_len
    K = 20 if args.steps is None else args.steps
    W = 3 if args.warmup is None else args.warmup
    log(f"[bench] workload {wl.name} T={T} steps={K} warmup={W}")
    weights = synth.make_weights(model, seed=0, logit_gain=args.logit_gain)
    x = synth.make_prompt(0, T)
    dec = Decoder(make_config(model, max_batch=1, max_ctx=T + 8, engine=not args.no_engine), weights)
    work = None
    for _ in range(max(W, 1)):
        nll, loss = dec.forward(x, work=work)
        work = dec.fwork
    dec.prefill([x])  # the segmentation, for the flop count (a host read, untimed)
    q = [int(v) for v in dec.row_boundaries(0)]
    dec.reset()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    w0 = time.perf_counter()
    for _ in range(K):
        nll, loss = dec.forward(x, work=work)
    ev1.record(stream)
    torch.cuda.synchronize()
    elapsed = max(time.perf_counter() - w0, ev0.elapsed_time(ev1) / 1000.0)
    value = K * T / elapsed
    lv = loss.double().cpu().numpy()
    log(f"[bench] timed: {K} forwards {elapsed * 1000:.1f} ms, {value:.0f} B/s, losses {lv}")

    lin, att = forward_flops(model, T, q)
    roofline, classes = None, {}
    if not args.no_timing_pass:
        dec.set_timing(True)
        cal_src = torch.empty(COPY_CAL_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        cal_dst = torch.empty_like(cal_src)
        torch.cuda.synchronize()
        cal_dst.copy_(cal_src)
        torch.cuda.synchronize()
        del cal_src, cal_dst
        for _ in range(K):
            dec.forward(x, work=work)
        torch.cuda.synchronize()
        classes = dec.read_timing()
        dec.set_timing(False)
        dom = max(classes, key=lambda c: classes[c][1])
        launches, ms, nbytes = classes[dom]
        flops = {"gemm": lin * K, "attention": att * K}.get(dom)
        if flops is not None:
            # bf16 weights: the linear layers run on bf16 MFMAs and the attention (float16
            # caches, head size 64) on float16 MFMAs, both 2.5 PFLOP/s dense; float32
            # models stay on the vector ALUs
            mfma = model.dtype == "bf16" and (dom == "gemm" or model.d_head == 64)
            peak = MFMA_BF16_PEAK_TFLOPS if mfma else VALU_FP32_PEAK_TFLOPS
            achieved = flops / (ms / 1000.0) / 1e12
            roofline = {"bound": "mfma" if mfma else "alu",
                        "kernel": f"{dom} (all launches of the class in the timed forwards)",
                        "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                        "frac": round(achieved / peak, 4), "traffic": measured_traffic(dom, wl.name),
                        "launches": launches, "avg_launch_us": round(ms * 1000.0 / max(launches, 1), 3),
                        "flops_per_launch": round(flops / max(launches, 1)),
                        "bytes_per_launch": round(nbytes / max(launches, 1))}
        log("[bench] kernel classes: " + ", ".join(f"{k}: {v[0]} launches {v[1]:.1f} ms" for k, v in classes.items()))

    cpu = None
    if args.cpu_steps > 0:
        import oracle

        W64 = oracle.to_float64(weights)
        Tc = 512
        c0 = time.perf_counter()
        oracle.forward_losses(W64, model, x[:Tc])
        cs = time.perf_counter() - c0
        cpu = {"value": round(Tc / cs, 2), "unit": "bytes/s", "cores": cpu_threads(), "kind": "oracle",
               "sample": f"one forward of the first {Tc} bytes of the sequence (float64, {cs:.1f}s)"}
        log(f"[bench] cpu oracle {Tc} bytes in {cs:.1f}s")
    out = {
        "metric": "full-sequence forward bytes/s", "value": round(value, 1), "unit": "bytes/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(elapsed * 1000.0 / K, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": model.dtype, "data": "synthetic",
        "config": {"workload": f"{wl.name}: d={model.d_model} heads={model.n_heads} layers enc/lm/nt/mb="
                               f"{model.n_enc}/{model.n_lm}/{model.n_nb}/{model.n_mb}, one {T}-byte sequence, "
                               f"{len(q)} segments, both heads at every position and the losses",
                   "seq_len": T, "segments": len(q), "weights": model.dtype,
                   "kv_cache": "f16" if model.dtype == "bf16" else "f32"},
        "roofline": roofline, "cpu_baseline": cpu,
        "flops_per_step": {"linear": lin, "attention": att},
        "kernel_classes": {k: {"launches": v[0], "ms": round(v[1], 3)} for k, v in classes.items()},
        "losses": [round(float(v), 4) for v in lv],
    }
    print(json.dumps(out), flush=True)


def prefill_flops(model, lens, qs):
    """Algorithmic flops of a batch prefill: (linear, attention).  Linear: 2 per weight
    per row (encoder and NT layers on every prompt byte, the LM module on BOS and every
    closed segment).  Attention: 4 d per visible (query, key) pair, causal per row in
    the encoder, NT decoder and LM module."""
    d, dff = model.d_model, model.d_ff
    per_layer = 4 * d * d + 3 * d * dff
    T = sum(lens)
    K1 = [len(q) + 1 for q in qs]
    linear = 2.0 * per_layer * (T * (model.n_enc + model.n_nb) + sum(K1) * model.n_lm)
    pairs = sum((model.n_enc + model.n_nb) * L * (L + 1) / 2 + model.n_lm * k * (k + 1) / 2 for L, k in zip(lens, K1))
    return linear, 4.0 * d * pairs


def cpu_cached_baseline(model, weights, prompt, n, tau, mode, seconds):
    """The float32 KV-cached CPU decoder (oracle/cached.py) on row 0 of the workload:
    one prefill (reported, untimed), then steps for about ``seconds`` on all BLAS
    threads, and from the same prefilled state again on one thread."""
    import copy

    from threadpoolctl import threadpool_limits

    from oracle.cached import CachedDecoder

    dec = CachedDecoder(weights, model, cap=len(prompt) + 4096)
    p0 = time.perf_counter()
    dec.prefill([int(b) for b in prompt])
    pre = time.perf_counter() - p0
    start = copy.deepcopy(dec)
    out = {"prefill_s": pre}
    for label, threads in (("all", None), ("one", 1)):
        d = copy.deepcopy(start)
        with threadpool_limits(limits=threads):
            got, steps = 0, 0
            c0 = time.perf_counter()
            while time.perf_counter() - c0 < seconds:
                if mode == "verify":
                    got += d.verify_step(n)["k"]
                else:
                    r = d.step(n, tau)
                    acc = [int(c) for c in r["cand"][: r["k"]]]
                    d.accept(acc)
                    got += len(acc)
                steps += 1
            cs = time.perf_counter() - c0
        out[label] = {"value": got / cs, "steps": steps, "seconds": cs, "cores": cpu_threads() if threads is None else 1}
    return out


def bench_decode(args, wl, K, W, logit_gain, cpu_seconds=0.0, weights=None):
    """The decode loop of one workload: value, roofline of the dominant kernel class,
    the batch prefill's matrix-core figure, and (cpu_seconds > 0) the CPU baselines."""
    import torch

    import synth
    from paper_2608_15454_amd import SELF_VERIFY, THRESHOLD, Decoder, make_config

    model = wl.model
    n = args.n or wl.n
    tau = wl.tau if args.tau is None else args.tau
    mode = SELF_VERIFY if wl.mode == "verify" else THRESHOLD
    ext = wl.mode == "external"
    B = wl.batch
    log(f"[bench] workload {wl.name} B={B} prompt={wl.prompt_len} n={n} tau={tau} logit_gain={logit_gain} "
        f"steps={K} warmup={W}")

    t0 = time.time()
    if weights is None:
        weights = synth.make_weights(model, seed=0, logit_gain=logit_gain)
    prompts = [synth.make_prompt(r, wl.prompt_len) for r in range(B)]
    max_ctx = wl.prompt_len + (max(K, W) + 2) * (n + 1) + 16
    max_n = max(n + 1 if ext else n, 8)
    dec = Decoder(make_config(model, max_batch=B, max_ctx=max_ctx, max_n=max_n, engine=not args.no_engine), weights)
    ver, vweights = None, None
    if ext:
        vweights = synth.make_weights(wl.verifier, seed=1, logit_gain=logit_gain)
        ver = Decoder(make_config(wl.verifier, max_batch=B, max_ctx=max_ctx, max_n=max_n, engine=not args.no_engine),
                      vweights)
    decs = [dec] + ([ver] if ext else [])
    log(f"[bench] weights + init {time.time() - t0:.1f}s")

    # sampled decoding: every step's uniforms, generated before any timed region
    samp = None
    if wl.temperature > 0:
        gen = torch.Generator(device="cuda")
        gen.manual_seed(0)
        U = torch.rand((max(K, W), B, 3 * n), generator=gen, device="cuda", dtype=torch.float32)
        samp = (wl.temperature, wl.top_p, U)

    def run(steps):
        if ext:
            run_external(dec, ver, steps, n, THRESHOLD)
        else:
            run_steps(dec, steps, n, tau, mode, samp)

    stream = torch.cuda.current_stream()

    def timed(fn):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        w0 = time.perf_counter()
        fn()
        ev1.record(stream)
        torch.cuda.synchronize()
        return max(time.perf_counter() - w0, ev0.elapsed_time(ev1) / 1000.0)

    pre_s = timed(lambda: [d.prefill(prompts) for d in decs])
    log(f"[bench] prefill {pre_s * 1000:.1f} ms")
    run(W)
    torch.cuda.synchronize()
    log("[bench] warm-up done")

    # ---- prefill again, timed, then the timed decode steps
    for d in decs:
        d.reset()
    pre_s = timed(lambda: [d.prefill(prompts) for d in decs])
    elapsed = timed(lambda: run(K))
    lens = [(ver if ext else dec).row_length(b) for b in range(B)]
    accepted = sum(L - wl.prompt_len for L in lens)
    value = accepted / elapsed
    log(f"[bench] timed: {K} steps {elapsed * 1000:.1f} ms, accepted {accepted} bytes, {value:.1f} B/s")

    # ---- kernel timing pass (identical prefill and steps, launches bracketed by HIP events)
    roofline, classes, timing_step_ms, prefill = None, {}, None, None
    if not args.no_timing_pass:
        for d in decs:
            d.reset()
            d.set_timing(True)
        for d in decs:
            d.prefill(prompts)
        pcls = {}
        for d in decs:
            for k, v in d.read_timing().items():
                c = pcls.get(k, (0, 0.0, 0.0))
                pcls[k] = (c[0] + v[0], c[1] + v[1], c[2] + v[2])
            d.set_timing(False)
            d.set_timing(True)  # clears the totals: the decode steps are counted alone
        qs = [[int(v) for v in dec.row_boundaries(b)] for b in range(B)]
        lin, att = prefill_flops(model, [wl.prompt_len] * B, qs)
        mfma = model.dtype == "bf16"
        peak = MFMA_BF16_PEAK_TFLOPS if mfma else VALU_FP32_PEAK_TFLOPS
        gemm_ms = pcls["gemm"][1]
        prefill = {
            "ms": round(pre_s * 1000.0, 3), "tflop": round((lin + att) / 1e12, 3),
            "achieved_tflops": round((lin + att) / pre_s / 1e12, 2),
            "frac_of_peak": round((lin + att) / pre_s / 1e12 / peak, 4),
            "linear": {"tflop": round(lin / 1e12, 3), "kernel_ms": round(gemm_ms, 3),
                       "achieved_tflops": round(lin / (gemm_ms / 1000.0) / 1e12, 2) if gemm_ms > 0 else None,
                       "frac_of_peak": round(lin / (gemm_ms / 1000.0) / 1e12 / peak, 4) if gemm_ms > 0 else None},
            "peak_tflops": peak, "unit": "TFLOP/s", "bound": "mfma" if mfma else "alu",
            "kernel_classes": {k: {"launches": v[0], "ms": round(v[1], 3)} for k, v in pcls.items()},
        }
        log(f"[bench] prefill {prefill['tflop']} TFLOP in {prefill['ms']} ms: {prefill['achieved_tflops']} TFLOP/s; "
            f"linear layers {prefill['linear']['achieved_tflops']} TFLOP/s in their kernels")
        cal_src = torch.empty(COPY_CAL_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        cal_dst = torch.empty_like(cal_src)
        torch.cuda.synchronize()
        cal_dst.copy_(cal_src)
        torch.cuda.synchronize()
        w1 = time.perf_counter()
        run(K)
        torch.cuda.synchronize()
        timing_step_ms = (time.perf_counter() - w1) * 1000.0 / K
        del cal_src, cal_dst
        classes = {}
        for d in decs:  # both handles' launches (external verification)
            for k, v in d.read_timing().items():
                c = classes.get(k, (0, 0.0, 0.0))
                classes[k] = (c[0] + v[0], c[1] + v[1], c[2] + v[2])
            d.set_timing(False)
        dom = max(classes, key=lambda c: classes[c][1])
        launches, ms, nbytes = classes[dom]
        achieved = nbytes / (ms / 1000.0) / 1e9 if ms > 0 else 0.0
        roofline = {
            "bound": "hbm", "kernel": f"{dom} (all launches of the class in the timed steps)",
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(dom, traffic_key(wl.name, logit_gain)),
            "launches": launches, "avg_launch_us": round(ms * 1000.0 / max(launches, 1), 3),
            "bytes_per_launch": round(nbytes / max(launches, 1)),
        }
        log(f"[bench] kernel classes: " + ", ".join(f"{k}: {v[0]} launches {v[1]:.1f} ms {v[2] / 1e9:.2f} GB"
                                                     for k, v in classes.items()))

    # ---- CPU baselines beside it
    cpu = None
    if cpu_seconds > 0 and not ext and not samp and model.boundary == "space":
        c = cpu_cached_baseline(model, weights, prompts[0], n, tau, wl.mode, cpu_seconds)
        cpu = {"value": round(c["all"]["value"], 3), "unit": "accepted bytes/s", "cores": c["all"]["cores"],
               "kind": "oracle",
               "sample": f"batch row 0 of the same workload: {c['all']['steps']} steps ({c['all']['seconds']:.1f}s) "
                         f"after its {wl.prompt_len}-byte prefill ({c['prefill_s']:.1f}s, untimed), float32 "
                         f"KV-cached decoder of the oracle package (oracle/cached.py)",
               "one_core": {"value": round(c["one"]["value"], 3), "cores": 1, "steps": c["one"]["steps"],
                            "seconds": round(c["one"]["seconds"], 2)}}
        log(f"[bench] cpu cached decoder: {cpu['value']} B/s on {cpu['cores']} threads, "
            f"{cpu['one_core']['value']} B/s on one")
    if cpu_seconds > 0 and args.cpu_steps > 0:
        import oracle

        W64 = oracle.to_float64(weights)
        x = [int(b) for b in prompts[0]]
        got = 0
        c0 = time.perf_counter()
        V64 = oracle.to_float64(vweights) if ext else None
        nsteps = args.cpu_steps if not ext else min(args.cpu_steps, 1)
        for got_steps in range(nsteps):
            if ext:
                r = oracle.verify_external(V64, wl.verifier, x, oracle.step(W64, model, x, n, tau)["cand"])
                acc = [int(c) for c in r["bytes"]]
            elif samp:
                u = samp[2][got_steps, 0].double().cpu().numpy()
                if mode == THRESHOLD:
                    r = oracle.step_sampled(W64, model, x, n, tau, wl.temperature, wl.top_p, u)
                    acc = [int(c) for c in r["cand"][: r["k"]]]
                else:
                    acc = [int(c) for c in oracle.verify_step_sampled(W64, model, x, n, wl.temperature, wl.top_p,
                                                                      u)["bytes"]]
            else:
                r = oracle.step(W64, model, x, n, tau) if mode == THRESHOLD else oracle.verify_step(W64, model, x, n)
                acc = [int(c) for c in r["cand"][: r["k"]]]
            x += acc
            got += len(acc)
        cs = time.perf_counter() - c0
        full = {"value": round(got / cs, 4), "unit": "accepted bytes/s", "cores": cpu_threads(), "kind": "oracle",
                "sample": f"{nsteps} steps of batch row 0 of the same workload (float64 full recompute, {cs:.1f}s)"}
        log(f"[bench] cpu oracle (full recompute) {got} bytes in {cs:.1f}s")
        if cpu is None:
            cpu = full
        else:
            cpu["full_recompute"] = full

    step_bytes = sum(v[2] for v in classes.values()) / K if classes else None
    return {
        "value": round(value, 2),
        "ms_per_step": round(elapsed * 1000.0 / K, 4),
        "steps": K, "warmup": W,
        "config": {
            "workload": f"{wl.name}: d={model.d_model} heads={model.n_heads} layers enc/lm/nt/mb="
                        f"{model.n_enc}/{model.n_lm}/{model.n_nb}/{model.n_mb} head={model.head}, "
                        + (f"verified by a next-byte model with layers enc/lm/nt={wl.verifier.n_enc}/"
                           f"{wl.verifier.n_lm}/{wl.verifier.n_nb}, " if ext else "")
                        + (f"sampled at temperature {wl.temperature} top-p {wl.top_p}, " if samp else "")
                        + (f"learned boundaries (probe scale {model.bp_scale}, bias {model.bp_bias}), "
                           if model.boundary == "learned" else "")
                        + f"batch {B}, prompt {wl.prompt_len} bytes, n={n}, tau={tau}",
            "batch": B, "prompt_len": wl.prompt_len, "n": n, "tau": tau, "mode": wl.mode,
            "weights": model.dtype, "kv_cache": "f16" if model.dtype == "bf16" else "f32", "accumulate": "f32",
            "logit_gain": logit_gain, "max_patch": model.max_patch, "boundary": model.boundary,
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "prefill": prefill,
        "steps_per_s": round(K / elapsed, 2),
        "mean_accepted_per_step": round(accepted / (K * B), 4),
        "step_algorithmic_bytes": round(step_bytes) if step_bytes else None,
        "step_hbm_frac": round(step_bytes / (elapsed / K) / 1e9 / HBM_PEAK_GBS, 4) if step_bytes else None,
        "timing_pass_ms_per_step": round(timing_step_ms, 4) if timing_step_ms else None,
        "kernel_classes": {k: {"launches": v[0], "ms": round(v[1], 3), "GB": round(v[2] / 1e9, 4)}
                           for k, v in classes.items()},
        "_weights": weights,
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU; the decode rows are independent and would shard "
              "by batch row with no per-step exchange, but no multi-GPU run is provided.", file=sys.stderr)
        sys.exit(2)

    import synth

    wl = synth.WORKLOADS[args.workload]
    if wl.mode == "forward":
        return bench_forward(args, wl)
    K = 1024 if args.steps is None else args.steps
    W = 16 if args.warmup is None else args.warmup
    head = bench_decode(args, wl, K, W, args.logit_gain, cpu_seconds=args.cpu_seconds)
    weights = head.pop("_weights")
    out = {"metric": "accepted bytes/sec per MI355X (MBP decode)", "value": head.pop("value"),
           "unit": "accepted bytes/s", "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": head.pop("ms_per_step"),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.model.dtype,
           "data": "synthetic"}
    head.pop("steps"), head.pop("warmup")
    out.update(head)
    if args.workload == "lca_d1024_b1" and not args.no_batch64:
        # the metric's batch-64 half: the same model and weights at batch 64, as the
        # workload specifies it (logit gain 1), and with ragged acceptance (gain 8)
        b64 = synth.WORKLOADS["lca_d1024_b64"]
        for key, gain in (("batch64", args.logit_gain), ("batch64_ragged", 8.0)):
            r = bench_decode(args, b64, K, W, gain, weights=weights if gain == args.logit_gain else None)
            r.pop("_weights")
            r.pop("cpu_baseline")
            out[key] = r
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
