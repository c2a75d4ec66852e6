"""CPU oracle of the MBP decode step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The HIP library never calls it, and it shares
no code with the library: plain NumPy, float64, stateless full recompute of
Algorithm 1 ("Multi-byte Prediction with LCA") at every step.
"""
from .model import (  # noqa: F401
    SPACE,
    to_float64,
    rms_norm,
    rope,
    causal_mask,
    lca_mask,
    attention,
    ffn,
    block,
    boundaries,
    boundary_logits,
    learned_boundaries,
    group_ids,
    group_start,
    downsample,
    trunk,
    head_logits,
    mb_window,
    mb_logits,
    step_logits,
    stack,
    top1,
    threshold_accept,
    step,
    verify_drafts,
    verify_step,
    verify_external,
    decoding_dist,
    sample_byte,
    step_sampled,
    speculative_accept,
    verify_step_sampled,
    generate_external,
    generate,
    greedy_generate,
    log_softmax,
    forward_full,
    boundary_loss,
    forward_losses,
)
