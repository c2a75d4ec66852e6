"""Plain float64 statement of the hierarchical byte LM with multi-byte prediction.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s ``cpu_baseline`` leg, never by the library.  Every function is the
definition written out, with no caching, blocking or fusion, so it can be checked
against the paper by eye.  Each docstring names the passage it follows.

Paper: "Dynamic Multi-Byte Prediction With Hierarchical Language Models".
Readings taken where the paper is silent or ambiguous (each is listed, with its
reason, in the design notes of this repository):

* n counts all candidate distributions of a step: 1 next-byte + (n-1) MB rows.
* The boundary byte opens the new group: byte i uses latent L(i) = #{boundaries <= i}.
* r2 is the LM-module input row: the MB input of group j is z_j = h'[j] + LMin[j].
* Window mode 0 (default): the MB layers run on the window only (previous group,
  current group, n-2 virtual rows); mode 1 runs them on the whole sequence.
* A segment also closes when it reaches ``max_patch`` bytes (0 = pure space rule).
* Attention score = q.k / sqrt(d_head) * attn_scale; RoPE rotates adjacent pairs.
* argmax ties resolve to the lowest byte value; acceptance compares P >= tau.
* Self-verify: c_1 is the next-byte greedy byte; c_m (m >= 2) is kept while it equals
  the greedy byte after x ++ c_1..c_{m-1}.  The correction byte at the first mismatch
  is the next step's c_1, so the emitted sequence is the greedy one.
* Learned boundaries: the predictor is a linear probe on the RMS-normalized encoder
  state, logit = w . h_e / RMS(h_e) + b; at inference byte i ends a segment when its
  logit is >= 0 (probability >= 0.5, no Gumbel noise), or at max_patch bytes.
* Training objective: sums over positions of the next-byte and MB negative
  log-likelihoods (MB row t predicts x_{t+2} under the full-sequence LCA mask), plus
  lambda_2 L_BP with k = the number of segment ends.
"""
from __future__ import annotations

import numpy as np

SPACE = 0x20


# ---------------------------------------------------------------- primitives --

def rms_norm(x, g, eps):
    """RMSNorm (Llama 3 blocks, model-architecture paragraph of the experimental
    setup; eps = 1e-6): x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(g, np.float64)


def rope(x, pos, base):
    """Rotary embedding (base 1e5, model-architecture paragraph).

    ``x``: [T, H, dh].  Pair (2i, 2i+1) of the row at position p is rotated by the
    angle p * base^(-2i/dh).
    """
    x = np.asarray(x, np.float64)
    dh = x.shape[-1]
    inv = base ** (-np.arange(0, dh, 2, dtype=np.float64) / dh)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x0 = x[..., 0::2]
    x1 = x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x0 * c - x1 * s
    out[..., 1::2] = x0 * s + x1 * c
    return out


def causal_mask(T):
    """Standard causal mask (encoder, LM module, NT decoder): i attends j iff j <= i."""
    return np.tril(np.ones((T, T), dtype=bool))


def lca_mask(G):
    """Latent Causal Attention mask (Figure 2 caption; Section 3).

    ``G[i]`` is the group (latent token) of row i.  Row i may attend to itself, to
    earlier rows of its own group, and to every row of the immediately preceding
    group; later rows and older groups are masked out.
    """
    G = np.asarray(G)
    T = len(G)
    m = np.zeros((T, T), dtype=bool)
    for i in range(T):
        for j in range(T):
            own_group_so_far = G[j] == G[i] and j <= i
            previous_group = G[j] == G[i] - 1
            m[i, j] = own_group_so_far or previous_group
    return m


def attention(x, P, mask, pos, n_heads, rope_base, attn_scale):
    """Multi-head self-attention with RoPE on q and k (8 KV heads = query heads in the
    paper; here as many KV heads as query heads), score scaled by attn_scale/sqrt(dh),
    masked positions excluded from the softmax."""
    x = np.asarray(x, np.float64)
    T, d = x.shape
    dh = d // n_heads
    q = (x @ P["wq"].T).reshape(T, n_heads, dh)
    k = (x @ P["wk"].T).reshape(T, n_heads, dh)
    v = (x @ P["wv"].T).reshape(T, n_heads, dh)
    q = rope(q, pos, rope_base).transpose(1, 0, 2)  # [H, T, dh]
    k = rope(k, pos, rope_base).transpose(1, 0, 2)
    v = v.transpose(1, 0, 2)
    o = np.empty((T, n_heads, dh))
    for h in range(n_heads):  # one head at a time: a [T(query), T(key)] score matrix
        scores = (q[h] @ k[h].T) * (attn_scale / np.sqrt(dh))
        scores = np.where(mask, scores, -np.inf)
        scores = scores - scores.max(axis=-1, keepdims=True)
        p = np.exp(scores)
        p = p / p.sum(axis=-1, keepdims=True)
        o[:, h, :] = p @ v[h]
    return o.reshape(T, d) @ P["wo"].T


def silu(x):
    return x / (1.0 + np.exp(-x))


def ffn(x, P):
    """SwiGLU feed-forward, d_inner = 4 d (Llama 3 style): W_d (SiLU(W_g x) * W_u x)."""
    return (silu(x @ P["w_gate"].T) * (x @ P["w_up"].T)) @ P["w_down"].T


def block(u, P, mask, pos, cfg):
    """Pre-norm Llama block: a = u + Attn(RMSNorm(u)); out = a + FFN(RMSNorm(a))."""
    a = u + attention(rms_norm(u, P["attn_norm"], cfg.rms_eps), P, mask, pos,
                      cfg.n_heads, cfg.rope_base, cfg.attn_scale)
    return a + ffn(rms_norm(a, P["ffn_norm"], cfg.rms_eps), P)


def to_float64(W):
    """The weight dict with every tensor as a float64 array (done once per model)."""
    return {k: np.asarray(v, np.float64) for k, v in W.items()}


def _params(W, prefix):
    parts = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
    return {p: np.asarray(W[f"{prefix}.{p}"], np.float64) for p in parts}


def stack(u, W, name, n_layers, mask, pos, cfg):
    h = np.asarray(u, np.float64)
    for i in range(n_layers):
        h = block(h, _params(W, f"{name}.{i}"), mask, pos, cfg)
    return h


# ------------------------------------------------------------- segmentation --

def boundaries(x, max_patch):
    """Boundary positions q_1 < q_2 < ... (0-based byte indices).

    A segment ends at a space byte (0x20), or when it reaches ``max_patch`` bytes
    (the boundary predictor of the encoder-module paragraph is replaced by this rule).
    """
    q = []
    prev = -1
    for i, b in enumerate(np.asarray(x)):
        if int(b) == SPACE or (max_patch > 0 and i - prev >= max_patch):
            q.append(i)
            prev = i
    return q


def boundary_logits(h_e, W, eps):
    """Boundary predictor of the encoder-module paragraph, read as a linear probe on the
    RMS-normalized encoder state: logit_i = w . h_e[i] / RMS(h_e[i]) + b, boundary
    probability sigmoid(logit_i)."""
    h = np.asarray(h_e, np.float64)
    r = np.sqrt(np.mean(h * h, axis=-1) + eps)
    return (h @ np.asarray(W["bp.w"], np.float64)) / r + float(np.asarray(W["bp.b"]).reshape(-1)[0])


def learned_boundaries(h_e, W, max_patch, eps):
    """Inference-time segmentation with the boundary predictor: byte i ends a segment
    when its boundary probability is >= 0.5 (logit >= 0; the Gumbel-sigmoid draw is a
    training device), or when the segment reaches ``max_patch`` bytes."""
    z = boundary_logits(h_e, W, eps)
    q, prev = [], -1
    for i in range(len(z)):
        if z[i] >= 0.0 or (max_patch > 0 and i - prev >= max_patch):
            q.append(i)
            prev = i
    return q


def group_ids(T, q):
    """L(i) = number of boundaries q_j <= i: the latent a byte is upsampled from
    (the boundary byte already uses the latent of the segment it closes)."""
    qa = np.asarray(q, dtype=np.int64).reshape(1, -1)
    return (qa <= np.arange(T, dtype=np.int64)[:, None]).sum(axis=1).astype(np.int64)


def group_start(j, q):
    """First byte of group j: 0 for j = 0, else the j-th boundary byte."""
    return 0 if j == 0 else q[j - 1]


def downsample(h_e, q):
    """Mean-pool each closed segment (encoder-module paragraph): latent j is the mean
    of h_e over bytes q_{j-1}+1 .. q_j (q_0 = -1); an open trailing segment gives none."""
    out = []
    prev = -1
    for qj in q:
        out.append(np.mean(h_e[prev + 1: qj + 1], axis=0))
        prev = qj
    d = h_e.shape[1]
    return np.array(out, dtype=np.float64).reshape(len(out), d)


# -------------------------------------------------------------------- model --

def trunk(W, cfg, x):
    """Encoder, boundaries, downsample, LM module and next-byte decoder over the whole
    byte sequence (Algorithm 1, first half; Section 2.2 module paragraphs).

    Returns h_e, the boundaries q, LMin = [BOS; h_down], h_lm = LMModule(LMin), the
    group ids L and the next-byte decoder output h1.
    """
    x = np.asarray(x, dtype=np.int64)
    T = len(x)
    pos = np.arange(T)
    E = np.asarray(W["emb"], np.float64)[x]
    h_e = stack(E, W, "enc", cfg.n_enc, causal_mask(T), pos, cfg)
    q = (learned_boundaries(h_e, W, cfg.max_patch, cfg.rms_eps) if cfg.boundary == "learned"
         else boundaries(x, cfg.max_patch))
    h_down = downsample(h_e, q)
    LMin = np.vstack([np.asarray(W["bos"], np.float64)[None, :], h_down])
    K1 = LMin.shape[0]
    h_lm = stack(LMin, W, "lm", cfg.n_lm, causal_mask(K1), np.arange(K1), cfg)
    L = group_ids(T, q)
    nt_in = h_lm[L] + h_e
    h1 = stack(nt_in, W, "nt", cfg.n_nb, causal_mask(T), pos, cfg)
    return {"h_e": h_e, "q": q, "LMin": LMin, "h_lm": h_lm, "L": L, "h1": h1}


def head_logits(h, g, W, eps):
    """Shared unembedding (Section 3: both heads share one unembedding matrix) after
    the head's final RMSNorm."""
    return rms_norm(h, g, eps) @ np.asarray(W["unembed"], np.float64).T


def mb_window(q, L, t, n, window_mode=0):
    """Rows the MB layers run on (Algorithm 1: duplicate the last position n-2 times,
    slice from the start of the previous segment).

    Returns the window start s, the positions P = s..t+n-2 (virtual rows t+1..t+n-2
    keep increasing positions) and their groups G (virtual rows belong to the current
    group g = L(t)).  Window mode 1 starts at byte 0 instead.
    """
    g = int(L[t])
    if window_mode == 0:
        s = group_start(g - 1, q) if g >= 1 else 0
    else:
        s = 0
    P = np.arange(s, t + n - 1)
    G = np.array([int(L[p]) if p <= t else g for p in P], dtype=np.int64)
    return s, P, G


def mb_logits(W, cfg, tr, n):
    """Rows 2..n of the step's candidate distributions from the MB head.

    LCA (Algorithm 1, second half; Section 3): z_j = h'[j] + LMin[j]; every byte of
    group j gets input z_j; the last position is duplicated n-2 times as virtual rows
    t+1..t+n-2 of the current group; the window starts at the first byte of the
    previous group; the MB layers run under the LCA mask; rows t..t+n-2 go to the
    head (row t predicts x_{t+2}, the MB target shifted by two).

    MLP (Section 4.1, MLP-MBP baseline): head m-1 is a residual pre-norm SwiGLU block
    on h1[t]; its output goes through the NT final norm and the shared unembedding.
    """
    if n < 2:
        return np.zeros((0, 256))
    x_len = tr["h1"].shape[0]
    t = x_len - 1
    if cfg.head == "mlp":
        h = tr["h1"][t]
        rows = []
        for m in range(2, n + 1):
            P = {k: np.asarray(W[f"mlp.{m - 2}.{k}"], np.float64) for k in ("norm", "w_gate", "w_up", "w_down")}
            y = h + ffn(rms_norm(h, P["norm"], cfg.rms_eps)[None, :], P)[0]
            rows.append(head_logits(y, W["nt_norm"], W, cfg.rms_eps))
        return np.array(rows)
    s, P, G = mb_window(tr["q"], tr["L"], t, n, cfg.window_mode)
    z = tr["h_lm"] + tr["LMin"]
    u = z[G]
    h2 = stack(u, W, "mb", cfg.n_mb, lca_mask(G), P, cfg)
    rows = h2[t - s: t - s + n - 1]
    return head_logits(rows, W["mb_norm"], W, cfg.rms_eps)


def step_logits(W, cfg, x, n):
    """The n x 256 logits of one step: row 1 from the next-byte head on h1[t]
    (always accepted), rows 2..n from the MB head."""
    tr = trunk(W, cfg, x)
    t = len(x) - 1
    l1 = head_logits(tr["h1"][t], W["nt_norm"], W, cfg.rms_eps)
    return np.vstack([l1[None, :], mb_logits(W, cfg, tr, n)])


def top1(logits):
    """Per row: the greedy byte (lowest index among equal maxima) and its softmax
    probability at temperature 1 over all 256 bytes."""
    logits = np.asarray(logits, np.float64)
    c = np.argmax(logits, axis=-1)
    mx = np.take_along_axis(logits, c[:, None], axis=-1)
    p = 1.0 / np.sum(np.exp(logits - mx), axis=-1)
    return c.astype(np.int64), p


def threshold_accept(prob, tau):
    """Byte acceptance (Section 3.1): the next-byte candidate is always accepted; MB
    candidates are accepted left to right while P >= tau; the first failure and all
    later candidates are discarded.  Returns the number of accepted bytes k."""
    k = 1
    while k < len(prob) and prob[k] >= tau:
        k += 1
    return k


def step(W, cfg, x, n, tau):
    """One threshold-acceptance step of Algorithm 1 on the byte sequence ``x``."""
    logits = step_logits(W, cfg, x, n)
    cand, prob = top1(logits)
    return {"logits": logits, "cand": cand, "prob": prob, "k": threshold_accept(prob, tau)}


def _nt_logits(W, cfg, x):
    """Next-byte head logits after the byte sequence x."""
    tr = trunk(W, cfg, x)
    return head_logits(tr["h1"][len(x) - 1], W["nt_norm"], W, cfg.rms_eps)


def _greedy_byte(W, cfg, x):
    return int(top1(_nt_logits(W, cfg, x)[None, :])[0][0])


def verify_drafts(W, cfg, x, drafts, seen=None):
    """Greedy speculative verification (Section 6.2, following Leviathan et al.): draft
    c_1 is kept; c_m (m >= 2) is kept while it equals the next-byte greedy byte after
    x ++ c_1..c_{m-1}.  Returns the number of kept drafts j and the greedy bytes seen
    (and appends the next-byte logits they came from to ``seen`` when it is a list)."""
    drafts = np.asarray(drafts, np.int64)
    j = 1
    gammas = []
    for m in range(2, len(drafts) + 1):
        lm = _nt_logits(W, cfg, np.concatenate([np.asarray(x, np.int64), drafts[: m - 1]]))
        if seen is not None:
            seen.append(lm)
        gm = int(top1(lm[None, :])[0][0])
        gammas.append(gm)
        if gm != int(drafts[m - 1]):
            break
        j += 1
    return j, gammas


def verify_step(W, cfg, x, n):
    """Self-verification step: drafts c_1..c_n from the next-byte and MB heads (c_1 is
    the greedy byte), verified by extra next-byte passes.  ``nt_seen`` holds the
    next-byte logits after each verified draft prefix."""
    s = step(W, cfg, x, n, tau=2.0)
    seen = []
    j, gammas = verify_drafts(W, cfg, x, s["cand"], seen)
    return {"logits": s["logits"], "cand": s["cand"], "prob": s["prob"], "k": j, "gamma": gammas,
            "nt_seen": np.array(seen).reshape(len(seen), 256)}


def verify_external(W, cfg, x, drafts):
    """External verification (Section 6, "Improving Baseline Throughput with MBP
    Models"): a separate next-byte model (the FxT baseline: encoder, LM module and
    next-byte decoder, no MB head) checks another model's drafts c_1..c_n with greedy
    speculative decoding.  g_m is the verifier's greedy byte after x ++ c_1..c_m
    (m = 0..n); the drafts are kept while c_{m+1} == g_m, and the verifier's greedy
    byte after the kept prefix is appended.  Returns k = j + 1 accepted bytes
    (j = 0..n kept drafts), the bytes, and the greedy bytes seen."""
    x = [int(b) for b in x]
    drafts = [int(c) for c in drafts]
    greedy = []
    j = 0
    while True:
        g = _greedy_byte(W, cfg, x + drafts[:j])
        greedy.append(g)
        if j == len(drafts) or g != drafts[j]:
            break
        j += 1
    return {"k": j + 1, "bytes": np.array(drafts[:j] + [greedy[j]], dtype=np.uint8), "greedy": greedy}


def generate_external(Wd, cfg_d, Wv, cfg_v, prompt, n_new, n):
    """Bytes emitted when the MBP model (Wd, cfg_d) drafts n candidates per step
    (next-byte head + MB head) and the verifier (Wv, cfg_v) checks them
    (verify_external); the last step is truncated."""
    x = [int(b) for b in prompt]
    out, steps = [], []
    while len(out) < n_new:
        drafts = step(Wd, cfg_d, x, n, tau=2.0)["cand"]
        r = verify_external(Wv, cfg_v, x, drafts)
        acc = [int(b) for b in r["bytes"][: n_new - len(out)]]
        steps.append({"k": r["k"], "drafts": np.asarray(drafts).copy(), "bytes": r["bytes"].copy()})
        out += acc
        x += acc
    return np.array(out, dtype=np.uint8), steps


# ------------------------------------------------------------ sampled decoding --
# Sampled decoding (the paper samples at temperature 0.7 with top-p 0.9 for one of its
# tasks and verifies drafts with speculative decoding, Section 6).  The uniforms are
# inputs: u[m] samples candidate m, u[n + m] decides the acceptance of draft m and
# u[2n + m] samples its replacement (verification), m = 0..n-1.

def decoding_dist(logits, temperature, top_p):
    """Distribution a byte is sampled from: softmax(logits / temperature) restricted to
    the nucleus (bytes ranked by probability, ties by lower byte value; a byte is in
    the nucleus while the probability ranked before it is below top_p) and
    renormalized."""
    z = np.asarray(logits, np.float64) / float(temperature)
    p = np.exp(z - z.max())
    p /= p.sum()
    before = np.empty(256)
    for i in range(256):
        ahead = (p > p[i]) | ((p == p[i]) & (np.arange(256) < i))
        before[i] = p[ahead].sum()
    q = np.where(before < top_p, p, 0.0)
    return q / q.sum()


def sample_byte(q, u):
    """Inverse CDF in byte order: the first byte whose cumulative mass exceeds u (the
    last byte of positive mass if rounding leaves none)."""
    c = np.cumsum(np.asarray(q, np.float64))
    hit = np.nonzero(c > u)[0]
    return int(hit[0]) if len(hit) else int(np.nonzero(np.asarray(q) > 0)[0][-1])


def step_sampled(W, cfg, x, n, tau, temperature, top_p, u):
    """Threshold acceptance on sampled candidates: candidate m is sampled from its
    row's decoding distribution with u[m]; P_m is its probability there; the rule of
    Section 3.1 then applies to P."""
    logits = step_logits(W, cfg, x, n)
    qs = [decoding_dist(logits[m], temperature, top_p) for m in range(n)]
    cand = np.array([sample_byte(qs[m], u[m]) for m in range(n)], np.int64)
    prob = np.array([qs[m][cand[m]] for m in range(n)])
    return {"logits": logits, "q": qs, "cand": cand, "prob": prob, "k": threshold_accept(prob, tau)}


def speculative_accept(p_rows, q_rows, cand, u, n):
    """Speculative sampling (Leviathan et al.) of drafts cand[1..n-1] (cand[0] is kept):
    draft m (m >= 2), drawn from q_rows[m-1], is kept when u[n+m-1] < p(c_m) / q(c_m)
    with p = p_rows[m-2], the target distribution after the previous drafts; at the first
    rejection a byte drawn from max(0, p - q) (normalized) with u[2n+m-1] replaces it and
    ends the step.  Returns the accepted bytes."""
    out = [int(cand[0])]
    for m in range(2, n + 1):
        pm, qm, c = np.asarray(p_rows[m - 2], np.float64), np.asarray(q_rows[m - 1], np.float64), int(cand[m - 1])
        if u[n + m - 1] < pm[c] / qm[c]:
            out.append(c)
            continue
        r = np.maximum(pm - qm, 0.0)
        out.append(sample_byte(r / r.sum(), u[2 * n + m - 1]))
        break
    return out


def verify_step_sampled(W, cfg, x, n, temperature, top_p, u):
    """Verification of sampled drafts (Section 6): c_1 is sampled from the next-byte
    head and kept; drafts c_2..c_n are sampled from the MB rows and checked by
    speculative sampling against the next-byte decoding distribution after the
    drafts before them.  Returns the accepted bytes (k of them)."""
    s = step_sampled(W, cfg, x, n, 2.0, temperature, top_p, u)
    p_rows = []
    for m in range(2, n + 1):
        seq = np.asarray(list(x) + [int(c) for c in s["cand"][: m - 1]], np.int64)
        tr = trunk(W, cfg, seq)
        p_rows.append(decoding_dist(head_logits(tr["h1"][-1], W["nt_norm"], W, cfg.rms_eps), temperature, top_p))
    out = speculative_accept(p_rows, s["q"], s["cand"], u, n)
    return {"logits": s["logits"], "cand": s["cand"], "prob": s["prob"], "p": p_rows, "q": s["q"], "k": len(out),
            "bytes": np.array(out, dtype=np.uint8)}


def generate(W, cfg, prompt, n_new, n, tau, mode="threshold"):
    """Run steps until ``n_new`` bytes are emitted; the last step is truncated."""
    x = [int(b) for b in prompt]
    out, steps = [], []
    while len(out) < n_new:
        r = step(W, cfg, x, n, tau) if mode == "threshold" else verify_step(W, cfg, x, n)
        k = min(r["k"], n_new - len(out))
        acc = [int(c) for c in r["cand"][:k]]
        steps.append({"k": r["k"], "cand": r["cand"].copy(), "prob": r["prob"].copy()})
        out += acc
        x += acc
    return np.array(out, dtype=np.uint8), steps


def greedy_generate(W, cfg, prompt, n_new):
    """Byte-by-byte next-byte decoding (the n = 1 case)."""
    x = [int(b) for b in prompt]
    out = []
    for _ in range(n_new):
        b = _greedy_byte(W, cfg, x)
        out.append(b)
        x.append(b)
    return np.array(out, dtype=np.uint8)


# ------------------------------------------------------ full-sequence forward --

def log_softmax(logits):
    """log of the softmax over the last axis (the log-sum-exp taken about the max)."""
    l = np.asarray(logits, np.float64)
    m = l.max(axis=-1, keepdims=True)
    return l - m - np.log(np.sum(np.exp(l - m), axis=-1, keepdims=True))


def forward_full(W, cfg, x):
    """Training-form forward over a whole byte sequence (Section 3, the MB head under
    the LCA mask; Section 2.2 modules): the trunk, then the MB layers over every byte
    at once with the full-sequence LCA mask (each byte sees its own group so far and
    the whole previous group), inputs z_{L(i)} = h'[L(i)] + LMin[L(i)].

    Returns the next-byte logits [T, 256] (row t predicts x_{t+1}) and the MB logits
    [T, 256] (row t predicts x_{t+2}), plus the trunk.
    """
    tr = trunk(W, cfg, x)
    T = len(x)
    l_nt = head_logits(tr["h1"], W["nt_norm"], W, cfg.rms_eps)
    out = {"trunk": tr, "nt": l_nt, "mb": None}
    if cfg.head == "lca" and cfg.n_mb > 0:
        z = tr["h_lm"] + tr["LMin"]
        h2 = stack(z[tr["L"]], W, "mb", cfg.n_mb, lca_mask(tr["L"]), np.arange(T), cfg)
        out["mb"] = head_logits(h2, W["mb_norm"], W, cfg.rms_eps)
    return out


def boundary_loss(k, T, alpha, beta):
    """L_BP of the encoder-module paragraph: zero while the boundary rate k/T lies in
    [beta, alpha], else its distance to the nearer bound."""
    r = k / T
    return max(r - alpha, 0.0) + max(beta - r, 0.0)


def forward_losses(W, cfg, x, lam0=1.0, lam1=1.0, lam2=1.0, alpha=1.0, beta=0.0):
    """The training objective of Section 3 (next-byte plus multi-byte terms) plus
    lambda_2 L_BP on one sequence: per-position
    negative log-likelihoods of the next-byte head (targets x_{t+1}, t < T-1) and of
    the MB head (targets x_{t+2}, t < T-2), their sums, L_LM = lam0 * sum_nt +
    lam1 * sum_mb, L_BP with k = the number of boundaries, and L_LM + lam2 * L_BP.
    Sums, not means, as the equation is written."""
    x = np.asarray(x, np.int64)
    T = len(x)
    f = forward_full(W, cfg, x)
    nll_nt = -np.take_along_axis(log_softmax(f["nt"][: T - 1]), x[1:, None], axis=1)[:, 0]
    if f["mb"] is not None and T > 2:
        nll_mb = -np.take_along_axis(log_softmax(f["mb"][: T - 2]), x[2:, None], axis=1)[:, 0]
    else:
        nll_mb = np.zeros(0)
    s_nt, s_mb = float(np.sum(nll_nt)), float(np.sum(nll_mb))
    l_lm = lam0 * s_nt + lam1 * s_mb
    l_bp = boundary_loss(len(f["trunk"]["q"]), T, alpha, beta)
    return {"nll_nt": nll_nt, "nll_mb": nll_mb, "sum_nt": s_nt, "sum_mb": s_mb, "l_lm": l_lm, "l_bp": l_bp,
            "total": l_lm + lam2 * l_bp, "k": len(f["trunk"]["q"]), "forward": f}
