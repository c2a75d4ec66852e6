"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: a closed form, a
hand-computed fixture under tests/golden/, a brute-force loop written differently, or
an invariant the paper states (causality of the LCA inputs, always-accepted next-byte
candidate, verification reproducing next-byte decoding).
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TINY = synth.WORKLOADS["tiny_f32"].model


def _bytes(text):
    return np.frombuffer(text.encode("latin-1"), dtype=np.uint8)


# ------------------------------------------------------------- primitives --

def test_rms_norm_constant_vector_closed_form():
    d, c, eps = 16, -3.0, 1e-6
    g = np.linspace(0.5, 2.0, d)
    out = oracle.rms_norm(np.full(d, c), g, eps)
    # mean(x^2) = c^2, so every entry is c / sqrt(c^2 + eps) * g_i
    expect = (c / math.sqrt(c * c + eps)) * g
    np.testing.assert_allclose(out, expect, rtol=1e-15, atol=0)


def test_rms_norm_unit_rms_and_eps_effect():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 64)) * 7.0
    y = oracle.rms_norm(x, np.ones(64), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-13)
    # eps only shrinks the output; the direction is unchanged
    y2 = oracle.rms_norm(x, np.ones(64), 1e-6)
    cos = np.sum(y * y2, -1) / np.linalg.norm(y, axis=-1) / np.linalg.norm(y2, axis=-1)
    np.testing.assert_allclose(cos, 1.0, rtol=1e-13)


def test_rope_basis_vectors_rotate_by_expected_angles():
    dh, base = 8, 1e5
    for p in (0, 1, 7, 1234):
        for pair in range(dh // 2):
            e = np.zeros((1, 1, dh))
            e[0, 0, 2 * pair] = 1.0
            out = oracle.rope(e, [p], base)[0, 0]
            theta = p * base ** (-(2.0 * pair) / dh)
            want = np.zeros(dh)
            want[2 * pair] = math.cos(theta)
            want[2 * pair + 1] = math.sin(theta)
            np.testing.assert_allclose(out, want, atol=1e-12)
            # the odd partner rotates to (-sin, cos)
            e2 = np.zeros((1, 1, dh))
            e2[0, 0, 2 * pair + 1] = 1.0
            out2 = oracle.rope(e2, [p], base)[0, 0]
            want2 = np.zeros(dh)
            want2[2 * pair] = -math.sin(theta)
            want2[2 * pair + 1] = math.cos(theta)
            np.testing.assert_allclose(out2, want2, atol=1e-12)


def test_rope_norm_and_relative_position():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((1, 3, 16))
    k = rng.standard_normal((1, 3, 16))
    for base in (1e4, 1e5):
        a = oracle.rope(q, [5], base)
        np.testing.assert_allclose(np.linalg.norm(a, axis=-1), np.linalg.norm(q, axis=-1), rtol=1e-13)
        dots = []
        for shift in (0, 3, 100, 4000):
            qa = oracle.rope(q, [9 + shift], base)
            ka = oracle.rope(k, [2 + shift], base)
            dots.append(np.sum(qa * ka, axis=-1))
        for dd in dots[1:]:
            np.testing.assert_allclose(dd, dots[0], rtol=1e-9, atol=1e-11)


def _rand_block(rng, d, dff, scale=0.2):
    return {
        "attn_norm": 1.0 + 0.1 * rng.standard_normal(d), "ffn_norm": 1.0 + 0.1 * rng.standard_normal(d),
        "wq": scale * rng.standard_normal((d, d)), "wk": scale * rng.standard_normal((d, d)),
        "wv": scale * rng.standard_normal((d, d)), "wo": scale * rng.standard_normal((d, d)),
        "w_gate": scale * rng.standard_normal((dff, d)), "w_up": scale * rng.standard_normal((dff, d)),
        "w_down": scale * rng.standard_normal((d, dff)),
    }


def test_attention_with_zero_query_key_is_mean_of_visible_values():
    rng = np.random.default_rng(3)
    T, d, H = 6, 8, 2
    P = _rand_block(rng, d, 4 * d)
    P["wq"][:] = 0.0
    P["wk"][:] = 0.0
    x = rng.standard_normal((T, d))
    for mask in (oracle.causal_mask(T), oracle.lca_mask([0, 0, 1, 1, 2, 2])):
        out = oracle.attention(x, P, mask, np.arange(T), H, 1e5, 1.0)
        v = x @ P["wv"].T
        mean_v = np.array([v[mask[i]].mean(axis=0) for i in range(T)])
        np.testing.assert_allclose(out, mean_v @ P["wo"].T, rtol=1e-12, atol=1e-12)


def test_attention_matches_scalar_loop():
    """Independent scalar-loop attention: per head, per query, explicit RoPE angles,
    dot products, max-subtracted exponentials and weighted sums."""
    rng = np.random.default_rng(4)
    T, d, H, base, scale = 5, 8, 2, 1e5, 1.0
    dh = d // H
    P = _rand_block(rng, d, 4 * d, scale=0.5)
    x = rng.standard_normal((T, d))
    pos = [3, 4, 5, 9, 10]
    mask = oracle.lca_mask([0, 1, 1, 2, 2])
    got = oracle.attention(x, P, mask, np.array(pos), H, base, scale)

    def matvec(Wm, v):
        return [sum(Wm[r][c] * v[c] for c in range(len(v))) for r in range(len(Wm))]

    def rot(vec, p):
        out = list(vec)
        for i in range(dh // 2):
            ang = p * base ** (-(2.0 * i) / dh)
            a, b = vec[2 * i], vec[2 * i + 1]
            out[2 * i] = a * math.cos(ang) - b * math.sin(ang)
            out[2 * i + 1] = a * math.sin(ang) + b * math.cos(ang)
        return out

    Q = [matvec(P["wq"], x[i]) for i in range(T)]
    Kx = [matvec(P["wk"], x[i]) for i in range(T)]
    V = [matvec(P["wv"], x[i]) for i in range(T)]
    concat = [[0.0] * d for _ in range(T)]
    for h in range(H):
        sl = slice(h * dh, (h + 1) * dh)
        for i in range(T):
            qi = rot(Q[i][sl], pos[i])
            scores = {}
            for j in range(T):
                if mask[i, j]:
                    kj = rot(Kx[j][sl], pos[j])
                    scores[j] = sum(a * b for a, b in zip(qi, kj)) / math.sqrt(dh) * scale
            mx = max(scores.values())
            w = {j: math.exp(s - mx) for j, s in scores.items()}
            z = sum(w.values())
            for c in range(dh):
                concat[i][h * dh + c] = sum(w[j] / z * V[j][sl][c] for j in w)
    want = np.array([matvec(P["wo"], concat[i]) for i in range(T)])
    np.testing.assert_allclose(got, want, rtol=1e-10, atol=1e-12)


def test_ffn_matches_scalar_loop_and_zero_down_projection():
    rng = np.random.default_rng(5)
    d, dff = 4, 16
    P = _rand_block(rng, d, dff, scale=0.7)
    x = rng.standard_normal((3, d))
    got = oracle.ffn(x, P)
    for r in range(3):
        hidden = []
        for j in range(dff):
            gj = sum(P["w_gate"][j][c] * x[r][c] for c in range(d))
            uj = sum(P["w_up"][j][c] * x[r][c] for c in range(d))
            hidden.append(gj / (1.0 + math.exp(-gj)) * uj)
        for o in range(d):
            want = sum(P["w_down"][o][j] * hidden[j] for j in range(dff))
            assert abs(got[r][o] - want) < 1e-12
    P["w_down"][:] = 0
    assert np.all(oracle.ffn(x, P) == 0)


def test_block_with_zero_weights_is_identity():
    rng = np.random.default_rng(6)
    d = 8
    P = {k: np.zeros_like(v) if k.startswith("w") else v for k, v in _rand_block(rng, d, 32).items()}
    u = rng.standard_normal((4, d))
    np.testing.assert_array_equal(oracle.block(u, P, oracle.causal_mask(4), np.arange(4), TINY.replace(n_heads=2, d_model=8)), u)


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _hand_block():
    """The hand-derived block fixture: its config (eps = 0 as derived) and parameters."""
    g = _golden("block_stack.json")
    cfg = TINY.replace(d_model=g["d_model"], n_heads=g["n_heads"], d_ff=2, rms_eps=0.0)
    P = [{k: np.asarray(v, np.float64) for k, v in g[name].items()} for name in ("P0", "P1")]
    return g, cfg, P


def test_block_hand_derived_one_token():
    """A one-token block: the softmax over a single key is 1, so attention reduces to
    W_o W_v (RMSNorm(u) g_attn); the expected vector is derived by hand in the fixture.
    Swapping the two norm gains, normalizing u instead of a before the FFN, a
    post-norm block or a dropped residual all change it."""
    g, cfg, (P0, _) = _hand_block()
    u = np.asarray(g["one_token"]["u"], np.float64)
    got = oracle.block(u, P0, oracle.causal_mask(1), np.arange(1), cfg)
    np.testing.assert_allclose(got, g["one_token"]["block_P0"], rtol=1e-14, atol=1e-14)
    # the same at the model's eps = 1e-6: the norms move by O(eps) only
    got_eps = oracle.block(u, P0, oracle.causal_mask(1), np.arange(1), cfg.replace(rms_eps=1e-6))
    np.testing.assert_allclose(got_eps, g["one_token"]["block_P0"], rtol=0, atol=1e-5)
    assert np.max(np.abs(got_eps - got)) > 0  # eps reaches the norms
    # a query attends to one key whatever its position: RoPE cannot change it
    got_p = oracle.block(u, P0, oracle.causal_mask(1), np.array([37]), cfg)
    np.testing.assert_allclose(got_p, got, rtol=1e-14, atol=1e-14)


def test_block_hand_derived_two_tokens_causal():
    """Two tokens with zero queries: every visible key gets the same weight, so row 0
    (which sees only itself under the causal mask) repeats the one-token result and
    row 1 averages both values; expected rows derived by hand in the fixture."""
    g, cfg, (P0, _) = _hand_block()
    P = dict(P0, wq=np.zeros_like(P0["wq"]))
    u = np.asarray(g["two_tokens"]["u"], np.float64)
    got = oracle.block(u, P, oracle.causal_mask(2), np.arange(2), cfg)
    np.testing.assert_allclose(got, g["two_tokens"]["block_P0_wq0"], rtol=1e-14, atol=1e-14)


def test_stack_applies_each_layers_own_parameters_in_order():
    """A two-layer stack with different parameters per layer equals the hand-derived
    composition block(block(u, P0), P1); reusing layer 0's parameters, reversing the
    order or skipping a layer each gives a different vector."""
    g, cfg, (P0, P1) = _hand_block()
    W = {}
    for i, P in enumerate((P0, P1)):
        for k, v in P.items():
            W[f"s.{i}.{k}"] = v
    u = np.asarray(g["one_token"]["u"], np.float64)
    want = np.asarray(g["one_token"]["stack_P0_P1"])
    got = oracle.stack(u, W, "s", 2, oracle.causal_mask(1), np.arange(1), cfg)
    np.testing.assert_allclose(got, want, rtol=1e-14, atol=1e-14)
    one = oracle.stack(u, W, "s", 1, oracle.causal_mask(1), np.arange(1), cfg)
    np.testing.assert_allclose(one, g["one_token"]["block_P0"], rtol=1e-14, atol=1e-14)
    # the wrong compositions are far from the expected vector
    m, pos = oracle.causal_mask(1), np.arange(1)
    for wrong in (oracle.block(oracle.block(u, P0, m, pos, cfg), P0, m, pos, cfg),
                  oracle.block(oracle.block(u, P1, m, pos, cfg), P0, m, pos, cfg)):
        assert np.max(np.abs(wrong - want)) > 0.1


# ------------------------------------------------------------ segmentation --


@pytest.mark.parametrize("case", _golden("segmentation.json")["cases"])
def test_boundaries_groups_segments(case):
    x = _bytes(case["text"])
    q = oracle.boundaries(x, case["max_patch"])
    assert q == case["q"]
    assert list(oracle.group_ids(len(x), q)) == case["L"]
    # mean pool over h_e[i] = i * 1: latent j is the midpoint of its segment
    h_e = np.repeat(np.arange(len(x), dtype=np.float64)[:, None], 3, axis=1)
    down = oracle.downsample(h_e, q)
    assert down.shape == (len(case["segments"]), 3)
    for j, (a, b) in enumerate(case["segments"]):
        np.testing.assert_allclose(down[j], (a + b) / 2.0, rtol=1e-15)


@pytest.mark.parametrize("case", _golden("segmentation.json")["windows"]["cases"])
def test_mb_window(case):
    x = _bytes(case["text"])
    q = oracle.boundaries(x, case["max_patch"])
    L = oracle.group_ids(len(x), q)
    s, P, G = oracle.mb_window(q, L, len(x) - 1, case["n"])
    assert s == case["s"]
    assert list(P) == case["P"]
    assert list(G) == case["G"]


@pytest.mark.parametrize("case", _golden("lca_masks.json")["cases"])
def test_lca_mask_hand_matrices(case):
    np.testing.assert_array_equal(oracle.lca_mask(case["G"]).astype(int), np.array(case["mask"]))


# ---------------------------------------------------------- whole-model pins --

def _zero_blocks(W):
    out = dict(W)
    for k, v in W.items():
        if k.split(".")[-1] in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"):
            out[k] = np.zeros_like(v)
    return out


def _rms(v, g, eps=1e-6):
    return v / math.sqrt(float(np.mean(v * v)) + eps) * g


@pytest.mark.parametrize("text,n", [("ab cd efg", 4), ("xyz", 3), ("a b c dd", 2), ("hello world  ok", 5)])
def test_zero_block_model_closed_form(text, n):
    """With every block matrix zero each block is the identity, so the whole step has
    a closed form: h_e = E, LMin = [BOS; segment means of E], h' = LMin,
    l_1 = U RMS(LMin[L(t)] + E[t]), and every MB row = U RMS(2 LMin[g])."""
    cfg = TINY.replace(max_patch=0)
    W = _zero_blocks(synth.make_weights(cfg, seed=11, gain_jitter=0.3))
    x = _bytes(text)
    t = len(x) - 1
    E = W["emb"].astype(np.float64)[x]
    q = [i for i, b in enumerate(x) if b == 0x20]
    lat = [W["bos"].astype(np.float64)]
    prev = -1
    for qj in q:
        lat.append(E[prev + 1: qj + 1].mean(axis=0))
        prev = qj
    g = sum(1 for qj in q if qj <= t)
    U = W["unembed"].astype(np.float64)
    l1 = U @ _rms(lat[g] + E[t], W["nt_norm"])
    lmb = U @ _rms(2.0 * lat[g], W["mb_norm"])
    got = oracle.step_logits(W, cfg, x, n)
    assert got.shape == (n, 256)
    np.testing.assert_allclose(got[0], l1, rtol=1e-12, atol=1e-13)
    for m in range(1, n):
        np.testing.assert_allclose(got[m], lmb, rtol=1e-12, atol=1e-13)


def test_zero_block_mlp_head_rows_equal_next_byte_row():
    cfg = TINY.replace(head="mlp", n_mb=3)
    W = _zero_blocks(synth.make_weights(cfg, seed=3, gain_jitter=0.2))
    got = oracle.step_logits(W, cfg, _bytes("abc de f"), 4)
    for m in range(1, 4):
        np.testing.assert_allclose(got[m], got[0], rtol=1e-13, atol=1e-14)


def test_mlp_head_with_zero_down_projection_equals_next_byte_head():
    cfg = TINY.replace(head="mlp", n_mb=3)
    W = synth.make_weights(cfg, seed=4, gain_jitter=0.2)
    x = synth.make_bytes(5, 40)
    full = oracle.step_logits(W, cfg, x, 4)
    W2 = dict(W)
    W2["mlp.1.w_down"] = np.zeros_like(W["mlp.1.w_down"])
    got = oracle.step_logits(W2, cfg, x, 4)
    np.testing.assert_allclose(got[2], got[0], rtol=1e-13, atol=1e-14)
    np.testing.assert_array_equal(got[[0, 1, 3]], full[[0, 1, 3]])
    assert not np.allclose(full[2], full[0])


def test_lm_module_with_zero_layers_is_identity():
    cfg = TINY.replace(n_lm=0)
    W = synth.make_weights(cfg, seed=8)
    x = synth.make_bytes(9, 30)
    tr = oracle.trunk(W, cfg, x)
    np.testing.assert_array_equal(tr["h_lm"], tr["LMin"])


def test_trunk_is_causal():
    """h1[i] depends only on x_0..x_i: changing later bytes (including adding spaces,
    which changes the later segmentation) leaves earlier rows unchanged."""
    W = synth.make_weights(TINY, seed=12, gain_jitter=0.2)
    x = synth.make_bytes(13, 50)
    y = x.copy()
    y[30:] = synth.make_bytes(14, 20)
    a = oracle.trunk(W, TINY, x)["h1"]
    b = oracle.trunk(W, TINY, y)["h1"]
    np.testing.assert_allclose(a[:30], b[:30], rtol=1e-12, atol=1e-13)
    assert not np.allclose(a[30:], b[30:])


def _current_group_start(x, max_patch):
    q = oracle.boundaries(x, max_patch)
    return q[-1] if q else 0


def test_mb_rows_do_not_depend_on_current_group_bytes():
    """Section 3: inputs inside the current latent token are duplicates plus residuals
    of the previous latent token, so the MB rows cannot see the bytes of the current
    group after its boundary; the next-byte row does."""
    cfg = TINY.replace(max_patch=0)
    W = synth.make_weights(cfg, seed=15, gain_jitter=0.2)
    x = _bytes("abc defgh ijk lmnop")
    y = _bytes("abc defgh ijk lQRSp")
    a = oracle.step_logits(W, cfg, x, 5)
    b = oracle.step_logits(W, cfg, y, 5)
    np.testing.assert_array_equal(a[1:], b[1:])
    assert np.max(np.abs(a[0] - b[0])) > 1e-3
    # a byte of the previous group does change the MB rows
    z = _bytes("abc defgh iZk lmnop")
    c = oracle.step_logits(W, cfg, z, 5)
    assert np.max(np.abs(a[1:] - c[1:])) > 1e-6


@pytest.mark.parametrize("window_mode", [0, 1])
def test_mb_rows_prefix_stable_in_n(window_mode):
    cfg = TINY.replace(window_mode=window_mode)
    W = synth.make_weights(cfg, seed=16, gain_jitter=0.2)
    x = synth.make_bytes(17, 60)
    prev = oracle.step_logits(W, cfg, x, 2)
    for n in range(3, 8):
        cur = oracle.step_logits(W, cfg, x, n)
        np.testing.assert_allclose(cur[:n - 1], prev, rtol=1e-11, atol=1e-12)
        prev = cur


def test_mb_rows_stable_when_one_non_boundary_byte_is_accepted():
    """Row t+m-2 of the MB window is the same row whether it is virtual (step t) or
    real (step t+1) while the group is unchanged: candidate m at t equals candidate
    m-1 at t+1."""
    cfg = TINY.replace(max_patch=0)
    W = synth.make_weights(cfg, seed=18, gain_jitter=0.2)
    x = _bytes("abc defgh ijk lm")
    n = 5
    a = oracle.step_logits(W, cfg, x, n)
    b = oracle.step_logits(W, cfg, np.append(x, np.uint8(ord("q"))), n)
    np.testing.assert_allclose(b[1:n - 1], a[2:n], rtol=1e-11, atol=1e-12)


def test_window_modes_agree_with_one_mb_layer():
    W = synth.make_weights(TINY, seed=19, gain_jitter=0.2)
    x = synth.make_bytes(20, 70)
    a = oracle.step_logits(W, TINY.replace(window_mode=0), x, 4)
    b = oracle.step_logits(W, TINY.replace(window_mode=1), x, 4)
    np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-12)
    cfg2 = TINY.replace(n_mb=2)
    W2 = synth.make_weights(cfg2, seed=19, gain_jitter=0.2)
    a2 = oracle.step_logits(W2, cfg2.replace(window_mode=0), x, 4)
    b2 = oracle.step_logits(W2, cfg2.replace(window_mode=1), x, 4)
    assert np.max(np.abs(a2[1:] - b2[1:])) > 1e-9


# ---------------------------------------------------------------- acceptance --

def test_top1_matches_brute_force_softmax():
    rng = np.random.default_rng(21)
    logits = rng.standard_normal((6, 256)) * 3
    logits[2, 10] = logits[2, 200] = logits[2].max() + 1.0  # tie: lowest index wins
    c, p = oracle.top1(logits)
    for r in range(6):
        row = [float(v) for v in logits[r]]
        best = 0
        for j in range(256):
            if row[j] > row[best]:
                best = j
        z = sum(math.exp(v) for v in row)
        assert c[r] == best
        assert abs(p[r] - math.exp(row[best]) / z) < 1e-14
    assert c[2] == 10


def test_threshold_acceptance_rule():
    assert oracle.threshold_accept([0.1, 0.9, 0.8, 0.2, 0.99], 0.75) == 3
    assert oracle.threshold_accept([0.1, 0.5, 0.99], 0.75) == 1
    assert oracle.threshold_accept([0.1, 0.75, 0.75], 0.75) == 3  # P >= tau accepts
    assert oracle.threshold_accept([0.3], 0.0) == 1
    assert oracle.threshold_accept([0.3, 0.2, 0.1], 0.0) == 3


@pytest.mark.parametrize("gain", [1.0, 25.0])
def test_tau_extremes_and_monotonicity(gain):
    W = synth.make_weights(TINY, seed=22, logit_gain=gain)
    x = synth.make_prompt(0, 64)
    n = 5
    logits = oracle.step_logits(W, TINY, x, n)
    _, prob = oracle.top1(logits)
    assert np.all(prob < 1.0)
    assert oracle.threshold_accept(prob, 1.0) == 1
    assert oracle.threshold_accept(prob, 0.0) == n
    ks = [oracle.threshold_accept(prob, tau) for tau in np.linspace(0, 1, 41)]
    assert all(a >= b for a, b in zip(ks, ks[1:]))
    assert all(1 <= k <= n for k in ks)


def test_generation_tau_one_accepts_one_byte_per_step():
    W = synth.make_weights(TINY, seed=23, logit_gain=20.0)
    out, steps = oracle.generate(W, TINY, synth.make_prompt(0, 48), 10, 4, 1.0)
    assert len(out) == 10 and len(steps) == 10
    assert all(s["k"] == 1 for s in steps)


def test_n1_and_threshold_generation_first_byte_is_greedy():
    W = synth.make_weights(TINY, seed=24)
    p = synth.make_prompt(1, 40)
    g = oracle.greedy_generate(W, TINY, p, 12)
    out1, _ = oracle.generate(W, TINY, p, 12, 1, 0.5)
    np.testing.assert_array_equal(out1, g)


# ------------------------------------------------------------- verification --

def test_verify_forced_drafts():
    W = synth.make_weights(TINY, seed=25, gain_jitter=0.2)
    x = synth.make_prompt(2, 40)
    g = oracle.greedy_generate(W, TINY, x, 6)
    j, _ = oracle.verify_drafts(W, TINY, x, g)
    assert j == 6
    for m in range(2, 7):
        bad = g.copy()
        bad[m - 1] = (int(bad[m - 1]) + 1) % 256
        j, _ = oracle.verify_drafts(W, TINY, x, bad)
        assert j == m - 1


@pytest.mark.parametrize("gain,n", [(1.0, 3), (30.0, 4), (30.0, 7)])
def test_verify_generation_equals_greedy(gain, n):
    W = synth.make_weights(TINY, seed=26, logit_gain=gain)
    p = synth.make_prompt(3, 40)
    g = oracle.greedy_generate(W, TINY, p, 14)
    out, steps = oracle.generate(W, TINY, p, 14, n, 0.0, mode="verify")
    np.testing.assert_array_equal(out, g)
    assert all(1 <= s["k"] <= n for s in steps)


# ---------------------------------------------------- external verification --
# A separate next-byte model (no MB head) checks another model's drafts; kept drafts
# plus the verifier's greedy byte after them (Section 6, external verification).

TINY_FXT = synth.TINY_FXT


def test_external_verify_perfect_and_wrong_drafts():
    Wv = synth.make_weights(TINY_FXT, seed=27, gain_jitter=0.2)
    x = synth.make_prompt(2, 40)
    g = oracle.greedy_generate(Wv, TINY_FXT, x, 7)
    r = oracle.verify_external(Wv, TINY_FXT, x, g[:6])
    assert r["k"] == 7
    np.testing.assert_array_equal(r["bytes"], g)  # 6 kept drafts + the 7th greedy byte
    for m in range(6):
        bad = g[:6].copy()
        bad[m] = (int(bad[m]) + 1) % 256
        r = oracle.verify_external(Wv, TINY_FXT, x, bad)
        assert r["k"] == m + 1
        np.testing.assert_array_equal(r["bytes"], g[: m + 1])  # the bonus byte replaces the bad draft


def test_external_verify_by_the_drafting_model_is_self_verify_plus_one_byte():
    W = synth.make_weights(TINY, seed=28, logit_gain=30.0)
    x = list(synth.make_prompt(4, 40))
    for n in (2, 4, 6):
        s = oracle.verify_step(W, TINY, x, n)
        r = oracle.verify_external(W, TINY, x, s["cand"])
        acc = [int(c) for c in s["cand"][: s["k"]]]
        assert r["k"] == s["k"] + 1
        assert [int(b) for b in r["bytes"][:-1]] == acc
        assert int(r["bytes"][-1]) == int(oracle.greedy_generate(W, TINY, x + acc, 1)[0])


@pytest.mark.parametrize("same,gain,n", [(False, 1.0, 3), (False, 30.0, 5), (True, 30.0, 4)])
def test_external_generation_equals_verifier_greedy(same, gain, n):
    Wd = synth.make_weights(TINY, seed=29, logit_gain=gain)
    cfg_v, Wv = (TINY, Wd) if same else (TINY_FXT, synth.make_weights(TINY_FXT, seed=30, logit_gain=gain))
    p = synth.make_prompt(5, 40)
    out, steps = oracle.generate_external(Wd, TINY, Wv, cfg_v, p, 14, n)
    np.testing.assert_array_equal(out, oracle.greedy_generate(Wv, cfg_v, p, 14))
    assert all(1 <= s["k"] <= n + 1 for s in steps)
    if same:  # the verifier's own drafts: its first draft is always its greedy byte
        assert all(s["k"] >= 2 for s in steps[:-1])


# --------------------------------------------------------------- sampling --
# Temperature / top-p sampling with given uniforms and speculative sampling of drafts.

def _row(vals):
    r = np.full(256, -1e30)
    r[: len(vals)] = vals
    return r


def test_decoding_dist_closed_forms():
    rng = np.random.default_rng(0)
    l = rng.normal(size=256) * 3
    for T in (0.5, 1.0, 2.0):
        e = np.exp(l / T - np.max(l / T))
        np.testing.assert_allclose(oracle.decoding_dist(l, T, 1.0), e / e.sum(), rtol=1e-12, atol=1e-15)
    q = oracle.decoding_dist(l, 0.7, 1e-12)  # the nucleus is the top byte alone
    assert q[int(np.argmax(l))] == 1.0 and q.sum() == 1.0
    # hand example: P = .4 .3 .2 .1; the mass before byte 1 is .4 < .65, before byte 2 .7
    q = oracle.decoding_dist(_row(np.log([4.0, 3.0, 2.0, 1.0])), 1.0, 0.65)
    np.testing.assert_allclose(q[:4], [4 / 7, 3 / 7, 0.0, 0.0], atol=1e-12)
    # ties rank by lower byte value: of two equal top bytes (2/7 each) only byte 3 is kept
    # at top_p .25 (the mass before byte 4 is 2/7 > .25)
    q = oracle.decoding_dist(_row(np.log([1.0, 1.0, 1.0, 2.0, 2.0])), 1.0, 0.25)
    np.testing.assert_allclose(q[:5], [0, 0, 0, 1, 0], atol=1e-12)


def test_sample_byte_inverse_cdf_counts():
    q = oracle.decoding_dist(np.random.default_rng(1).normal(size=256) * 2, 0.8, 0.9)
    N = 20000
    counts = np.bincount([oracle.sample_byte(q, (k + 0.5) / N) for k in range(N)], minlength=256)
    assert np.all(np.abs(counts - q * N) <= 1.0 + 1e-9)
    assert counts[q == 0].sum() == 0


def test_sampled_step_with_a_one_byte_nucleus_is_greedy():
    W = synth.make_weights(TINY, seed=31, logit_gain=5.0)
    x = synth.make_prompt(6, 40)
    u = np.random.default_rng(2).random(12)
    s = oracle.step_sampled(W, TINY, x, 4, 0.5, 0.7, 1e-12, u)
    g = oracle.step(W, TINY, x, 4, 0.5)
    np.testing.assert_array_equal(s["cand"], g["cand"])
    assert s["k"] == 4 and np.all(s["prob"] == 1.0)
    # one-hot p and q: a rejected draft is replaced by the next-byte greedy byte, so the
    # step gives greedy verification's bytes plus that byte when a draft is rejected
    for n in (2, 4, 6):
        v = oracle.verify_step_sampled(W, TINY, x, n, 0.7, 1e-12, np.random.default_rng(n).random(3 * n))
        gv = oracle.verify_step(W, TINY, x, n)
        acc = [int(c) for c in gv["cand"][: gv["k"]]]
        assert [int(b) for b in v["bytes"][: gv["k"]]] == acc
        if gv["k"] < n:
            assert v["k"] == gv["k"] + 1
            assert int(v["bytes"][-1]) == int(oracle.greedy_generate(W, TINY, list(x) + acc, 1)[0])
        else:
            assert v["k"] == n


def test_speculative_accept_output_law_is_the_target():
    """The byte after c_1 has the target distribution p whatever the draft
    distribution q (the property speculative sampling guarantees): enumerate the draft
    over q and the two uniforms on grids."""
    rng = np.random.default_rng(3)
    for _ in range(3):
        p = rng.dirichlet(np.ones(8) * 0.7)
        q = rng.dirichlet(np.ones(8) * 0.7)
        N = 400
        law = np.zeros(8)
        for c in range(8):
            for a in range(N):
                for r in range(N):
                    u = np.zeros(6)
                    u[3], u[5] = (a + 0.5) / N, (r + 0.5) / N
                    out = oracle.speculative_accept([p], [None, q], [0, c], u, 2)
                    law[out[1]] += q[c] / (N * N)
        np.testing.assert_allclose(law, p, atol=3.0 / N)


# ------------------------------------------------------- learned boundaries --
# Boundary predictor at inference: logit = w . h_e / RMS(h_e) + b, a boundary where
# the probability is >= 0.5 (logit >= 0) or the segment reaches max_patch bytes.

LEARNED = TINY.replace(boundary="learned")


def _nospace(seed, length):
    x = synth.make_prompt(seed, length).copy()
    x[x == oracle.SPACE] = 65
    return x


def test_learned_boundaries_limits():
    x = _nospace(20, 70)
    W = synth.make_weights(LEARNED, seed=32)
    W["bp.w"] = np.zeros_like(W["bp.w"])
    W["bp.b"] = np.array([-1.0], np.float32)  # never: only the length cap remains
    assert oracle.trunk(W, LEARNED, x)["q"] == oracle.boundaries(x, LEARNED.max_patch)
    W["bp.b"] = np.array([1.0], np.float32)  # always
    assert oracle.trunk(W, LEARNED, x)["q"] == list(range(len(x)))


def test_learned_boundaries_are_causal_and_scale_free():
    W = synth.make_weights(LEARNED, seed=33)
    x = synth.make_prompt(21, 60)
    longer = np.concatenate([x, synth.make_prompt(22, 20)])
    q1 = oracle.trunk(W, LEARNED, x)["q"]
    q2 = [i for i in oracle.trunk(W, LEARNED, longer)["q"] if i < len(x)]
    assert q1 == q2 and 0 < len(q1) < len(x)
    h = oracle.trunk(W, LEARNED, x)["h_e"]
    np.testing.assert_allclose(oracle.boundary_logits(3.7 * h, W, 0.0), oracle.boundary_logits(h, W, 0.0), atol=1e-12)


def test_learned_boundaries_hand_computed():
    """Constructed states, d = 4, w = (1/4, 0, 0, 0), b = -1/4: the logits by hand,
    a logit of exactly 0 ends a segment, and max_patch = 2 closes a 2-byte segment."""
    W = {"bp.w": np.array([0.25, 0.0, 0.0, 0.0]), "bp.b": np.array([-0.25])}
    h = np.array([[1, 1, 1, 1], [-1, 1, 1, 1], [-1, 1, 1, 1], [4, 0, 0, 0], [-1, 1, 1, 1], [5, 5, 5, 5]], np.float64)
    np.testing.assert_allclose(oracle.boundary_logits(h, W, 0.0), [0.0, -0.5, -0.5, 0.25, -0.5, 0.0], atol=1e-15)
    assert oracle.learned_boundaries(h, W, 0, 0.0) == [0, 3, 5]
    assert oracle.learned_boundaries(h, W, 2, 0.0) == [0, 2, 3, 5]


# ------------------------------------------------------ full-sequence forward --

MB2 = TINY.replace(n_mb=2)


def test_log_softmax_is_scipys():
    from scipy.special import log_softmax as ref
    rng = np.random.default_rng(5)
    l = rng.normal(size=(7, 256)) * 30
    np.testing.assert_allclose(oracle.log_softmax(l), ref(l, axis=-1), atol=1e-12)


def test_forward_losses_uniform_logits_closed_form():
    """A zero unembedding gives all-zero logits: every NLL is log 256."""
    W = synth.make_weights(TINY, seed=40)
    W["unembed"] = np.zeros_like(W["unembed"])
    x = synth.make_prompt(30, 40)
    r = oracle.forward_losses(W, TINY, x, lam0=0.5, lam1=2.0, lam2=0.0)
    assert len(r["nll_nt"]) == 39 and len(r["nll_mb"]) == 38
    np.testing.assert_allclose(r["nll_nt"], np.log(256.0), atol=1e-12)
    np.testing.assert_allclose(r["nll_mb"], np.log(256.0), atol=1e-12)
    np.testing.assert_allclose(r["l_lm"], (0.5 * 39 + 2.0 * 38) * np.log(256.0), rtol=1e-12)


def test_boundary_loss_closed_forms():
    assert oracle.boundary_loss(30, 100, 0.4, 0.2) == 0.0
    assert abs(oracle.boundary_loss(50, 100, 0.4, 0.2) - 0.1) < 1e-15
    assert abs(oracle.boundary_loss(10, 100, 0.4, 0.2) - 0.1) < 1e-15
    W = synth.make_weights(TINY, seed=41)
    x = synth.make_prompt(31, 60)
    r = oracle.forward_losses(W, TINY, x, lam2=3.0, alpha=0.05, beta=0.0)
    assert r["k"] == len(oracle.boundaries(x, TINY.max_patch))
    np.testing.assert_allclose(r["total"], r["l_lm"] + 3.0 * (r["k"] / 60 - 0.05), rtol=1e-12)


def test_forward_nll_is_the_definition():
    """One position by hand: -log of the softmax probability of the target byte."""
    W = oracle.to_float64(synth.make_weights(TINY, seed=42, logit_gain=20.0))
    x = synth.make_prompt(32, 30)
    r = oracle.forward_losses(W, TINY, x)
    l = r["forward"]["nt"][11]
    p = np.exp(l - l.max()) / np.sum(np.exp(l - l.max()))
    np.testing.assert_allclose(r["nll_nt"][11], -np.log(p[x[12]]), rtol=1e-12)
    l = r["forward"]["mb"][11]
    p = np.exp(l - l.max()) / np.sum(np.exp(l - l.max()))
    np.testing.assert_allclose(r["nll_mb"][11], -np.log(p[x[13]]), rtol=1e-12)


def test_forward_rows_equal_decode_rows():
    """Every position of the full-sequence forward is the decode step on the prefix:
    next-byte row t = the step's row 1 after x[:t+1]; MB row t = its row 2 with the
    MB layers run over the whole sequence (window mode 1).  With two MB layers the
    windowed step (mode 0) differs, so the check tells the two masks apart."""
    W = oracle.to_float64(synth.make_weights(MB2, seed=43, gain_jitter=0.2))
    x = synth.make_prompt(33, 48)
    f = oracle.forward_full(W, MB2, x)
    full = MB2.replace(window_mode=1)
    differs = False
    for t in (0, 5, 17, 30, 47):
        st = oracle.step_logits(W, full, x[: t + 1], 2)
        np.testing.assert_allclose(f["nt"][t], st[0], atol=1e-10)
        np.testing.assert_allclose(f["mb"][t], st[1], atol=1e-10)
        differs |= np.max(np.abs(oracle.step_logits(W, MB2, x[: t + 1], 2)[1] - st[1])) > 1e-6
    assert differs
