"""Float32 KV-cached CPU decoder of the MBP step -- TEST INFRASTRUCTURE ONLY.

The CPU baseline that ``bench.py`` times beside the GPU (and nothing else uses): the
same method as ``oracle.model`` (Algorithm 1 with the readings listed there), run
the way a CPU implementation would run it, with per-layer key/value caches for the
encoder, the LM module and the next-byte decoder, the LM module run only on the
segments a commit closes, and the MB window recomputed from the cached latents at
every step.  float32 throughout (the bf16 weights upcast exactly).  Checked against
the float64 full recompute of ``oracle.model`` by the CPU tests.
"""
from __future__ import annotations

import numpy as np

from .model import SPACE


def _rms(x, g, eps):
    ms = np.mean(x * x, axis=-1, keepdims=True, dtype=np.float32)
    return (x / np.sqrt(ms + np.float32(eps))) * g


def _silu(x):
    return x / (np.float32(1.0) + np.exp(-x))


class _Cache:
    """Rotated keys and values of one layer: [cap, H, dh] each, the first n rows valid."""

    def __init__(self, cap, H, dh):
        self.k = np.zeros((cap, H, dh), np.float32)
        self.v = np.zeros((cap, H, dh), np.float32)
        self.n = 0


class CachedDecoder:
    """One sequence: prefill(prompt), then step(n, tau) + accept(bytes) (threshold
    acceptance) or verify_step(n) (self-verification, which commits what it keeps)."""

    def __init__(self, W, cfg, cap):
        if cfg.boundary != "space" or cfg.window_mode != 0:
            raise ValueError("the cached decoder covers the space rule and the window of Algorithm 1")
        self.cfg = cfg
        W = {k: np.asarray(v, np.float32) for k, v in W.items()}
        self.W = W
        d, H = cfg.d_model, cfg.n_heads
        self.d, self.H, self.dh = d, H, d // H
        self.cap = cap
        half = self.dh // 2
        inv = (np.float64(cfg.rope_base) ** (-np.arange(0, self.dh, 2, dtype=np.float64) / self.dh))
        ang = np.arange(cap + 16, dtype=np.float64)[:, None] * inv[None, :]
        self.cos = np.cos(ang).astype(np.float32).reshape(-1, 1, half)
        self.sin = np.sin(ang).astype(np.float32).reshape(-1, 1, half)
        self.scale = np.float32(cfg.attn_scale / np.sqrt(self.dh))

        def layers(name, n):
            out = []
            for i in range(n):
                P = {p: W[f"{name}.{i}.{p}"] for p in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate",
                                                       "w_up", "w_down")}
                P["wqkv_t"] = np.ascontiguousarray(np.concatenate([P["wq"], P["wk"], P["wv"]], 0).T)
                P["wo_t"] = np.ascontiguousarray(P["wo"].T)
                P["wgu_t"] = np.ascontiguousarray(np.concatenate([P["w_gate"], P["w_up"]], 0).T)
                P["wd_t"] = np.ascontiguousarray(P["w_down"].T)
                out.append(P)
            return out

        self.enc = layers("enc", cfg.n_enc)
        self.lm = layers("lm", cfg.n_lm)
        self.nt = layers("nt", cfg.n_nb)
        self.mb = layers("mb", cfg.n_mb) if cfg.head == "lca" else []
        self.unembed_t = np.ascontiguousarray(W["unembed"].T)
        self.reset()

    def reset(self):
        cfg, H, dh = self.cfg, self.H, self.dh
        self.x = []          # committed bytes
        self.q = []          # boundary positions
        self.he = np.zeros((self.cap, self.d), np.float32)
        self.lmin = np.zeros((self.cap + 1, self.d), np.float32)
        self.hlm = np.zeros((self.cap + 1, self.d), np.float32)
        self.k_lat = 0       # latent rows through the LM module (BOS included)
        self.c_enc = [_Cache(self.cap, H, dh) for _ in self.enc]
        self.c_lm = [_Cache(self.cap + 1, H, dh) for _ in self.lm]
        self.c_nt = [_Cache(self.cap, H, dh) for _ in self.nt]
        self.h1 = None

    # ---------------------------------------------------------------- blocks --
    def _rope(self, x, pos):
        c, s = self.cos[pos], self.sin[pos]
        x0, x1 = x[..., 0::2], x[..., 1::2]
        out = np.empty_like(x)
        out[..., 0::2] = x0 * c - x1 * s
        out[..., 1::2] = x0 * s + x1 * c
        return out

    def _attend(self, q, k, v, mask):
        """q [m, H, dh], k/v [T, H, dh], mask [m, T] (True = visible) -> [m, d]."""
        m = q.shape[0]
        out = np.empty((m, self.H, self.dh), np.float32)
        for h in range(self.H):
            s = (q[:, h, :] @ k[:, h, :].T) * self.scale
            s = np.where(mask, s, -np.inf)
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[:, h, :] = p @ v[:, h, :]
        return out.reshape(m, self.d)

    def _ffn(self, a, P):
        y = _rms(a, P["ffn_norm"], self.cfg.rms_eps)
        gu = y @ P["wgu_t"]
        f = self.cfg.d_ff
        return a + (_silu(gu[:, :f]) * gu[:, f:]) @ P["wd_t"]

    def _cached_stack(self, u, layers, caches, pos):
        """Causal stack over new rows u [m, d] at positions pos (consecutive, after the
        cached ones); their keys and values are appended to the caches."""
        h = u
        m = h.shape[0]
        for P, c in zip(layers, caches):
            x = _rms(h, P["attn_norm"], self.cfg.rms_eps)
            qkv = (x @ P["wqkv_t"]).reshape(m, 3, self.H, self.dh)
            q = self._rope(qkv[:, 0], pos)
            c.k[c.n: c.n + m] = self._rope(qkv[:, 1], pos)
            c.v[c.n: c.n + m] = qkv[:, 2]
            c.n += m
            T = c.n
            mask = np.arange(T)[None, :] <= (T - m + np.arange(m))[:, None]
            h = h + self._attend(q, c.k[:T], c.v[:T], mask) @ P["wo_t"]
            h = self._ffn(h, P)
        return h

    def _plain_stack(self, u, layers, mask, pos):
        h = u
        m = h.shape[0]
        for P in layers:
            x = _rms(h, P["attn_norm"], self.cfg.rms_eps)
            qkv = (x @ P["wqkv_t"]).reshape(m, 3, self.H, self.dh)
            q, k = self._rope(qkv[:, 0], pos), self._rope(qkv[:, 1], pos)
            h = h + self._attend(q, k, qkv[:, 2], mask) @ P["wo_t"]
            h = self._ffn(h, P)
        return h

    # ---------------------------------------------------------------- commit --
    def _group(self, i):
        return int(np.searchsorted(self.q, i, side="right"))

    def commit(self, new):
        """Append bytes: encoder, segmentation, LM module on the closed segments, NT."""
        cfg = self.cfg
        new = [int(b) for b in new]
        if not new:
            return
        t0 = len(self.x)
        pos = np.arange(t0, t0 + len(new))
        E = self.W["emb"][np.asarray(new)]
        self.he[pos] = self._cached_stack(E, self.enc, self.c_enc, pos)
        lat_rows = []
        if self.k_lat == 0:  # BOS opens a fresh sequence's latent list
            self.lmin[0] = self.W["bos"]
            lat_rows.append(0)
        for i, b in zip(pos, new):
            self.x.append(b)
            prev = self.q[-1] if self.q else -1
            if b == SPACE or (cfg.max_patch > 0 and i - prev >= cfg.max_patch):
                self.q.append(int(i))
                j = len(self.q)
                self.lmin[j] = self.he[prev + 1: i + 1].mean(axis=0, dtype=np.float32)
                lat_rows.append(j)
        if lat_rows:
            lp = np.asarray(lat_rows)
            self.hlm[lp] = self._cached_stack(self.lmin[lp], self.lm, self.c_lm, lp)
            self.k_lat = lat_rows[-1] + 1
        L = np.asarray([self._group(i) for i in pos])
        h = self._cached_stack(self.hlm[L] + self.he[pos], self.nt, self.c_nt, pos)
        self.h1 = h[-1]

    def prefill(self, prompt):
        self.reset()
        self.commit(prompt)

    # ------------------------------------------------------------------ step --
    def _head(self, h, g):
        return _rms(h, g, self.cfg.rms_eps) @ self.unembed_t

    def logits(self, n):
        cfg = self.cfg
        t = len(self.x) - 1
        rows = [self._head(self.h1[None, :], self.W["nt_norm"])[0]]
        if n >= 2 and cfg.head == "mlp":
            for m in range(2, n + 1):
                P = {k: self.W[f"mlp.{m - 2}.{k}"] for k in ("norm", "w_gate", "w_up", "w_down")}
                y = _rms(self.h1[None, :], P["norm"], cfg.rms_eps)
                hm = self.h1 + ((_silu(y @ P["w_gate"].T) * (y @ P["w_up"].T)) @ P["w_down"].T)[0]
                rows.append(self._head(hm[None, :], self.W["nt_norm"])[0])
        elif n >= 2:
            g = self._group(t)
            s = (0 if g < 2 else self.q[g - 2]) if g >= 1 else 0
            P = np.arange(s, t + n - 1)
            G = np.array([self._group(p) if p <= t else g for p in P])
            mask = ((G[None, :] == G[:, None]) & (P[None, :] <= P[:, None])) | (G[None, :] == G[:, None] - 1)
            z = self.hlm + self.lmin
            h2 = self._plain_stack(z[G], self.mb, mask, P)
            rows += list(self._head(h2[t - s: t - s + n - 1], self.W["mb_norm"]))
        return np.array(rows, np.float32)

    def step(self, n, tau):
        l = self.logits(n)
        c = np.argmax(l, axis=1)
        p = 1.0 / np.sum(np.exp(l - l[np.arange(n), c][:, None]), axis=1)
        k = 1
        while k < n and p[k] >= tau:
            k += 1
        return {"logits": l, "cand": c, "prob": p, "k": k}

    def verify_step(self, n):
        """Self-verification: drafts c_1..c_n from one step; c_1 is committed, then
        each next draft is kept (and committed) while it equals the next-byte greedy
        byte after the drafts before it.  The kept drafts are committed on return:
        the caller does not call accept."""
        r = self.step(n, 2.0)
        c = [int(v) for v in r["cand"]]
        j = 1
        self.commit(c[:1])
        while j < n:
            gm = int(np.argmax(self._head(self.h1[None, :], self.W["nt_norm"])[0]))
            if gm != c[j]:
                break
            self.commit(c[j: j + 1])
            j += 1
        r["k"] = j
        return r

    def accept(self, acc):
        self.commit(acc)
