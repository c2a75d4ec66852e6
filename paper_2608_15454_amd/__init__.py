"""Python binding of the MBP decode library (libmbp.so, HIP for gfx950).

Argument marshalling only: every step of the decode path runs in the library's
kernels.  PyTorch supplies device memory (weights, workspace, outputs) and the
stream.  There is no CPU fallback: if the library is missing, loading fails.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "MbpConfig", "MbpError", "Decoder", "lib", "lib_path", "make_config", "weight_manifest",
    "HEAD_LCA", "HEAD_MLP", "F32", "BF16", "F16", "THRESHOLD", "SELF_VERIFY",
    "OK", "EINVAL", "ECAPACITY", "EHIP", "ESTATE",
]

OK, EINVAL, ECAPACITY, EHIP, ESTATE = 0, -1, -2, -3, -4
HEAD_LCA, HEAD_MLP = 0, 1
F32, BF16, F16 = 0, 1, 2
THRESHOLD, SELF_VERIFY = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))


def lib_path() -> str:
    return os.path.join(_HERE, "libmbp.so")


class LossParams(ctypes.Structure):
    """Mirror of mbp_loss_params."""
    _fields_ = [("lambda0", ctypes.c_float), ("lambda1", ctypes.c_float), ("lambda2", ctypes.c_float),
                ("alpha", ctypes.c_float), ("beta", ctypes.c_float)]


class MbpConfig(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("d_ff", ctypes.c_int32),
        ("n_enc", ctypes.c_int32), ("n_lm", ctypes.c_int32), ("n_nb", ctypes.c_int32), ("n_mb", ctypes.c_int32),
        ("head", ctypes.c_int32), ("dtype", ctypes.c_int32),
        ("max_batch", ctypes.c_int32), ("max_ctx", ctypes.c_int32), ("max_latents", ctypes.c_int32),
        ("max_n", ctypes.c_int32), ("max_patch", ctypes.c_int32), ("max_window", ctypes.c_int32),
        ("max_chunk", ctypes.c_int32),
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float), ("attn_scale", ctypes.c_float),
        ("window_mode", ctypes.c_int32), ("kv_dtype", ctypes.c_int32), ("no_engine", ctypes.c_int32),
        ("boundary_mode", ctypes.c_int32),
    ]


class KernelTime(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64), ("ms", ctypes.c_double), ("bytes", ctypes.c_double)]


KCLASSES = ("gemv", "gemm", "attention", "other", "engine")

_lib = None


def lib():
    """Load libmbp.so (built by ``__graft_entry__.build()``); raise if it is absent."""
    global _lib
    if _lib is not None:
        return _lib
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"MBP HIP library not built ({path} missing); run __graft_entry__.build()")
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    cfgp = ctypes.POINTER(MbpConfig)
    L.mbp_weight_count.argtypes = [cfgp]
    L.mbp_weight_count.restype = ctypes.c_int32
    L.mbp_weight_info.argtypes = [cfgp, ctypes.c_int32, ctypes.c_char_p, ctypes.c_size_t,
                                  ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
    L.mbp_weight_info.restype = ctypes.c_int
    L.mbp_workspace_bytes.argtypes = [cfgp]
    L.mbp_workspace_bytes.restype = ctypes.c_size_t
    L.mbp_init.argtypes = [cfgp, ctypes.POINTER(P), ctypes.c_int32, P, ctypes.c_size_t, P, ctypes.POINTER(P)]
    L.mbp_init.restype = ctypes.c_int
    L.mbp_prefill.argtypes = [P, P, P, ctypes.c_int32]
    L.mbp_prefill.restype = ctypes.c_int
    L.mbp_decode_step.argtypes = [P, ctypes.c_int32, ctypes.c_float, ctypes.c_int32, P, P, P]
    L.mbp_decode_step.restype = ctypes.c_int
    L.mbp_decode_step_sampled.argtypes = [P, ctypes.c_int32, ctypes.c_float, ctypes.c_int32, ctypes.c_float,
                                          ctypes.c_float, P, P, P, P]
    L.mbp_decode_step_sampled.restype = ctypes.c_int
    L.mbp_verify_draft.argtypes = [P, P, ctypes.c_int32, P, P]
    L.mbp_verify_draft.restype = ctypes.c_int
    L.mbp_last_accepted.argtypes = [P, P, P]
    L.mbp_last_accepted.restype = ctypes.c_int
    L.mbp_accept.argtypes = [P, P, P]
    L.mbp_accept.restype = ctypes.c_int
    L.mbp_get_logits.argtypes = [P, P]
    L.mbp_get_logits.restype = ctypes.c_int
    L.mbp_row_length.argtypes = [P, ctypes.c_int32]
    L.mbp_row_length.restype = ctypes.c_int32
    L.mbp_row_boundaries.argtypes = [P, ctypes.c_int32, P, ctypes.c_int32]
    L.mbp_row_boundaries.restype = ctypes.c_int32
    L.mbp_forward_workspace_bytes.argtypes = [P, ctypes.c_int32]
    L.mbp_forward_workspace_bytes.restype = ctypes.c_size_t
    L.mbp_forward.argtypes = [P, P, ctypes.c_int32, P, P, ctypes.c_size_t, P, P]
    L.mbp_forward.restype = ctypes.c_int
    L.mbp_forward_static.argtypes = [P, P, ctypes.c_int32, P, P, P]
    L.mbp_forward_static.restype = ctypes.c_int
    L.mbp_forward_static_max_bytes.argtypes = []
    L.mbp_forward_static_max_bytes.restype = ctypes.c_size_t
    L.mbp_reset.argtypes = [P]
    L.mbp_reset.restype = ctypes.c_int
    L.mbp_destroy.argtypes = [P]
    L.mbp_destroy.restype = None
    L.mbp_last_error.argtypes = [P]
    L.mbp_last_error.restype = ctypes.c_char_p
    L.mbp_set_timing.argtypes = [P, ctypes.c_int32]
    L.mbp_set_timing.restype = ctypes.c_int
    L.mbp_read_timing.argtypes = [P, ctypes.POINTER(KernelTime)]
    L.mbp_read_timing.restype = ctypes.c_int
    _lib = L
    return L


class MbpError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"mbp error {code}: {msg}")
        self.code = code


def make_config(model, *, max_batch, max_ctx, max_latents=None, max_n=8, max_window=0, max_chunk=0,
                kv_dtype=None, engine=True) -> MbpConfig:
    """Fill an MbpConfig from any object with the model attributes (d_model, n_heads,
    d_ff, n_enc, n_lm, n_nb, n_mb, head 'lca'|'mlp', dtype 'f32'|'bf16', rope_base,
    rms_eps, attn_scale, max_patch, window_mode).  KV caches default to float16 for
    bfloat16 models (same bytes, 3 more mantissa bits) and float32 otherwise."""
    c = MbpConfig()
    c.d_model, c.n_heads, c.d_ff = model.d_model, model.n_heads, model.d_ff
    c.n_enc, c.n_lm, c.n_nb, c.n_mb = model.n_enc, model.n_lm, model.n_nb, model.n_mb
    c.head = HEAD_LCA if model.head == "lca" else HEAD_MLP
    c.dtype = BF16 if model.dtype == "bf16" else F32
    c.max_batch, c.max_ctx = max_batch, max_ctx
    c.max_latents = max_latents if max_latents is not None else max_ctx
    c.max_n, c.max_patch, c.max_window, c.max_chunk = max_n, model.max_patch, max_window, max_chunk
    c.rope_base, c.rms_eps, c.attn_scale = model.rope_base, model.rms_eps, model.attn_scale
    c.window_mode = model.window_mode
    if kv_dtype is None:
        kv_dtype = F16 if model.dtype == "bf16" else F32
    c.kv_dtype = kv_dtype
    c.no_engine = 0 if engine else 1
    c.boundary_mode = 1 if getattr(model, "boundary", "space") == "learned" else 0
    return c


def weight_manifest(cfg: MbpConfig):
    """The library's manifest: list of (name, (rows, cols))."""
    L = lib()
    n = L.mbp_weight_count(ctypes.byref(cfg))
    if n < 0:
        raise MbpError(n, "invalid config")
    out = []
    buf = ctypes.create_string_buffer(128)
    r, c = ctypes.c_int64(), ctypes.c_int64()
    for i in range(n):
        rc = L.mbp_weight_info(ctypes.byref(cfg), i, buf, 128, ctypes.byref(r), ctypes.byref(c))
        if rc:
            raise MbpError(rc, "weight_info")
        out.append((buf.value.decode(), (r.value, c.value)))
    return out


class Decoder:
    """One library handle with its device weights and workspace (torch tensors)."""

    def __init__(self, cfg: MbpConfig, weights: dict, device="cuda"):
        import torch

        self.torch = torch
        self.cfg = cfg
        self.L = lib()
        self.device = torch.device(device)
        man = weight_manifest(cfg)
        wdt = torch.bfloat16 if cfg.dtype == BF16 else torch.float32
        self.weights = []
        for name, (rows, cols) in man:
            a = np.asarray(weights[name], dtype=np.float32)
            if a.size != rows * cols:
                raise ValueError(f"weight {name}: size {a.size} != {rows}x{cols}")
            t = torch.from_numpy(np.ascontiguousarray(a).reshape(-1)).to(self.device).to(wdt).contiguous()
            self.weights.append(t)
        self.ws_bytes = self.L.mbp_workspace_bytes(ctypes.byref(cfg))
        if self.ws_bytes == 0:
            raise MbpError(EINVAL, "invalid config")
        self.workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        ptrs = (ctypes.c_void_p * len(self.weights))(*[t.data_ptr() for t in self.weights])
        self.stream = torch.cuda.current_stream(self.device)
        self.h = ctypes.c_void_p()
        rc = self.L.mbp_init(ctypes.byref(cfg), ptrs, len(self.weights), ctypes.c_void_p(self.workspace.data_ptr()),
                             self.ws_bytes, ctypes.c_void_p(self.stream.cuda_stream), ctypes.byref(self.h))
        if rc:
            raise MbpError(rc, "mbp_init failed")
        B, nmax = cfg.max_batch, cfg.max_n
        self.cand = torch.zeros((B, nmax), dtype=torch.uint8, device=self.device)
        self.prob = torch.zeros((B, nmax), dtype=torch.float32, device=self.device)
        self.accept_len = torch.zeros((B,), dtype=torch.int32, device=self.device)
        self.vout = torch.zeros((B, nmax), dtype=torch.uint8, device=self.device)
        self.logits_buf = torch.zeros((B, nmax, 256), dtype=torch.float32, device=self.device)
        self.batch = 0
        self.n = 0

    def _check(self, rc):
        if rc:
            msg = self.L.mbp_last_error(self.h)
            raise MbpError(rc, msg.decode() if msg else "")

    def close(self):
        if self.h:
            self.L.mbp_destroy(self.h)
            self.h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, prompts):
        prompts = [np.ascontiguousarray(p, dtype=np.uint8) for p in prompts]
        flat = np.concatenate(prompts)
        lens = np.array([len(p) for p in prompts], dtype=np.int32)
        self._check(self.L.mbp_prefill(self.h, flat.ctypes.data, lens.ctypes.data, len(prompts)))
        self.batch = len(prompts)

    def forward(self, seq, lam0=1.0, lam1=1.0, lam2=1.0, alpha=1.0, beta=0.0, work=None):
        """Full-sequence forward of one byte sequence (mbp_forward).  Returns device
        tensors nll [2, T] and loss [6]; every row is forgotten afterwards.  ``work``:
        a device uint8 tensor to reuse as the workspace (allocated when too small)."""
        torch = self.torch
        seq = np.ascontiguousarray(seq, dtype=np.uint8)
        T = len(seq)
        need = self.L.mbp_forward_workspace_bytes(ctypes.byref(self.cfg), T)
        if need == 0:
            raise MbpError(EINVAL, "forward workspace size")
        if work is None or work.numel() < need:
            work = torch.empty(need, dtype=torch.uint8, device=self.device)
        self.fwork = work
        nll = torch.zeros((2, T), dtype=torch.float32, device=self.device)
        loss = torch.zeros((6,), dtype=torch.float32, device=self.device)
        lp = LossParams(lam0, lam1, lam2, alpha, beta)
        self._check(self.L.mbp_forward(self.h, seq.ctypes.data, T, ctypes.byref(lp),
                                       ctypes.c_void_p(work.data_ptr()), work.numel(),
                                       ctypes.c_void_p(nll.data_ptr()), ctypes.c_void_p(loss.data_ptr())))
        self.batch = 0
        return nll, loss

    def forward_static(self, seq, lam0=1.0, lam1=1.0, lam2=1.0, alpha=1.0, beta=0.0):
        """forward() on the library's fixed scratch array (mbp_forward_static): no
        workspace is passed or allocated.  Returns device tensors nll [2, T], loss [6]."""
        torch = self.torch
        seq = np.ascontiguousarray(seq, dtype=np.uint8)
        T = len(seq)
        nll = torch.zeros((2, T), dtype=torch.float32, device=self.device)
        loss = torch.zeros((6,), dtype=torch.float32, device=self.device)
        lp = LossParams(lam0, lam1, lam2, alpha, beta)
        self._check(self.L.mbp_forward_static(self.h, seq.ctypes.data, T, ctypes.byref(lp),
                                              ctypes.c_void_p(nll.data_ptr()), ctypes.c_void_p(loss.data_ptr())))
        self.batch = 0
        return nll, loss

    def decode_step(self, n, tau, mode=THRESHOLD):
        """Enqueue one step; returns device views (cand [B,n], prob [B,n], accept_len [B])."""
        B = self.batch
        cand = self.cand.view(-1)[: B * n]
        prob = self.prob.view(-1)[: B * n]
        self._check(self.L.mbp_decode_step(self.h, n, float(tau), mode, ctypes.c_void_p(cand.data_ptr()),
                                           ctypes.c_void_p(prob.data_ptr()),
                                           ctypes.c_void_p(self.accept_len.data_ptr())))
        self.n = n
        return cand.view(B, n), prob.view(B, n), self.accept_len[:B]

    def decode_step_sampled(self, n, tau, mode, temperature, top_p, uniforms):
        """decode_step with candidates sampled at ``temperature`` / ``top_p`` with the
        device float uniforms [B, 3n]; returns the same device views as decode_step."""
        import torch

        B = self.batch
        uniforms = uniforms.contiguous()
        assert uniforms.dtype == torch.float32 and uniforms.numel() == B * 3 * n
        cand = self.cand.view(-1)[: B * n]
        prob = self.prob.view(-1)[: B * n]
        self._check(self.L.mbp_decode_step_sampled(self.h, n, float(tau), mode, float(temperature), float(top_p),
                                                   ctypes.c_void_p(uniforms.data_ptr()),
                                                   ctypes.c_void_p(cand.data_ptr()), ctypes.c_void_p(prob.data_ptr()),
                                                   ctypes.c_void_p(self.accept_len.data_ptr())))
        self.n = n
        return cand.view(B, n), prob.view(B, n), self.accept_len[:B]

    def verify_draft(self, draft):
        """External verification of another model's drafts (device uint8 [B, n], on this
        decoder's stream); returns device views (accepted bytes [B, n+1], accept_len [B])."""
        B = self.batch
        draft = draft.contiguous()
        n = int(draft.shape[1])
        out = self.vout.view(-1)[: B * (n + 1)]
        self._check(self.L.mbp_verify_draft(self.h, ctypes.c_void_p(draft.data_ptr()), n,
                                            ctypes.c_void_p(out.data_ptr()),
                                            ctypes.c_void_p(self.accept_len.data_ptr())))
        self.n = n + 1
        return out.view(B, n + 1), self.accept_len[:B]

    def last_accepted(self):
        B, nmax = self.batch, self.cfg.max_n
        out = np.zeros((B, nmax), dtype=np.uint8)
        lens = np.zeros((B,), dtype=np.int32)
        self._check(self.L.mbp_last_accepted(self.h, out.ctypes.data, lens.ctypes.data))
        return out, lens

    def accept(self, override=None):
        """Commit the step's accepted bytes, or ``override`` (list of byte arrays, one per row)."""
        if override is None:
            self._check(self.L.mbp_accept(self.h, None, None))
            return
        B, nmax = self.batch, self.cfg.max_n
        buf = np.zeros((B, nmax), dtype=np.uint8)
        lens = np.zeros((B,), dtype=np.int32)
        for b, row in enumerate(override):
            row = np.asarray(row, dtype=np.uint8).reshape(-1)
            buf[b, : min(len(row), nmax)] = row[:nmax]
            lens[b] = len(row)  # the library rejects lengths above max_n
        self._check(self.L.mbp_accept(self.h, buf.ctypes.data, lens.ctypes.data))

    def logits(self):
        B, n = self.batch, self.n
        view = self.logits_buf.view(-1)[: B * n * 256]
        self._check(self.L.mbp_get_logits(self.h, ctypes.c_void_p(view.data_ptr())))
        return view.view(B, n, 256)

    def row_length(self, row):
        r = self.L.mbp_row_length(self.h, row)
        if r < 0:
            raise MbpError(r, "row_length")
        return r

    def row_boundaries(self, row):
        """Positions of the bytes of ``row`` that closed a segment (numpy int32)."""
        n = self.L.mbp_row_boundaries(self.h, row, None, 0)
        if n < 0:
            raise MbpError(n, "row_boundaries")
        q = np.zeros(max(n, 1), dtype=np.int32)
        r = self.L.mbp_row_boundaries(self.h, row, q.ctypes.data_as(ctypes.c_void_p), n)
        if r < 0:
            raise MbpError(r, "row_boundaries")
        return q[:n]

    def reset(self):
        self._check(self.L.mbp_reset(self.h))
        self.batch = 0

    def set_timing(self, on: bool):
        self._check(self.L.mbp_set_timing(self.h, 1 if on else 0))

    def read_timing(self):
        """{class: (launches, ms, algorithmic bytes)} since timing was enabled."""
        out = (KernelTime * len(KCLASSES))()
        self._check(self.L.mbp_read_timing(self.h, out))
        return {k: (out[i].launches, out[i].ms, out[i].bytes) for i, k in enumerate(KCLASSES)}
