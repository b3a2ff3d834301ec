"""Python binding of the DVI decode-step engine (libdvi.so).

PyTorch supplies device memory (weights, LoRA factors, the workspace) and the
stream; every step of the decode path runs in the HIP kernels behind the C ABI.
Names follow the C entry points: prefill / draft / verify / commit /
update_drafter.
"""
from __future__ import annotations

import ctypes
import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _abi
from .schedule import KLRLSchedule


@dataclasses.dataclass
class EngineConfig:
    n_layers: int
    split_k: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    bf16: bool
    max_batch: int
    max_seq: int
    max_k_spec: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    lora_rank: int = 16
    lora_gamma: float = 1.0
    buffer_rows: int = 256

    @classmethod
    def from_shape(cls, shape, max_batch: int, max_seq: int, max_k_spec: int, buffer_rows: int = 256):
        """From any object with the model-shape attributes (n_layers, split_k, d_model, ...)."""
        return cls(n_layers=shape.n_layers, split_k=shape.split_k, d_model=shape.d_model,
                   n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                   ffn_dim=shape.ffn_dim, vocab=shape.vocab, bf16=shape.bf16, max_batch=max_batch,
                   max_seq=max_seq, max_k_spec=max_k_spec, rms_eps=shape.rms_eps,
                   rope_theta=shape.rope_theta, lora_rank=shape.lora_rank, lora_gamma=shape.lora_gamma,
                   buffer_rows=buffer_rows)

    def to_c(self) -> _abi.Config:
        return _abi.Config(self.n_layers, self.split_k, self.d_model, self.n_heads, self.n_kv_heads,
                           self.head_dim, self.ffn_dim, self.vocab, self.rms_eps, self.rope_theta,
                           self.max_batch, self.max_seq, self.max_k_spec, self.lora_rank, self.lora_gamma,
                           self.buffer_rows, _abi.BF16 if self.bf16 else _abi.FP32)


def workspace_bytes(cfg: EngineConfig) -> int:
    c = cfg.to_c()
    return int(_abi.load().dvi_workspace_bytes(ctypes.byref(c)))


def _dev(a, device) -> torch.Tensor:
    """Host array (numpy uint16 bf16 bits / float32) -> device tensor holding the same bytes."""
    if isinstance(a, torch.Tensor):
        return a.to(device).contiguous()
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device)
    return torch.from_numpy(a).to(device)


def _p(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.data_ptr()


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


class Engine:
    """One decode context on one GPU.

    weights: object with attributes tok_emb, layers (list of dicts with attn_norm, wq, wk, wv,
    wo, mlp_norm, w_gate, w_up, w_down), final_norm, lm_head, lora_A, lora_B holding numpy
    arrays (bf16 bit patterns as uint16, or float32) or torch tensors.
    """

    def __init__(self, cfg: EngineConfig, weights, device: str = "cuda:0"):
        self.cfg = cfg
        self.device = torch.device(device)
        self.lib = _abi.load()
        torch.cuda.set_device(self.device)
        # The engine's own stream (default priority): the null stream cannot be captured into the
        # HIP graphs that replay the draft and verify passes.  It starts after the work already
        # queued on the current stream (the weight uploads below are ordered by the wait in front
        # of dvi_create).
        self.stream = torch.cuda.Stream(self.device)
        L = cfg.n_layers
        # frozen weights: only needed until dvi_create has copied them into the workspace
        frozen = {"tok_emb": _dev(weights.tok_emb, self.device), "final_norm": _dev(weights.final_norm, self.device),
                  "lm_head": _dev(weights.lm_head, self.device)}
        names = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")
        per_layer = {n: [_dev(weights.layers[l][n], self.device) for l in range(L)] for n in names}
        self.lora_A = _dev(np.asarray(weights.lora_A, np.float32), self.device)
        self.lora_B = _dev(np.asarray(weights.lora_B, np.float32), self.device)
        arrs = {n: (ctypes.c_void_p * L)(*[t.data_ptr() for t in per_layer[n]]) for n in names}
        cw = _abi.Weights(frozen["tok_emb"].data_ptr(),
                          *[ctypes.cast(arrs[n], ctypes.POINTER(ctypes.c_void_p)) for n in names],
                          frozen["final_norm"].data_ptr(), frozen["lm_head"].data_ptr(),
                          self.lora_A.data_ptr(), self.lora_B.data_ptr())
        self._ccfg = cfg.to_c()
        nbytes = int(self.lib.dvi_workspace_bytes(ctypes.byref(self._ccfg)))
        if nbytes == 0:
            raise _abi.DVIError(_abi.ERR_ARG, "invalid configuration")
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = (self.workspace.data_ptr() + 255) & ~255
        for t in (self.workspace, self.lora_A, self.lora_B):
            t.record_stream(self.stream)
        self.stream.wait_stream(torch.cuda.current_stream(self.device))
        ctx = ctypes.c_void_p()
        st = self.lib.dvi_create(ctypes.byref(self._ccfg), ctypes.byref(cw), base, nbytes,
                                 self.stream.cuda_stream, ctypes.byref(ctx))
        self.ctx = ctx.value
        if st != _abi.OK:
            msg = self.lib.dvi_last_error(self.ctx).decode() if self.ctx else "dvi_create failed"
            if self.ctx:
                self.lib.dvi_destroy(self.ctx)
                self.ctx = None
            raise _abi.DVIError(st, msg)
        del frozen, per_layer, arrs
        self.batch = 0
        self.k_spec = 0
        self.opt_step = 0
        self.baseline = 0.0
        self.updates = 0

    def close(self):
        if getattr(self, "ctx", None):
            self.stream.synchronize()
            self.lib.dvi_destroy(self.ctx)
            self.ctx = None

    def set_sampling(self, tau: float, seed: int = 0):
        """Draw every draft from softmax(z / tau) with seeded Gumbel-max noise (tau = 0: argmax
        drafting, the default).  Commits are unchanged: they are greedy decoding's."""
        self._check(self.lib.dvi_set_sampling(self.ctx, float(tau), int(seed) & 0xFFFFFFFFFFFFFFFF))

    def set_graphs(self, enable: bool):
        """Replay the draft and verify passes as captured HIP graphs (the default) or launch
        every kernel directly; results are bitwise the same."""
        self._check(self.lib.dvi_set_graphs(self.ctx, 1 if enable else 0))

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ------------------------------------------------------------------ helpers
    def _check(self, st: int):
        if st != _abi.OK:
            raise _abi.DVIError(st, self.lib.dvi_last_error(self.ctx).decode())

    def status_of(self, fn, *args) -> int:
        """Call a raw C entry point and return its status (for error-path tests)."""
        return getattr(self.lib, fn)(self.ctx, *args)

    # ------------------------------------------------------------------ decode step
    def prefill(self, ids, lens=None) -> np.ndarray:
        """ids [B, P]; lens [B] (default: P for every sequence) -- sequence b's prompt is
        ids[b, :lens[b]]."""
        ids = _i32(ids)
        if ids.ndim == 1:
            ids = ids[None]
        B, P = ids.shape
        lens = np.full(B, P, np.int32) if lens is None else _i32(lens).reshape(B)
        first = np.empty(B, np.int32)
        st = self.lib.dvi_prefill(self.ctx, B, ids.ctypes.data, lens.ctypes.data, P, first.ctypes.data)
        if st in (_abi.OK, _abi.ERR_NUMERIC):  # the prefill ran (a non-finite head logit is reported after it)
            self.batch = B
            self.k_spec = 1   # read_logits() now returns the prefill head's row per sequence
        self._check(st)
        return first

    def draft(self, k_spec: int, forced=None, want: bool = False) -> Optional[np.ndarray]:
        out = np.empty((self.batch, k_spec), np.int32) if want else None
        f = _i32(forced).reshape(self.batch, k_spec) if forced is not None else None
        self._check(self.lib.dvi_draft(self.ctx, k_spec, f.ctypes.data if f is not None else None,
                                       out.ctypes.data if out is not None else None))
        self.k_spec = k_spec
        return out

    def verify(self, want: bool = False):
        if not want:
            self._check(self.lib.dvi_verify(self.ctx, None, None))
            return None
        tg = np.empty((self.batch, self.k_spec), np.int32)
        m = np.empty(self.batch, np.int32)
        self._check(self.lib.dvi_verify(self.ctx, tg.ctypes.data, m.ctypes.data))
        return tg, m

    def commit(self, max_new=None, forced=None):
        tok = np.empty((self.batch, self.k_spec), np.int32)
        n = np.empty(self.batch, np.int32)
        m = np.empty(self.batch, np.int32)
        mx = _i32(max_new) if max_new is not None else None
        f = _i32(forced).reshape(self.batch, self.k_spec) if forced is not None else None
        self._check(self.lib.dvi_commit(self.ctx, mx.ctypes.data if mx is not None else None,
                                        f.ctypes.data if f is not None else None,
                                        tok.ctypes.data, n.ctypes.data, m.ctypes.data))
        return tok, n, m

    def decode_steps(self, k_spec: int, n_steps: int, max_new=None):
        """n_steps draft/verify/commit steps in one call (no host sync between them): tokens
        [n_steps, batch, k_spec] (-1 past n), n [n_steps, batch], m [n_steps, batch]."""
        tok = np.empty((n_steps, self.batch, k_spec), np.int32)
        n = np.empty((n_steps, self.batch), np.int32)
        m = np.empty((n_steps, self.batch), np.int32)
        mx = _i32(max_new) if max_new is not None else None
        self._check(self.lib.dvi_decode_steps(self.ctx, k_spec, n_steps, mx.ctypes.data if mx is not None else None,
                                              tok.ctypes.data, n.ctypes.data, m.ctypes.data))
        self.k_spec = k_spec
        return tok, n, m

    def abort(self):
        self._check(self.lib.dvi_abort_step(self.ctx))

    # ------------------------------------------------------------------ drafter update
    def update_drafter(self, c_kl, c_ce, c_pg, c_ent=0.0, tau=1.0, baseline=0.0, lr=1e-3,
                       beta1=0.9, beta2=0.999, eps=1e-8, opt_step=None, grads: bool = False):
        g_A = torch.empty_like(self.lora_A) if grads else None
        g_B = torch.empty_like(self.lora_B) if grads else None
        if grads:
            self.stream.wait_stream(torch.cuda.current_stream(self.device))
        if lr != 0.0 and opt_step is None:
            self.opt_step += 1
            opt_step = self.opt_step
        args = _abi.UpdateArgs(c_kl, c_ce, c_pg, c_ent, tau, baseline, lr, beta1, beta2, eps,
                               int(opt_step or 0), _p(g_A), _p(g_B))
        stats = _abi.UpdateStats()
        self._check(self.lib.dvi_update_drafter(self.ctx, ctypes.byref(args), ctypes.byref(stats)))
        out = {k: getattr(stats, k) for k, _ in _abi.UpdateStats._fields_}
        if grads:
            out["grad_A"], out["grad_B"] = g_A, g_B
        return out

    # ------------------------------------------------------------------ inspection
    def read_kv(self, layer: int, seq: int, pos0: int, npos: int):
        c = self.cfg
        dt = np.uint16 if c.bf16 else np.float32
        k = np.empty((c.n_kv_heads, npos, c.head_dim), dt)
        v = np.empty_like(k)
        self._check(self.lib.dvi_read_kv(self.ctx, layer, seq, pos0, npos, k.ctypes.data, v.ctypes.data))
        return k, v

    def read_logits(self) -> np.ndarray:
        out = np.empty((self.batch, self.k_spec, self.cfg.vocab), np.float32)
        self._check(self.lib.dvi_read_logits(self.ctx, out.ctypes.data))
        return out

    def read_draft_logits(self) -> np.ndarray:
        out = np.empty((self.batch, self.cfg.vocab), np.float32)
        self._check(self.lib.dvi_read_draft_logits(self.ctx, out.ctypes.data))
        return out

    def lengths(self) -> np.ndarray:
        out = np.empty(self.batch, np.int32)
        self._check(self.lib.dvi_read_lengths(self.ctx, out.ctypes.data))
        return out

    def buffer_info(self):
        v, n = ctypes.c_int32(), ctypes.c_int32()
        self._check(self.lib.dvi_buffer_info(self.ctx, ctypes.byref(v), ctypes.byref(n)))
        return v.value, n.value

    def read_buffer(self, row0: int, nrows: int) -> Dict[str, np.ndarray]:
        c = self.cfg
        out = {"h": np.empty((nrows, c.d_model), np.float32), "a": np.empty(nrows, np.int32),
               "logits": np.empty((nrows, c.vocab), np.float32), "r": np.empty(nrows, np.int8),
               "fresh": np.empty(nrows, np.int8), "i": np.empty(nrows, np.int32), "prev": np.empty(nrows, np.int32)}
        self._check(self.lib.dvi_read_buffer(self.ctx, row0, nrows, *[out[k].ctypes.data for k in
                                                                      ("h", "a", "logits", "r", "fresh", "i", "prev")]))
        return out

    def write_buffer(self, h, a, logits, r, fresh):
        h = np.ascontiguousarray(h, np.float32)
        a, lg = _i32(a), np.ascontiguousarray(logits, np.float32)
        r, fr = np.ascontiguousarray(r, np.int8), np.ascontiguousarray(fresh, np.int8)
        self._check(self.lib.dvi_write_buffer(self.ctx, h.shape[0], h.ctypes.data, a.ctypes.data, lg.ctypes.data,
                                              r.ctypes.data, fr.ctypes.data))

    def probe(self, which: str):
        """Time every launch of one kernel class with HIP events (see dvi_probe_kernel)."""
        self._check(self.lib.dvi_probe_kernel(self.ctx, _abi.PROBES[which]))

    def probe_read(self):
        t, n, b = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
        self._check(self.lib.dvi_probe_read(self.ctx, ctypes.byref(t), ctypes.byref(n), ctypes.byref(b)))
        return {"ms": t.value, "launches": n.value, "bytes": b.value}

    def read_rate(self, nbytes: int, reps: int = 5) -> float:
        """Streaming-read reference: GB/s of the fastest of reps reads of a fresh device buffer
        (see dvi_measure_read_rate)."""
        buf = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.stream.wait_stream(torch.cuda.current_stream(self.device))
        v = ctypes.c_double()
        self._check(self.lib.dvi_measure_read_rate(self.ctx, buf.data_ptr(), nbytes, reps, ctypes.byref(v)))
        del buf
        return v.value

    def timings(self) -> Dict[str, float]:
        vals = [ctypes.c_double() for _ in range(4)]
        self._check(self.lib.dvi_get_timings(self.ctx, *[ctypes.byref(v) for v in vals]))
        return dict(zip(("draft", "verify", "commit", "update"), [v.value for v in vals]))

    # ------------------------------------------------------------------ driver
    def generate(self, prompts, n_new: int, k_spec: int, update_every: int = 0,
                 schedule: Optional[KLRLSchedule] = None, lr: float = 1e-3, on_step=None, lens=None):
        """Prefill then decode until every sequence has n_new tokens (the first from the prefill).

        Returns (tokens [B, n_new], info) with per-step accept lengths m and commit counts n.
        update_every > 0 runs a drafter update after every update_every decode steps, with
        coefficients from the KL->RL schedule.  lens: per-sequence prompt lengths (see prefill)."""
        first = self.prefill(prompts, lens)
        B = self.batch
        out: List[List[int]] = [[int(t)] for t in first]
        remaining = np.full(B, n_new - 1, np.int32)
        ms, ns, upd = [], [], []
        step = 0
        sched = schedule or KLRLSchedule()
        while remaining.max() > 0:
            self.draft(k_spec)
            self.verify()
            tok, n, m = self.commit(max_new=remaining)
            for b in range(B):
                out[b].extend(int(t) for t in tok[b, :n[b]])
            remaining -= n
            ms.append(m.copy())
            ns.append(n.copy())
            step += 1
            if on_step is not None:
                on_step(self, step)
            if update_every and step % update_every == 0 and k_spec > 1:
                c = sched.coeffs(self.updates, self.baseline)
                st = self.update_drafter(c["c_kl"], c["c_ce"], c["c_pg"], c["c_ent"], c["tau"],
                                         self.baseline, lr=lr)
                upd.append(st)
                if st["fresh"] > 0:
                    self.baseline = sched.ema(self.baseline, st["fresh_accepted"] / st["fresh"])
                self.updates += 1
        return np.array(out, np.int32), {"m": np.array(ms), "n": np.array(ns), "updates": upd, "steps": step}
