"""CPU oracle for DVI's self-speculative decode step (arxiv 2510.05421).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything here.  The
product path (``paper_2510_05421_amd``) never imports this package, and this
package never imports the product path: the two share no code, only the
seeded inputs from ``synth``.

Contents
  model.c    float64 decoder forward, heads (Section 3.1)
  dvi.py     greedy autoregressive decoding (the definition of the committed
             output) and the DVI draft/verify/commit/log rollout (Section 3.3)
  update.py  the KL->RL drafter objective, its gradient, Adam and the schedule
             (Section 3.4)
  sampling.py  seeded stochastic drafting (t~ ~ p_theta, Section 3.3) by
             Gumbel-max with Philox4x64-10 uniforms

What pins each part (tests/test_oracle_pins.py, tests/test_oracle_update_pins.py):
  layers / heads      a float64 reference assembled from torch.nn.functional
                      (rms_norm, linear, scaled_dot_product_attention, silu) with a
                      complex-number rotary embedding; GQA == MHA with shared kv
                      weights; block == token-by-token (bitwise); scipy softmax for
                      one attention row; A_s = 0 draft head == target head
  greedy_ar           the definition itself (argmax of the pinned forward); the gap it
                      records per token is its logits row's top-2 gap
  top2_gap            hand values (a tie for the maximum gives 0), a sorted-values brute
                      force on batched rows with repeats and on 32000-wide rows
  dvi_generate        losslessness (== greedy_ar for random LoRA, forced-wrong and
                      forced-right drafts, k_spec 1/2/4/8); every m forced by
                      construction; brute-force m; split k = L accepts everything;
                      buffer count / reward pattern; rolled-back cache bitwise equal
                      across different rejected drafts and to the AR cache; each logged
                      row's prev_id is the token whose state drafted it, and its h_hat is
                      reproduced bitwise by a fresh forward ending in that token
  loss_and_grad       finite differences per term; scipy rel_entr / entropy for the
                      loss terms; closed-form dL/dz for masked CE; row sums of
                      dL/dz = 0; KL = 0 and gradient 0 at z = logits/tau; A_s = 0 =>
                      dB = 0; gamma = 0 => no gradient; torch autograd
  adam_step           torch.optim.Adam
  sampling            Philox4x64-10 == numpy's Philox bit generator (bit for bit);
                      sampled drafts follow softmax(z / tau) (chi-square); the rollout
                      with sampled drafts == greedy_ar (tests/test_oracle_sampling.py)
  Schedule            closed-form values.  The schedule's constants (lambda0,
                      lambda_kl_min, lambda_pg_max, w_rl, T_warmup, T_ramp, EMA rate)
                      are not given in the paper: parity unpinned for those values.
  acceptance / MAT    on synthetic weights: parity unpinned (the paper's numbers
                      need its model and data)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile model.c with gcc: -O2, OpenMP, no fast-math, no FMA contraction."""
    src = os.path.join(_HERE, "model.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                               "-fno-fast-math", "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


class _Model(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("bf16", ctypes.c_int32),
        ("eps", ctypes.c_double), ("theta", ctypes.c_double),
        ("tok_emb", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
        ("attn_norm", ctypes.POINTER(ctypes.c_void_p)), ("wq", ctypes.POINTER(ctypes.c_void_p)),
        ("wk", ctypes.POINTER(ctypes.c_void_p)), ("wv", ctypes.POINTER(ctypes.c_void_p)),
        ("wo", ctypes.POINTER(ctypes.c_void_p)), ("mlp_norm", ctypes.POINTER(ctypes.c_void_p)),
        ("wg", ctypes.POINTER(ctypes.c_void_p)), ("wu", ctypes.POINTER(ctypes.c_void_p)),
        ("wd", ctypes.POINTER(ctypes.c_void_p)),
    ]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        lib = ctypes.CDLL(_SO)
        P, i32, dbl = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double
        mp = ctypes.POINTER(_Model)
        lib.orc_embed.argtypes = [mp, P, i32, P]
        lib.orc_layers.argtypes = [mp, P, P, i32, i32, i32, i32, i32, P]
        lib.orc_final_norm.argtypes = [mp, P, i32, P]
        lib.orc_target_logits.argtypes = [mp, P, i32, P]
        lib.orc_draft_logits.argtypes = [mp, P, i32, P, P, i32, dbl, P]
        for f in (lib.orc_embed, lib.orc_layers, lib.orc_final_norm, lib.orc_target_logits,
                  lib.orc_draft_logits):
            f.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


class OracleModel:
    """Frozen backbone + the two vocabulary heads, on the CPU in float64."""

    def __init__(self, weights):
        self.w = weights
        s = weights.shape
        self.shape = s
        lib = _load()
        L = s.n_layers

        def arr(name):
            a = (ctypes.c_void_p * L)(*[_ptr(weights.layers[l][name]) for l in range(L)])
            return a

        self._arrs = {n: arr(n) for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm",
                                          "w_gate", "w_up", "w_down")}
        self._m = _Model(
            n_layers=L, d=s.d_model, n_heads=s.n_heads, n_kv_heads=s.n_kv_heads,
            head_dim=s.head_dim, ffn=s.ffn_dim, vocab=s.vocab, bf16=int(s.bf16),
            eps=s.rms_eps, theta=s.rope_theta,
            tok_emb=_ptr(weights.tok_emb), final_norm=_ptr(weights.final_norm),
            lm_head=_ptr(weights.lm_head),
            attn_norm=ctypes.cast(self._arrs["attn_norm"], ctypes.POINTER(ctypes.c_void_p)),
            wq=ctypes.cast(self._arrs["wq"], ctypes.POINTER(ctypes.c_void_p)),
            wk=ctypes.cast(self._arrs["wk"], ctypes.POINTER(ctypes.c_void_p)),
            wv=ctypes.cast(self._arrs["wv"], ctypes.POINTER(ctypes.c_void_p)),
            wo=ctypes.cast(self._arrs["wo"], ctypes.POINTER(ctypes.c_void_p)),
            mlp_norm=ctypes.cast(self._arrs["mlp_norm"], ctypes.POINTER(ctypes.c_void_p)),
            wg=ctypes.cast(self._arrs["w_gate"], ctypes.POINTER(ctypes.c_void_p)),
            wu=ctypes.cast(self._arrs["w_up"], ctypes.POINTER(ctypes.c_void_p)),
            wd=ctypes.cast(self._arrs["w_down"], ctypes.POINTER(ctypes.c_void_p)),
        )
        self._lib = lib

    # --- state -----------------------------------------------------------------------
    def new_cache(self, s_max: int):
        """Per-sequence K and V caches, float64 [n_layers, s_max, kv_dim]."""
        s = self.shape
        return (np.zeros((s.n_layers, s_max, s.kv_dim)), np.zeros((s.n_layers, s_max, s.kv_dim)))

    # --- forward pieces ----------------------------------------------------------------
    def embed(self, tokens) -> np.ndarray:
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        h = np.empty((tok.size, self.shape.d_model))
        self._lib.orc_embed(ctypes.byref(self._m), _ptr(tok), tok.size, _ptr(h))
        return h

    def layers(self, cache, h: np.ndarray, pos0: int, l0: int, l1: int) -> np.ndarray:
        """Layers [l0, l1) (0-based) on rows of h at positions pos0.. ; returns new h."""
        kc, vc = cache
        h = np.array(h, dtype=np.float64, order="C", copy=True)
        n = h.shape[0]
        assert pos0 + n <= kc.shape[1], "cache too small"
        self._lib.orc_layers(ctypes.byref(self._m), _ptr(kc), _ptr(vc), kc.shape[1], pos0, n,
                             l0, l1, _ptr(h))
        return h

    def final_norm(self, h: np.ndarray) -> np.ndarray:
        h = np.ascontiguousarray(h, dtype=np.float64)
        out = np.empty_like(h)
        self._lib.orc_final_norm(ctypes.byref(self._m), _ptr(h), h.shape[0], _ptr(out))
        return out

    def target_logits(self, hn: np.ndarray) -> np.ndarray:
        hn = np.ascontiguousarray(hn, dtype=np.float64)
        out = np.empty((hn.shape[0], self.shape.vocab))
        self._lib.orc_target_logits(ctypes.byref(self._m), _ptr(hn), hn.shape[0], _ptr(out))
        return out

    def draft_logits(self, hn: np.ndarray, A: np.ndarray, B: np.ndarray, gamma: float) -> np.ndarray:
        hn = np.ascontiguousarray(hn, dtype=np.float64)
        A = np.ascontiguousarray(A, dtype=np.float64)
        B = np.ascontiguousarray(B, dtype=np.float64)
        out = np.empty((hn.shape[0], self.shape.vocab))
        self._lib.orc_draft_logits(ctypes.byref(self._m), _ptr(hn), hn.shape[0], _ptr(A), _ptr(B),
                                   A.shape[1], float(gamma), _ptr(out))
        return out


def argmax_lowest(z: np.ndarray) -> np.ndarray:
    """Greedy choice per row; equal maxima go to the lowest token id."""
    return np.argmax(z, axis=-1).astype(np.int32)   # numpy returns the first occurrence


def top2_gap(z: np.ndarray) -> np.ndarray:
    part = np.partition(z, -2, axis=-1)
    return part[..., -1] - part[..., -2]


from . import dvi, update  # noqa: E402,F401
