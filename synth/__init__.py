"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

Holds no arithmetic of the method: it draws weights, prompts and replay
buffers from a counter-based generator (``synth.c``), so every array is a pure
function of (seed, stream, index) and both sides receive identical bits.

Model shapes are those of the five workloads the decode step is measured on
(tiny 4-layer decoder, 1B-, 7B- and 13B-shaped Llama-style decoders); weights
follow the initialisation those workloads name: embeddings N(0,1), every other
matrix N(0,0.02), the two residual-output projections (attention out and MLP
down) N(0, 0.02/sqrt(2L)), norm gains 1, LoRA A_s = 0 and B_s ~ N(0,0.02).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Dict, List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "libsynth.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile synth.c into libsynth.so (plain gcc, OpenMP)."""
    src = os.path.join(_HERE, "synth.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
                               "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build(force=False)
        lib = ctypes.CDLL(_SO)
        u64, i64, i32, dbl, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_double, ctypes.c_void_p)
        lib.synth_normal_f32.argtypes = [u64, u64, dbl, i64, vp]
        lib.synth_normal_bf16.argtypes = [u64, u64, dbl, i64, vp]
        lib.synth_uniform_int.argtypes = [u64, u64, i32, i64, vp]
        lib.synth_uniform_f64.argtypes = [u64, u64, i64, vp]
        lib.synth_bits.argtypes = [u64, u64, i64, vp]
        lib.synth_mix64.argtypes = [u64]
        lib.synth_mix64.restype = u64
        for f in (lib.synth_normal_f32, lib.synth_normal_bf16, lib.synth_uniform_int,
                  lib.synth_uniform_f64, lib.synth_bits):
            f.restype = None
        _lib = lib
    return _lib


def normal(seed: int, stream: int, std: float, shape, bf16: bool) -> np.ndarray:
    """std*N(0,1) array; bf16=True returns uint16 bf16 bit patterns, else float32."""
    n = int(np.prod(shape))
    out = np.empty(shape, dtype=np.uint16 if bf16 else np.float32)
    fn = _load().synth_normal_bf16 if bf16 else _load().synth_normal_f32
    fn(seed, stream, float(std), n, out.ctypes.data)
    return out


def uniform_int(seed: int, stream: int, hi: int, shape) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(shape, dtype=np.int32)
    _load().synth_uniform_int(seed, stream, int(hi), n, out.ctypes.data)
    return out


def uniform(seed: int, stream: int, shape) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(shape, dtype=np.float64)
    _load().synth_uniform_f64(seed, stream, n, out.ctypes.data)
    return out


def raw_bits(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, dtype=np.uint64)
    _load().synth_bits(seed, stream, n, out.ctypes.data)
    return out


def mix64(z: int) -> int:
    return int(_load().synth_mix64(z))


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32 (pure bit placement)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bf16 bit patterns (data preparation only)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


# --------------------------------------------------------------------------------------
# Model shapes
# --------------------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    split_k: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    bf16: bool
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    lora_rank: int = 16
    lora_gamma: float = 1.0

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_params(self) -> int:
        d, f = self.d_model, self.ffn_dim
        return (d * self.q_dim + 2 * d * self.kv_dim + self.q_dim * d + 3 * d * f + 2 * d)

    def weight_bytes_per_param(self) -> int:
        return 2 if self.bf16 else 4


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    prompt_len: int
    new_tokens: int
    k_spec: tuple
    update_every: int = 0       # decode steps between drafter updates (0: never)
    buffer_rows: int = 256


TINY = ModelShape("tiny", 4, 2, 256, 4, 4, 64, 1024, 4096, bf16=False)
SHAPE_1B = ModelShape("1b", 16, 8, 2048, 32, 8, 64, 8192, 32000, bf16=True)
SHAPE_7B = ModelShape("7b", 32, 16, 4096, 32, 32, 128, 11008, 32000, bf16=True)
SHAPE_13B = ModelShape("13b", 40, 20, 5120, 40, 40, 128, 13824, 32000, bf16=True)

WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", TINY, 1, 32, 64, (4,)),
    "1b": Workload("1b", SHAPE_1B, 1, 256, 256, (5,)),
    "7b": Workload("7b", SHAPE_7B, 1, 512, 512, (4, 6, 8)),
    "7b_b8": Workload("7b_b8", SHAPE_7B, 8, 2048, 256, (8,)),
    "13b": Workload("13b", SHAPE_13B, 1, 1024, 512, (6,), update_every=8, buffer_rows=256),
    # the 7B shape at the split the paper itself runs (drafter = layers 1..2 of 32), same weights
    "7b_k2": Workload("7b_k2", SHAPE_7B.replace(name="7b_k2", split_k=2), 1, 512, 512, (4,)),
}


def shrunk(shape: ModelShape, n_layers: int = 4, split_k: int = 2) -> ModelShape:
    """Same widths (d, heads, F, V, dtype), fewer layers: for fast oracle parity."""
    return shape.replace(name=shape.name + "_L%d" % n_layers, n_layers=n_layers, split_k=split_k)


# stream ids: one per tensor, fixed
S_EMB, S_HEAD, S_LORA_B, S_LORA_A, S_PROMPT, S_BUFFER = 0, 1, 2, 3, 4, 5
_LAYER_BASE = 16
_LAYER_TENSORS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def layer_stream(layer: int, name: str) -> int:
    return _LAYER_BASE + layer * 8 + _LAYER_TENSORS.index(name)


@dataclasses.dataclass
class Weights:
    """Host arrays: uint16 bf16 bits (bf16 shapes) or float32 (fp32 shapes).

    Matrices are row-major [out_features, in_features]."""
    shape: ModelShape
    tok_emb: np.ndarray
    layers: List[Dict[str, np.ndarray]]
    final_norm: np.ndarray
    lm_head: np.ndarray
    lora_A: np.ndarray      # float32 [V, r]
    lora_B: np.ndarray      # float32 [r, d]

    def as_f32(self, a: np.ndarray) -> np.ndarray:
        return bf16_bits_to_f32(a) if self.shape.bf16 else a


def _ones(n: int, bf16: bool) -> np.ndarray:
    return np.full(n, 0x3F80, dtype=np.uint16) if bf16 else np.ones(n, dtype=np.float32)


def make_weights(shape: ModelShape, seed: int = 0, lora_A_std: float = 0.0) -> Weights:
    """Random-init weights of the given shape (see module docstring)."""
    bf = shape.bf16
    d, L = shape.d_model, shape.n_layers
    std, out_std = 0.02, 0.02 / np.sqrt(2.0 * L)
    layers = []
    for l in range(L):
        layers.append({
            "attn_norm": _ones(d, bf),
            "wq": normal(seed, layer_stream(l, "wq"), std, (shape.q_dim, d), bf),
            "wk": normal(seed, layer_stream(l, "wk"), std, (shape.kv_dim, d), bf),
            "wv": normal(seed, layer_stream(l, "wv"), std, (shape.kv_dim, d), bf),
            "wo": normal(seed, layer_stream(l, "wo"), out_std, (d, shape.q_dim), bf),
            "mlp_norm": _ones(d, bf),
            "w_gate": normal(seed, layer_stream(l, "w_gate"), std, (shape.ffn_dim, d), bf),
            "w_up": normal(seed, layer_stream(l, "w_up"), std, (shape.ffn_dim, d), bf),
            "w_down": normal(seed, layer_stream(l, "w_down"), out_std, (d, shape.ffn_dim), bf),
        })
    lora_A = (normal(seed, S_LORA_A, lora_A_std, (shape.vocab, shape.lora_rank), False)
              if lora_A_std > 0 else np.zeros((shape.vocab, shape.lora_rank), np.float32))
    return Weights(
        shape=shape,
        tok_emb=normal(seed, S_EMB, 1.0, (shape.vocab, d), bf),
        layers=layers,
        final_norm=_ones(d, bf),
        lm_head=normal(seed, S_HEAD, std, (shape.vocab, d), bf),
        lora_A=lora_A,
        lora_B=normal(seed, S_LORA_B, std, (shape.lora_rank, d), False),
    )


def make_prompts(vocab: int, batch: int, prompt_len: int, seed: int = 0) -> np.ndarray:
    """Uniform random prompt ids, int32 [batch, prompt_len]."""
    return uniform_int(seed, S_PROMPT, vocab, (batch, prompt_len))


@dataclasses.dataclass
class Buffer:
    """A synthetic replay buffer, for update parity: rows of (h_hat_k, a, logits_phi, r, fresh)."""
    h: np.ndarray        # float32 [n, d], bf16-representable values
    a: np.ndarray        # int32 [n]
    logits: np.ndarray   # float32 [n, V]
    r: np.ndarray        # int8 [n]   (1 accepted, 0 first reject)
    fresh: np.ndarray    # int8 [n]


def make_buffer(d: int, vocab: int, n: int, seed: int = 0, accept_p: float = 0.6,
                fresh_p: float = 0.5, logit_std: float = 1.5) -> Buffer:
    base = S_BUFFER * 1000
    h = bf16_bits_to_f32(normal(seed, base + 0, 1.0, (n, d), True))
    logits = normal(seed, base + 1, logit_std, (n, vocab), False)
    a = uniform_int(seed, base + 2, vocab, (n,))
    r = (uniform(seed, base + 3, (n,)) < accept_p).astype(np.int8)
    fresh = (uniform(seed, base + 4, (n,)) < fresh_p).astype(np.int8)
    return Buffer(h=h, a=a, logits=logits, r=r, fresh=fresh)
