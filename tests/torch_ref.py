"""An independent float64 reference of the decoder, assembled from PyTorch library
routines (rms_norm, linear, scaled_dot_product_attention, silu) and a complex-number
form of the rotary embedding.  Used only to pin the oracle's forward pass: it shares
no code with the oracle and is written in a different form (whole-sequence masked
attention instead of a per-position loop, complex rotation instead of rotate-half)."""
import numpy as np
import torch
import torch.nn.functional as F

import synth


def _w(weights, a):
    return torch.from_numpy(np.asarray(weights.as_f32(a), np.float64))


def rope_complex(x: torch.Tensor, pos: torch.Tensor, theta: float) -> torch.Tensor:
    """x [T, heads, hd]: pair (x_i, x_{i+hd/2}) as the complex number x_i + 1j x_{i+hd/2},
    multiplied by exp(1j * pos * theta^(-2i/hd))."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * torch.arange(half, dtype=torch.float64) / hd)
    ang = pos.to(torch.float64)[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)[:, None, :]
    c = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([c.real, c.imag], dim=-1)


def forward(weights, tokens, n_layers=None):
    """Hidden states after each layer for one full causal sequence (positions 0..T-1)."""
    s = weights.shape
    L = s.n_layers if n_layers is None else n_layers
    tok = torch.as_tensor(np.asarray(tokens, np.int64))
    T = tok.numel()
    h = _w(weights, weights.tok_emb)[tok]
    pos = torch.arange(T)
    outs = []
    for l in range(L):
        lw = weights.layers[l]
        a = F.rms_norm(h, (s.d_model,), weight=_w(weights, lw["attn_norm"]), eps=s.rms_eps)
        q = F.linear(a, _w(weights, lw["wq"])).view(T, s.n_heads, s.head_dim)
        k = F.linear(a, _w(weights, lw["wk"])).view(T, s.n_kv_heads, s.head_dim)
        v = F.linear(a, _w(weights, lw["wv"])).view(T, s.n_kv_heads, s.head_dim)
        q, k = rope_complex(q, pos, s.rope_theta), rope_complex(k, pos, s.rope_theta)
        rep = s.n_heads // s.n_kv_heads
        k = k.repeat_interleave(rep, dim=1)
        v = v.repeat_interleave(rep, dim=1)
        o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True)
        o = o.transpose(0, 1).reshape(T, s.q_dim)
        h = h + F.linear(o, _w(weights, lw["wo"]))
        b = F.rms_norm(h, (s.d_model,), weight=_w(weights, lw["mlp_norm"]), eps=s.rms_eps)
        h = h + F.linear(F.silu(F.linear(b, _w(weights, lw["w_gate"]))) * F.linear(b, _w(weights, lw["w_up"])),
                         _w(weights, lw["w_down"]))
        outs.append(h.clone())
    return outs


def target_logits(weights, h):
    s = weights.shape
    hn = F.rms_norm(torch.as_tensor(h), (s.d_model,), weight=_w(weights, weights.final_norm), eps=s.rms_eps)
    return F.linear(hn, _w(weights, weights.lm_head)).numpy()


def randomize_norms(weights, seed=0):
    """Norm gains drawn away from 1, so a dropped gain is visible."""
    rng = np.random.default_rng(seed)
    bf = weights.shape.bf16

    def gains(n):
        g = rng.uniform(0.5, 1.5, n).astype(np.float32)
        return synth.f32_to_bf16_bits(g) if bf else g

    for lw in weights.layers:
        lw["attn_norm"] = gains(weights.shape.d_model)
        lw["mlp_norm"] = gains(weights.shape.d_model)
    weights.final_norm = gains(weights.shape.d_model)
    return weights
