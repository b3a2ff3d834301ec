"""Drafter-head objective, gradient, optimiser step and schedule (Section 3.4).

TEST INFRASTRUCTURE ONLY (see the package docstring).  Plain numpy float64.

Objective on the LoRA parameters theta = {A_s, B_s} of the draft head
  z_i = W^(S) h_i + gamma * A_s (B_s h_i),  p_i = softmax(z_i),
  q_i = softmax(logits^phi_i / tau)     (tempered target distribution)
with three terms, as the text composes L_fast and L_policy:
  * online distillation KL(p_i || q_i)            (the lambda_kl / beta(t) term)
  * reward-masked cross-entropy -log p_i(a_i), averaged over accepted rows
    (the term the text calls L_pg)
  * on-policy REINFORCE -(r_i - b) log p_i(a_i) over fresh rows (L_policy)
  * optional entropy bonus -w_ent H[p_i].
Readings (listed in the design notes): the KL and entropy terms average over
all valid rows, the masked CE over accepted rows (0 if none), the policy term
over fresh rows; the beta(t) KL of L_policy is folded into the single KL
coefficient; the undefined w_ce L_CE is the reward-masked CE term.
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class Coeffs:
    c_kl: float
    c_ce: float
    c_pg: float
    c_ent: float = 0.0
    tau: float = 1.0
    baseline: float = 0.0


@dataclasses.dataclass
class LossOut:
    loss: float
    kl: float      # mean over valid rows of KL(p||q)
    ce: float      # mean over accepted rows of -log p(a)
    pg: float      # mean over fresh rows of -(r-b) log p(a)
    entropy: float
    dA: np.ndarray
    dB: np.ndarray
    g: np.ndarray  # dLoss/dz, [n, V]


def log_softmax(x: np.ndarray) -> np.ndarray:
    mx = np.max(x, axis=-1, keepdims=True)
    y = x - mx
    return y - np.log(np.sum(np.exp(y), axis=-1, keepdims=True))


def draft_logits(W: np.ndarray, A: np.ndarray, B: np.ndarray, gamma: float, h: np.ndarray):
    """z = W h + gamma A (B h) for each row of h; returns (z, u = B h)."""
    u = h @ B.T
    return h @ W.T + gamma * (u @ A.T), u


def objective(W, A, B, gamma, h, a, logits_phi, r, fresh, c: Coeffs):
    """Loss value only (used by the finite-difference pins)."""
    z, _ = draft_logits(W, A, B, gamma, h)
    return _terms(z, a, logits_phi, r, fresh, c)[0]


def _terms(z, a, logits_phi, r, fresh, c: Coeffs):
    n = z.shape[0]
    logp = log_softmax(z)
    p = np.exp(logp)
    logq = log_softmax(np.asarray(logits_phi, np.float64) / c.tau)
    kl = np.sum(p * (logp - logq), axis=1)
    ent = -np.sum(p * logp, axis=1)
    lpa = logp[np.arange(n), a]
    r = np.asarray(r, np.float64)
    fr = np.asarray(fresh, np.float64)
    n_acc = float(r.sum())
    n_fr = float(fr.sum())
    alpha = c.c_kl / n
    beta = c.c_ce * r / max(n_acc, 1.0) + c.c_pg * (r - c.baseline) * fr / max(n_fr, 1.0)
    eps = c.c_ent / n
    loss = float(np.sum(alpha * kl - beta * lpa - eps * ent))
    return loss, logp, p, logq, kl, ent, lpa, alpha, beta, eps, n_acc, n_fr


def loss_and_grad(W, A, B, gamma, h, a, logits_phi, r, fresh, c: Coeffs) -> LossOut:
    """Loss and its gradient with respect to A_s and B_s.

    Per row, dLoss/dz = alpha p (log p - log q - KL) + beta (p - e_a)
                        + eps p (log p + H);
    then dA = gamma sum_i g_i u_i^T and dB = sum_i (gamma A^T g_i) h_i^T.
    """
    W = np.asarray(W, np.float64)
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    h = np.asarray(h, np.float64)
    a = np.asarray(a, np.int64)
    z, u = draft_logits(W, A, B, gamma, h)
    loss, logp, p, logq, kl, ent, lpa, alpha, beta, eps, n_acc, n_fr = _terms(z, a, logits_phi, r, fresh, c)
    n = z.shape[0]
    onehot = np.zeros_like(p)
    onehot[np.arange(n), a] = 1.0
    g = (alpha * p * (logp - logq - kl[:, None]) + beta[:, None] * (p - onehot)
         + eps * p * (logp + ent[:, None]))
    dA = gamma * (g.T @ u)
    du = gamma * (g @ A)
    dB = du.T @ h
    r64 = np.asarray(r, np.float64)
    fr = np.asarray(fresh, np.float64)
    ce = float(-(lpa * r64).sum() / max(n_acc, 1.0))
    pg = float(-((r64 - c.baseline) * fr * lpa).sum() / max(n_fr, 1.0))
    return LossOut(loss, float(kl.mean()), ce, pg, float(ent.mean()), dA, dB, g)


@dataclasses.dataclass
class AdamState:
    mA: np.ndarray
    vA: np.ndarray
    mB: np.ndarray
    vB: np.ndarray
    step: int = 0


def adam_init(A, B) -> AdamState:
    return AdamState(np.zeros_like(A, dtype=np.float64), np.zeros_like(A, dtype=np.float64),
                     np.zeros_like(B, dtype=np.float64), np.zeros_like(B, dtype=np.float64), 0)


def adam_step(param, grad, m, v, t, lr, b1=0.9, b2=0.999, eps=1e-8):
    """Adam (Kingma & Ba, 2015), bias-corrected, step t >= 1.  Returns new (param, m, v)."""
    m = b1 * m + (1 - b1) * grad
    v = b2 * v + (1 - b2) * grad * grad
    mh = m / (1 - b1 ** t)
    vh = v / (1 - b2 ** t)
    return param - lr * mh / (np.sqrt(vh) + eps), m, v


@dataclasses.dataclass
class Schedule:
    """KL->RL schedule over update count t (Section 3.4).

    rho(t) = clamp((t - T_warmup) / T_ramp, 0, 1)
    lambda_pg = rho * lambda_pg_max;  lambda_kl = lambda0 - rho (lambda0 - lambda_kl_min)
    The policy term ramps in with the same rho (weight w_rl).
    """
    lambda0: float = 1.0
    lambda_kl_min: float = 0.5
    lambda_pg_max: float = 1.0
    w_rl: float = 0.5
    w_ent: float = 0.0
    t_warmup: int = 4
    t_ramp: int = 4

    def rho(self, t: int) -> float:
        return min(max((t - self.t_warmup) / float(self.t_ramp), 0.0), 1.0)

    def coeffs(self, t: int, baseline: float, tau: float = 1.0) -> Coeffs:
        rho = self.rho(t)
        return Coeffs(c_kl=self.lambda0 - rho * (self.lambda0 - self.lambda_kl_min),
                      c_ce=rho * self.lambda_pg_max, c_pg=rho * self.w_rl, c_ent=self.w_ent,
                      tau=tau, baseline=baseline)


def ema_baseline(b: float, fresh_rewards, rate: float = 0.9) -> float:
    """b <- rate b + (1 - rate) mean(fresh rewards); unchanged if there are none."""
    fr = np.asarray(fresh_rewards, np.float64)
    if fr.size == 0:
        return b
    return rate * b + (1.0 - rate) * float(fr.mean())
