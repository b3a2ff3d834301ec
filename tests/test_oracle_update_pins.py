"""Pins for the oracle's drafter objective, gradient, Adam step and schedule (Section 3.4)."""
import numpy as np
import pytest
import scipy.special
import scipy.stats
import torch

from oracle import update as U

V, D, R, N = 7, 5, 2, 6


def _case(seed=0, gamma=0.8):
    rng = np.random.default_rng(seed)
    W = rng.normal(0, 0.5, (V, D))
    A = rng.normal(0, 0.5, (V, R))
    B = rng.normal(0, 0.5, (R, D))
    h = rng.normal(0, 1, (N, D))
    a = rng.integers(0, V, N)
    lg = rng.normal(0, 1.5, (N, V))
    r = np.array([1, 1, 0, 1, 0, 1], np.int8)
    fresh = np.array([1, 0, 1, 1, 0, 0], np.int8)
    return W, A, B, gamma, h, a, lg, r, fresh


COEFFS = [
    U.Coeffs(1.0, 0.0, 0.0),                        # KL only
    U.Coeffs(0.0, 1.0, 0.0),                        # masked CE only
    U.Coeffs(0.0, 0.0, 1.0, baseline=0.3),          # policy gradient only
    U.Coeffs(0.0, 0.0, 0.0, c_ent=1.0),             # entropy only
    U.Coeffs(0.7, 0.9, 0.4, c_ent=0.05, tau=1.7, baseline=0.45),
]


@pytest.mark.parametrize("c", COEFFS)
def test_gradient_matches_finite_differences(c):
    W, A, B, g, h, a, lg, r, fr = _case(1)
    out = U.loss_and_grad(W, A, B, g, h, a, lg, r, fr, c)
    eps = 1e-6
    for P, dP in ((A, out.dA), (B, out.dB)):
        num = np.zeros_like(P)
        for idx in np.ndindex(P.shape):
            old = P[idx]
            P[idx] = old + eps
            lp = U.objective(W, A, B, g, h, a, lg, r, fr, c)
            P[idx] = old - eps
            lm = U.objective(W, A, B, g, h, a, lg, r, fr, c)
            P[idx] = old
            num[idx] = (lp - lm) / (2 * eps)
        assert np.allclose(dP, num, rtol=1e-6, atol=1e-8)


def test_loss_terms_match_library_routines():
    W, A, B, g, h, a, lg, r, fr = _case(2)
    z = h @ (W + g * A @ B).T
    p = scipy.special.softmax(z, axis=1)
    tau = 1.3
    q = scipy.special.softmax(lg / tau, axis=1)
    kl = scipy.special.rel_entr(p, q).sum(axis=1)
    ent = scipy.stats.entropy(p, axis=1)
    lpa = np.log(p[np.arange(N), a])
    out = U.loss_and_grad(W, A, B, g, h, a, lg, r, fr, U.Coeffs(1.0, 1.0, 1.0, c_ent=1.0, tau=tau, baseline=0.2))
    assert np.isclose(out.kl, kl.mean(), rtol=1e-12)
    assert np.isclose(out.entropy, ent.mean(), rtol=1e-12)
    assert np.isclose(out.ce, -lpa[r == 1].mean(), rtol=1e-12)
    assert np.isclose(out.pg, -((r - 0.2) * lpa)[fr == 1].mean(), rtol=1e-12)
    expect = kl.mean() + out.ce + out.pg - ent.mean()
    assert np.isclose(out.loss, expect, rtol=1e-12)


def test_kl_hand_value_and_zero_at_match():
    # z = [0, ln 3] -> p = [1/4, 3/4]; logits_phi = 0 -> q = [1/2, 1/2]
    W = np.array([[0.0], [np.log(3.0)]])
    A, B = np.zeros((2, 1)), np.zeros((1, 1))
    h = np.ones((1, 1))
    out = U.loss_and_grad(W, A, B, 1.0, h, np.array([0]), np.zeros((1, 2)), np.array([0]), np.array([0]),
                          U.Coeffs(1.0, 0.0, 0.0))
    assert np.isclose(out.kl, 0.25 * np.log(0.5) + 0.75 * np.log(1.5), rtol=1e-14)
    # z = logits_phi / tau exactly -> KL = 0 and gradient 0
    W, A, B, g, h, a, lg, r, fr = _case(3)
    tau = 2.0
    z = h @ (W + g * A @ B).T
    out = U.loss_and_grad(W, A, B, g, h, a, z * tau, r, fr, U.Coeffs(1.0, 0.0, 0.0, tau=tau))
    assert abs(out.kl) < 1e-14
    assert np.abs(out.dA).max() < 1e-13 and np.abs(out.dB).max() < 1e-13
    assert out.kl >= 0


def test_closed_form_dz_and_row_sums():
    W, A, B, g, h, a, lg, r, fr = _case(4)
    z = h @ (W + g * A @ B).T
    p = scipy.special.softmax(z, axis=1)
    onehot = np.eye(V)[a]
    # masked CE only: dL/dz_i = (r_i / n_acc) (p_i - e_{a_i})
    out = U.loss_and_grad(W, A, B, g, h, a, lg, r, fr, U.Coeffs(0.0, 1.0, 0.0))
    assert np.allclose(out.g, (r / r.sum())[:, None] * (p - onehot), rtol=1e-12, atol=1e-14)
    # every term's dL/dz sums to zero over the vocabulary (softmax shift invariance)
    for c in COEFFS:
        o = U.loss_and_grad(W, A, B, g, h, a, lg, r, fr, c)
        assert np.abs(o.g.sum(axis=1)).max() < 1e-14


def test_lora_chain_rule_special_cases():
    W, A, B, g, h, a, lg, r, fr = _case(5)
    c = COEFFS[-1]
    o = U.loss_and_grad(W, np.zeros_like(A), B, g, h, a, lg, r, fr, c)
    assert np.all(o.dB == 0.0)
    o = U.loss_and_grad(W, A, B, 0.0, h, a, lg, r, fr, c)
    assert np.all(o.dA == 0.0) and np.all(o.dB == 0.0)


def test_no_accepted_rows_gives_zero_ce():
    W, A, B, g, h, a, lg, r, fr = _case(6)
    o = U.loss_and_grad(W, A, B, g, h, a, lg, np.zeros(N, np.int8), fr, U.Coeffs(0.0, 1.0, 0.0))
    assert o.ce == 0.0 and np.all(o.dA == 0.0)


def test_torch_autograd_agrees():
    W, A, B, g, h, a, lg, r, fr = _case(7)
    c = COEFFS[-1]
    At = torch.tensor(A, requires_grad=True)
    Bt = torch.tensor(B, requires_grad=True)
    z = torch.tensor(h) @ (torch.tensor(W) + g * At @ Bt).T
    logp = torch.log_softmax(z, 1)
    logq = torch.log_softmax(torch.tensor(lg) / c.tau, 1)
    kl = torch.nn.functional.kl_div(logq, logp, log_target=True, reduction="none").sum(1)
    p = logp.exp()
    ent = -(p * logp).sum(1)
    lpa = logp[torch.arange(N), torch.tensor(a)]
    rt, ft = torch.tensor(r, dtype=torch.float64), torch.tensor(fr, dtype=torch.float64)
    loss = (c.c_kl * kl.mean() - c.c_ce * (rt * lpa).sum() / rt.sum()
            - c.c_pg * ((rt - c.baseline) * ft * lpa).sum() / ft.sum() - c.c_ent * ent.mean())
    loss.backward()
    o = U.loss_and_grad(W, A, B, g, h, a, lg, r, fr, c)
    assert np.isclose(o.loss, loss.item(), rtol=1e-12)
    assert np.allclose(o.dA, At.grad.numpy(), rtol=1e-10, atol=1e-13)
    assert np.allclose(o.dB, Bt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_adam_matches_torch_optim():
    rng = np.random.default_rng(8)
    p = rng.normal(size=(4, 3))
    pt = torch.tensor(p.copy(), requires_grad=True)
    opt = torch.optim.Adam([pt], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    m = np.zeros_like(p)
    v = np.zeros_like(p)
    for t in range(1, 6):
        gr = rng.normal(size=p.shape)
        pt.grad = torch.tensor(gr)
        opt.step()
        p, m, v = U.adam_step(p, gr, m, v, t, 1e-2)
    assert np.allclose(p, pt.detach().numpy(), rtol=1e-12, atol=1e-14)


def test_schedule_closed_form():
    s = U.Schedule(lambda0=1.0, lambda_kl_min=0.5, lambda_pg_max=1.0, w_rl=0.5, t_warmup=4, t_ramp=4)
    c = s.coeffs(2, 0.0)
    assert (c.c_kl, c.c_ce, c.c_pg) == (1.0, 0.0, 0.0)          # warmup: KL only
    c = s.coeffs(6, 0.0)                                         # half-way up the ramp
    assert np.isclose(c.c_kl, 0.75) and np.isclose(c.c_ce, 0.5) and np.isclose(c.c_pg, 0.25)
    c = s.coeffs(100, 0.0)
    assert (c.c_kl, c.c_ce, c.c_pg) == (0.5, 1.0, 0.5)
    assert U.ema_baseline(0.0, [1, 1, 0, 1], 0.9) == pytest.approx(0.075)
    assert U.ema_baseline(0.3, [], 0.9) == 0.3
