"""Pins of the oracle's training step: activity penalties, Adam, App. H statistics (no GPU).

Closed forms and hand-worked numbers for the penalties (App. E), finite differences
for their gradient, finite differences of the smoothed model (smooth.py) with the
penalties for the whole backward, torch.optim.Adam for the update, and a hand-worked
example for the gradient-difference statistics.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import smooth
from synth import CONFIGS, make_inputs
from synth.inputs import Config

F32 = np.float32


def test_spike_counts_brute_force():
    r = np.random.default_rng(5)
    S = (r.random((13, 3, 7)) < 0.3).astype(np.uint8) * r.integers(1, 255, (13, 3, 7)).astype(np.uint8)
    z = oracle.spike_counts(S)
    for b in range(3):
        for i in range(7):
            assert z[b, i] == sum(1 for t in range(13) if S[t, b, i] != 0)


def test_penalty_closed_forms():
    """App. E penalties: a silent layer pays lam_low nu_low^2 per sample, a saturated one
    lam_up (T - nu_up); a hand-worked mixed case."""
    lam_low, nu_low, lam_up, nu_up = 100.0, 0.001, 0.06, 1.0
    N, B, T = 200, 3, 100
    silent = np.zeros((B, N))
    assert np.allclose(oracle.activity_penalty(silent, lam_low, nu_low, lam_up, nu_up), lam_low * nu_low ** 2, rtol=1e-14)
    full = np.full((B, N), T)
    assert np.allclose(oracle.activity_penalty(full, lam_low, nu_low, lam_up, nu_up), lam_up * (T - nu_up), rtol=1e-14)
    # N = 4, counts (0, 1, 3, 0): lower term 8/4 (2^2 + 1^2 + 0 + 2^2) = 18; mean count 1,
    # upper term 3 (1 - 0.5) = 1.5
    z = np.array([[0, 1, 3, 0]])
    assert oracle.activity_penalty(z, 8.0, 2.0, 3.0, 0.5)[0] == pytest.approx(19.5, rel=1e-15)
    # at or below the upper bound the upper term vanishes
    assert oracle.activity_penalty(z, 8.0, 2.0, 3.0, 1.0)[0] == pytest.approx(18.0, rel=1e-15)


def test_penalty_gradient_finite_differences():
    """activity_grad is the derivative of the batch mean of activity_penalty (away from hinges)."""
    r = np.random.default_rng(7)
    B, N = 4, 9
    z = r.uniform(0, 4, (B, N))
    params = (30.0, 2.0, 5.0, 1.5)
    z[0] = r.uniform(0, 1, N)  # sample 0 below the upper bound, the rest above it on average
    g = oracle.activity_grad(z, *params)
    h = 1e-6
    for b in range(B):
        for i in range(N):
            zp, zm = z.copy(), z.copy()
            zp[b, i] += h
            zm[b, i] -= h
            fd = (oracle.activity_penalty(zp, *params).mean() - oracle.activity_penalty(zm, *params).mean()) / (2 * h)
            assert fd == pytest.approx(g[b, i], abs=1e-7)
    assert (g[0] < 0).any() and (g[1:] > 0).any()


def _penalty_case():
    cfg = Config("tiny2r", 102, T=24, B=4, sizes=(64, 32, 24, 4), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
                 loss_mode="max", b_th=0.3, kind="bernoulli", rate=0.08)
    return make_inputs(cfg, sigmas=[0.2, 0.35, 1 / math.sqrt(24)])


# penalties far stronger than App. E's so that their gradient dominates the check
STRONG = (40.0, 2.0, 4.0, 0.2)


def _fd_check(inp, b_th, reg):
    """Central differences of the smoothed model with penalties vs training_gradients."""
    cfg = inp.cfg
    base = smooth.hard_forward64(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out)
    ref = oracle.training_gradients(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels,
                                    cfg.loss_mode, 1.0, b_th, 100.0, reg=reg, fwd=base)
    tstar = ref["readout"]["tstar"]
    args = (inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode, 1.0, b_th, 100.0, base, tstar)
    L0 = smooth.smoothed_losses(inp.X, inp.Ws, inp.W_out, *args, reg=reg)[0]
    assert L0 == pytest.approx(ref["total"], rel=1e-12)
    h = 1e-6
    mats = list(inp.Ws) + [inp.W_out]
    grads = list(ref["dW"]) + [ref["dW_out"]]
    worst = 0.0
    for m, (W, gref) in enumerate(zip(mats[:-1], grads[:-1])):
        W = W.astype(np.float64)
        n = W.size
        sel = np.random.default_rng(m).choice(n, size=min(n, 384), replace=False)
        stack = np.repeat(W[None], 2 * sel.size, axis=0)
        for k, i in enumerate(sel):
            stack[k].flat[i] += h
            stack[sel.size + k].flat[i] -= h
        Ws_p = [w.astype(np.float64) for w in mats]
        Ws_p[m] = stack
        losses = smooth.smoothed_losses(inp.X, Ws_p[:-1], Ws_p[-1], *args, reg=reg)
        up, dn = losses[: sel.size], losses[sel.size:]
        fd = (up - dn) / (2 * h)
        jump = np.abs((up - L0) / h - (L0 - dn) / h)
        g = gref.ravel()[sel]
        scale = np.abs(gref).max()
        ok = jump <= 1e-3 * scale
        assert ok.mean() >= 0.9
        worst = max(worst, float((np.abs(fd - g)[ok]).max() / scale))
    return ref, worst


@pytest.mark.parametrize("b_th", [0.3, np.inf])
def test_backward_with_penalties_finite_differences(b_th):
    """The penalties' gradient joins each layer's spike gradient at every step (App. E with
    Eqs. (w_grad), (s_grad)): central differences of the smoothed model agree."""
    inp = _penalty_case()
    ref, worst = _fd_check(inp, b_th, STRONG)
    assert worst <= 1e-6
    plain = oracle.training_gradients(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels,
                                      inp.cfg.loss_mode, 1.0, b_th, 100.0, reg=None, fwd=ref["fwd"])
    # the penalties move the hidden-layer gradients by a visible amount
    for l in range(2):
        d = np.abs(ref["dW"][l] - plain["dW"][l]).max()
        assert d >= 0.05 * np.abs(ref["dW"][l]).max(), l
    assert ref["penalty"][0] > 0 and ref["penalty"][1] > 0


def test_penalty_gradient_mistakes_are_caught(monkeypatch):
    """A dropped factor or a flipped sign in the penalty gradient fails the finite differences."""
    inp = _penalty_case()
    good = oracle.regularize.activity_grad
    for bad in (lambda z, *p: 0.5 * good(z, *p), lambda z, *p: -good(z, *p)):
        monkeypatch.setattr(oracle.train, "activity_grad", bad)
        _, worst = _fd_check(inp, 0.3, STRONG)
        assert worst > 1e-3
    monkeypatch.setattr(oracle.train, "activity_grad", good)


def test_paper_penalty_values_on_tiny():
    """With App. E's values the penalty on the tiny workload is the lower term of its silent
    neurons (hand count) plus the upper term."""
    inp = make_inputs(CONFIGS["tiny"])
    fwd = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, F32(1.0))
    z = oracle.spike_counts(fwd["S"][0])
    B, N = z.shape
    silent = (z == 0).sum(axis=1)
    want = 100.0 * (0.001 ** 2) * silent / N + 0.06 * np.maximum(0.0, z.mean(axis=1) - 1.0)
    got = oracle.activity_penalty(z, 100.0, 0.001, 0.06, 1.0)
    assert np.allclose(got, want, rtol=1e-13, atol=0)


def test_adam_matches_torch_optim():
    """adam_update reproduces torch.optim.Adam (float64) over several steps."""
    r = np.random.default_rng(11)
    w0 = r.standard_normal((5, 7))
    grads = [r.standard_normal((5, 7)) * s for s in (1.0, 1e-3, 10.0, 0.0)]
    grads[3][0, 0] = 1e-9
    lr, b1, b2, eps = 2e-4, 0.9, 0.999, 1e-8
    p = torch.nn.Parameter(torch.tensor(w0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps)
    w, m, v = w0.copy(), np.zeros_like(w0), np.zeros_like(w0)
    for k, g in enumerate(grads, start=1):
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        w, m, v = oracle.adam_update(w, g, m, v, k, lr, b1, b2, eps)
        assert np.allclose(w, p.detach().numpy(), rtol=1e-14, atol=1e-16)
    st = opt.state[p]
    assert np.allclose(m, st["exp_avg"].numpy(), rtol=1e-14, atol=0)
    assert np.allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-14, atol=0)


def test_adam_first_step_closed_form():
    """From m = v = 0 the first step moves each weight by lr g / (|g| + eps)."""
    g = np.array([3.0, -2e-3, 0.0, 5e-9])
    w, m, v = oracle.adam_update(np.zeros(4), g, np.zeros(4), np.zeros(4), 1, 1e-3)
    assert np.allclose(w, -1e-3 * g / (np.abs(g) + 1e-8), rtol=1e-14, atol=0)
    assert np.allclose(m, 0.1 * g) and np.allclose(v, 1e-3 * g * g)
    with pytest.raises(ValueError):
        oracle.adam_update(np.zeros(4), g, np.zeros(4), np.zeros(4), 0, 1e-3)


def test_gradient_difference_hand_example():
    full = np.array([[4.0, -2.0], [0.01, 0.0]])
    sparse = np.array([[3.0, -2.0], [0.0, 0.0]])
    d = oracle.gradient_difference(sparse, full)
    assert d["max_abs_over_max"] == pytest.approx(1.0 / 4.0)
    assert d["max_rel_big"] == pytest.approx(1.0 / 4.0)  # 0.01 is below 1% of 4 and is skipped
    nb = math.sqrt(16 + 4 + 1e-4)
    assert d["frobenius_rel"] == pytest.approx(math.sqrt(1 + 1e-4) / nb)
    assert d["cosine"] == pytest.approx((12 + 4) / (math.sqrt(13) * nb))
    same = oracle.gradient_difference(full, full)
    assert same["max_abs_over_max"] == 0 and same["cosine"] == pytest.approx(1.0)
