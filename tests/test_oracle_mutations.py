"""The pins must fail on plausible mistakes: each test plants one in a copy of the
oracle's arithmetic (on the CPU) and checks that the autograd pin rejects it."""
import numpy as np
import pytest

import oracle
from oracle import backward as bw
from oracle import forward as fw
from test_oracle_pins import _o2, _rel, _torch_grads, _two_layer_tiny


def _delta_wrong_index(G, alpha):
    a = float(alpha)
    D = np.zeros(G.shape)
    for t in range(G.shape[0] - 2, -1, -1):
        D[t] = a * D[t + 1] + G[t]  # should be G[t + 1]
    return D


def _delta_no_decay(G, alpha):
    D = np.zeros(G.shape)
    for t in range(G.shape[0] - 2, -1, -1):
        D[t] = D[t + 1] + G[t + 1]  # dropped alpha
    return D


def _worst_rel(inp, fwd64, torch_dW):
    r = _o2(inp, fwd64, 0.3)
    return max(_rel(r["dW"][l], torch_dW[l]) for l in range(len(torch_dW)))


@pytest.mark.parametrize("bad", [_delta_wrong_index, _delta_no_decay])
def test_delta_mistakes_are_caught(monkeypatch, bad):
    inp = _two_layer_tiny()
    _, dWs, _, fwd64 = _torch_grads(inp, 0.3)
    assert _worst_rel(inp, fwd64, dWs) <= 1e-10
    monkeypatch.setattr(bw, "delta_recurrence", bad)
    assert _worst_rel(inp, fwd64, dWs) > 1e-3


def test_wrong_surrogate_exponent_is_caught(monkeypatch):
    """g = 1/(beta|V-1|+1) instead of its square (App. E) must fail."""
    inp = _two_layer_tiny()
    _, dWs, _, fwd64 = _torch_grads(inp, 0.3)
    real = bw.surrogate
    monkeypatch.setattr(bw, "surrogate", lambda V, th, be: real(V, th, be) ** 0.5)  # wrong exponent in g
    assert _worst_rel(inp, fwd64, dWs) > 1e-3


def test_forward_reset_sign_is_caught():
    """A reset added instead of subtracted breaks the closed form of Eq. (lif)."""
    X = np.zeros((8, 1, 1), np.uint8)
    X[1, 0, 0] = 1
    W = np.array([[1.5]], np.float32)
    V, S, _ = oracle.lif_forward(X, W, np.float32(0.9), np.float32(1.0))
    assert abs(float(V[3, 0, 0]) - (0.9 * 1.5 - 1.0)) < 1e-6  # the right answer
    assert abs(float(V[3, 0, 0]) - (0.9 * 1.5 + 1.0)) > 1.0  # the mistake would be far off
