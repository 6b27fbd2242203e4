"""Pins of the convolutional oracle (oracle/conv.py) against library routines (no GPU).

The Toeplitz matrix against torch.nn.functional.conv2d, the forward against a float64 torch
recurrence, the pooling against torch.nn.functional.max_pool2d, and the whole gradient against
torch autograd of the same network (conv2d, max_pool2d, readout, cross-entropy) with the
Heaviside forward and the banded surrogate backward.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import conv

F32 = np.float32


def _case(T=12, B=3, H=6, W=6, C=2, Fo=5, Cls=4, rate=0.15, seed=0, sigma=0.6):
    r = np.random.default_rng(seed)
    X = (r.random((T, B, H, W, C)) < rate).astype(np.uint8)
    Wc = (r.standard_normal((3, 3, C, Fo)) * sigma).astype(F32)
    Np = (H // 2) * (W // 2) * Fo
    Wo = (r.standard_normal((Np, Cls)) / math.sqrt(Np)).astype(F32)
    y = r.integers(0, Cls, B).astype(np.int32)
    return X, Wc, Wo, y


def _oihw(Wc):
    return torch.tensor(np.transpose(Wc, (3, 2, 0, 1)).astype(np.float64))  # [F, C, 3, 3]


def test_toeplitz_is_conv2d():
    X, Wc, _, _ = _case(T=1, B=4)
    x = X[0].astype(np.float64)  # [B, H, W, C]
    B, H, W, C = x.shape
    Fo = Wc.shape[3]
    got = x.reshape(B, -1) @ conv.toeplitz(Wc, H, W).astype(np.float64)
    ref = torch.nn.functional.conv2d(torch.tensor(x).permute(0, 3, 1, 2), _oihw(Wc), padding=1)
    assert np.allclose(got.reshape(B, H, W, Fo), ref.permute(0, 2, 3, 1).numpy(), rtol=1e-12, atol=1e-12)


def test_forward_matches_float64_recurrence():
    X, Wc, Wo, _ = _case(T=16)
    a = F32(math.exp(-0.1))
    f = conv.conv_network_forward(X, Wc, Wo, a, a)
    x = torch.tensor(X, dtype=torch.float64).permute(0, 1, 4, 2, 3)  # [T, B, C, H, W]
    T, B = X.shape[:2]
    v = torch.zeros(B, Wc.shape[3], X.shape[2], X.shape[3], dtype=torch.float64)
    for t in range(T):
        V = f["V"][t].transpose(0, 3, 1, 2)
        assert np.allclose(V, v.numpy(), atol=2e-5)
        s = v > 1.0
        far = (v - 1.0).abs().numpy() > 1e-4
        assert np.array_equal(f["S"][t].transpose(0, 3, 1, 2)[far], s.numpy()[far].astype(np.uint8))
        v = float(a) * v + torch.nn.functional.conv2d(x[t], _oihw(Wc), padding=1) - torch.tensor(
            f["S"][t].transpose(0, 3, 1, 2), dtype=torch.float64)
    assert f["S"].any() and not f["S"].all()


def test_pool_matches_torch():
    r = np.random.default_rng(3)
    S = (r.random((5, 2, 8, 6, 7)) < 0.3).astype(np.uint8)
    P, arg = conv.maxpool_spikes(S)
    t = torch.tensor(S, dtype=torch.float64).reshape(10, 8, 6, 7).permute(0, 3, 1, 2)
    out, idx = torch.nn.functional.max_pool2d(t, 2, return_indices=True)
    assert np.array_equal(P.reshape(10, 4, 3, 7), out.permute(0, 2, 3, 1).numpy().astype(np.uint8))
    # torch's index is the flat position in the 8x6 map; the window element it names
    idx = idx.permute(0, 2, 3, 1).numpy()
    yy, xx = idx // 6, idx % 6
    py, px = np.meshgrid(np.arange(4), np.arange(3), indexing="ij")
    want = (yy - 2 * py[None, :, :, None]) * 2 + (xx - 2 * px[None, :, :, None])
    assert np.array_equal(arg.reshape(10, 4, 3, 7), want)
    # an empty window routes to its top-left element
    assert (arg[P == 0] == 0).all()


def _torch_conv_grads(X, Wc, Wo, y, b_th, beta=100.0, alpha=math.exp(-0.1), mode="max", pen=None):
    class Spike(torch.autograd.Function):
        @staticmethod
        def forward(ctx, v):
            ctx.save_for_backward(v)
            return (v > 1.0).to(v.dtype)

        @staticmethod
        def backward(ctx, gout):
            (v,) = ctx.saved_tensors
            d = (v - 1.0).abs()
            return gout * (1.0 / (beta * d + 1.0) ** 2) * (d < b_th).to(v.dtype)

    a = float(F32(alpha))
    x = torch.tensor(X, dtype=torch.float64).permute(0, 1, 4, 2, 3)  # [T, B, C, H, W]
    T, B = X.shape[:2]
    wc = _oihw(Wc).requires_grad_(True)
    wo = torch.tensor(Wo.astype(np.float64), requires_grad=True)
    v = torch.zeros(B, Wc.shape[3], X.shape[2], X.shape[3], dtype=torch.float64)
    vo = torch.zeros(B, Wo.shape[1], dtype=torch.float64)
    tr = torch.zeros(x.shape[1:], dtype=torch.float64)
    tro = torch.zeros(B, wo.shape[0], dtype=torch.float64)
    vol, vl, sl, tl, tol = [], [], [], [], []
    sg = []
    for t in range(T):
        s = Spike.apply(v)
        sg.append(s)
        p = torch.nn.functional.max_pool2d(s, 2).permute(0, 2, 3, 1).reshape(B, -1)  # channels last
        vol.append(vo)
        vl.append(v.detach())
        sl.append(s.detach())
        tl.append(tr)
        tol.append(tro)
        if t < T - 1:
            v = a * v + torch.nn.functional.conv2d(x[t], wc, padding=1) - s.detach()
            vo = a * vo + p @ wo
            tr = a * tr + x[t]
            tro = a * tro + p.detach()
    Vo = torch.stack(vol)
    cl = lambda z: torch.stack(z).permute(0, 1, 3, 4, 2).numpy()  # noqa: E731  -> channels last
    S64 = cl(sl).astype(np.uint8)
    P, arg = conv.maxpool_spikes(S64)
    fwd = {"V": cl(vl), "S": S64, "trace": cl(tl), "P": P, "arg": arg, "V_out": Vo.detach().numpy(),
           "trace_out": torch.stack(tol).numpy()}
    if mode == "max":
        logits = Vo.gather(0, torch.argmax(Vo.detach(), dim=0, keepdim=True))[0]
    else:
        logits = Vo.sum(0)
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    if pen is not None:  # App. E activity penalties on the spike counts, (1/B) sum over samples
        lam_low, nu_low, lam_up, nu_up = pen
        zeta = torch.stack(sg).sum(0).reshape(B, -1)
        n = zeta.shape[1]
        r = (lam_low / n) * torch.clamp(nu_low - zeta, min=0.0).pow(2).sum(1) \
            + lam_up * torch.clamp(zeta.mean(1) - nu_up, min=0.0)
        loss = loss + r.mean()
    loss.backward()
    return float(loss.detach()), wc.grad.permute(2, 3, 1, 0).numpy(), wo.grad.numpy(), fwd


@pytest.mark.parametrize("b_th,mode", [(0.3, "max"), (np.inf, "max"), (0.3, "sum")])
def test_gradient_matches_torch_autograd(b_th, mode):
    """dWc and dW_out of the truncated-surrogate BPTT through conv, pooling and readout equal
    torch autograd (reset detached, Sec. 2.2)."""
    X, Wc, Wo, y = _case(T=14, B=3, H=6, W=6, C=2, Fo=5, rate=0.2, sigma=0.8, seed=11)
    a = F32(math.exp(-0.1))
    loss, gWc, gWo, f = _torch_conv_grads(X, Wc, Wo, y, b_th, mode=mode)
    assert (f["S"].sum() > 20) and (f["P"].sum() < f["P"].size)
    r = conv.conv_network_backward(f, Wc, Wo, a, y, mode, 1.0, b_th, 100.0)
    assert r["loss"] == pytest.approx(loss, rel=1e-9)
    assert np.allclose(r["dWc"], gWc, rtol=1e-7, atol=1e-9 * np.abs(gWc).max())
    assert np.allclose(r["dW_out"], gWo, rtol=1e-7, atol=1e-9 * np.abs(gWo).max())
    assert np.abs(r["dWc"]).max() > 0


def test_weight_grad_is_toeplitz_chain_rule():
    """conv_weight_grad equals dW of the equivalent fully connected layer (trace^T G on the
    Toeplitz matrix's entries) summed over the positions that share each filter weight."""
    r = np.random.default_rng(5)
    T, B, H, W, C, Fo = 3, 2, 5, 4, 2, 3
    G = r.standard_normal((T, B, H, W, Fo))
    tr = r.standard_normal((T, B, H, W, C))
    full = tr.reshape(T * B, -1).T @ G.reshape(T * B, -1)  # [H W C, H W F]
    want = np.zeros((3, 3, C, Fo))
    for y in range(H):
        for x in range(W):
            for ky in range(3):
                for kx in range(3):
                    yi, xi = y + ky - 1, x + kx - 1
                    if 0 <= yi < H and 0 <= xi < W:
                        want[ky, kx] += full[(yi * W + xi) * C:(yi * W + xi + 1) * C, (y * W + x) * Fo:(y * W + x + 1) * Fo]
    assert np.allclose(conv.conv_weight_grad(G, tr), want, rtol=1e-12, atol=1e-12)


def test_wrong_pool_routing_is_caught():
    """Routing each window's gradient to its last maximal element instead fails the autograd pin."""
    X, Wc, Wo, y = _case(T=14, B=3, H=6, W=6, C=2, Fo=5, rate=0.2, sigma=0.8, seed=11)
    good = conv.maxpool_spikes

    def last_max(S):
        P, _ = good(S)
        T, B, H, W, Fo = S.shape
        s = (S != 0).reshape(T, B, H // 2, 2, W // 2, 2, Fo)
        win = np.stack([s[:, :, :, 0, :, 0], s[:, :, :, 0, :, 1], s[:, :, :, 1, :, 0], s[:, :, :, 1, :, 1]], -1)
        return P, 3 - np.argmax(win[..., ::-1], axis=-1)

    _, gWc, _, f = _torch_conv_grads(X, Wc, Wo, y, np.inf)
    _, f["arg"] = last_max(f["S"])
    a = F32(math.exp(-0.1))
    r = conv.conv_network_backward(f, Wc, Wo, a, y, "max", 1.0, np.inf, 100.0)
    assert not np.allclose(r["dWc"], gWc, rtol=1e-3)


def test_activity_penalty_gradient_matches_torch_autograd():
    """With the activity penalties of App. E on the conv layer's spike counts, dWc (through the
    spike-count coefficient joining every conv spike's gradient) equals torch autograd of
    cross-entropy + (1/B) sum_b R(zeta_b); bounds chosen so both hinges are active."""
    X, Wc, Wo, y = _case(T=14, B=3, H=6, W=6, C=2, Fo=5, rate=0.2, sigma=0.8, seed=11)
    pen = (3.0, 2.0, 0.7, 0.4)
    a = F32(math.exp(-0.1))
    loss, gWc, gWo, f = _torch_conv_grads(X, Wc, Wo, y, 0.3, pen=pen)
    zeta = oracle.spike_counts(f["S"].reshape(14, 3, -1))
    assert (zeta < pen[1]).any() and (zeta.mean(axis=1) > pen[3]).any()
    coef = oracle.activity_grad(zeta, *pen)
    r = conv.conv_network_backward(f, Wc, Wo, a, y, "max", 1.0, 0.3, 100.0, reg=coef.reshape(3, 6, 6, 5))
    pen_total = float(np.mean(oracle.activity_penalty(zeta, *pen)))
    assert r["loss"] + pen_total == pytest.approx(loss, rel=1e-9)
    assert np.allclose(r["dWc"], gWc, rtol=1e-7, atol=1e-9 * np.abs(gWc).max())
    assert np.allclose(r["dW_out"], gWo, rtol=1e-7, atol=1e-9 * np.abs(gWo).max())
    plain = conv.conv_network_backward(f, Wc, Wo, a, y, "max", 1.0, 0.3, 100.0)
    assert not np.allclose(plain["dWc"], gWc, rtol=1e-3)  # the penalty term is not negligible
