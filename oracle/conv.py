"""Spiking convolutional layer with 2x2 max pooling (the convolutional experiment of Sec. 3,
network details in App. E); oracle, test use only.

Network: input spikes X [T, B, H, W, C] (channels last) -> a convolutional LIF layer of F
filters, 3x3, stride 1, zero padding 1 -> 2x2 max pooling of its spikes -> flattened -> the
non-spiking LIF readout (infinite threshold) -> cross-entropy (loss.py).

Readings adopted:
* The convolutional layer is a LIF layer whose input current is the convolution: Sec. 2's
  definitions hold with W replaced by the layer's Toeplitz matrix (toeplitz() writes it out), so
  the forward is forward.lif_forward on that matrix (weighted inputs summed over spiking inputs
  in ascending flattened input index (y', x', c), float32, from +0.0).
* Padding 1: with 28x28 inputs, 64 filters and the 2x2 pool this gives the 64 * 14 * 14 = 12544
  readout inputs the appendix states (no padding would give 10816).
* Max pooling of binary spikes is their OR. Its gradient goes to the first maximal element of
  the window in row-major order (as PyTorch's max pooling does): the first spiking element,
  else the window's top-left element.
* The readout integrates the pooled spikes; its trace is theirs.
* Layouts: activations channels last, neuron index n = (y * W + x) * F + f; filters
  Wc [3, 3, C, F] indexed (ky, kx, c, f), output (y, x) reading input (y + ky - 1, x + kx - 1).
Everything in the backward is float64.
"""
from __future__ import annotations

import numpy as np

from .active import active_mask, surrogate
from .backward import layer_backward
from .forward import lif_forward
from .loss import readout_grad

F32 = np.float32
F64 = np.float64


def toeplitz(Wc: np.ndarray, H: int, W: int) -> np.ndarray:
    """[H*W*C, H*W*F] float32 matrix of the 3x3, stride 1, padding 1 convolution:
    M[(y'*W + x')*C + c, (y*W + x)*F + f] = Wc[y' - y + 1, x' - x + 1, c, f] for |y'-y|, |x'-x| <= 1."""
    Wc = np.asarray(Wc, F32)
    _, _, C, Fo = Wc.shape
    M = np.zeros((H * W * C, H * W * Fo), F32)
    for y in range(H):
        for x in range(W):
            out = (y * W + x) * Fo
            for ky in range(3):
                for kx in range(3):
                    yi, xi = y + ky - 1, x + kx - 1
                    if 0 <= yi < H and 0 <= xi < W:
                        inp = (yi * W + xi) * C
                        M[inp:inp + C, out:out + Fo] = Wc[ky, kx]
    return M


def maxpool_spikes(S: np.ndarray):
    """2x2 max pooling of spikes [T, B, H, W, F]: pooled spikes [T, B, H/2, W/2, F] uint8 and the
    window position (0..3, row-major: (0,0), (0,1), (1,0), (1,1)) of the first maximal element."""
    T, B, H, W, Fo = S.shape
    s = (np.asarray(S) != 0).reshape(T, B, H // 2, 2, W // 2, 2, Fo)
    win = np.stack([s[:, :, :, 0, :, 0], s[:, :, :, 0, :, 1], s[:, :, :, 1, :, 0], s[:, :, :, 1, :, 1]], axis=-1)
    P = win.any(axis=-1).astype(np.uint8)
    arg = np.argmax(win, axis=-1).astype(np.int64)  # first True, or 0 when none
    return P, arg


def conv_network_forward(X, Wc, W_out, alpha, alpha_out, theta=1.0):
    """X [T, B, H, W, C] spikes. Returns V, S [T, B, H, W, F], the input trace [T, B, H, W, C],
    P and arg of the pooling, V_out and the readout's trace of P [T, B, (H/2)(W/2)F]."""
    T, B, H, W, C = X.shape
    Fo = Wc.shape[3]
    V, S, tr = lif_forward(X.reshape(T, B, H * W * C), toeplitz(Wc, H, W), alpha, F32(theta))
    V = V.reshape(T, B, H, W, Fo)
    S = S.reshape(T, B, H, W, Fo)
    P, arg = maxpool_spikes(S)
    V_out, _, tr_out = lif_forward(P.reshape(T, B, -1), W_out, alpha_out, np.inf)
    return {"V": V, "S": S, "trace": tr.reshape(T, B, H, W, C), "P": P, "arg": arg, "V_out": V_out,
            "trace_out": tr_out}


def route_to_conv(eps_P: np.ndarray, arg: np.ndarray, H: int, W: int) -> np.ndarray:
    """Gradient w.r.t. the pooled spikes [T, B, H/2, W/2, F] to the conv layer's spikes
    [T, B, H, W, F]: each window's gradient goes to the element the pooling picked."""
    T, B, h, w, Fo = eps_P.shape
    out = np.zeros((T, B, h, 2, w, 2, Fo), F64)
    for k, (dy, dx) in enumerate(((0, 0), (0, 1), (1, 0), (1, 1))):
        out[:, :, :, dy, :, dx] = np.where(arg == k, eps_P, 0.0)
    return out.reshape(T, B, H, W, Fo)


def conv_weight_grad(G: np.ndarray, trace: np.ndarray) -> np.ndarray:
    """dWc[ky, kx, c, f] = sum over (t, b, y, x) of G[t,b,y,x,f] * trace[t,b,y+ky-1,x+kx-1,c]
    (zero outside the map): Eq. (w_grad) with the Toeplitz matrix's shared weights summed."""
    T, B, H, W, Fo = G.shape
    C = trace.shape[4]
    tp = np.zeros((T, B, H + 2, W + 2, C), F64)
    tp[:, :, 1:H + 1, 1:W + 1] = trace
    G2 = np.asarray(G, F64).reshape(-1, Fo)
    dW = np.zeros((3, 3, C, Fo), F64)
    for ky in range(3):
        for kx in range(3):
            dW[ky, kx] = tp[:, :, ky:ky + H, kx:kx + W].reshape(-1, C).T @ G2
    return dW


def conv_network_backward(fwd: dict, Wc, W_out, alpha_out, labels, mode: str, theta, b_th, beta,
                          absolute: bool = False, reg=None):
    """Truncated-surrogate gradient of the conv network (float64): loss, dWc [3, 3, C, F],
    dW_out, eps_P (w.r.t. pooled spikes), eps (w.r.t. conv spikes), G, mask, g. With
    absolute=True the magnitude envelope (as backward.network_backward). reg ([B, H, W, F],
    d penalty / d spike count from regularize.activity_grad, App. E) joins the gradient w.r.t.
    every conv spike S[t] before the surrogate gate, as the spike count sums S over t."""
    T, B, H, W, Fo = fwd["V"].shape
    ro = readout_grad(fwd["V_out"], labels, mode)
    G_out = ro["G_abs"] if absolute else ro["G"]
    Wo = np.abs(W_out) if absolute else W_out
    dW_out, eps_P = layer_backward(G_out, Wo, fwd["trace_out"], alpha_out, grad_in=True)
    eps_P = eps_P.reshape(T, B, H // 2, W // 2, Fo)
    eps = route_to_conv(eps_P, fwd["arg"], H, W)
    if reg is not None:
        r = np.asarray(reg, np.float64).reshape(B, H, W, Fo)
        eps = eps + (np.abs(r) if absolute else r)[None]
    mask = active_mask(fwd["V"], theta, b_th)
    g = surrogate(fwd["V"], theta, beta)
    G = eps * g * mask
    dWc = conv_weight_grad(G, fwd["trace"])
    return {"loss": ro["loss"], "readout": ro, "dWc": dWc, "dW_out": dW_out, "eps_P": eps_P, "eps": eps, "G": G,
            "mask": mask, "g": g}
