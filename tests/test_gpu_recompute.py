"""Trace recompute (snn_trace_checkpoints + snn_sparse_dw_spikes) on the GPU.

The checkpoints equal the forward's stored input trace at every K-th step bit for bit; dW
computed from the spikes and checkpoints (float64 accumulation) equals dW computed from the stored
trace (same CSR; float32 accumulation per chunk of rows on the matrix cores) within 3e-5 of the
error envelope sum |G| trace, and stays within the oracle's envelope. Cases cover sample
counts that are not multiples of 8 or 128, step counts that are not multiples of K, K = 1, K > T,
narrow and wide layers, and the stress workload's layers at full size.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2105_08810_amd import pipeline, snn
from synth import CONFIGS, make_inputs
from synth.inputs import Config

pytestmark = pytest.mark.gpu
TOL = 1e-4


def _np(t):
    return t.detach().cpu().numpy()


def _inputs(T, B, sizes, rate=0.3, seed=301, b_th=0.4):
    cfg = Config(f"rc{T}x{B}", seed, T=T, B=B, sizes=sizes, tau_ratio_hidden=0.1, tau_ratio_out=0.1, loss_mode="max",
                 b_th=b_th, kind="bernoulli", rate=rate)
    rates = [rate] + [0.2] * (len(sizes) - 2)
    sig = [1.2 / math.sqrt(r * n) for r, n in zip(rates, sizes[:-2])] + [1 / math.sqrt(sizes[-2])]
    return make_inputs(cfg, sigmas=sig)


def _layers(net, csrs, epss, K):
    """Per LIF layer: (dW from the stored trace, dW from spikes + checkpoints, checkpoints, s_in)."""
    out = []
    for l in range(net.L):
        s_in = net.X if l == 0 else net.S[l - 1]
        ck = snn.trace_checkpoints(s_in, net.alphas[l], K)
        n_out = net.Ws[l].shape[1]
        ref = snn.sparse_dw(net.trace[l], csrs[l], epss[l], n_out)
        got = snn.sparse_dw_spikes(s_in, ck, K, net.alphas[l], csrs[l], epss[l], n_out)
        out.append((ref, got, ck, _env(net.trace[l], csrs[l], epss[l], n_out)))
    torch.cuda.synchronize()
    return out


def _check_ck(net, ck, l, K):
    tr = _np(net.trace[l])
    c = _np(ck)
    T = tr.shape[0]
    assert c.shape[0] == -(-T // K)
    same = c.view(np.uint32) == tr[::K].view(np.uint32)
    assert same.all(), f"checkpoints of layer {l}: {int((~same).sum())} differ"


def _env(trace, csr, eps, n_out):
    """The error envelope sum |G| trace of a dW (g >= 0 and traces >= 0: the same sparse dW of |eps|)."""
    return snn.sparse_dw(trace, csr, eps.abs(), n_out)


def _check_dw(ref, got, env, what):
    """Two float32 sums of the same terms: within 3e-5 of the envelope (a float32 sum of n terms is
    within about n 2^-24 of it; the stored-trace dW sums at most a few hundred terms per chunk)."""
    x, y = _np(got).astype(np.float64), _np(ref).astype(np.float64)
    bad = np.abs(x - y) > 3e-5 * _np(env).astype(np.float64) + 1e-30
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} differ from the stored-trace dW"


@pytest.mark.parametrize("T,B,sizes,K", [(37, 3, (61, 37, 29, 5), 5), (20, 13, (40, 70, 9), 1),
                                         (9, 5, (130, 33, 3), 16), (33, 200, (24, 96, 7), 8)])
def test_recompute_matches_stored_trace_and_oracle(T, B, sizes, K):
    print(f"\n[case] recompute T={T} B={B} sizes={sizes} K={K}", flush=True)
    inp = _inputs(T, B, sizes)
    cfg = inp.cfg
    net = pipeline.from_inputs(inp).forward()
    ro = net.readout(dense=True)
    csrs = net.compact(0.4)
    _, _, epss = net.sparse_backward(csrs, ro)
    f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))
    args = (inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode, cfg.theta, 0.4, cfg.beta)
    r = oracle.network_backward(f, *args)
    env = oracle.network_backward(f, *args, absolute=True)
    for l, (ref, got, ck, e) in enumerate(_layers(net, csrs, epss, K)):
        _check_ck(net, ck, l, K)
        _check_dw(ref, got, e, f"dW[{l}]")
        err = np.abs(_np(got).astype(np.float64) - r["dW"][l])
        assert not (err > TOL * env["dW"][l] + 1e-30).any(), f"dW[{l}] outside the oracle envelope"
        assert np.abs(r["dW"][l]).max() > 0


@pytest.mark.parametrize("K", [16, 32])
def test_recompute_full_size_stress(K):
    """The stress workload at full size (T=500, B=256, 3 x 1024, B_th = 0.2): checkpoints bit-exact,
    dW of every LIF layer from spikes equal to dW from the stored trace."""
    print(f"\n[case] recompute full-size stress K={K}", flush=True)
    inp = make_inputs(CONFIGS["stress"])
    net = pipeline.from_inputs(inp).forward(0.2)
    ro = net.readout(dense=True)
    csrs = net.compact(0.2)
    _, _, epss = net.sparse_backward(csrs, ro)
    for l, (ref, got, ck, e) in enumerate(_layers(net, csrs, epss, K)):
        _check_ck(net, ck, l, K)
        _check_dw(ref, got, e, f"stress dW[{l}]")


@pytest.mark.parametrize("aux", [False, True])
def test_network_recompute_mode(aux):
    """Network(recompute_k=K) stores no LIF input trace: its sparse backward (spike gradient beside
    the spikes-based dW) gives the stored-trace network's dW (up to accumulation order) and the
    same spike gradients bit for bit; the dense baseline refuses to run without traces."""
    print(f"\n[case] network recompute aux={aux}", flush=True)
    inp = _inputs(41, 19, (50, 80, 70, 6), b_th=0.4)
    ref = pipeline.from_inputs(inp).forward(0.4)
    net = pipeline.from_inputs(inp)
    net.recompute_k = 8
    net.forward(0.4)
    assert all(t is None for t in net.trace) and len(net.ck) == net.L
    side = torch.cuda.Stream() if aux else None
    outs = []
    for n in (ref, net):
        ro = n.readout(dense=False)
        csrs = n.compact(0.4)
        outs.append(n.sparse_backward(csrs, ro, aux_stream=side) + (csrs,))
    torch.cuda.synchronize()
    (dW_a, dWo_a, eps_a, cs_a), (dW_b, dWo_b, eps_b, cs_b) = outs
    assert torch.equal(dWo_a, dWo_b)
    for l in range(net.L):
        env = _env(ref.trace[l], cs_a[l], eps_a[l], ref.Ws[l].shape[1])
        _check_dw(dW_a[l], dW_b[l], env, f"network dW[{l}]")
        n = cs_a[l].nnz()
        assert n == cs_b[l].nnz() and torch.equal(eps_a[l][:n], eps_b[l][:n]), f"eps[{l}]"
    with pytest.raises(ValueError):
        net.dense_backward(0.4)
