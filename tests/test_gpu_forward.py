"""LIF forward through the C ABI against the oracle, bit for bit, on shapes chosen to reach each
variant of the fused forward kernel: spike rows of one segment (the trace from the staged spike
bytes) or of several (trace blocks beside the fused blocks), one or two float4 groups of columns
per lane, several column groups per sample, partial column groups, wavefronts with columns past
the layer's width, spike rows that are not whole 4-byte words, dense spike rows, a last time tile
that is not full, and the two-kernel path (widths whose bitset words straddle samples, grids of
fewer than two blocks per CU).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2105_08810_amd import snn

pytestmark = pytest.mark.gpu
F32 = np.float32


def _case(T, B, n_in, n_out, rate, seed):
    rng = np.random.default_rng(seed)
    X = (rng.random((T, B, n_in)) < rate).astype(np.uint8)
    alpha = F32(np.exp(-0.1))
    m = max(1.0, rate * n_in)
    W = (rng.standard_normal((n_in, n_out)) * (0.6 * math.sqrt(1 - float(alpha) ** 2) / math.sqrt(m))).astype(F32)
    W += F32(0.05)  # a positive drift, so that neurons cross the threshold and reset
    return X, W, alpha


def _bits_from(V, theta, b_th):
    T, B, N = V.shape
    act = oracle.active_mask(V, theta, b_th).reshape(T, B * N)
    n64 = (B * N + 63) // 64
    pad = np.zeros((T, n64 * 64), dtype=bool)
    pad[:, :B * N] = act
    w = np.packbits(pad.reshape(T, n64, 64), axis=2, bitorder="little")
    return w.view(np.uint64).reshape(T, n64).view(np.int64)


def _run(X, W, alpha, theta, b_th):
    T, B, n_in = X.shape
    n_out = W.shape[1]
    x = torch.from_numpy(X).cuda()
    w = torch.from_numpy(W).cuda()
    V = torch.empty((T, B, n_out), dtype=torch.float32, device="cuda")
    S = torch.empty((T, B, n_out), dtype=torch.uint8, device="cuda")
    tr = torch.empty((T, B, n_in), dtype=torch.float32, device="cuda")
    if b_th is None:
        snn.snn_lif_forward(x, w, T, B, n_in, n_out, alpha, theta, V, S, tr)
        bits = None
    else:
        bits = torch.empty(snn.snn_active_bits_words(T, B, n_out), dtype=torch.int64, device="cuda")
        snn.snn_lif_forward_active(x, w, T, B, n_in, n_out, alpha, theta, b_th, V, S, tr, bits)
    torch.cuda.synchronize()
    return V.cpu().numpy(), S.cpu().numpy(), tr.cpu().numpy(), None if bits is None else bits.cpu().numpy()


# The fused form runs when the grid has at least two blocks per CU (B x column groups >= 512 on
# 256 CUs), hence the batch sizes; the last two cases take the two-kernel form.
@pytest.mark.parametrize("T,B,n_in,n_out,rate,b_th", [
    (37, 256, 1024, 1024, 0.02, 0.2),  # one segment, two column groups of 512, a partial last tile
    (20, 512, 1030, 256, 0.03, 0.2),   # spike rows not whole words: trace blocks, one group of 256
    (18, 512, 2312, 320, 0.01, 0.3),   # several segments; wavefronts 5..7 of the group past the width
    (33, 512, 64, 100, 0.2, None),     # no bitset: a wavefront with columns past the width
    (4, 512, 1024, 512, 0.9, 0.2),     # dense spike rows (lists of up to 1024 entries)
    (9, 64, 700, 3968, 0.05, 0.25),    # eight column groups, the last one partial
    (1, 512, 256, 128, 0.1, 0.2),      # a single step: no tile at all
    (16, 3, 300, 200, 0.05, 0.2),      # bitset words straddle samples: the two-kernel form
    (21, 4, 1024, 1024, 0.02, 0.2),    # too few blocks for the fused form
])
def test_forward_variants_bit_exact(T, B, n_in, n_out, rate, b_th):
    X, W, alpha = _case(T, B, n_in, n_out, rate, seed=T * 7919 + n_in)
    theta = F32(1.0)
    V, S, tr, bits = _run(X, W, alpha, theta, b_th)
    rV, rS, rtr = oracle.lif_forward(X, W, alpha, theta)
    assert (rS[1:] != 0).any() or T == 1, "the case should spike"
    assert np.array_equal(V.view(np.uint32), rV.view(np.uint32)), "V differs from the oracle"
    assert np.array_equal(S, rS), "spikes differ from the oracle"
    assert np.array_equal(tr.view(np.uint32), rtr.view(np.uint32)), "trace differs from the oracle"
    if bits is not None:
        assert np.array_equal(bits.reshape(T, -1), _bits_from(rV, theta, F32(b_th))), "active bitset differs"


@pytest.mark.parametrize("T,B,n_in,n_out,rate,b_th", [
    (37, 256, 1024, 1024, 0.02, 0.2),  # fused, trace from the staged spike bytes (two groups of 512)
    (20, 512, 1030, 256, 0.03, 0.2),   # fused with trace blocks beside it
    (33, 512, 64, 100, 0.2, None),     # fused, no bitset, columns past the width
    (9, 64, 700, 3968, 0.05, 0.25),    # eight column groups, the last one partial
    (1, 512, 256, 128, 0.1, 0.2),      # a single step
    (16, 3, 300, 200, 0.05, 0.2),      # the two-kernel form
    (21, 4, 1024, 1024, 0.02, None),   # the two-kernel form without a bitset
])
def test_forward_output_trace_bit_exact(T, B, n_in, n_out, rate, b_th):
    """snn_lif_forward_traces: the trace of the layer's own spikes, written beside V, equals bit for
    bit the input trace that the oracle forms from those spikes with the next layer's leak (Eq.
    (w_grad)), and V, spikes, input trace and bitset are those of the other forward entry points."""
    X, W, alpha = _case(T, B, n_in, n_out, rate, seed=T * 104729 + n_out)
    theta = F32(1.0)
    alpha_next = F32(np.exp(-1.0 / 15.0))  # not this layer's leak
    V0, S0, tr0, bits0 = _run(X, W, alpha, theta, b_th)
    x = torch.from_numpy(X).cuda()
    w = torch.from_numpy(W).cuda()
    V = torch.empty((T, B, n_out), dtype=torch.float32, device="cuda")
    S = torch.empty((T, B, n_out), dtype=torch.uint8, device="cuda")
    tr = torch.empty((T, B, n_in), dtype=torch.float32, device="cuda")
    to = torch.full((T, B, n_out), float("nan"), dtype=torch.float32, device="cuda")
    bits = None if b_th is None else torch.empty(snn.snn_active_bits_words(T, B, n_out), dtype=torch.int64,
                                                 device="cuda")
    snn.snn_lif_forward_traces(x, w, T, B, n_in, n_out, alpha, theta, 0.0 if b_th is None else b_th, V, S, tr, to,
                               alpha_next, bits)
    torch.cuda.synchronize()
    assert np.array_equal(V.cpu().numpy().view(np.uint32), V0.view(np.uint32))
    assert np.array_equal(S.cpu().numpy(), S0)
    assert np.array_equal(tr.cpu().numpy().view(np.uint32), tr0.view(np.uint32))
    if b_th is not None:
        assert np.array_equal(bits.cpu().numpy(), bits0)
    rS = oracle.lif_forward(X, W, alpha, theta)[1]
    assert (rS[:-1] != 0).any() or T == 1, "the case should spike"
    ref = oracle.lif_forward(rS, np.zeros((n_out, 1), F32), alpha_next, theta)[2]
    assert np.array_equal(to.cpu().numpy().view(np.uint32), ref.view(np.uint32)), "output trace differs"
