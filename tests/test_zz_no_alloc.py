"""snn_active_compact_bits_noalloc (the compaction with its scratch in the library's own device
array) against snn_active_compact_bits with a caller workspace: the same CSR, g and nnz, bit for
bit, on two calls in a row, the second with a smaller input (the array keeps the first call's
contents), and again after a call with a capacity too small for the active set."""
import pytest
import torch

from paper_2105_08810_amd import pipeline, snn
from synth import CONFIGS, make_inputs

pytestmark = pytest.mark.gpu


def _layer(name, batch, b_th, l):
    net = pipeline.from_inputs(make_inputs(CONFIGS[name], batch)).forward(b_th)
    torch.cuda.synchronize()
    return net.bits[l], net.V[l], net.theta, net.beta


def _both(bits, V, theta, beta, cap):
    T, B, N = V.shape
    dev = V.device
    out = []
    for noalloc in (False, True):
        rp = torch.full((T * B + 1,), -7, dtype=torch.int32, device=dev)
        ci = torch.full((max(cap, 1),), -7, dtype=torch.int32, device=dev)
        g = torch.full((max(cap, 1),), -7.0, dtype=torch.float32, device=dev)
        nnz = torch.full((1,), -7, dtype=torch.int64, device=dev)
        if noalloc:
            snn.snn_active_compact_bits_noalloc(bits, V, T, B, N, theta, beta, rp, ci, g, cap, nnz)
        else:
            ws = snn.workspace(snn.snn_active_compact_bits_workspace(T, B, N), dev)
            snn.snn_active_compact_bits(bits, V, T, B, N, theta, beta, rp, ci, g, cap, nnz, ws)
        torch.cuda.synchronize()
        out.append((rp, ci, g, nnz))
    return out


def _same(a, b, what):
    (rp, ci, g, nnz), (rp2, ci2, g2, nnz2) = a, b
    assert int(nnz.item()) == int(nnz2.item()), what
    assert torch.equal(rp, rp2), what
    assert torch.equal(ci, ci2), what  # slots past nnz keep the fill value on both sides
    assert torch.equal(g.view(torch.int32), g2.view(torch.int32)), what


def test_noalloc_matches_workspace_form():
    cases = [("stress", list(range(8)), 0.2, 0), ("latency", list(range(16)), 0.2, 0)]  # second call smaller
    print(f"\n[case] noalloc compaction {[c[:1] + (len(c[1]),) for c in cases]}", flush=True)
    for name, batch, b_th, l in cases:
        bits, V, theta, beta = _layer(name, batch, b_th, l)
        T, B, N = V.shape
        assert T * B * 4 < (8 << 20)
        ref_nnz = None
        for cap in (None, 5):  # a capacity that fits, then one that overflows (entries dropped)
            if cap is None:
                probe = _both(bits, V, theta, beta, 1)
                ref_nnz = int(probe[0][3].item())
                assert ref_nnz > 5, (name, ref_nnz)
                cap = ref_nnz
            a, b = _both(bits, V, theta, beta, cap)
            _same(a, b, f"{name} cap={cap}")
            assert int(a[3].item()) == ref_nnz


def test_noalloc_second_call_smaller_after_larger():
    """Large call, then a small one, then the large one again: each equals the workspace form."""
    big = _layer("stress", list(range(8)), 0.2, 1)
    small = _layer("tiny", None, 0.2, 0)
    print(f"\n[case] noalloc big {tuple(big[1].shape)} then small {tuple(small[1].shape)}", flush=True)
    for k, (bits, V, theta, beta) in enumerate((big, small, big)):
        n = int(_both(bits, V, theta, beta, 1)[0][3].item())
        a, b = _both(bits, V, theta, beta, max(n, 1))
        _same(a, b, f"call {k}")
