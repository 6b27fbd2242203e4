"""The training step on the GPU (through the C ABI) against the CPU oracle.

Activity penalties (App. E): spike counts bit-exact, the coefficient and the penalty to float32
rounding of the oracle's float64 values. Gradient add: bit-exact against the one float32 add it
defines. Adam: within the rounding of its float32 arithmetic. Whole steps: gradients with the
penalties inside the 1e-4 envelope of the oracle's, and the Adam step exact to float32 rounding
on the gradients the GPU produced.
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
F32 = np.float32
F64 = np.float64
U = 2.0 ** -24  # float32 unit roundoff


def _np(t):
    return t.detach().cpu().numpy()


def _f32(*xs):
    """Hyper-parameters as the float32 values the C ABI receives, widened to float64 for the oracle."""
    return tuple(float(F32(x)) for x in xs)


def _spikes(T, B, N, p, seed):
    r = np.random.default_rng(seed)
    S = (r.random((T, B, N)) < p).astype(np.uint8)
    return S * r.choice(np.array([1, 7, 255], np.uint8), size=S.shape)  # any nonzero byte is a spike


REG_CASES = [
    # T, B, N, spike prob, (lam_low, nu_low, lam_up, nu_up)
    (20, 4, 32, 0.05, (100.0, 0.001, 0.06, 1.0)),
    (100, 8, 200, 0.02, (100.0, 0.001, 0.06, 1.0)),
    (37, 5, 13, 0.3, (40.0, 3.5, 4.0, 5.0)),  # B*N odd: byte-wise count
    (1, 1, 1, 1.0, (2.0, 1.5, 3.0, 0.25)),
    (1000, 3, 64, 0.01, (100.0, 12.0, 0.06, 10.0)),  # many chunks
    (500, 256, 1024, 0.015, (100.0, 0.001, 0.06, 1.0)),  # a full stress-sized layer
]


@pytest.mark.parametrize("T,B,N,p,reg", REG_CASES)
def test_activity_reg_matches_oracle(T, B, N, p, reg):
    S_h = _spikes(T, B, N, p, seed=T * 7 + N)
    S = torch.from_numpy(S_h).cuda()
    coef, pen, zeta = snn.activity_reg(S, *reg, want_zeta=True)
    torch.cuda.synchronize()
    z_ref = oracle.spike_counts(S_h)
    assert np.array_equal(_np(zeta).astype(np.int64), z_ref)
    r = _f32(*reg)
    c_ref = oracle.activity_grad(z_ref, *r)
    assert np.allclose(_np(coef), c_ref, rtol=U, atol=1e-45)
    p_ref = oracle.activity_penalty(z_ref, *r).mean()
    assert abs(float(pen.item()) - p_ref) <= U * abs(p_ref) + 1e-45


def test_activity_reg_unaligned_spikes():
    """A spike tensor that starts off a 4-byte boundary takes the byte-wise count."""
    T, B, N = 30, 4, 64
    S_h = _spikes(T, B, N, 0.1, seed=3)
    buf = torch.zeros(S_h.size + 1, dtype=torch.uint8, device="cuda")
    buf[1:] = torch.from_numpy(S_h.ravel()).cuda()
    S = buf[1:].view(T, B, N)
    coef, pen, zeta = snn.activity_reg(S, 100.0, 2.0, 0.06, 0.5, want_zeta=True)
    torch.cuda.synchronize()
    z_ref = oracle.spike_counts(S_h)
    assert np.array_equal(_np(zeta).astype(np.int64), z_ref)
    assert np.allclose(_np(coef), oracle.activity_grad(z_ref, *_f32(100.0, 2.0, 0.06, 0.5)), rtol=U, atol=1e-45)


@pytest.mark.parametrize("T,B,N,dens", [(20, 4, 32, 0.3), (50, 7, 101, 0.05), (3, 2, 4, 1.0), (10, 3, 9, 0.0)])
def test_activity_reg_grad_csr(T, B, N, dens):
    """eps[e] += coef[b, col] at every CSR entry, one float32 add; entries past the capacity untouched."""
    r = np.random.default_rng(T + N)
    V = r.uniform(0.5, 1.5, (T, B, N)).astype(F32)
    b_th = dens * 0.5 if dens < 1 else 1.0
    rp, ci, _ = oracle.active_csr(V, 1.0, b_th, 100.0)
    nnz = int(rp[-1])
    coef_h = r.standard_normal((B, N)).astype(F32)
    eps_h = r.standard_normal(nnz + 5).astype(F32)
    rows = np.repeat(np.arange(T * B), np.diff(rp))
    want = eps_h.copy()
    want[:nnz] = (eps_h[:nnz] + coef_h[rows % B, ci]).astype(F32)
    csr = snn.Csr(torch.from_numpy(rp.astype(np.int32)).cuda(), torch.from_numpy(
        np.concatenate([ci, np.zeros(5, np.int64)]).astype(np.int32)).cuda(), None, None, nnz + 5)
    eps = torch.from_numpy(eps_h).cuda()
    snn.activity_reg_grad(torch.from_numpy(coef_h).cuda(), T, eps, csr)
    torch.cuda.synchronize()
    assert np.array_equal(_np(eps).view(np.uint32), want.view(np.uint32))
    if nnz > 1:  # a capacity below nnz stops the add there
        eps2 = torch.from_numpy(eps_h).cuda()
        csr.capacity = nnz // 2
        snn.activity_reg_grad(torch.from_numpy(coef_h).cuda(), T, eps2, csr)
        torch.cuda.synchronize()
        w2 = eps_h.copy()
        w2[: nnz // 2] = want[: nnz // 2]
        assert np.array_equal(_np(eps2).view(np.uint32), w2.view(np.uint32))


@pytest.mark.parametrize("T,B,N", [(20, 4, 32), (7, 3, 5)])
def test_activity_reg_grad_dense(T, B, N):
    r = np.random.default_rng(N)
    coef_h = r.standard_normal((B, N)).astype(F32)
    eps_h = r.standard_normal((T, B, N)).astype(F32)
    eps = torch.from_numpy(eps_h).cuda()
    snn.activity_reg_grad(torch.from_numpy(coef_h).cuda(), T, eps)
    torch.cuda.synchronize()
    want = (eps_h + coef_h[None]).astype(F32)
    assert np.array_equal(_np(eps).view(np.uint32), want.view(np.uint32))


def _adam_bound(w, g, m, v, k, lr, b1, b2, eps, m_ref, v_ref, w_ref):
    """Rounding bounds of the float32 Adam step against the float64 one (same float32 inputs):
    a few unit roundoffs of each term's magnitude, the update's relative error carried by
    step_size, 1/sqrt(1-b2^k), the division and the square root."""
    bm = 4 * U * (b1 * np.abs(m) + (1 - b1) * np.abs(g)) + 1e-45
    bv = 4 * U * (b2 * np.abs(v) + (1 - b2) * g * g) + 1e-45
    upd = np.abs(w - w_ref)
    bw = U * np.abs(w_ref) + 16 * U * upd + 1e-45
    return bm, bv, bw


@pytest.mark.parametrize("n", [4096, 1027, 1])
@pytest.mark.parametrize("k", [1, 2, 50])
def test_adam_matches_oracle(n, k):
    r = np.random.default_rng(n + k)
    w = r.standard_normal(n).astype(F32)
    g = (r.standard_normal(n) * 10.0 ** r.integers(-6, 2, n)).astype(F32)
    g[::7] = 0.0
    m = (r.standard_normal(n) * 1e-2).astype(F32) if k > 1 else np.zeros(n, F32)
    v = (r.random(n) * 1e-3).astype(F32) if k > 1 else np.zeros(n, F32)
    lr, b1, b2, eps = 2e-4, 0.9, 0.999, 1e-8
    W_d, g_d, m_d, v_d = (torch.from_numpy(x.copy()).cuda() for x in (w, g, m, v))
    snn.adam_step(W_d, g_d, m_d, v_d, k, lr, (b1, b2), eps)
    torch.cuda.synchronize()
    L = _f32(lr, b1, b2, eps)
    w_ref, m_ref, v_ref = oracle.adam_update(w, g, m, v, k, *L)
    bm, bv, bw = _adam_bound(w.astype(F64), g.astype(F64), m.astype(F64), v.astype(F64), k, *L, m_ref, v_ref, w_ref)
    assert (np.abs(_np(m_d) - m_ref) <= bm).all()
    assert (np.abs(_np(v_d) - v_ref) <= bv).all()
    assert (np.abs(_np(W_d) - w_ref) <= bw).all()


# ------------------------------------------------------------------ whole training steps

STRONG = (40.0, 2.0, 4.0, 0.2)
APP_E = (100.0, 0.001, 0.06, 1.0)


def _two_layer():
    cfg = Config("tiny2t", 103, T=40, B=8, sizes=(96, 48, 40, 5), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
                 loss_mode="max", b_th=0.3, kind="bernoulli", rate=0.08)
    return make_inputs(cfg, sigmas=[0.2, 0.3, 1 / math.sqrt(40)])


def _check_grads(inp, grads, b_th, reg):
    cfg = inp.cfg
    args = (inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode, cfg.theta, b_th, cfg.beta)
    r = oracle.training_gradients(*args, reg=_f32(*reg) if reg else None)
    env = oracle.network_backward(r["fwd"], inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode,
                                  cfg.theta, b_th, cfg.beta, absolute=True, reg=r["coef"])
    refs = list(r["dW"]) + [r["dW_out"]]
    envs = list(env["dW"]) + [env["dW_out"]]
    for k, (x, want, e) in enumerate(zip(grads, refs, envs)):
        err = np.abs(_np(x).astype(F64) - want)
        assert (err <= 1e-4 * e + 1e-30).all(), (k, float((err / np.maximum(e, 1e-300)).max()))
    return r


@pytest.mark.parametrize("sparse,b_th", [(True, 0.3), (False, 0.3), (False, math.inf)])
@pytest.mark.parametrize("reg", [STRONG, APP_E, None])
def test_training_gradients_match_oracle(sparse, b_th, reg):
    """Gradients of CE + penalties through the sparse chain (and the dense and full-surrogate
    ones) against the oracle, inside the 1e-4 envelope."""
    inp = _two_layer()
    net = pipeline.from_inputs(inp)
    pen = pipeline.Penalty(*reg) if reg else None
    opt = pipeline.Adam(net.params(), lr=0.0)  # lr 0: weights stay, only the gradients matter here
    out = net.train_step(opt, b_th, pen, sparse=sparse)
    torch.cuda.synchronize()
    r = _check_grads(inp, out["grads"], b_th, reg)
    assert abs(float(out["ce"].item()) - r["ce"]) <= 1e-5 * max(1.0, r["ce"])
    want_pen = sum(r["penalty"])
    assert abs(float(out["penalty"].item()) - want_pen) <= 4 * U * abs(want_pen) + 1e-30


def test_three_adam_steps_track_the_oracle():
    """Each step: the GPU's gradients at its current weights match the oracle's there, and the
    weights after the step equal the oracle's Adam step applied to the GPU's gradients."""
    inp = _two_layer()
    net = pipeline.from_inputs(inp)
    lr = 1e-3
    opt = pipeline.Adam(net.params(), lr=lr)
    pen = pipeline.Penalty(*STRONG)
    L = _f32(lr, 0.9, 0.999, 1e-8)
    for k in range(1, 4):
        before = [_np(p).copy() for p in net.params()]
        m0 = [_np(m).copy() for m in opt.m]
        v0 = [_np(v).copy() for v in opt.v]
        out = net.train_step(opt, 0.3, pen, sparse=True)
        torch.cuda.synchronize()
        inp.Ws, inp.W_out = before[:-1], before[-1]
        _check_grads(inp, out["grads"], 0.3, STRONG)
        for j, p in enumerate(net.params()):
            g = _np(out["grads"][j]).astype(F64)
            w_ref, m_ref, v_ref = oracle.adam_update(before[j], g, m0[j], v0[j], k, *L)
            _, _, bw = _adam_bound(before[j].astype(F64), g, m0[j].astype(F64), v0[j].astype(F64), k, *L, m_ref,
                                   v_ref, w_ref)
            assert (np.abs(_np(p) - w_ref) <= bw).all(), (k, j)
        assert any(not np.array_equal(_np(p), b) for p, b in zip(net.params(), before))
