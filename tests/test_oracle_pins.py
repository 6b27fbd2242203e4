"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test names the passage it checks. None of them re-types the oracle's own
formula: they use closed forms, brute force, finite differences of an
independent smoothed model, PyTorch autograd, limits, and the App. C example.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import smooth
from synth import CONFIGS, make_inputs
from synth.inputs import Config

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32 = np.float32


def _tiny(batch=None):
    return make_inputs(CONFIGS["tiny"], batch)


def _two_layer_tiny():
    """Two LIF layers (64 -> 32 -> 24) + readout 24 -> 4, to exercise LIF -> LIF grad_in."""
    cfg = Config("tiny2", 101, T=24, B=4, sizes=(64, 32, 24, 4), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
                 loss_mode="max", b_th=0.3, kind="bernoulli", rate=0.08)
    return make_inputs(cfg, sigmas=[0.2, 0.35, 1 / math.sqrt(24)])


def _fwd(inp):
    return oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, F32(inp.cfg.theta))


# ------------------------------------------------------------------ forward

def test_summation_order_matches_elementwise_loop():
    """Eq. (lif): the vectorised weighted input equals the one-term-at-a-time float32 sum."""
    r = np.random.default_rng(0)
    x = r.random((7, 40)) < 0.2
    W = r.standard_normal((40, 9)).astype(F32)
    a = oracle.summed_inputs(x, W)
    b = oracle.summed_inputs_loop(x, W)
    assert a.dtype == F32 and np.array_equal(a.view(np.uint32), b.view(np.uint32))


def _closed_form_V(X, S_out, W, alpha):
    """Eq. (lif_unrolled) in float64 with the oracle's own spikes."""
    a = float(alpha)
    x = (X != 0).astype(np.float64)
    s = S_out.astype(np.float64)
    T = x.shape[0]
    V = np.zeros((T, x.shape[1], W.shape[1]))
    for t in range(T - 1):
        tr = sum(a ** (t - k) * x[k] for k in range(t + 1))
        rs = sum(a ** (t - k) * s[k] for k in range(t + 1))
        V[t + 1] = tr @ W.astype(np.float64) - rs
    return V


@pytest.mark.parametrize("name,batch", [("tiny", None), ("latency", [0, 1]), ("audio", [3]), ("event", [5]),
                                        ("stress", [2])])
def test_P1_forward_matches_unrolled_closed_form(name, batch):
    """P1: the float32 recursion agrees with Eq. (lif_unrolled) evaluated in float64."""
    inp = make_inputs(CONFIGS[name], batch)
    if name in ("event", "stress"):  # keep the O(T^2) closed form cheap
        inp.X = inp.X[:120]
    f = _fwd(inp)
    x = inp.X
    for l, W in enumerate(inp.Ws):
        V64 = _closed_form_V(x, f["S"][l], W, inp.alphas[l])
        err = np.abs(f["V"][l].astype(np.float64) - V64)
        assert err.max() <= 1e-5 * (1.0 + np.abs(V64).max()), (name, l, err.max())
        # spikes are the strict threshold of the float32 V (Eq. (spike_fn))
        assert np.array_equal(f["S"][l], (f["V"][l] > F32(1.0)).astype(np.uint8))
        x = f["S"][l]
    # the trace is the filtered input of Eq. (lif_unrolled)
    a = float(inp.alphas[0])
    xs = (inp.X != 0).astype(np.float64)
    for t in (0, 1, 7, inp.X.shape[0] - 1):
        ref = sum(a ** (t - k - 1) * xs[k] for k in range(t)) if t else np.zeros_like(xs[0])
        assert np.abs(f["trace"][0][t] - ref).max() <= 1e-5 * (1 + np.abs(ref).max())


def test_P2_single_spike_closed_forms():
    """P2: alpha convention (+alpha), one-step delay, soft reset by 1 one step after the spike."""
    T, t0 = 30, 4
    alpha = F32(math.exp(-0.1))
    X = np.zeros((T, 1, 2), np.uint8)
    X[t0, 0, 0] = 1
    w_small, w_big = F32(0.7), F32(1.6)
    W = np.array([[w_small, w_big], [0.0, 0.0]], F32)
    V, S, tr = oracle.lif_forward(X, W, alpha, F32(1.0))
    a = float(alpha)
    for t in range(T):
        ref = float(w_small) * a ** (t - t0 - 1) if t > t0 else 0.0
        assert abs(float(V[t, 0, 0]) - ref) <= 1e-6 * max(1.0, abs(ref))
        assert S[t, 0, 0] == 0
        tref = a ** (t - t0 - 1) if t > t0 else 0.0
        assert abs(float(tr[t, 0, 0]) - tref) <= 1e-6
    assert V[t0 + 1, 0, 1] == w_big and S[t0 + 1, 0, 1] == 1
    assert abs(float(V[t0 + 2, 0, 1]) - (a * float(w_big) - 1.0)) <= 1e-6
    assert S[: t0 + 1, 0, 1].sum() == 0 and S[t0 + 2:, 0, 1].sum() == 0
    assert np.all(S[0] == 0)  # V[0] = 0 never spikes


def test_readout_never_spikes():
    inp = _tiny()
    f = _fwd(inp)
    V, S, _ = oracle.lif_forward(f["S"][0], inp.W_out, inp.alpha_out, np.inf)
    assert S.sum() == 0 and np.array_equal(V, f["V_out"])


# ------------------------------------------------------------------ active set

def test_P3_compaction_brute_force():
    """P3: Definition 1 (strict) and the CSR order, enumerated element by element."""
    inp = _tiny()
    V = _fwd(inp)["V"][0]
    T, B, N = V.shape
    for b_th in (0.2, 0.05, 1.5, np.inf):
        row_ptr, col, g = oracle.active_csr(V, 1.0, b_th, 100.0)
        k = 0
        for r in range(T * B):
            assert row_ptr[r] == k
            for j in range(N):
                v = float(V[r // B, r % B, j])
                d = abs(np.float32(v) - np.float32(1.0))
                if d < np.float32(b_th):
                    assert col[k] == j
                    assert g[k] == pytest.approx(1.0 / (100.0 * abs(v - 1.0) + 1.0) ** 2, rel=1e-15)
                    k += 1
        assert row_ptr[-1] == k == col.size


def test_band_edges_and_nan():
    """Equality is inactive (strict '<'); NaN is never active nor spiking."""
    V = np.array([[[1.2, 0.8, 1.0, np.nan, 1.19999, 0.80001]]], F32)
    m = oracle.active_mask(V, 1.0, F32(0.2))
    d = np.abs(V - F32(1.0))
    assert list(m[0, 0]) == [bool(x < F32(0.2)) for x in d[0, 0]]
    assert not m[0, 0, 3]
    assert not (V[0, 0, 3] > F32(1.0))


# ------------------------------------------------------------------ backward pins

def _torch_grads(inp, b_th, beta=100.0, band=True):
    """fp64 autograd of the LIF network with a Heaviside forward and g*1[band] backward,
    the reset detached (Sec. 2.2). Returns loss, [dW_l], dW_out and the fp64 trajectory."""

    class Spike(torch.autograd.Function):
        @staticmethod
        def forward(ctx, v):
            ctx.save_for_backward(v)
            return (v > 1.0).to(v.dtype)

        @staticmethod
        def backward(ctx, gout):
            (v,) = ctx.saved_tensors
            d = (v - 1.0).abs()
            g = 1.0 / (beta * d + 1.0) ** 2
            if band:
                g = g * (d < b_th).to(v.dtype)
            return gout * g

    cfg = inp.cfg
    x = torch.tensor(inp.X != 0, dtype=torch.float64)
    T = x.shape[0]
    Ws = [torch.tensor(W, dtype=torch.float64, requires_grad=True) for W in inp.Ws]
    Wo = torch.tensor(inp.W_out, dtype=torch.float64, requires_grad=True)
    Vs, trs = [], []
    for W, a in zip(Ws, inp.alphas):
        a = float(a)
        v = torch.zeros(x.shape[1], W.shape[1], dtype=torch.float64)
        outs, vl = [], []
        tr = torch.zeros(x.shape[1], x.shape[2], dtype=torch.float64)
        tl = []
        for t in range(T):
            s = Spike.apply(v)
            outs.append(s)
            vl.append(v)
            tl.append(tr)
            if t < T - 1:
                v = a * v + x[t] @ W - s.detach()
                tr = a * tr + x[t]
        Vs.append(torch.stack(vl).detach().numpy())
        trs.append(torch.stack(tl).detach().numpy())
        x = torch.stack(outs)
    ao = float(inp.alpha_out)
    vo = torch.zeros(x.shape[1], Wo.shape[1], dtype=torch.float64)
    vol, tol = [], []
    tr = torch.zeros(x.shape[1], x.shape[2], dtype=torch.float64)
    for t in range(T):
        vol.append(vo)
        tol.append(tr)
        if t < T - 1:
            vo = ao * vo + x[t] @ Wo
            tr = ao * tr + x[t].detach()
    Vo = torch.stack(vol)
    if cfg.loss_mode == "max":
        idx = torch.argmax(Vo.detach(), dim=0, keepdim=True)  # first maximal index
        logits = Vo.gather(0, idx)[0]
    else:
        logits = Vo.sum(0)
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(inp.labels, dtype=torch.long))
    loss.backward()
    fwd = {"V": Vs, "trace": trs, "V_out": Vo.detach().numpy(), "trace_out": torch.stack(tol).detach().numpy()}
    return float(loss.detach()), [W.grad.numpy() for W in Ws], Wo.grad.numpy(), fwd


def _o2(inp, fwd, b_th, beta=100.0):
    return oracle.network_backward(fwd, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels,
                                   inp.cfg.loss_mode, 1.0, b_th, beta)


def _rel(a, b):
    return float(np.abs(a - b).max() / max(np.abs(b).max(), 1e-300))


@pytest.mark.parametrize("which", ["tiny", "tiny2", "latency8", "audio8"])
@pytest.mark.parametrize("b_th", [0.2, np.inf])
def test_P5_P6_matches_torch_autograd(which, b_th):
    """P5: O2 equals fp64 autograd of the same model; P6: B_th = inf is full surrogate BPTT."""
    if which == "tiny":
        inp = _tiny()
    elif which == "tiny2":
        inp = _two_layer_tiny()
    elif which == "latency8":
        inp = make_inputs(CONFIGS["latency"], range(8))
    else:
        inp = make_inputs(CONFIGS["audio"], range(8))
    loss, dWs, dWo, fwd64 = _torch_grads(inp, b_th, band=np.isfinite(b_th))
    ref = _o2(inp, fwd64, b_th)
    assert ref["loss"] == pytest.approx(loss, rel=1e-12)
    assert _rel(ref["dW_out"], dWo) <= 1e-10
    for l in range(len(dWs)):
        assert np.abs(dWs[l]).max() > 0
        assert _rel(ref["dW"][l], dWs[l]) <= 1e-10, l


def test_P6_zero_band_gives_no_gradient():
    """P6: B_th = 0 leaves no active neuron, so every LIF gradient is zero."""
    inp = _two_layer_tiny()
    f = _fwd(inp)
    r = _o2(inp, f, 0.0)
    for l in range(len(inp.Ws)):
        assert not r["mask"][l].any()
        assert np.all(r["dW"][l] == 0)
        row_ptr, col, _ = oracle.active_csr(f["V"][l], 1.0, 0.0, 100.0)
        assert row_ptr[-1] == 0 and col.size == 0
    assert np.abs(r["dW_out"]).max() > 0  # the readout gradient does not depend on the band


def test_P4_finite_differences_of_smoothed_model():
    """P4: central differences of the smoothed-surrogate model equal O2 (Eqs. (w_grad), (s_grad))."""
    for inp, b_th in ((_tiny(), 0.2), (_two_layer_tiny(), 0.3), (_tiny(), np.inf)):
        cfg = inp.cfg
        base = smooth.hard_forward64(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out)
        ref = _o2(inp, base, b_th)
        tstar = ref["readout"]["tstar"]
        args = (inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode, 1.0, b_th, 100.0, base, tstar)
        h = 1e-6
        L0 = smooth.smoothed_losses(inp.X, inp.Ws, inp.W_out, *args)[0]
        assert L0 == pytest.approx(ref["loss"], rel=1e-13)
        mats = list(inp.Ws) + [inp.W_out]
        grads = list(ref["dW"]) + [ref["dW_out"]]
        checked = total = 0
        for m, (W, gref) in enumerate(zip(mats, grads)):
            W = W.astype(np.float64)
            n = W.size
            fd = np.zeros(n)
            jump = np.zeros(n)
            for s in range(0, n, 128):
                idx = np.arange(s, min(n, s + 128))
                stack = np.repeat(W[None], 2 * idx.size, axis=0)
                for k, i in enumerate(idx):
                    stack[k].flat[i] += h
                    stack[idx.size + k].flat[i] -= h
                Ws_p = [w.astype(np.float64) for w in mats]
                Ws_p[m] = stack
                losses = smooth.smoothed_losses(inp.X, Ws_p[:-1], Ws_p[-1], *args)
                up, dn = losses[: idx.size], losses[idx.size:]
                fd[idx] = (up - dn) / (2 * h)
                fwd_d, bwd_d = (up - L0) / h, (L0 - dn) / h
                jump[idx] = np.abs(fwd_d - bwd_d)
            g = gref.ravel()
            scale = np.abs(g).max()
            # a band edge or arg-max switch inside [w-h, w+h] shows as a jump between the
            # one-sided slopes far above the curvature term h*L''
            ok = jump <= 1e-3 * scale
            err = np.abs(fd - g)[ok]
            assert err.max() <= 1e-6 * scale + 1e-9, (m, err.max(), scale)
            checked += ok.sum()
            total += n
        assert checked >= 0.95 * total


def _full_literal_and_events(inp, b_th):
    """Run O1 and O3 layer by layer with the same epsilons as O2 and return all three."""
    cfg = inp.cfg
    fwd = smooth.hard_forward64(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out)
    o2 = _o2(inp, fwd, b_th)
    L = len(inp.Ws)
    ro = o2["readout"]
    out_active_ro = ro["G"] != 0
    # readout layer (derivative factor 1)
    in_act = o2["mask"][L - 1]
    S_top = fwd["V"][L - 1] > 1.0  # hard spikes of the top LIF layer
    S_top = np.concatenate([np.zeros_like(S_top[:1]), S_top[1:]]) if False else (fwd["V"][L - 1] > 1.0)
    res = {"o2": o2, "o1": {}, "o3": {}}
    dW1, e1 = oracle.layer_backward_literal(ro["G"], np.ones_like(ro["G"]), S_top, inp.W_out, inp.alpha_out)
    res["o1"]["dW_out"], res["o1"]["eps_top"] = dW1, e1
    dW3, e3, c3 = oracle.layer_backward_events(ro["G"], out_active_ro, fwd["trace_out"], inp.W_out,
                                               inp.alpha_out, in_active=in_act)
    res["o3"]["dW_out"], res["o3"]["eps_top"], res["o3"]["counts_out"] = dW3, e3, c3
    for l in range(L - 1, -1, -1):
        G = o2["G"][l]
        x_in = inp.X if l == 0 else (fwd["V"][l - 1] > 1.0)
        g_trunc = o2["g"][l] * o2["mask"][l]
        dW1, e1 = oracle.layer_backward_literal(o2["eps"][l], g_trunc, x_in, inp.Ws[l], inp.alphas[l])
        res["o1"][l] = (dW1, e1)
        dW3, e3, c3 = oracle.layer_backward_events(G, o2["mask"][l], fwd["trace"][l], inp.Ws[l], inp.alphas[l],
                                                   in_active=o2["mask"][l - 1] if l > 0 else None)
        res["o3"][l] = (dW3, e3, c3)
    return res


@pytest.mark.parametrize("b_th", [0.3, np.inf])
def test_P7_event_driven_and_literal_equal_memoised(b_th):
    """P7 (Proposition 1: sparse = dense-truncated) and O1 (literal sums) = O2, fp64."""
    inp = _two_layer_tiny()
    r = _full_literal_and_events(inp, b_th)
    o2 = r["o2"]
    L = len(inp.Ws)
    assert _rel(r["o1"]["dW_out"], o2["dW_out"]) <= 1e-12
    assert _rel(r["o3"]["dW_out"], o2["dW_out"]) <= 1e-12
    top_mask = o2["mask"][L - 1]
    assert _rel(r["o1"]["eps_top"], o2["eps"][L - 1]) <= 1e-12
    assert _rel(r["o3"]["eps_top"][top_mask], o2["eps"][L - 1][top_mask]) <= 1e-12
    assert np.all(r["o3"]["eps_top"][~top_mask] == 0)
    for l in range(L):
        dW1, e1 = r["o1"][l]
        dW3, e3, _ = r["o3"][l]
        assert _rel(dW1, o2["dW"][l]) <= 1e-12
        assert _rel(dW3, o2["dW"][l]) <= 1e-12
        if l > 0:
            m = o2["mask"][l - 1]
            assert _rel(e3[m], o2["eps"][l - 1][m]) <= 1e-12
            assert _rel(e1, o2["eps"][l - 1]) <= 1e-12


def test_P8_appendix_c_schedule():
    """P8: the App. C example -- visited and written times, values, and the update bound."""
    with open(os.path.join(GOLDEN, "appc_schedule.json")) as f:
        gold = json.load(f)
    T = 10
    alpha = math.exp(-0.1)
    r = np.random.default_rng(7)
    G = {t: float(r.standard_normal()) for t in gold["t_j"]}
    vals, visited, n = oracle.skip_delta(G, gold["t_i"], alpha, T)
    assert visited == gold["computed_in_order"]
    assert sorted(vals) == sorted(gold["written"])
    for t in gold["not_required"]:
        assert t not in visited
    assert n <= len(gold["t_i"]) + len(gold["t_j"])
    for t, v in vals.items():
        ref = sum(alpha ** (k - t - 1) * G.get(k, 0.0) for k in range(t + 1, T))
        assert v == pytest.approx(ref, rel=1e-14)


def test_P9_single_pair_closed_forms():
    """P9: one input spike at t0 and one active output at t1 > t0."""
    T, t0, t1 = 16, 3, 9
    alpha = 0.9
    eps, w, gval = 0.37, -0.8, 0.25
    G = np.zeros((T, 1, 1))
    G[t1, 0, 0] = eps * gval
    trace = np.zeros((T, 1, 1))
    for t in range(t0 + 1, T):
        trace[t, 0, 0] = alpha ** (t - t0 - 1)
    W = np.array([[w]])
    dW, eps_in = oracle.layer_backward(G, W, trace, alpha)
    assert dW[0, 0] == pytest.approx(eps * gval * alpha ** (t1 - t0 - 1), rel=1e-14)
    for t in range(T):
        ref = w * alpha ** (t1 - t - 1) * eps * gval if t < t1 else 0.0
        assert eps_in[t, 0, 0] == pytest.approx(ref, rel=1e-14, abs=1e-300)


def test_P10_op_counts_and_linearity():
    """P10: Table 1 counts (nnz_out*N_in for dW, nnz_in*N_out for grad_in); linearity in eps."""
    inp = _two_layer_tiny()
    r = _full_literal_and_events(inp, 0.3)
    o2 = r["o2"]
    for l in range(len(inp.Ws)):
        c = r["o3"][l][2]
        n_in, n_out = inp.Ws[l].shape
        assert c["madds_w"] == int(o2["mask"][l].sum()) * n_in
        if l > 0:
            assert c["madds_s"] == int(o2["mask"][l - 1].sum()) * n_out
            assert c["delta_updates"] <= n_out * inp.cfg.T * inp.cfg.B
    f = _fwd(inp)
    rng = np.random.default_rng(3)
    W, tr, a = inp.Ws[1], f["trace"][1], inp.alphas[1]
    G1 = rng.standard_normal(o2["G"][1].shape) * o2["mask"][1]
    G2 = rng.standard_normal(o2["G"][1].shape) * o2["mask"][1]
    dA, eA = oracle.layer_backward(G1, W, tr, a)
    dB, eB = oracle.layer_backward(G2, W, tr, a)
    dC, eC = oracle.layer_backward(2.0 * G1 - 3.0 * G2, W, tr, a)
    assert _rel(dC, 2 * dA - 3 * dB) <= 1e-12 and _rel(eC, 2 * eA - 3 * eB) <= 1e-12


@pytest.mark.parametrize("mode", ["max", "sum"])
def test_P11_cross_entropy_gradient(mode):
    """P11: dL/da = (p - y)/B against torch's cross_entropy (App. E loss)."""
    rng = np.random.default_rng(11)
    V = rng.standard_normal((9, 5, 7)).astype(F32)
    y = rng.integers(0, 7, size=5)
    a, _ = oracle.readout_logits(V, mode)
    loss, d = oracle.cross_entropy(a, y)
    at = torch.tensor(a, requires_grad=True)
    lt = torch.nn.functional.cross_entropy(at, torch.tensor(y))
    lt.backward()
    assert loss == pytest.approx(float(lt), rel=1e-14)
    assert np.abs(d - at.grad.numpy()).max() <= 1e-15
    ro = oracle.readout_grad(V, y, mode)
    assert ro["row_ptr"][-1] == (5 * 7 if mode == "max" else 9 * 5 * 7)
    if mode == "max":
        t = np.argmax(V, axis=0)
        assert np.all(ro["G"][t, np.arange(5)[:, None], np.arange(7)[None]] == d)
