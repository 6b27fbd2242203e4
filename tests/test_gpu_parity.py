"""GPU path (through the C ABI) against the CPU oracle, element by element.

Bar: spikes, V, traces and active-set CSR bit-exact; gradients within 1e-4 of the oracle's
magnitude envelope, |x - r| <= 1e-4 * r_abs, where r_abs is the same contraction taken with
absolute values (so cancellation cannot hide or fake an error).
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
F64 = np.float64


def _oracle(inp, b_th):
    cfg = inp.cfg
    f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))
    args = (inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode, cfg.theta, b_th, cfg.beta)
    r = oracle.network_backward(f, *args)
    env = oracle.network_backward(f, *args, absolute=True)
    csrs = [oracle.active_csr(V, cfg.theta, b_th, cfg.beta) for V in f["V"]]
    return f, r, env, csrs


def _gpu(inp, b_th, dense=True, aux=None):
    net = pipeline.from_inputs(inp).forward()
    ro = net.readout(dense=True)
    csrs = net.compact(b_th)
    dWs, dW_out, epss = net.sparse_backward(csrs, ro, aux_stream=aux)
    out = {"net": net, "ro": ro, "csrs": csrs, "dW": dWs, "dW_out": dW_out, "eps": epss}
    if dense:
        ddW, ddW_out, deps = net.dense_backward(b_th, ro)
        out.update(ddW=ddW, ddW_out=ddW_out, deps=deps)
    torch.cuda.synchronize()
    return out


def _np(t):
    return t.detach().cpu().numpy()


def assert_bits(x, r, what):
    x, r = np.asarray(x), np.asarray(r)
    assert x.shape == r.shape, (what, x.shape, r.shape)
    if x.dtype == np.float32:
        same = x.view(np.uint32) == r.view(np.uint32)
    else:
        same = x == r
    if not same.all():
        k = np.argwhere(~same)[0]
        raise AssertionError(f"{what}: {int((~same).sum())} of {same.size} differ, first at {tuple(k)}: "
                             f"{x[tuple(k)]!r} vs {r[tuple(k)]!r}")


def assert_env(x, r, env, what, tol=TOL):
    x = np.asarray(x, F64)
    assert x.shape == np.shape(r), (what, x.shape, np.shape(r))
    if x.size == 0:
        return 0.0
    err = np.abs(x - r)
    bad = err > tol * env + 1e-30
    if bad.any():
        ratio = (err / np.maximum(env, 1e-300)).max()
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} outside 1e-4 envelope, worst err/env {ratio:.3g}")
    return float(err.max() / max(np.abs(r).max(), 1e-300))


def check_all(inp, b_th, g, ref, dense=True):
    f, r, env, ocsr = ref
    net = g["net"]
    # forward, bit for bit
    for l in range(net.L):
        assert_bits(_np(net.V[l]), f["V"][l], f"V[{l}]")
        assert_bits(_np(net.S[l]), f["S"][l], f"S[{l}]")
        assert_bits(_np(net.trace[l]), f["trace"][l], f"trace[{l}]")
    assert_bits(_np(net.V_out), f["V_out"], "V_out")
    assert_bits(_np(net.trace_out), f["trace_out"], "trace_out")
    # active sets, bit for bit; g to float32 rounding
    for l, (c, (rp, ci, gg)) in enumerate(zip(g["csrs"], ocsr)):
        nnz = c.nnz()
        assert nnz == rp[-1], (l, nnz, rp[-1])
        assert_bits(_np(c.row_ptr).astype(np.int64), rp, f"row_ptr[{l}]")
        assert_bits(_np(c.col_idx)[:nnz].astype(np.int64), ci, f"col_idx[{l}]")
        assert np.allclose(_np(c.g)[:nnz], gg, rtol=2e-6, atol=0), f"g[{l}]"
    # readout
    ro_csr, ro_eps, loss = g["ro"][0], g["ro"][1], g["ro"][2]
    rro = r["readout"]
    assert abs(float(loss.item()) - rro["loss"]) <= 1e-5 * max(1.0, abs(rro["loss"]))
    assert_bits(_np(ro_csr.row_ptr).astype(np.int64), rro["row_ptr"], "readout row_ptr")
    assert_bits(_np(ro_csr.col_idx).astype(np.int64), rro["col_idx"], "readout col_idx")
    # dL/da = (softmax(a) - y)/B at the read entries, against its envelope (p + y)/B
    n_ro = int(rro["row_ptr"][-1])
    env_ro = oracle.csr_values(rro["G_abs"], rro["row_ptr"], rro["col_idx"])
    assert_env(_np(ro_eps)[:n_ro], rro["eps"], env_ro, "readout eps")
    # sparse gradients
    assert_env(_np(g["dW_out"]), r["dW_out"], env["dW_out"], "dW_out")
    for l in range(net.L):
        assert_env(_np(g["dW"][l]), r["dW"][l], env["dW"][l], f"dW[{l}]")
        rp, ci, _ = ocsr[l]
        nnz = int(rp[-1])
        ref_e = oracle.csr_values(r["eps"][l], rp, ci)
        env_e = oracle.csr_values(env["eps"][l], rp, ci)
        assert_env(_np(g["eps"][l])[:nnz], ref_e, env_e, f"eps[{l}] at active entries")
    if dense:
        assert_env(_np(g["ddW_out"]), r["dW_out"], env["dW_out"], "dense dW_out")
        for l in range(net.L):
            assert_env(_np(g["ddW"][l]), r["dW"][l], env["dW"][l], f"dense dW[{l}]")
            assert_env(_np(g["deps"][l]), r["eps"][l], env["eps"][l], f"dense eps[{l}]")


_CACHE = {}


def _case(name, batch=None):
    key = (name, None if batch is None else tuple(batch))
    if key not in _CACHE:
        _CACHE[key] = make_inputs(CONFIGS[name], batch)
    return _CACHE[key]


def _ragged():
    cfg = Config("ragged", 201, T=37, B=3, sizes=(61, 37, 29, 5), tau_ratio_hidden=0.15, tau_ratio_out=0.1,
                 loss_mode="max", b_th=0.3, kind="bernoulli", rate=0.1)
    return make_inputs(cfg, sigmas=[0.25, 0.3, 1 / math.sqrt(29)])


def _ragged_sum():
    cfg = Config("ragged_sum", 202, T=9, B=5, sizes=(130, 70, 3), tau_ratio_hidden=0.2, tau_ratio_out=0.1,
                 loss_mode="sum", b_th=0.25, kind="bernoulli", rate=0.15)
    return make_inputs(cfg, sigmas=[0.2, 1 / math.sqrt(70)])


@pytest.mark.parametrize("name,batch,b_th", [
    ("tiny", None, 0.2),
    ("tiny", None, math.inf),
    ("latency", None, 0.2),
    ("audio", None, 0.2),
    ("event", None, 0.05),
    ("event", None, 0.2),
    ("event", None, 0.5),
    ("stress", list(range(8)), 0.02),
    ("stress", list(range(8)), 0.05),
    ("stress", list(range(8)), 0.1),
    ("stress", list(range(8)), 0.2),
    ("stress", list(range(8)), 0.35),
    ("stress", list(range(8)), 0.5),
    ("stress", list(range(8)), 0.8),
    ("stress", list(range(8)), 1.2),
    ("deep", list(range(32)), 0.2),
    ("deep", list(range(16)), 0.95),
    ("latency_train", list(range(32)), 0.2),
])
def test_parity_configs(name, batch, b_th):
    print(f"\n[case] {name} batch={'all' if batch is None else len(batch)} b_th={b_th}", flush=True)
    inp = _case(name, batch)
    ref = _oracle(inp, b_th)
    g = _gpu(inp, b_th, dense=True)
    check_all(inp, b_th, g, ref, dense=True)


@pytest.mark.parametrize("maker,b_th", [(_ragged, 0.3), (_ragged, math.inf), (_ragged_sum, 0.25)])
def test_parity_ragged_shapes(maker, b_th):
    """Sizes that are not multiples of 4, 64 or any tile (unaligned paths, partial tiles)."""
    inp = maker()
    print(f"\n[case] {inp.cfg.name} b_th={b_th}", flush=True)
    check_all(inp, b_th, _gpu(inp, b_th), _oracle(inp, b_th))


def test_zero_band_is_empty():
    inp = _case("tiny")
    ref = _oracle(inp, 0.0)
    g = _gpu(inp, 0.0)
    for c in g["csrs"]:
        assert c.nnz() == 0
    for l in range(len(inp.Ws)):
        assert np.all(_np(g["dW"][l]) == 0) and np.all(_np(g["ddW"][l]) == 0)
    check_all(inp, 0.0, g, ref)


def test_degenerate_time_and_batch():
    """T = 1 (no update at all), T = 2 and B = 1."""
    for T, B in ((1, 2), (2, 1), (3, 1)):
        cfg = Config(f"deg{T}{B}", 203, T=T, B=B, sizes=(16, 8, 3), tau_ratio_hidden=0.1, tau_ratio_out=0.1,
                     loss_mode="max", b_th=2.0, kind="bernoulli", rate=0.5)
        inp = make_inputs(cfg, sigmas=[0.6, 0.5])
        check_all(inp, 2.0, _gpu(inp, 2.0), _oracle(inp, 2.0))


def test_compaction_capacity_overflow_is_safe():
    """A capacity below nnz: the true nnz is reported and nothing past capacity is written."""
    inp = _case("latency", list(range(16)))
    net = pipeline.from_inputs(inp).forward()
    V = net.V[0]
    T, B, N = V.shape
    full = snn.active_compact(V, 1.0, 0.2, 100.0)
    nnz = full.nnz()
    cap = nnz // 2
    col = torch.full((cap + 64,), -7, dtype=torch.int32, device="cuda")
    gg = torch.full((cap + 64,), -7.0, dtype=torch.float32, device="cuda")
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device="cuda")
    nnz_dev = torch.empty(1, dtype=torch.int64, device="cuda")
    ws = snn.workspace(snn.snn_active_compact_workspace(T, B, N))
    snn.snn_active_compact(V, T, B, N, 1.0, 0.2, 100.0, row_ptr, col, gg, cap, nnz_dev, ws)
    torch.cuda.synchronize()
    assert int(nnz_dev.item()) == nnz
    assert torch.equal(col[:cap], full.col_idx[:cap]) and torch.equal(gg[:cap], full.g[:cap])
    assert bool((col[cap:] == -7).all()) and bool((gg[cap:] == -7.0).all())
    # the backward reads such a CSR safely (entries past capacity are ignored)
    eps = torch.ones(cap, dtype=torch.float32, device="cuda")
    trunc = snn.Csr(row_ptr, col[:cap].contiguous(), gg[:cap].contiguous(), nnz_dev, cap)
    dW, _ = snn.sparse_backward(net.Ws[0], net.trace[0], net.alphas[0], trunc, eps)
    torch.cuda.synchronize()
    assert torch.isfinite(dW).all()


@pytest.mark.parametrize("width", [200, 400, 600])
def test_dw_truncated_csr_each_path(width):
    """A CSR whose compaction overflowed its capacity (half of nnz): dW sums exactly the entries
    below the capacity, element by element against a float64 sum over them, on each dW path
    (200 outputs: CSR-direct; 400: slab records; 600: matrix cores)."""
    inp = _wide((width,), 40, 10, T=30, B=8)
    print(f"\n[case] truncated CSR dW, 40->{width}", flush=True)
    net = pipeline.from_inputs(inp).forward()
    V = net.V[0]
    T, B, N = V.shape
    full = snn.active_compact(V, 1.0, 0.2, 100.0)
    cap = full.nnz() // 2
    assert cap > 64
    col = torch.full((cap,), -7, dtype=torch.int32, device="cuda")
    gg = torch.full((cap,), -7.0, dtype=torch.float32, device="cuda")
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device="cuda")
    nnz_dev = torch.empty(1, dtype=torch.int64, device="cuda")
    ws = snn.workspace(snn.snn_active_compact_workspace(T, B, N))
    snn.snn_active_compact(V, T, B, N, 1.0, 0.2, 100.0, row_ptr, col, gg, cap, nnz_dev, ws)
    eps = torch.from_numpy(np.random.default_rng(width).standard_normal(cap).astype(np.float32)).cuda()
    trunc = snn.Csr(row_ptr, col, gg, nnz_dev, cap)
    dW = snn.sparse_dw(net.trace[0], trunc, eps, N)
    torch.cuda.synchronize()
    rp = np.minimum(_np(row_ptr).astype(np.int64), cap)
    rows = np.repeat(np.arange(T * B), np.diff(rp))
    G = (_np(eps) * _np(gg)).astype(np.float32).astype(np.float64)  # the kernels form G in float32
    tr = _np(net.trace[0]).reshape(T * B, -1).astype(np.float64)[rows]
    ref = np.zeros((tr.shape[1], N))
    mag = np.zeros((tr.shape[1], N))
    np.add.at(ref.T, _np(col), G[:, None] * tr)
    np.add.at(mag.T, _np(col), np.abs(G)[:, None] * np.abs(tr))
    x = _np(dW).astype(np.float64)
    bad = np.abs(x - ref) > 2e-6 * mag + 1e-30
    assert not bad.any(), f"{int(bad.sum())} elements differ from the sum over the entries below capacity"


def test_run_to_run_determinism():
    inp = _case("latency", list(range(32)))
    a = _gpu(inp, 0.2, dense=False)
    b = _gpu(inp, 0.2, dense=False)
    for l in range(len(inp.Ws)):
        assert torch.equal(a["net"].V[l], b["net"].V[l])
        assert torch.equal(a["csrs"][l].row_ptr, b["csrs"][l].row_ptr)
        n = a["csrs"][l].nnz()
        assert torch.equal(a["csrs"][l].col_idx[:n], b["csrs"][l].col_idx[:n])
        assert torch.equal(a["eps"][l][:n], b["eps"][l][:n])  # grad_in sums in a fixed order


def test_matrix_core_dw_is_reproducible():
    """The matrix-core dW (stress layers: 1024 outputs at about 2% active) accumulates each window's
    entries in a fixed order and sums the chunk partials in chunk order in float64: two runs give
    the same dW bit for bit. (The float64 LDS atomics of the other dW paths commit in any order;
    their float32 results differ only where a float64 sum falls within ~1e-16 of a rounding
    boundary.)"""
    inp = _case("stress", list(range(8)))
    a = _gpu(inp, 0.2, dense=False)
    b = _gpu(inp, 0.2, dense=False)
    for l in range(len(inp.Ws)):
        assert torch.equal(a["dW"][l], b["dW"][l]), f"dW[{l}]"


@pytest.mark.parametrize("name,batch,b_th", [("latency", list(range(32)), 0.2), ("stress", list(range(8)), 0.2),
                                             ("tiny", None, math.inf)])
def test_aux_stream_overlap(name, batch, b_th):
    """The spike gradient on a second stream beside dW: same results as on one stream, and
    work enqueued afterwards on the main stream sees both."""
    print(f"\n[case] aux stream {name} b_th={b_th}", flush=True)
    inp = _case(name, batch)
    aux = torch.cuda.Stream()
    a = _gpu(inp, b_th, dense=False, aux=aux)
    check_all(inp, b_th, a, _oracle(inp, b_th), dense=False)
    b = _gpu(inp, b_th, dense=False)
    for l in range(len(inp.Ws)):
        n = a["csrs"][l].nnz()
        assert torch.equal(a["eps"][l][:n], b["eps"][l][:n])  # fixed summation order on either stream


@pytest.mark.parametrize("maker,b_th", [(_ragged, 0.3), (lambda: _case("deep", list(range(6))), 0.2)])
def test_pipelined_schedule_matches_layerwise(maker, b_th):
    """With an auxiliary stream and two or more LIF layers, Network.sparse_backward runs the
    spike-gradient chain on the current stream and every dW on the auxiliary stream: the same
    dW, readout dW and spike gradients, bit for bit, as the layer-by-layer schedule."""
    inp = maker()
    print(f"\n[case] pipelined schedule {inp.cfg.name} b_th={b_th}", flush=True)
    a = _gpu(inp, b_th, dense=False, aux=torch.cuda.Stream())
    b = _gpu(inp, b_th, dense=False)
    assert torch.equal(a["dW_out"], b["dW_out"])
    for l in range(len(inp.Ws)):
        assert torch.equal(a["dW"][l], b["dW"][l]), f"dW[{l}]"
        n = a["csrs"][l].nnz()
        assert torch.equal(a["eps"][l][:n], b["eps"][l][:n]), f"eps[{l}]"
    check_all(inp, b_th, a, _oracle(inp, b_th), dense=False)


@pytest.mark.parametrize("name,batch,b_th", [("latency", list(range(16)), math.inf), ("stress", [0, 1], 0.8),
                                             ("ragged_sum", None, math.inf)])
def test_compaction_long_rows(name, batch, b_th):
    """Rows with more active entries than the count pass stages (every entry active, wide
    bands), on aligned and unaligned widths: CSR bit-exact against the oracle."""
    print(f"\n[case] long rows {name} b_th={b_th}", flush=True)
    inp = _ragged_sum() if name == "ragged_sum" else _case(name, batch)
    cfg = inp.cfg
    f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))
    net = pipeline.from_inputs(inp).forward()
    csrs = net.compact(b_th)
    torch.cuda.synchronize()
    longest = 0
    for l, V in enumerate(f["V"]):
        rp, ci, g = oracle.active_csr(V, cfg.theta, b_th, cfg.beta)
        c = csrs[l]
        n = c.nnz()
        assert n == int(rp[-1])
        assert_bits(_np(c.row_ptr).astype(np.int64), rp.astype(np.int64), f"row_ptr[{l}]")
        assert_bits(_np(c.col_idx[:n]).astype(np.int64), ci.astype(np.int64), f"col_idx[{l}]")
        assert_env(_np(c.g[:n]).astype(F64), g, np.abs(g), f"g[{l}]", tol=2e-6)
        longest = max(longest, int(np.diff(rp).max()))
    assert longest > 64  # the re-read path ran


@pytest.mark.parametrize("name,batch,b_th", [("latency", list(range(32)), 0.2), ("stress", list(range(8)), 0.2)])
def test_split_calls_match_combined(name, batch, b_th):
    """snn_sparse_dw and snn_sparse_grad_in, on two streams, give the combined call's results."""
    print(f"\n[case] split calls {name} b_th={b_th}", flush=True)
    inp = _case(name, batch)
    g = _gpu(inp, b_th, dense=False)
    net, csrs, ro = g["net"], g["csrs"], g["ro"]
    T, B, L = net.T, net.B, net.L
    aux = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    eps = g["eps"][L - 1]  # eps of the top hidden layer from the combined readout call
    for l in range(L - 1, -1, -1):
        W = net.Ws[l]
        if l > 0:
            aux.wait_stream(main)
            with torch.cuda.stream(aux):
                eps_in = snn.sparse_grad_in(W, net.alphas[l], T, B, csrs[l], eps, csrs[l - 1], share_cu=True,
                                            stream=aux)
        dW = snn.sparse_dw(net.trace[l], csrs[l], eps, W.shape[1])
        main.wait_stream(aux)
        torch.cuda.synchronize()
        ref_dW = g["dW"][l]
        assert torch.allclose(dW, ref_dW, rtol=1e-6, atol=1e-7 * float(ref_dW.abs().max())), f"dW[{l}]"
        if l > 0:
            n = csrs[l - 1].nnz()
            assert torch.equal(eps_in[:n], g["eps"][l - 1][:n]), f"eps[{l - 1}]"  # fixed order: bit-equal
            eps = eps_in


def _sample_entries(csr, T, B, b):
    """CSR positions, times and columns of sample b's entries (rows t*B + b), in CSR order."""
    rp = _np(csr.row_ptr).astype(np.int64)
    rows = np.arange(T) * B + b
    lo, hi = rp[rows], rp[rows + 1]
    idx = np.concatenate([np.arange(x, z) for x, z in zip(lo, hi)] + [np.zeros(0, np.int64)]).astype(np.int64)
    col = _np(csr.col_idx)[idx].astype(np.int64)
    return idx, np.repeat(np.arange(T), hi - lo), col, hi - lo


def _pin_dw(trace, csr, n_out, picks, what):
    """The dW call of the bench (structure-only layout, then the call with the gradients) on the
    full-size trace and CSR, with eps zero at every entry but the sampled ones, which carry eps
    from the oracle. Samples add up in dW, so the result is the sum of the oracle's per-sample dW,
    checked element by element within the summed envelope.
    picks: list of (idx, eps, dW, env) per sample: CSR positions and the oracle's eps there, and the
    oracle's dW and its envelope for that sample alone, all scaled to the batch mean."""
    T, B, n_in = trace.shape
    eps = torch.zeros(max(csr.capacity, 1), dtype=torch.float32, device=trace.device)
    idx = np.concatenate([p[0] for p in picks])
    val = np.concatenate([p[1] for p in picks]).astype(np.float32)
    eps[torch.from_numpy(idx).to(trace.device)] = torch.from_numpy(val).to(trace.device)
    ws = snn.workspace(snn.snn_sparse_dw_workspace(T, B, n_in, n_out, csr.capacity))
    snn.sparse_dw_layout((T, B, n_in), csr, n_out, ws)
    dW = snn.sparse_dw_prepared(trace, csr, eps, n_out, ws)
    ref = sum(p[2] for p in picks)
    env = sum(p[3] for p in picks)
    assert np.abs(ref).max() > 0, what
    assert_env(_np(dW), ref, env, what)


def _full_size_check(cfg, b_th, net, ro, csrs, eps_l, samples):
    """Per sampled b, against the oracle run on sample b alone (samples are independent in the
    forward, the compaction and the spike gradient; its loss gradient scaled by 1/B): V, spikes,
    traces, CSR rows and g bit-exact or to float32 rounding, eps of every layer within the
    envelope. Then every dW (the readout's too) pinned to the oracle through _pin_dw."""
    T, B, L = net.T, net.B, net.L
    picks = [[] for _ in range(L + 1)]
    for b in samples:
        sub = make_inputs(cfg, [b])
        f = oracle.network_forward(sub.X, sub.Ws, sub.W_out, sub.alphas, sub.alpha_out, np.float32(cfg.theta))
        args = (sub.Ws, sub.W_out, sub.alphas, sub.alpha_out, sub.labels, cfg.loss_mode, cfg.theta, b_th, cfg.beta)
        r = oracle.network_backward(f, *args)
        env = oracle.network_backward(f, *args, absolute=True)
        assert_bits(_np(net.V_out[:, b]), f["V_out"][:, 0], f"V_out b={b}")
        for l in range(L):
            assert_bits(_np(net.V[l][:, b]), f["V"][l][:, 0], f"V[{l}] b={b}")
            assert_bits(_np(net.S[l][:, b]), f["S"][l][:, 0], f"S[{l}] b={b}")
            assert_bits(_np(net.trace[l][:, b]), f["trace"][l][:, 0], f"trace[{l}] b={b}")
            idx, t_of, col, counts = _sample_entries(csrs[l], T, B, b)
            ref_rp, ref_ci, ref_g = oracle.active_csr(f["V"][l], cfg.theta, b_th, cfg.beta)
            assert_bits(counts, np.diff(ref_rp).astype(np.int64), f"row counts[{l}] b={b}")
            assert_bits(col, ref_ci.astype(np.int64), f"col_idx[{l}] b={b}")
            g = _np(csrs[l].g)[idx].astype(F64)
            assert np.allclose(g, ref_g, rtol=2e-6, atol=0), f"g[{l}] b={b}"
            ref_e = r["eps"][l][t_of, 0, col] / B
            assert_env(_np(eps_l[l])[idx].astype(F64), ref_e, env["eps"][l][t_of, 0, col] / B, f"eps[{l}] b={b}")
            picks[l].append((idx, ref_e, r["dW"][l] / B, env["dW"][l] / B))
        # the readout's read entries of sample b and dL/da there
        rro = r["readout"]
        idx, t_of, col, counts = _sample_entries(ro[0], T, B, b)
        assert_bits(counts, np.diff(rro["row_ptr"]).astype(np.int64), f"readout row counts b={b}")
        assert_bits(col, rro["col_idx"], f"readout col_idx b={b}")
        env_ro = oracle.csr_values(rro["G_abs"], rro["row_ptr"], rro["col_idx"])
        assert_env(_np(ro[1])[idx].astype(F64), rro["eps"] / B, env_ro / B, f"readout eps b={b}")
        picks[L].append((idx, rro["eps"] / B, r["dW_out"] / B, env["dW_out"] / B))
    for l in range(L):
        _pin_dw(net.trace[l], csrs[l], net.Ws[l].shape[1], picks[l], f"dW[{l}] of samples {samples}")
    _pin_dw(net.trace_out, ro[0], net.W_out.shape[1], picks[L], f"dW_out of samples {samples}")


def test_full_size_stress_sampled():
    """The stress workload at full size (T=500, B=256, 3 x 1024) in the bench's launch
    configuration: the spike-gradient chain on one stream, every layer's dW (structure-only layout
    first) on a second stream. Sampled b checked against the oracle run on sample b alone, and each
    dW call of the bench's plan pinned to the oracle's dW of the sampled samples."""
    cfg = CONFIGS["stress"]
    b_th = cfg.b_th
    print(f"\n[case] full-size stress b_th={b_th}", flush=True)
    inp = make_inputs(cfg)
    net = pipeline.from_inputs(inp).forward(b_th)
    ro = net.readout(dense=True)
    csrs = net.compact(b_th)
    dW, dW_out, eps_l = net.sparse_backward(csrs, ro, aux_stream=torch.cuda.Stream())
    ddW, _, _ = net.dense_backward(b_th, ro)
    torch.cuda.synchronize()
    assert (net.T, net.B) == (500, 256)
    _full_size_check(cfg, b_th, net, ro, csrs, eps_l, (0, 137, 255))
    # the full batch's dW against the dense matrix-core chain (itself pinned on the smaller cases)
    for l in range(net.L):
        x, y = _np(dW[l]).astype(F64), _np(ddW[l]).astype(F64)
        bad = np.abs(x - y) > 1e-4 * (np.abs(x) + np.abs(y)) + 1e-5 * np.abs(y).max()
        assert not bad.any(), f"dW[{l}]: {int(bad.sum())} elements differ from the dense path"


@pytest.mark.parametrize("name,b_th", [("latency", 0.2), ("event", 0.05), ("event", 0.5), ("audio", 0.2),
                                        ("deep", 0.2)])
def test_full_size_sampled(name, b_th):
    """Every other fully connected workload at its full size (B = 256, its own T and widths),
    through Network.sparse_backward with an auxiliary stream: the launch configuration of the
    bench (the pipelined schedule for the five-layer network, the readout's spike gradient beside
    its dW for one LIF layer). Sampled b checked against the oracle as for the stress workload,
    each dW call pinned to the oracle's dW of the sampled samples."""
    cfg = CONFIGS[name]
    print(f"\n[case] full-size {name} b_th={b_th}", flush=True)
    inp = make_inputs(cfg)
    net = pipeline.from_inputs(inp).forward(b_th)
    ro = net.readout(dense=True)
    csrs = net.compact(b_th)
    dW, dW_out, eps_l = net.sparse_backward(csrs, ro, aux_stream=torch.cuda.Stream())
    ddW, ddW_out, _ = net.dense_backward(b_th, ro)
    torch.cuda.synchronize()
    assert net.B == 256
    _full_size_check(cfg, b_th, net, ro, csrs, eps_l, (0, 101, 255))
    for x, y, what in [(dW[l], ddW[l], f"dW[{l}]") for l in range(net.L)] + [(dW_out, ddW_out, "dW_out")]:
        x, y = _np(x).astype(F64), _np(y).astype(F64)
        assert np.abs(y).max() > 0, what
        bad = np.abs(x - y) > 1e-4 * (np.abs(x) + np.abs(y)) + 1e-5 * np.abs(y).max()
        assert not bad.any(), f"{what}: {int(bad.sum())} elements differ from the dense path"


def _wide(hidden, n_in, n_ro, T=8, B=2):
    sizes = (n_in, *hidden, n_ro)
    cfg = Config(f"wide{'x'.join(map(str, hidden))}", 204, T=T, B=B, sizes=sizes, tau_ratio_hidden=0.1,
                 tau_ratio_out=0.1, loss_mode="max", b_th=0.4, kind="bernoulli", rate=0.3)
    rates = [0.3] + [0.2] * len(hidden)  # input rate, then about the hidden spike rate
    sig = [1.2 / math.sqrt(r * n) for r, n in zip(rates, sizes[:-2])] + [1 / math.sqrt(sizes[-2])]
    return make_inputs(cfg, sigmas=sig)


@pytest.mark.parametrize("hidden,n_in,n_ro", [((2000, 4096), 48, 3), ((1500,), 40, 1100), ((700, 3000), 33, 7)])
def test_parity_wide_layers(hidden, n_in, n_ro):
    """Wide layers: the forward's 8- and 16-group gathers, the spike gradient's 32- and 64-group
    walks (LIF to LIF with 4096 outputs, a 1100-class readout), unaligned widths."""
    inp = _wide(hidden, n_in, n_ro)
    print(f"\n[case] wide {n_in}->{hidden}->{n_ro}", flush=True)
    check_all(inp, 0.4, _gpu(inp, 0.4), _oracle(inp, 0.4))


@pytest.mark.parametrize("hidden,n_in,n_ro,T,B", [((600, 1000), 52, 520, 37, 3), ((1000,), 1024, 512, 300, 4)])
def test_parity_matrix_core_widths(hidden, n_in, n_ro, T, B):
    """Layers of 512..1024 outputs take the matrix-core dW: widths that leave wavefronts and lane
    groups without columns (520, 600, 1000), a partial 64-input tile (52 inputs), a partial window
    of rows (111 rows) and several windows and chunks (1200 rows)."""
    inp = _wide(hidden, n_in, n_ro, T=T, B=B)
    print(f"\n[case] matrix-core widths {n_in}->{hidden}->{n_ro} T={T} B={B}", flush=True)
    check_all(inp, 0.4, _gpu(inp, 0.4), _oracle(inp, 0.4))


@pytest.mark.parametrize("b_th", [0.6, 1.2])
def test_parity_csr_direct_dw_dense_rows(b_th):
    """The CSR-direct dW (layers of up to 300 outputs and 1024 inputs) with most neurons active:
    batches of 8 rows with more than 64 entries take their rest in pieces of 64 (second pass),
    two hidden layers so the spike gradient walk runs between them."""
    inp = _wide((200, 150), 40, 10, T=30, B=4)
    print(f"\n[case] CSR-direct dW dense rows 40->(200, 150)->10 b_th={b_th}", flush=True)
    g = _gpu(inp, b_th)
    per_row = [c.nnz() / (30 * 4) for c in g["csrs"]]
    assert max(per_row) > 8, per_row  # more than 64 entries per batch of 8 rows on average
    check_all(inp, b_th, g, _oracle(inp, b_th))


@pytest.mark.parametrize("hidden,n_ro", [((24, 31), 3), ((31,), 8), ((24,), 9), ((40, 17), 16), ((32,), 32),
                                          ((29,), 33)])
def test_parity_narrow_outputs(hidden, n_ro):
    """Layers of at most 32 outputs (hidden LIF layers and readouts) take the spike gradient's
    narrow path (dense G, per-output delta, one lane per input-active entry); 33 outputs and up
    take the walk. Widths at and beside each register-block boundary (8, 16, 32)."""
    inp = _wide(hidden, 37, n_ro, T=41, B=3)
    print(f"\n[case] narrow 37->{hidden}->{n_ro}", flush=True)
    check_all(inp, 0.4, _gpu(inp, 0.4), _oracle(inp, 0.4))


@pytest.mark.parametrize("name,b_th", [("tiny", 0.2), ("tiny", math.inf), ("latency", 0.2), ("event", 0.05),
                                       ("audio", 0.2), ("ragged", 0.3), ("ragged_sum", 0.25), ("wide", 0.4),
                                       ("stress8", 0.02), ("stress8", 0.8)])
def test_fused_active_bits(name, b_th):
    """Active sets marked by the forward, compacted from the bitsets: CSR bit-exact against the
    oracle and g bit-equal to the compaction that reads V; V and spikes unchanged."""
    inp = {"ragged": _ragged, "ragged_sum": _ragged_sum, "wide": lambda: _wide((700, 3000), 33, 7),
           "stress8": lambda: _case("stress", list(range(8)))}.get(name, lambda: _case(name))()
    cfg = inp.cfg
    print(f"\n[case] fused bits {cfg.name} b_th={b_th}", flush=True)
    f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))
    net = pipeline.from_inputs(inp).forward(b_th)
    fused = net.compact(b_th)
    plain = [snn.active_compact(net.V[l], net.theta, b_th, net.beta) for l in range(net.L)]
    torch.cuda.synchronize()
    for l in range(net.L):
        assert_bits(_np(net.V[l]), f["V"][l], f"V[{l}]")
        rp, ci, g = oracle.active_csr(f["V"][l], cfg.theta, b_th, cfg.beta)
        n = fused[l].nnz()
        assert n == int(rp[-1])
        assert_bits(_np(fused[l].row_ptr).astype(np.int64), rp.astype(np.int64), f"row_ptr[{l}]")
        assert_bits(_np(fused[l].col_idx[:n]).astype(np.int64), ci.astype(np.int64), f"col_idx[{l}]")
        assert torch.equal(fused[l].g[:n], plain[l].g[:n]), f"g[{l}]"


def test_fused_bits_capacity_overflow():
    inp = _case("latency", list(range(16)))
    net = pipeline.from_inputs(inp).forward(0.2)
    V, bits = net.V[0], net.bits[0]
    T, B, N = V.shape
    full = snn.active_compact_bits(bits, V, 1.0, 100.0)
    nnz = full.nnz()
    cap = nnz // 3
    col = torch.full((cap + 64,), -7, dtype=torch.int32, device="cuda")
    gg = torch.full((cap + 64,), -7.0, dtype=torch.float32, device="cuda")
    row_ptr = torch.empty(T * B + 1, dtype=torch.int32, device="cuda")
    nnz_dev = torch.empty(1, dtype=torch.int64, device="cuda")
    ws = snn.workspace(snn.snn_active_compact_bits_workspace(T, B, N))
    snn.snn_active_compact_bits(bits, V, T, B, N, 1.0, 100.0, row_ptr, col, gg, cap, nnz_dev, ws)
    torch.cuda.synchronize()
    assert int(nnz_dev.item()) == nnz
    assert torch.equal(col[:cap], full.col_idx[:cap]) and torch.equal(gg[:cap], full.g[:cap])
    assert bool((col[cap:] == -7).all()) and bool((gg[cap:] == -7.0).all())


def test_graph_replays_match_eager():
    """Readout loss, compaction and the sparse backward chain captured once as HIP graphs and
    replayed three times; between replays the weights change and the forward runs eagerly. Each
    replay equals an eager run on the same state: CSR, loss and spike gradients bit for bit, dW
    to float64-accumulation order (its LDS adds are unordered)."""
    inp = _case("deep", list(range(16)))
    net = pipeline.from_inputs(inp).allocate()
    b_th = 0.2
    net.forward(b_th)
    caps = [2 * c.nnz() + 4096 for c in net.compact(b_th)]
    g_ro = pipeline.Graphed(lambda: net.readout())
    g_cmp = pipeline.Graphed(lambda: net.compact(b_th, caps))
    g_bwd = pipeline.Graphed(lambda: net.sparse_backward(g_cmp.out, g_ro.out))
    gen = torch.Generator(device="cuda").manual_seed(7)
    for rep in range(3):
        print(f"\n[case] graph replay {rep}", flush=True)
        with torch.no_grad():
            for W in net.Ws:
                W.mul_(1.0 + 0.02 * torch.randn(W.shape, device=W.device, generator=gen))
        net.forward(b_th)
        ro_g = g_ro()
        cs_g = g_cmp()
        dW_g, dWo_g, eps_g = g_bwd()
        torch.cuda.synchronize()
        snap = {"loss": ro_g[2].clone(), "rp": [c.row_ptr.clone() for c in cs_g],
                "col": [c.col_idx.clone() for c in cs_g], "nnz": [c.nnz() for c in cs_g],
                "dW": [d.clone() for d in dW_g], "dWo": dWo_g.clone(), "eps": [e.clone() for e in eps_g]}
        ro_e = net.readout()
        cs_e = net.compact(b_th, caps)
        dW_e, dWo_e, eps_e = net.sparse_backward(cs_e, ro_e)
        torch.cuda.synchronize()
        assert torch.equal(snap["loss"], ro_e[2])
        for l in range(net.L):
            n = cs_e[l].nnz()
            assert n == snap["nnz"][l] and n <= caps[l]
            assert torch.equal(snap["rp"][l], cs_e[l].row_ptr)
            assert torch.equal(snap["col"][l][:n], cs_e[l].col_idx[:n])
            assert torch.equal(snap["eps"][l][:n], eps_e[l][:n])
            d = (snap["dW"][l] - dW_e[l]).abs().max().item()
            assert d <= 1e-6 * dW_e[l].abs().max().item() + 1e-30, (l, d)
        assert (snap["dWo"] - dWo_e).abs().max().item() <= 1e-6 * dWo_e.abs().max().item() + 1e-30


@pytest.mark.parametrize("maker", [_ragged, lambda: _case("stress", [0, 1, 2])])
def test_dw_layout_then_prepared_equals_one_call(maker):
    """snn_sparse_dw_layout (structure only, run before eps exists) followed by
    snn_sparse_dw_prepared gives snn_sparse_dw's dW bit for bit, for narrow (<= 32 outputs) and
    slab layers alike; the layout can be reused with a second eps."""
    inp = maker()
    print(f"\n[case] dW layout + prepared {inp.cfg.name}", flush=True)
    g = _gpu(inp, 0.3, dense=False)
    net, csrs = g["net"], g["csrs"]
    T, B = net.T, net.B
    for l in range(net.L):
        n_in, n_out = net.Ws[l].shape
        ws = snn.workspace(snn.snn_sparse_dw_workspace(T, B, n_in, n_out, csrs[l].capacity))
        snn.sparse_dw_layout((T, B, n_in), csrs[l], n_out, ws)
        for eps in (g["eps"][l], 2.0 * g["eps"][l]):
            got = snn.sparse_dw_prepared(net.trace[l], csrs[l], eps, n_out, ws)
            ref = snn.sparse_dw(net.trace[l], csrs[l], eps, n_out)
            torch.cuda.synchronize()
            assert torch.equal(got, ref), f"dW[{l}]"
