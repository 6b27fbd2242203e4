"""Benchmark of the sparse spiking BPTT path on one MI355X.

One step = the whole path over one batch of the workload: LIF forward of every layer and
the readout, readout loss, active-set compaction of every LIF layer, the sparse backward
chain, and the dense matrix-core baseline chain. HIP events time each part; the headline is
the sparse backward (compaction + sparse backward of every LIF layer; the readout's own
backward and the loss are outside both chains, as are the forward passes).

Schedule of the LIF layers' backward: with two or more LIF layers the spike gradients form a chain
on the main stream, each followed by its layer's dW call; the dW calls' structure-only layouts and
the compactions of the layers below the top two run on a side stream from the start of the chain
(`--dw-streams N` puts the dW calls on streams beside the chain instead). With one LIF layer
everything runs on one stream. HIP events bracket every dW call and spike gradient; dW is the
dominant kernel and the roofline object is computed from its calls' durations.

Prints ONE JSON line. `value` = active neuron-steps per second of the sparse backward
(sum over LIF layers of the active entries, divided by its time); the dense time and the
speedup are in the same line. Inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--workload stress] [--b-th 0.2] [--no-cpu]
    python bench.py --sweep            one JSON line per B_th of the workload's sweep
    python bench.py --copy-probe MB    device copies of known size (counter calibration)
    python bench.py --train            training runs, sparse vs full-surrogate gradient (App. E, H)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F32_TFLOPS = 157.3  # dense fp32 matrix-core peak
CPU_TARGET_S = 10.0  # seconds of oracle work timed for the CPU baseline
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_sparse_dw_stress.json")
CSRC = os.path.join(ROOT, "paper_2105_08810_amd", "csrc")


DW_SOURCES = ("common.h", "runtime.hip", "sparse_backward.hip", "dw_mfma.hip")  # the dW call's kernels


def csrc_digest() -> str:
    """Digest of the dW call's sources: a traffic record is used only while they are unchanged."""
    h = hashlib.sha256()
    for name in DW_SOURCES:
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def algorithmic(T, B, n_in, n_out, nnz_out, r_out, nnz_in=None):
    """Gathered bytes and flops of one layer's sparse backward, split into (dW, spike gradient).

    dW: trace rows with at least one active output, the output CSR (index, g, eps), the row
    pointers and the dW write; 2 flops per multiply-add. Spike gradient: W once, the input
    CSR index, the eps_in write and its row pointers; 2 flops per multiply-add plus the delta
    recurrence.
    """
    TB = T * B
    by_dw = 4 * n_in * r_out + 12 * nnz_out + 4 * (TB + 1) + 4 * n_in * n_out
    fl_dw = 2 * nnz_out * n_in
    by_gi = fl_gi = 0
    if nnz_in is not None:
        by_gi = 4 * n_in * n_out + 8 * nnz_in + 4 * (TB + 1)
        fl_gi = 2 * nnz_in * n_out + 2 * TB * n_out
    return by_dw, fl_dw, by_gi, fl_gi


def forward_bytes(T, B, sizes, bits):
    """Bytes the forward moves once each: per LIF layer the input spikes (u8) and W read, V (f32),
    spikes (u8) and the input trace (f32) written, and the active bitset when the forward marks it;
    the readout (infinite threshold) the same without the bitset."""
    TB, total = T * B, 0
    for l in range(len(sizes) - 1):
        n_in, n_out = sizes[l], sizes[l + 1]
        total += TB * n_in + 4 * n_in * n_out + 4 * TB * n_out + TB * n_out + 4 * TB * n_in
        if bits and l < len(sizes) - 2:
            total += T * ((B * n_out + 63) // 64) * 8
    return total


def cpu_baseline(cfg, b_th, n_samples):
    """The oracle's backward (compaction + dense-truncated BPTT, fp64 BLAS) on a batch subset."""
    import oracle
    from synth import make_inputs
    try:
        from threadpoolctl import threadpool_info
        blas = [(d.get("internal_api"), d.get("num_threads")) for d in threadpool_info()]
    except Exception:  # pragma: no cover
        blas = []
    n_samples = min(n_samples, cfg.B, 2 if cfg.conv else cfg.B)
    if cfg.conv:
        from oracle import conv as oconv
        from synth.inputs import make_conv_inputs
        inp = make_conv_inputs(cfg, list(range(n_samples)))
        f = oconv.conv_network_forward(inp.X, inp.Wc, inp.W_out, cfg.alpha, cfg.alpha_out, cfg.theta)

        def unit():
            rp, _, _ = oracle.active_csr(f["V"].reshape(cfg.T, n_samples, -1), cfg.theta, b_th, cfg.beta)
            oconv.conv_network_backward(f, inp.Wc, inp.W_out, cfg.alpha_out, inp.labels, cfg.loss_mode, cfg.theta,
                                        b_th, cfg.beta)
            return int(rp[-1])
    else:
        inp = make_inputs(cfg, list(range(n_samples)))
        f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))

        def unit():
            n = 0
            for V in f["V"]:
                rp, _, _ = oracle.active_csr(V, cfg.theta, b_th, cfg.beta)
                n += int(rp[-1])
            oracle.network_backward(f, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode,
                                    cfg.theta, b_th, cfg.beta)
            return n
    # the timed unit is repeated until about CPU_TARGET_S of work has been measured
    reps, dt, nnz = 0, 0.0, 0
    while reps == 0 or (dt < CPU_TARGET_S and reps < 200):
        t0 = time.perf_counter()
        nnz += unit()
        dt += time.perf_counter() - t0
        reps += 1
    threads = max([n for _, n in blas if n] or [1])
    return {"value": nnz / dt, "unit": "active neuron-steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{cfg.name} workload, batch samples 0..{n_samples - 1} of {cfg.B}, B_th={b_th}: "
                      f"compaction + fp64 backward of all layers, {reps} runs, {dt:.2f} s, {nnz} active entries",
            "host_cpus": len(os.sched_getaffinity(0)), "blas": blas}


def copy_probe(mb):
    """Device-to-device copies of a known size (for scaling the HBM byte counters)."""
    import torch
    n = mb * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4, "copies": 5}))


def _grad_difference(a, b):
    """App. H statistics of a sparse gradient a against the full-surrogate gradient b (host arrays):
    max |a - b| / max |b|, the largest per-weight relative difference among weights with
    |b| >= 1% of max |b|, the relative Frobenius norm of a - b, and the cosine of a and b."""
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    d = np.abs(a - b)
    sc = np.abs(b).max()
    big = np.abs(b) >= 0.01 * sc
    nb, na = np.linalg.norm(b), np.linalg.norm(a)
    return {"max_abs_over_max": float(d.max() / sc) if sc > 0 else 0.0,
            "max_rel_big": float((d[big] / np.abs(b[big])).max()) if big.any() else 0.0,
            "frobenius_rel": float(np.linalg.norm(a - b) / nb) if nb > 0 else 0.0,
            "cosine": float(a @ b / (na * nb)) if na > 0 and nb > 0 else 0.0}


def train_experiment(args):
    """Training runs (App. E): the sparse gradient (the workload's B_th, or each band of
    --train-bth) and full-surrogate BPTT (dense chain, B_th = inf) from the same initial weights
    over the same batches, with the activity penalties and Adam. Prints one JSON line with the loss and test-accuracy
    trajectories, the active fraction per layer, the time per training step of both, and the
    App. H gradient-difference statistics at the initial and at the final sparse weights.
    The step time is host wall time from the call to the end of the step's work (it includes
    the host reads of each layer's active-set size); the phases are HIP events."""
    import torch
    from paper_2105_08810_amd import pipeline, snn
    from synth import CONFIGS, make_inputs
    from synth.inputs import make_labels, make_spikes
    snn.lib()
    cfg = CONFIGS[args.train_workload]
    B, T, P = cfg.B, cfg.T, args.train_batches
    dev = torch.device("cuda:0")
    t0 = time.time()
    shape = (T, B, *cfg.conv[:3]) if cfg.conv else (T, B, cfg.sizes[0])  # conv: [T, B, H, W, C]

    def spikes(idx):
        return torch.from_numpy(make_spikes(cfg, idx).reshape(shape)).to(dev)

    Xs = [spikes(range(k * B, (k + 1) * B)) for k in range(P)]
    Ys = [torch.from_numpy(make_labels(cfg, range(k * B, (k + 1) * B))).to(dev) for k in range(P)]
    held = 10 ** 6  # held-out samples come from far above the training indices
    Xt = [spikes(range(held + k * B, held + (k + 1) * B)) for k in range(2)]
    Yt = [torch.from_numpy(make_labels(cfg, range(held + k * B, held + (k + 1) * B))).to(dev) for k in range(2)]
    gen_s = time.time() - t0
    if cfg.conv:
        from synth.inputs import make_conv_inputs
        cin = make_conv_inputs(cfg, range(B))

        def new_net():
            return pipeline.ConvNetwork(
                X=torch.from_numpy(cin.X).to(dev), Wc=torch.from_numpy(cin.Wc).to(dev),
                W_out=torch.from_numpy(cin.W_out).to(dev), alpha=float(cfg.alpha), alpha_out=float(cfg.alpha_out),
                labels=torch.from_numpy(cin.labels).to(dev), loss_mode=0 if cfg.loss_mode == "max" else 1,
                theta=float(cfg.theta), beta=float(cfg.beta)).allocate()
    else:
        inp0 = make_inputs(cfg, range(B))

        def new_net():
            return pipeline.from_inputs(inp0, "cuda:0").allocate()
    pen = pipeline.Penalty(nu_up=args.nu_up)
    aux = torch.cuda.Stream()

    def grads_at(net, k, b_th):
        """Gradients at the net's weights on batch k: sparse with band b_th, or full surrogate (inf)."""
        net.X, net.labels = Xs[k], Ys[k]
        opt = pipeline.Adam(net.params(), lr=0.0)
        out = net.train_step(opt, b_th, pen, sparse=math.isfinite(b_th), aux_stream=aux)
        return [g.cpu().numpy() for g in out["grads"]]

    def diff(net, b_th):
        gs, gf = grads_at(net, 0, b_th), grads_at(net, 0, math.inf)
        return [_grad_difference(a, b) for a, b in zip(gs, gf)]

    def accuracy(net):
        hits = 0
        for X, Y in zip(Xt, Yt):
            net.X = X
            net.forward()
            logits = net.V_out.max(dim=0).values if net.loss_mode == 0 else net.V_out.sum(dim=0)
            hits += int((logits.argmax(dim=1).to(torch.int32) == Y).sum().item())
        return hits / (len(Xt) * B)

    bths = [float(x) for x in args.train_bth.split(",")] if args.train_bth else [cfg.b_th]
    result = {"mode": "train", "workload": cfg.name, "description": cfg.description, "steps": args.train_steps,
              "batches_in_training_set": P, "lr": args.lr, "betas": [0.9, 0.999],
              "penalty": vars(pen), "b_th_sparse": bths, "data": "synthetic", "input_gen_s": gen_s}
    runs = [(f"sparse_bth_{b:g}", True, b) for b in bths] + [("full_surrogate", False, math.inf)]
    nets = {}
    for name, sparse, b_th in runs:
        net = new_net()
        if name == runs[0][0]:
            result["grad_difference_init"] = diff(net, b_th)
        opt = pipeline.Adam(net.params(), lr=args.lr)
        acc0 = accuracy(net)
        ce, pn, nnz, ms, acc, phases = [], [], [], [], [acc0], []
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        for step in range(args.train_steps):
            k = step % P
            net.X, net.labels = Xs[k], Ys[k]
            w0 = time.perf_counter()
            out = net.train_step(opt, b_th, pen, sparse=sparse, aux_stream=aux, events=ev)
            ev[5].synchronize()
            ms.append((time.perf_counter() - w0) * 1e3)
            phases.append([ev[i].elapsed_time(ev[i + 1]) for i in range(5)])
            ce.append(float(out["ce"].item()))
            pn.append(float(out["penalty"].item()))
            if sparse:
                nnz.append([int(c.item()) for c in out["nnz"]])
            if k == P - 1:
                acc.append(accuracy(net))
        nets[name] = (net, b_th)
        ph = np.median(np.array(phases), axis=0)
        r = {"b_th": b_th if math.isfinite(b_th) else "inf", "ce": ce, "penalty": pn,
             "test_accuracy_per_epoch": acc, "train_step_ms_median": float(np.median(ms)),
             "train_step_ms_iqr": [float(np.percentile(ms, 25)), float(np.percentile(ms, 75))],
             "phase_ms_median": dict(zip(("forward", "loss_and_penalties", "compaction", "backward", "adam"),
                                         map(float, ph))),
             "initial_test_accuracy": acc0}
        if sparse:
            sizes = cfg.sizes[1:-1]
            r["active_fraction_per_layer"] = [[n / (T * B * sizes[l]) for l, n in enumerate(row)] for row in nnz]
        result[name] = r
    first_net, first_bth = nets[runs[0][0]]
    result["grad_difference_end_sparse_weights"] = diff(first_net, first_bth)
    result["train_step_speedup"] = result["full_surrogate"]["train_step_ms_median"] / result[runs[0][0]][
        "train_step_ms_median"]
    print(json.dumps(result), flush=True)


class ConvRunner:
    """The convolutional workload: conv LIF layer, 2x2 spike pooling, readout. Sparse chain =
    compaction of the conv layer (and the pooled entries) + the readout's backward at the pooled
    entries + routing to the conv entries + the sparse filter gradient; dense chain = the dense
    readout backward + dense routing + the dense filter gradient."""

    def __init__(self, cfg, args):
        import torch
        from paper_2105_08810_amd import pipeline, snn
        from synth.inputs import make_conv_inputs
        self.torch, self.snn = torch, snn
        self.cfg, self.args = cfg, args
        inp = make_conv_inputs(cfg)
        dev = torch.device("cuda:0")
        self.net = pipeline.ConvNetwork(
            X=torch.from_numpy(inp.X).to(dev), Wc=torch.from_numpy(inp.Wc).to(dev),
            W_out=torch.from_numpy(inp.W_out).to(dev), alpha=float(cfg.alpha), alpha_out=float(cfg.alpha_out),
            labels=torch.from_numpy(inp.labels).to(dev), loss_mode=0 if cfg.loss_mode == "max" else 1,
            theta=float(cfg.theta), beta=float(cfg.beta)).allocate()
        T, B, H, W, C, F = self.net.dims
        self.ws_sp = snn.workspace(snn.snn_conv_sparse_dw_workspace(T, B, H, W, C, F))
        self.ws_dn = snn.workspace(snn.snn_conv_dense_dw_workspace(T, B, H, W, C, F))
        # --conv-csr: the chain through the conv layer's CSR, its compaction on a second stream
        # beside the pooled entries' compaction and the readout's backward (--serial: one stream)
        self.aux = None if args.serial else torch.cuda.Stream()  # default priority

    def prepare(self, b_th):
        self.b_th = b_th
        self.net.forward(b_th)
        cs = self.net.compact(b_th)
        self.caps = [c.capacity for c in cs]
        self.conv_nnz = cs[0].nnz()  # the conv layer's active entries (counted before the timed steps)

    def measured_memory(self):
        """Eq. (memory_saved) from the allocator: the peak bytes allocated while each chain's backward
        runs (from the readout's gradient at its read entries to the filter gradient), above what
        was allocated before it, plus the per-entry record of the forward that the chain reads: V
        [T, B, H W F] (float32) for the dense chain, the conv and pooled active bitsets for the
        sparse one. Returns [(sparse, dense, saved %)] for the conv layer."""
        torch, net = self.torch, self.net
        T, B, H, W, C, F = net.dims
        dev = net.X.device
        ro = net.readout(dense=True)
        TB, N = T * B, H * W * F

        def peak(fn):
            torch.cuda.synchronize()
            base = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            keep = fn()
            torch.cuda.synchronize()
            used = torch.cuda.max_memory_allocated(dev) - base
            del keep
            return used

        if self.args.conv_csr:
            sparse = peak(lambda: net.compact_and_backward(self.b_th, ro, self.caps))
        else:
            sparse = peak(lambda: net.pooled_backward(self.b_th, ro, self.caps[1]))
        sparse += net.bits.numel() * net.bits.element_size() + net.pbits.numel() * net.pbits.element_size()
        dense = peak(lambda: net.dense_backward(self.b_th, ro)) + 4 * TB * N
        return [(sparse, dense, 100.0 * (dense - sparse) / dense)]

    def events(self):
        mk = lambda: self.torch.cuda.Event(enable_timing=True)  # noqa: E731
        return {k: mk() for k in ("fwd0", "fwd1", "cmp0", "conv0", "conv1", "pool0", "pool1", "bw1", "dn0", "dn1")}

    def step(self, ev, dense=True):
        net = self.net
        with_dense = dense and not self.args.no_dense
        ev["fwd0"].record()
        net.forward(self.b_th)
        ev["fwd1"].record()
        ro = net.readout(dense=with_dense)
        ev["cmp0"].record()  # the sparse chain: compaction to dWc
        if self.args.conv_csr:
            cs, _ = net.compact_and_backward(self.b_th, ro, self.caps, ws=self.ws_sp, aux_stream=self.aux, events=ev)
        else:
            pool, _ = net.pooled_backward(self.b_th, ro, self.caps[1], ws=self.ws_sp, events=ev)
            cs = [None, pool]
        ev["bw1"].record()
        if with_dense:
            ev["dn0"].record()
            net.dense_backward(self.b_th, ro, ws=self.ws_dn)
            ev["dn1"].record()
        return cs

    def run(self, steps, warmup, dense=True):
        torch = self.torch
        for _ in range(warmup):
            self.step(self.events(), dense)
        torch.cuda.synchronize()
        evs = [self.events() for _ in range(steps)]
        t0 = time.perf_counter()
        for k in range(steps):
            cs = self.step(evs[k], dense)
        torch.cuda.synchronize()
        return evs, cs, time.perf_counter() - t0

    def summarize(self, evs, cs, wall, dense=True):
        med = lambda a: float(np.median(a))  # noqa: E731
        span = lambda a, b: np.array([e[a].elapsed_time(e[b]) for e in evs])  # noqa: E731
        T, B, H, W, C, F = self.net.dims
        csr_chain = self.args.conv_csr
        # the compaction kernels' own spans
        t_cmp = (span("conv0", "conv1") if csr_chain else 0.0) + span("pool0", "pool1")
        t_sparse = span("cmp0", "bw1")
        with_dense = dense and not self.args.no_dense
        nnz = cs[0].nnz() if csr_chain else self.conv_nnz
        nnz_pool = cs[1].nnz()
        N = H * W * F
        TB = T * B
        Np = self.net.Np
        bits = TB * ((B * N + 63) // 64) // B * 8
        # gathered bytes: pooled bits (conv bitset and picks read, pooled bitset written) and CSR,
        # the readout's backward at the pooled entries; then either the filter gradient from the
        # pooled entries (their picks, V, eps and 3x3xC input patches) or the conv layer's
        # compaction (bitset, CSR, g, V at active entries), routing and the filter gradient from it
        sparse_bytes = bits + TB * Np + TB * Np // 8 + 4 * (TB + 1) + 4 * nnz_pool + 2 * TB * Np
        # the pooled active set, each byte once: conv bitset and picks read, pooled bitset written
        # (route) and read back, row pointers and columns written (compaction)
        pool_bytes = bits + TB * Np + TB * Np // 8 + 4 * (TB + 1) + 4 * nnz_pool
        t_pool = span("pool0", "pool1")
        pool_gbs = pool_bytes / (med(t_pool) * 1e-3) / 1e9
        if csr_chain:
            sparse_bytes += bits + 12 * nnz + 4 * (TB + 1) + 4 * nnz_pool + 12 * nnz
        else:
            sparse_bytes += nnz_pool * (4 + 4 + 1 + 4 + 36 * C)
        out = {
            "metric": "sparse backward ms/batch + active neuron-steps/s, speedup vs dense BPTT",
            "value": nnz / (med(t_sparse) * 1e-3),
            "unit": "active neuron-steps/s",
            "n_gpus": 1, "steps": len(evs), "warmup": self.args.warmup, "ms_per_step": med(span("fwd0", "dn1" if with_dense else "bw1")),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
            "config": {"workload": f"{self.cfg.name}: {self.cfg.description}; B_th={self.b_th}", "T": T, "B": B,
                       "H": H, "W": W, "C": C, "F": F, "b_th": self.b_th},
            "sparse_backward_ms": med(t_sparse),
            "sparse_backward_ms_iqr": [float(np.percentile(t_sparse, 25)), float(np.percentile(t_sparse, 75))],
            "compaction_ms": med(t_cmp),
            "sparse_chain": ("conv-layer CSR (its compaction beside the readout's backward), routing, filter gradient"
                             if csr_chain else "pooled entries only: readout backward, filter gradient of the picked "
                             "conv neurons (no conv-layer compaction)"),
            "dense_backward_ms": med(span("dn0", "dn1")) if with_dense else None,
            "forward_ms": med(span("fwd0", "fwd1")),
            "active_fraction": [nnz / (TB * N)],
            "pooled_active_entries": nnz_pool,
            "nnz": [nnz],
            "sparse_backward_gathered_bytes": sparse_bytes,
            "sparse_backward_hbm_frac": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "roofline": {
                "bound": "hbm", "achieved": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9 / HBM_PEAK_GBS, "traffic": None,
                "kernel": "the whole sparse chain (one launch sequence per step): " + (
                    "conv-layer compaction, routing, filter gradient" if csr_chain else
                    "pooled active set, the readout's backward at the pooled entries, the filter gradient and "
                    "its reduction"),
                "algorithmic_bytes_per_launch": sparse_bytes, "launch_ms": med(t_sparse),
                "pooled_active_set": {"kernel": "snn_pool_route_bits + snn_active_compact_bits",
                                      "algorithmic_bytes": pool_bytes, "ms": med(t_pool), "achieved_gbs": pool_gbs,
                                      "frac": pool_gbs / HBM_PEAK_GBS},
            },
            "value_pooled_entries": nnz_pool / (med(t_sparse) * 1e-3),
            "memory_sparse_dense_bytes_analytic": [(12 * nnz + 4 * (TB + 1) if csr_chain else 0) + 8 * nnz_pool +
                                                   4 * (TB + 1), 4 * TB * N + 4 * TB * self.net.Np],
            "wall_s_timed": wall,
        }
        m = out["memory_sparse_dense_bytes_analytic"]
        out["memory_saved_pct_analytic"] = [100.0 * (m[1] - m[0]) / m[1]]
        if with_dense:
            out["speedup_vs_dense"] = out["dense_backward_ms"] / out["sparse_backward_ms"]
            out["overall_speedup_fwd_plus_bwd"] = (out["forward_ms"] + out["dense_backward_ms"]) / (
                out["forward_ms"] + out["sparse_backward_ms"])
        return out


class Runner:
    """Device state of one workload and the timed step."""

    def __init__(self, cfg, args):
        import torch
        from paper_2105_08810_amd import pipeline, snn
        from synth import make_inputs
        self.torch, self.snn, self.pipeline = torch, snn, pipeline
        self.cfg, self.args = cfg, args
        self.graphs = {}
        inp = make_inputs(cfg)
        self.net = net = pipeline.from_inputs(inp, "cuda:0").allocate()
        self.T, self.B, self.L = net.T, net.B, net.L
        self.sizes = list(cfg.sizes)
        net.forward()
        self.main = torch.cuda.current_stream()
        self.aux = self.main if args.serial else torch.cuda.Stream()  # default priority
        T, B, L, sizes = self.T, self.B, self.L, self.sizes
        n_extra = max(1, args.dw_streams - 1)  # extra dW streams the pipelined schedule may take
        self.dw_extra = [] if args.serial else [torch.cuda.Stream() for _ in range(n_extra)]
        self.n_dw = 1
        self.ws_dn = None if args.no_dense else snn.workspace(
            max(snn.snn_dense_backward_workspace(T, B, sizes[l], sizes[l + 1]) for l in range(L + 1)))
        self.ws_gi = snn.workspace(max(snn.snn_sparse_grad_in_workspace(T, B, sizes[l + 1]) for l in range(L + 1)))
        self.ro = net.readout(dense=not args.no_dense)
        self.dW_out = torch.empty_like(net.W_out)
        # dW calls on their own stream beside the spike-gradient chain when there is a chain to
        # overlap (two or more LIF layers); layer by layer otherwise
        sched = args.schedule
        self.pipelined = sched == "pipelined" or (sched == "auto" and L >= 2)
        self.ws_ro = snn.workspace(snn.snn_sparse_backward_workspace(T, B, sizes[L], sizes[L + 1],
                                                                     self.ro[0].capacity))

    def prepare(self, b_th):
        """Size compaction outputs and workspaces for one band (the first compaction counts)."""
        snn, T, B, L, sizes = self.snn, self.T, self.B, self.L, self.sizes
        self.b_th = b_th
        self.graphs = {}  # captured for this band on first use
        self.net.forward(None if self.args.unfused else b_th)
        csrs = self.net.compact(b_th)
        self.caps = [c.capacity for c in csrs]
        # dW streams of the pipelined schedule: one by default, the dW calls in line with the spike
        # gradients. Beside them on a second stream each spike gradient shares the GPU with a dW
        # call: deep 0.48-0.55 ms against 0.44-0.45 in line (its walks 0.08 against 0.035 ms),
        # stress 2.83 against 2.47 ms (the walk is gather-bound, the dW call LDS- and
        # matrix-core-bound, yet together they slow each other more than they overlap).
        self.n_dw = min(1 + len(self.dw_extra), self.args.dw_streams or 1)
        K = self.args.recompute
        if K:  # trace recompute: dW from the input spikes and checkpoints of the trace every K steps
            self.ws_dw = [snn.workspace(snn.snn_sparse_dw_spikes_workspace(T, B, sizes[l], sizes[l + 1],
                                                                           self.caps[l], K)) for l in range(L)]
            nck = snn.snn_trace_checkpoint_count(T, K)
            self.ck = [self.torch.empty((nck, B, sizes[l]), dtype=self.torch.float32, device="cuda:0")
                       for l in range(L)]
        else:
            self.ws_dw = [snn.workspace(snn.snn_sparse_dw_workspace(T, B, sizes[l], sizes[l + 1], self.caps[l]))
                          for l in range(L)]
        self.dW = [self.torch.empty((sizes[l], sizes[l + 1]), dtype=self.torch.float32, device="cuda:0")
                   for l in range(L)]
        self.eps = [self.torch.empty(self.caps[l], dtype=self.torch.float32, device="cuda:0") for l in range(L)]
        # the walk keeps to two blocks per CU when the dW beside it is the longer job
        self.share = [False] + [3.0 * self.caps[l] * sizes[l] >= 2.0 * self.caps[l - 1] * sizes[l + 1]
                                for l in range(1, L)]

    def region(self, key, stream, fn):
        """Run fn's library calls on stream: directly, or (with --graph) as a HIP graph captured on
        first use and replayed after that. Returns what fn returns (static under a graph)."""
        torch = self.torch
        if not self.args.graph:
            with torch.cuda.stream(stream):
                return fn()
        if key not in self.graphs:
            self.graphs[key] = self.pipeline.Graphed(fn, stream)
        return self.graphs[key](stream)

    def step(self, ev, dense=True):
        """One pass of the whole path. ev: dict of event lists, recorded in order (outside any graph)."""
        snn, net = self.snn, self.net
        T, B, L = self.T, self.B, self.L
        main, aux = self.main, self.aux
        R = self.region
        E = lambda k: ev[k]  # noqa: E731
        with_dense = dense and not self.args.no_dense
        E("fwd0").record(main)
        R("fwd", main, lambda: net.forward(None if self.args.unfused else self.b_th))
        E("fwd1").record(main)
        K = self.args.recompute
        if K:
            def checkpoints():
                for l in range(L):
                    snn.trace_checkpoints(net.X if l == 0 else net.S[l - 1], net.alphas[l], K, ck=self.ck[l])
            R("ck", main, checkpoints)
            E("ck1").record(main)
        r = R("readout" + ("d" if with_dense else ""), main, lambda: net.readout(dense=with_dense))
        use_aux = not (self.args.serial or self.args.graph)
        E("cmp0").record(main)
        self.deferred = self.pipelined and use_aux and L >= 3 and not K and self.n_dw == 1
        if self.deferred:
            # one stream of dW calls and spike gradients: the top two layers' active sets now (the
            # readout's and the top layer's spike gradients need them), the others on the side
            # stream beside the chain, each before the spike gradient that needs it (stress: 2.51
            # -> 2.48 ms). With the dW calls on a second stream the chain's waits cost more than the
            # overlap saves (deep: 0.475 -> 0.515 ms), so there they are all compacted first.
            top = R("compact", main, lambda: [net.compact_layer(l, self.b_th, self._cap(l)) for l in (L - 2, L - 1)])
            cs = [None] * (L - 2) + top
        else:
            cs = R("compact", main, lambda: net.compact(self.b_th, self.caps))
        E("cmp1").record(main)
        if self.pipelined and use_aux:
            self._layers_pipelined(ev, r, cs, K)
        else:
            self._layers_layerwise(ev, r, cs, K, use_aux)
        if with_dense:
            def dense_chain():
                _, e = snn.dense_backward_ref(net.W_out, net.trace_out, net.V_out, r[3], net.alpha_out, math.inf,
                                              math.inf, net.beta, grad_in=True, ws=self.ws_dn)
                return e
            e_top = R("dense_ro", main, dense_chain)

            def dense_layers():
                e = e_top
                for l in range(L - 1, -1, -1):
                    _, e = snn.dense_backward_ref(net.Ws[l], net.trace[l], net.V[l], e, net.alphas[l], net.theta,
                                                  self.b_th, net.beta, grad_in=l > 0, ws=self.ws_dn)
                return e
            E("dn0").record(main)
            R("dense", main, dense_layers)
            E("dn1").record(main)
        return cs

    def _cap(self, l):
        return self.caps[l] if self.caps else None

    def _dw_call(self, l, eps, K, prepared=False):
        snn, net = self.snn, self.net
        if prepared:
            return lambda: snn.sparse_dw_prepared(net.trace[l], self.cs[l], eps, net.Ws[l].shape[1], self.ws_dw[l],
                                                  dW=self.dW[l])
        if K:
            return lambda: snn.sparse_dw_spikes(net.X if l == 0 else net.S[l - 1], self.ck[l], K, net.alphas[l],
                                                self.cs[l], eps, net.Ws[l].shape[1], ws=self.ws_dw[l], dW=self.dW[l])
        return lambda: snn.sparse_dw(net.trace[l], self.cs[l], eps, net.Ws[l].shape[1], ws=self.ws_dw[l],
                                     dW=self.dW[l])

    def _gi_call(self, l, eps, share):
        snn, net = self.snn, self.net
        return lambda: snn.sparse_grad_in(net.Ws[l], net.alphas[l], self.T, self.B, self.cs[l], eps, self.cs[l - 1],
                                          share_cu=share, ws=self.ws_gi, eps_in=self.eps[l - 1])

    def _layers_pipelined(self, ev, r, cs, K):
        """The spike gradients form a chain (each layer's needs the one above); a layer's dW needs only
        its own eps, and its structure-only layout only the active sets. The layouts (and the lower
        layers' compactions) run on a side stream from the start of the chain. By default the dW
        calls run on main between the spike gradients; with --dw-streams N > 1 each dW runs on a dW
        stream as soon as its eps is there, beside the chain."""
        snn, net, main, side, R = self.snn, self.net, self.main, self.aux, self.region
        T, B, L = self.T, self.B, self.L
        self.cs = cs
        inline = self.n_dw == 1  # dW calls in line with the spike gradients
        # the dW streams: the extra ones first, so that the top layer's dW waits only for its own
        # layout, not behind every layout queued on the side stream
        dw_streams = [main] if inline else (self.dw_extra + [side])[:self.n_dw]
        eps = R("ro_gi", main, lambda: snn.sparse_grad_in(net.W_out, net.alpha_out, T, B, r[0], r[1], cs[L - 1],
                                                         share_cu=not inline, ws=self.ws_gi, eps_in=self.eps[L - 1]))
        ev["ro1"].record(main)
        # From here on every kernel is LIF-layer work (timed); the layouts start here too, so that
        # none of them hides behind the readout's spike gradient.
        side.wait_stream(main)
        laid = [None] * L
        made = [None] * L  # active sets compacted on the side stream (inside the measured chain)
        if not K:
            for l in range(L - 1, -1, -1):  # top layer first: its dW comes first
                if cs[l] is None:
                    cs[l] = R(f"cmp{l}", side, lambda l=l: net.compact_layer(l, self.b_th, self._cap(l)))
                    made[l] = self.torch.cuda.Event()
                    made[l].record(side)
                R(f"lay{l}", side, lambda l=l: snn.sparse_dw_layout((T, B, self.sizes[l]), cs[l], self.sizes[l + 1],
                                                                   self.ws_dw[l]))
                laid[l] = self.torch.cuda.Event()
                laid[l].record(side)
        if inline:
            # One stream: each layer's spike gradient first (it needs no layout, so the chain starts
            # while the layouts run on the side stream), then its dW. One event per boundary: a timing
            # event is a barrier packet that costs the stream several microseconds.
            mark = ev["ro1"]  # recorded at the current boundary of main
            for l in range(L - 1, -1, -1):
                i = L - 1 - l
                ev["lay0"][i] = mark
                if l > 0:
                    ev["gi0"][i] = mark
                    if made[l - 1] is not None:
                        main.wait_event(made[l - 1])
                    R(f"gi{l}", main, self._gi_call(l, eps, False))
                    ev["gi1"][i].record(main)
                    mark = ev["gi1"][i]
                ev["dw0"][i] = mark
                if laid[l] is not None:
                    main.wait_event(laid[l])
                R(f"dw{l}", main, self._dw_call(l, eps, K, prepared=not K))
                ev["dw1"][i].record(main)
                mark = ev["lay1"][i] = ev["dw1"][i]
                if l > 0:
                    eps = self.eps[l - 1]
            main.wait_stream(side)
            ev["bw1"].record(main)
            R("ro_dw", main, lambda: snn.sparse_dw(net.trace_out, r[0], r[1], net.W_out.shape[1], ws=self.ws_ro,
                                                  dW=self.dW_out))
            return
        mark = ev["ro1"]  # timing events only where a span needs one (each is a barrier packet)
        for l in range(L - 1, -1, -1):
            i = L - 1 - l  # top layer first
            sd = dw_streams[i % len(dw_streams)]
            if sd is not main:
                sd.wait_stream(main)  # eps of layer l is ready
            if laid[l] is not None:
                sd.wait_event(laid[l])
            ev["dw0"][i].record(sd)
            ev["lay0"][i] = ev["dw0"][i]
            R(f"dw{l}", sd, self._dw_call(l, eps, K, prepared=not K))
            ev["dw1"][i].record(sd)
            ev["lay1"][i] = ev["dw1"][i]
            if l > 0:
                ev["gi0"][i] = mark
                if made[l - 1] is not None:
                    main.wait_event(made[l - 1])
                R(f"gi{l}", main, self._gi_call(l, eps, not inline))
                ev["gi1"][i].record(main)
                mark = ev["gi1"][i]
                eps = self.eps[l - 1]
        for sd in [side] + dw_streams:
            if sd is not main:
                main.wait_stream(sd)
        ev["bw1"].record(main)  # end of the LIF layers' backward
        # the readout's dW, outside the measured chain (as the readout's loss and forward are)
        R("ro_dw", main, lambda: snn.sparse_dw(net.trace_out, r[0], r[1], net.W_out.shape[1], ws=self.ws_ro,
                                              dW=self.dW_out))

    def _layers_layerwise(self, ev, r, cs, K, use_aux):
        """Layer by layer: the readout's backward, then each LIF layer's spike gradient (on the second
        stream) beside its dW, the next layer starting when both are done. With one LIF layer there is
        no spike gradient to overlap: everything runs on the main stream (the readout's own spike
        gradient too, as the join of a second stream costs more than the overlap saves), and a timing
        event is recorded only where one is needed (each is a barrier packet of several
        microseconds on the stream)."""
        snn, net, main, aux, R = self.snn, self.net, self.main, self.aux, self.region
        L = self.L
        self.cs = cs
        fork = use_aux and L > 1 and aux is not main
        eps = R("ro_bwd", main, lambda: snn.sparse_backward(net.W_out, net.trace_out, net.alpha_out, r[0], r[1],
                                                             inp=cs[L - 1], ws=self.ws_ro,
                                                             aux_stream=aux if fork else None)[1])
        ev["ro1"].record(main)
        mark = ev["ro1"]  # the event at the current boundary of main
        for l in range(L - 1, -1, -1):
            i = L - 1 - l
            ev["lay0"][i] = mark
            if l > 0:
                if fork:
                    aux.wait_stream(main)
                    ev["gi0"][i].record(aux)
                    R(f"gi{l}", aux, self._gi_call(l, eps, self.share[l]))
                    ev["gi1"][i].record(aux)
                else:
                    ev["gi0"][i] = mark
                    R(f"gi{l}", main, self._gi_call(l, eps, False))
                    ev["gi1"][i].record(main)
                    mark = ev["gi1"][i]
            ev["dw0"][i] = mark
            R(f"dw{l}", main, self._dw_call(l, eps, K))
            ev["dw1"][i].record(main)
            mark = ev["dw1"][i]
            if l > 0:
                if fork:
                    main.wait_stream(aux)
                    ev["lay1"][i].record(main)
                    mark = ev["lay1"][i]
                eps = self.eps[l - 1]
            ev["lay1"][i] = mark
        ev["bw1"] = mark

    def memory(self, nnz):
        """Per LIF layer, the analytic figure: bytes each backward chain allocates beyond the shared
        forward state (CSR, eps, dW and workspaces against the dense gradient buffers), and the
        memory saved, 100 (dense - sparse) / dense."""
        snn, T, B, L, sizes = self.snn, self.T, self.B, self.L, self.sizes
        TB = T * B
        out = []
        for l in range(L):
            n_in, n_out = sizes[l], sizes[l + 1]
            sparse = 4 * (TB + 1) + 12 * nnz[l] + 4 * n_in * n_out  # CSR (index, g), eps, dW
            sparse += snn.snn_sparse_dw_workspace(T, B, n_in, n_out, nnz[l])
            dense = 4 * TB * n_out + 4 * n_in * n_out + snn.snn_dense_backward_workspace(T, B, n_in, n_out)
            if l > 0:
                sparse += 4 * nnz[l - 1] + snn.snn_sparse_grad_in_workspace(T, B, n_out)
                dense += 4 * TB * n_in
            out.append((sparse, dense, 100.0 * (dense - sparse) / dense))
        return out

    def measured_memory(self):
        """Eq. (memory_saved) from the allocator, per LIF layer: the peak bytes allocated while the
        layer's backward step runs in each chain, above what was allocated before it (the forward
        state and the incoming spike gradient). The sparse step makes its active set (CSR, g), then
        allocates dW, the spike gradient at the active entries of the layer below and its
        workspaces; the dense step allocates dW, the dense spike gradient and its workspace. Each
        step also reads one per-entry record the forward kept for it, counted too: V [T, B, N]
        (float32) for the dense step, the active bitset (one bit per entry) for the sparse one
        (V itself when the compaction reads V). Returns [(sparse, dense, saved %)] per layer."""
        torch, snn, net = self.torch, self.snn, self.net
        T, B, L, TB = self.T, self.B, self.L, self.T * self.B
        b_th = self.b_th
        dev = net.X.device
        fused = not self.args.unfused
        out = []

        def peak(fn):
            torch.cuda.synchronize()
            base = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            keep = fn()
            torch.cuda.synchronize()
            used = torch.cuda.max_memory_allocated(dev) - base
            del keep
            return used

        for l in range(L):
            n_in, n_out = net.Ws[l].shape
            below = net.compact_layer(l - 1, b_th, self.caps[l - 1]) if l > 0 else None  # made by that layer's step
            eps_s = torch.zeros(self.caps[l], dtype=torch.float32, device=dev)
            sparse = peak(lambda: (lambda c: snn.sparse_backward(net.Ws[l], net.trace[l], net.alphas[l], c, eps_s,
                                                                   inp=below) + (c,))(
                net.compact_layer(l, b_th, self.caps[l])))
            sparse += T * ((B * n_out + 63) // 64) * 8 if fused else 4 * TB * n_out
            del eps_s, below
            eps_d = torch.zeros((T, B, n_out), dtype=torch.float32, device=dev)
            dense = peak(lambda: snn.dense_backward_ref(net.Ws[l], net.trace[l], net.V[l], eps_d, net.alphas[l],
                                                        net.theta, b_th, net.beta, grad_in=l > 0))
            dense += 4 * TB * n_out
            del eps_d
            out.append((sparse, dense, 100.0 * (dense - sparse) / dense))
        return out

    def events(self):
        mk = lambda: self.torch.cuda.Event(enable_timing=True)  # noqa: E731
        ev = {k: mk() for k in ("fwd0", "fwd1", "ck1", "cmp0", "cmp1", "ro1", "bw1", "dn0", "dn1")}
        for k in ("lay0", "lay1", "gi0", "gi1", "dw0", "dw1"):
            ev[k] = [mk() for _ in range(self.L)]
        return ev

    def run(self, steps, warmup, dense=True):
        torch = self.torch
        for _ in range(warmup):
            self.step(self.events(), dense)
        torch.cuda.synchronize()
        evs = [self.events() for _ in range(steps)]
        t0 = time.perf_counter()
        for k in range(steps):
            cs = self.step(evs[k], dense)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return evs, cs, wall

    def summarize(self, evs, cs, wall, dense=True):
        T, B, L, sizes = self.T, self.B, self.L, self.sizes
        cfg = self.cfg

        def span(a, b, i=None):
            if i is None:
                return np.array([e[a].elapsed_time(e[b]) for e in evs])
            return np.array([e[a][i].elapsed_time(e[b][i]) for e in evs])

        med = lambda a: float(np.median(a))  # noqa: E731
        t_fwd = span("fwd0", "fwd1")
        t_layers = [np.array([e["lay0"][i].elapsed_time(e["lay1"][i]) for e in evs]) for i in range(L)]
        t_dw = [span("dw0", "dw1", i) for i in range(L)]
        t_gi = [np.array([e["gi0"][i].elapsed_time(e["gi1"][i]) for e in evs]) for i in range(L - 1)]
        t_cmp = span("cmp0", "cmp1")
        t_sparse = t_cmp + span("ro1", "bw1")  # compaction + the LIF layers (readout excluded, as in the dense chain)
        t_step = np.array([e["fwd0"].elapsed_time(e["dn1"] if dense and not self.args.no_dense else e["lay1"][L - 1])
                           for e in evs])

        nnz = [c.nnz() for c in cs]
        r_out = [int((c.row_ptr[1:] > c.row_ptr[:-1]).sum().item()) for c in cs]
        per = [algorithmic(T, B, sizes[l], sizes[l + 1], nnz[l], r_out[l], nnz[l - 1] if l > 0 else None)
               for l in range(L)]
        dw_ms = [med(t) for t in reversed(t_dw)]  # layer order
        dw_flops = sum(p[1] for p in per)
        dw_bytes = sum(p[0] for p in per)
        dw_s = sum(dw_ms) * 1e-3
        dw_gbs = dw_bytes / dw_s / 1e9  # algorithmic bytes per launch / average launch time
        value = sum(nnz) / (med(t_sparse) * 1e-3)
        mem = self.memory(nnz)
        # whole sparse backward on its gathered bytes (compaction: V read... here the bitset, the
        # CSR and g written; layers: dW and spike-gradient bytes), against the HBM peak
        cmp_bytes = sum(4 * (T * B + 1) + 8 * nnz[l] + (4 * T * B * sizes[l + 1] if self.args.unfused else
                                                          T * ((B * sizes[l + 1] + 63) // 64) * 8 + 4 * nnz[l])
                        for l in range(L))
        sparse_bytes = cmp_bytes + sum(p[0] + p[2] for p in per)
        # dense chain: dW GEMM of every LIF layer and the spike-gradient GEMM of all but the first
        dense_flops = sum(2 * T * B * sizes[l] * sizes[l + 1] * (2 if l > 0 else 1) for l in range(L))
        fwd_bytes = forward_bytes(T, B, sizes, not self.args.unfused)
        use_aux = not (self.args.serial or self.args.graph)
        traffic = None
        if os.path.exists(TRAFFIC_FILE):
            with open(TRAFFIC_FILE) as f:
                tr = json.load(f)
            if tr.get("csrc_digest") == csrc_digest() and tr.get("workload") == f"{cfg.name}:{self.b_th}":
                traffic = tr.get("hbm_bytes_per_launch")
        out = {
            "metric": "sparse backward ms/batch + active neuron-steps/s, speedup vs dense BPTT",
            "value": value,
            "unit": "active neuron-steps/s",
            "n_gpus": 1,
            "steps": len(evs),
            "warmup": self.args.warmup,
            "ms_per_step": med(t_step),
            "higher_is_better": True,
            "scaling": "weak",
            "vs_baseline": None,
            "dtype": "f32",
            "data": "synthetic",
            "config": {"workload": f"{cfg.name}: {cfg.description}; B_th={self.b_th}", "T": T, "B": B,
                       "sizes": sizes, "b_th": self.b_th, "alpha": float(cfg.alpha), "beta": cfg.beta,
                       "compaction": ("from V" if self.args.unfused else "from the forward's active bitsets")
                       + ("; compaction_ms covers the top two layers, the others run on a side stream inside the "
                          "chain's span" if getattr(self, "deferred", False) else "")},
            "sparse_backward_ms": med(t_sparse),
            "sparse_backward_ms_iqr": [float(np.percentile(t_sparse, 25)), float(np.percentile(t_sparse, 75))],
            "compaction_ms": med(t_cmp),
            "sparse_layer_ms": [med(t) for t in reversed(t_layers)],
            "sparse_dw_ms": dw_ms,
            "sparse_grad_in_ms": [med(t) for t in reversed(t_gi)],
            "dense_backward_ms": med(span("dn0", "dn1")) if dense and not self.args.no_dense else None,
            "forward_ms": med(t_fwd),
            "forward_hbm_frac": fwd_bytes / (med(t_fwd) * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "forward_bytes": fwd_bytes,
            "active_fraction": [n / (T * B * sizes[l + 1]) for l, n in enumerate(nnz)],
            "memory_saved_pct_analytic": [m[2] for m in mem],
            "backward_bytes_sparse_dense_analytic": [[m[0], m[1]] for m in mem],
            "nnz": nnz,
            "roofline": {
                "bound": "hbm", "achieved": dw_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": dw_gbs / HBM_PEAK_GBS, "traffic": traffic,
                "kernel": ("snn_sparse_dw_prepared (mdw_gate + mdw_kernel + mdw_reduce) of each LIF layer; the "
                           "structure-only layouts run on a side stream inside the timed chain" if self.pipelined
                           and use_aux
                           else "snn_sparse_dw (layout + mdw_gate + mdw_kernel + mdw_reduce) of each LIF layer"),
                "algorithmic_bytes_per_launch": dw_bytes / L, "algorithmic_flops_per_launch": dw_flops / L,
                "launches": L, "launch_ms": dw_ms,
                "alu_view": {"resource": "fp32 matrix cores (v_mfma_f32_4x4x1f32)", "achieved": dw_flops / dw_s / 1e12,
                             "peak": MFMA_F32_TFLOPS, "unit": "TFLOP/s",
                             "frac": dw_flops / dw_s / 1e12 / MFMA_F32_TFLOPS},
                "chain_hbm_frac": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9 / HBM_PEAK_GBS,
            },
            "sparse_backward_gathered_bytes": sparse_bytes,
            "sparse_backward_hbm_gbs": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9,
            "sparse_backward_hbm_frac": sparse_bytes / (med(t_sparse) * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "wall_s_timed": wall,
        }
        K = self.args.recompute
        if K:
            nck = self.snn.snn_trace_checkpoint_count(T, K)
            out["trace_recompute"] = {
                "K": K, "checkpoint_ms": med(span("fwd1", "ck1")),
                "stored_trace_bytes": sum(4 * T * B * sizes[l] for l in range(L)),
                "checkpoint_bytes": sum(4 * nck * B * sizes[l] for l in range(L)),
                "dw_kernel": "dw_slab_spikes_kernel (trace rebuilt in registers from the input spikes)"}
            out["roofline"]["kernel"] = "snn_sparse_dw_spikes (slab records + dw_slab_spikes_kernel + chunk reduction)"
            out["roofline"]["alu_view"]["resource"] = "float64 LDS adds (multiply on the VALU)"
            out["roofline"]["traffic"] = None
        if out["dense_backward_ms"] is not None:
            out["dense_mfma_tflops"] = dense_flops / (out["dense_backward_ms"] * 1e-3) / 1e12
            out["dense_mfma_frac"] = out["dense_mfma_tflops"] / MFMA_F32_TFLOPS
            out["speedup_vs_dense"] = out["dense_backward_ms"] / out["sparse_backward_ms"]
            out["overall_speedup_fwd_plus_bwd"] = (out["forward_ms"] + out["dense_backward_ms"]) / (
                out["forward_ms"] + out["sparse_backward_ms"])
        return out


def build_parser() -> argparse.ArgumentParser:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)  # stress: ~2 s of timed GPU work
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="stress")
    ap.add_argument("--b-th", type=float, default=None)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-samples", type=int, default=16)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--serial", action="store_true", help="everything on one stream")
    ap.add_argument("--conv-csr", action="store_true",
                    help="conv workload: the sparse chain through the conv layer's CSR and routing instead of the "
                         "pooled entries alone")
    ap.add_argument("--unfused", action="store_true",
                    help="compaction reads V instead of the active bitsets the forward marks")
    ap.add_argument("--sweep", action="store_true", help="one JSON line per B_th of the workload's sweep")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB")
    ap.add_argument("--no-memory", action="store_true",
                    help="skip the allocator-peak memory measurement after the timed steps (for counter runs that "
                         "should hold the timed step's dispatches only)")
    ap.add_argument("--schedule", choices=("auto", "pipelined", "layerwise"), default="auto",
                    help="LIF layers' backward: pipelined (the dW layouts and the lower layers' compactions on a "
                         "side stream beside the spike-gradient chain) or layer by layer (auto: pipelined for two or "
                         "more LIF layers)")
    ap.add_argument("--dw-streams", type=int, default=0, metavar="N",
                    help="pipelined schedule: streams the dW calls take in turn, layer by layer (default 1: "
                         "in line with the spike gradients)")
    ap.add_argument("--recompute", type=int, default=0, metavar="K",
                    help="trace recompute: dW rebuilds the input trace from the spikes and checkpoints every K steps")
    ap.add_argument("--graph", action="store_true",
                    help="each library call of the step captured once as a HIP graph and replayed")
    ap.add_argument("--train", action="store_true",
                    help="training runs, sparse vs full surrogate (App. E); prints one JSON line")
    ap.add_argument("--train-workload", default="latency_train",
                    help="latency_train (784-200-10), deep (five LIF layers of 300) or conv (conv layer + pooling)")
    ap.add_argument("--train-steps", type=int, default=600)
    ap.add_argument("--train-batches", type=int, default=20, help="batches in the synthetic training set")
    ap.add_argument("--lr", type=float, default=2e-4)
    ap.add_argument("--nu-up", type=float, default=1.0)
    ap.add_argument("--train-bth", default="", help="comma-separated bands of the sparse runs (default: the workload's)")
    return ap


def main():
    args = build_parser().parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the path is single-device here (multi-GPU is design only)",
              file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.train:
        train_experiment(args)
        return

    from paper_2105_08810_amd import snn
    from synth import CONFIGS
    snn.lib()
    cfg = CONFIGS[args.workload]
    if cfg.conv and args.recompute:
        print("--recompute applies to the fully connected workloads", file=sys.stderr)
        sys.exit(2)
    run = ConvRunner(cfg, args) if cfg.conv else Runner(cfg, args)
    points = cfg.sweep() if args.sweep else (cfg.b_th if args.b_th is None else args.b_th,)
    dense_ms = None
    for k, b_th in enumerate(points):
        run.prepare(b_th)
        dense = not args.no_dense and (k == 0 or not args.sweep)  # the dense chain's cost does not depend on B_th
        evs, cs, wall = run.run(args.steps, args.warmup, dense)
        out = run.summarize(evs, cs, wall, dense)
        if not args.no_memory:
            mem = run.measured_memory()
            out["memory_saved_pct"] = [m[2] for m in mem]
            out["backward_peak_bytes_sparse_dense"] = [[m[0], m[1]] for m in mem]
        if dense:
            dense_ms = out["dense_backward_ms"]
        elif dense_ms is not None:
            out["dense_backward_ms"] = dense_ms
            out["speedup_vs_dense"] = dense_ms / out["sparse_backward_ms"]
            out["overall_speedup_fwd_plus_bwd"] = (out["forward_ms"] + dense_ms) / (
                out["forward_ms"] + out["sparse_backward_ms"])
        if not args.no_cpu and not args.sweep:
            out["cpu_baseline"] = cpu_baseline(cfg, b_th, args.cpu_samples)
        print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
