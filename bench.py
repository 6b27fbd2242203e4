"""Benchmark of the sparse spiking BPTT path on one MI355X.

One step = the whole path over one batch of the workload: LIF forward of every layer and
the readout, readout loss, active-set compaction of every LIF layer, the sparse backward
chain, and the dense matrix-core baseline chain. HIP events on the launch stream time each
part; the headline is the sparse backward (compaction + snn_sparse_backward of every LIF
layer; the readout's own backward and the loss are outside both chains).

Prints ONE JSON line. `value` = active neuron-steps per second of the sparse backward
(sum over LIF layers of the active entries, divided by its time); the dense time and the
speedup are in the same line. Inputs are resident in HBM before timing starts.

    python bench.py [--steps K] [--warmup W] [--workload stress] [--b-th 0.2] [--no-cpu]
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
FP32_PEAK_TFLOPS = 157.3
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_sparse_backward_stress.json")
CSRC = os.path.join(ROOT, "paper_2105_08810_amd", "csrc")


def csrc_digest() -> str:
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def algorithmic(T, B, n_in, n_out, nnz_out, r_out, nnz_in=None):
    """Gathered bytes and flops of one layer's sparse backward.

    bytes: trace rows with at least one active output, the output CSR (index, g, eps), the
    row pointers and the dW write; with a spike gradient also W once, the input CSR index and
    the eps_in write, and its row pointers. flops: 2 per multiply-add of the sparse dW and
    grad_in sums plus the delta recurrence.
    """
    TB = T * B
    by = 4 * n_in * r_out + 12 * nnz_out + 4 * (TB + 1) + 4 * n_in * n_out
    fl = 2 * nnz_out * n_in
    if nnz_in is not None:
        by += 4 * n_in * n_out + 8 * nnz_in + 4 * (TB + 1)
        fl += 2 * nnz_in * n_out + 2 * TB * n_out
    return by, fl


def cpu_baseline(cfg, b_th, n_samples):
    """The oracle's backward (compaction + dense-truncated BPTT, fp64 BLAS) on a batch subset."""
    import oracle
    from synth import make_inputs
    try:
        from threadpoolctl import threadpool_info
        blas = [(d.get("internal_api"), d.get("num_threads")) for d in threadpool_info()]
    except Exception:  # pragma: no cover
        blas = []
    inp = make_inputs(cfg, list(range(n_samples)))
    f = oracle.network_forward(inp.X, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, np.float32(cfg.theta))
    t0 = time.perf_counter()
    nnz = 0
    for V in f["V"]:
        rp, _, _ = oracle.active_csr(V, cfg.theta, b_th, cfg.beta)
        nnz += int(rp[-1])
    oracle.network_backward(f, inp.Ws, inp.W_out, inp.alphas, inp.alpha_out, inp.labels, cfg.loss_mode,
                            cfg.theta, b_th, cfg.beta)
    dt = time.perf_counter() - t0
    threads = max([n for _, n in blas if n] or [1])
    return {"value": nnz / dt, "unit": "active neuron-steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{cfg.name} workload, batch samples 0..{n_samples - 1} of {cfg.B}, B_th={b_th}: "
                      f"compaction + fp64 backward of all layers, {dt:.2f} s, {nnz} active entries",
            "host_cpus": len(os.sched_getaffinity(0)), "blas": blas}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="stress")
    ap.add_argument("--b-th", type=float, default=None)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-samples", type=int, default=16)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--serial", action="store_true", help="no auxiliary stream in the sparse backward")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the path is single-device here (multi-GPU is design only)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2105_08810_amd import pipeline, snn
    from synth import CONFIGS, make_inputs

    snn.lib()
    cfg = CONFIGS[args.workload]
    b_th = cfg.b_th if args.b_th is None else args.b_th
    inp = make_inputs(cfg)
    net = pipeline.from_inputs(inp, "cuda:0").allocate()
    T, B, L = net.T, net.B, net.L
    sizes = list(cfg.sizes)

    # size everything once (the first compaction counts; inputs are fixed so nnz is too)
    net.forward()
    ro = net.readout(dense=not args.no_dense)
    csrs = net.compact(b_th)
    caps = [c.capacity for c in csrs]
    ws_sp = [snn.workspace(snn.snn_sparse_backward_workspace(T, B, sizes[l], sizes[l + 1], caps[l]))
             for l in range(L)]
    ws_ro = snn.workspace(snn.snn_sparse_backward_workspace(T, B, sizes[L], sizes[L + 1], ro[0].capacity))
    ws_dn = None if args.no_dense else snn.workspace(
        max(snn.snn_dense_backward_workspace(T, B, sizes[l], sizes[l + 1]) for l in range(L + 1)))
    stream = torch.cuda.current_stream()
    aux = None if args.serial else torch.cuda.Stream()  # default priority

    def step(ev):
        ev[0].record(stream)
        net.forward()
        ev[1].record(stream)
        r = net.readout(dense=not args.no_dense)
        ev[2].record(stream)
        cs = net.compact(b_th, caps)
        ev[3].record(stream)
        dW_out, eps = snn.sparse_backward(net.W_out, net.trace_out, net.alpha_out, r[0], r[1], inp=cs[L - 1],
                                          ws=ws_ro, aux_stream=aux)
        ev[4].record(stream)
        for l in range(L - 1, -1, -1):
            ev[5 + 2 * (L - 1 - l)].record(stream)
            _, eps = snn.sparse_backward(net.Ws[l], net.trace[l], net.alphas[l], cs[l], eps,
                                         inp=cs[l - 1] if l > 0 else None, ws=ws_sp[l], aux_stream=aux)
            ev[6 + 2 * (L - 1 - l)].record(stream)
        k = 5 + 2 * L
        if not args.no_dense:
            _, e = snn.dense_backward_ref(net.W_out, net.trace_out, net.V_out, r[3], net.alpha_out, math.inf,
                                          math.inf, net.beta, grad_in=True, ws=ws_dn)
            ev[k].record(stream)
            for l in range(L - 1, -1, -1):
                _, e = snn.dense_backward_ref(net.Ws[l], net.trace[l], net.V[l], e, net.alphas[l], net.theta, b_th,
                                              net.beta, grad_in=l > 0, ws=ws_dn)
            ev[k + 1].record(stream)
        else:
            ev[k].record(stream)
            ev[k + 1].record(stream)
        return cs

    n_ev = 7 + 2 * L
    for _ in range(args.warmup):
        step([torch.cuda.Event(enable_timing=True) for _ in range(n_ev)])
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(n_ev)] for _ in range(args.steps)]
    t_wall0 = time.perf_counter()
    for k in range(args.steps):
        cs = step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall0

    def span(a, b):
        return np.array([e[a].elapsed_time(e[b]) for e in evs])  # ms

    t_fwd = span(0, 1)
    t_cmp = span(2, 3)
    t_layers = [span(5 + 2 * i, 6 + 2 * i) for i in range(L)]  # top layer first
    t_sparse = t_cmp + sum(t_layers)
    t_dense = span(5 + 2 * L, 6 + 2 * L)
    t_step = span(0, 6 + 2 * L)

    # active entries and algorithmic bytes (bookkeeping outside the timed steps)
    nnz = [c.nnz() for c in cs]
    r_out = [int((c.row_ptr[1:] > c.row_ptr[:-1]).sum().item()) for c in cs]
    by_l, fl_l = [], []
    for l in range(L):
        by, fl = algorithmic(T, B, sizes[l], sizes[l + 1], nnz[l], r_out[l], nnz[l - 1] if l > 0 else None)
        by_l.append(by)
        fl_l.append(fl)
    med = lambda a: float(np.median(a))  # noqa: E731
    t_bwd_kernels = sum(med(t) for t in t_layers)  # snn_sparse_backward of all LIF layers
    gb = sum(by_l)
    achieved = gb / (t_bwd_kernels * 1e-3) / 1e9
    flops = sum(fl_l)
    value = sum(nnz) / (med(t_sparse) * 1e-3)

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("csrc_digest") == csrc_digest() and tr.get("workload") == f"{cfg.name}:{b_th}":
            traffic = tr.get("bytes_per_step")

    out = {
        "metric": "sparse backward ms/batch + active neuron-steps/s, speedup vs dense BPTT",
        "value": value,
        "unit": "active neuron-steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": med(t_step),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.description}; B_th={b_th}", "T": T, "B": B,
                   "sizes": sizes, "b_th": b_th, "alpha": float(cfg.alpha), "beta": cfg.beta},
        "sparse_backward_ms": med(t_sparse),
        "sparse_backward_ms_iqr": [float(np.percentile(t_sparse, 25)), float(np.percentile(t_sparse, 75))],
        "compaction_ms": med(t_cmp),
        "sparse_layer_ms": [med(t) for t in reversed(t_layers)],
        "dense_backward_ms": None if args.no_dense else med(t_dense),
        "speedup_vs_dense": None if args.no_dense else med(t_dense) / med(t_sparse),
        "forward_ms": med(t_fwd),
        "overall_speedup_fwd_plus_bwd": None if args.no_dense else (med(t_fwd) + med(t_dense)) / (
            med(t_fwd) + med(t_sparse)),
        "active_fraction": [n / (T * B * sizes[l + 1]) for l, n in enumerate(nnz)],
        "nnz": nnz,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "snn_sparse_backward, all LIF layers per step",
                     "algorithmic_bytes": gb, "algorithmic_flops": flops,
                     "alu_frac": flops / (t_bwd_kernels * 1e-3) / 1e12 / FP32_PEAK_TFLOPS,
                     "launch_ms": t_bwd_kernels},
        "wall_s_timed": wall,
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(cfg, b_th, args.cpu_samples)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
