"""bench.py's host-side logic and its output contract.

CPU: the one-GPU guard, the algorithmic byte and flop counts against a hand count, and the
App. H statistics against the oracle's. GPU: one short run of the default line on the tiny
workload and of the training mode, checked for the fields the line must carry.
"""
import json
import math
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env=None, timeout=600):
    e = dict(os.environ)
    e.update(env or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          env=e, timeout=timeout)


@pytest.mark.parametrize("args,env", [(["--gpus", "2"], None), ([], {"WORLD_SIZE": "4"})])
def test_more_than_one_gpu_is_refused(args, env):
    r = _run(args, env)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_recompute_is_refused_for_conv():
    r = _run(["--workload", "conv", "--recompute", "8"])
    assert r.returncode == 2
    assert "fully connected" in r.stderr


def test_algorithmic_counts_by_hand():
    # T=2, B=3, 5 inputs, 4 outputs; 7 active outputs on 4 rows, 6 input-active entries
    by_dw, fl_dw, by_gi, fl_gi = bench.algorithmic(2, 3, 5, 4, nnz_out=7, r_out=4, nnz_in=6)
    assert by_dw == 4 * 5 * 4 + 12 * 7 + 4 * 7 + 4 * 5 * 4
    assert fl_dw == 2 * 7 * 5
    assert by_gi == 4 * 5 * 4 + 8 * 6 + 4 * 7
    assert fl_gi == 2 * 6 * 4 + 2 * 6 * 4
    assert bench.algorithmic(2, 3, 5, 4, 7, 4)[2:] == (0, 0)


def test_grad_difference_matches_oracle():
    r = np.random.default_rng(2)
    full = r.standard_normal((30, 20))
    sparse = full + 0.05 * r.standard_normal((30, 20))
    sparse[full == full.max()] = 0.0
    a = bench._grad_difference(sparse, full)
    b = oracle.gradient_difference(sparse, full)
    for k in b:
        assert a[k] == pytest.approx(b[k], rel=1e-12)


def test_roofline_peaks():
    assert bench.HBM_PEAK_GBS == 8000.0
    assert bench.MFMA_F32_TFLOPS == 157.3


def test_forward_bytes_by_hand():
    # T=2, B=3; 5 inputs, one LIF layer of 4, readout of 2; bitsets marked for the LIF layer only
    TB = 6
    lif = TB * 5 + 4 * 5 * 4 + 4 * TB * 4 + TB * 4 + 4 * TB * 5
    ro = TB * 4 + 4 * 4 * 2 + 4 * TB * 2 + TB * 2 + 4 * TB * 4
    bits = 2 * ((3 * 4 + 63) // 64) * 8
    assert bench.forward_bytes(2, 3, [5, 4, 2], bits=False) == lif + ro
    assert bench.forward_bytes(2, 3, [5, 4, 2], bits=True) == lif + ro + bits


@pytest.mark.gpu
def test_bench_line_on_tiny():
    r = _run(["--workload", "tiny", "--steps", "3", "--warmup", "1"])
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in line, k
    assert line["n_gpus"] == 1 and line["steps"] == 3 and line["warmup"] == 1
    assert line["config"]["workload"].startswith("tiny")
    rl = line["roofline"]
    assert rl["bound"] == "hbm" and rl["peak"] == bench.HBM_PEAK_GBS and rl["unit"] == "GB/s" and 0 < rl["frac"] < 1
    assert math.isclose(rl["frac"], rl["achieved"] / rl["peak"], rel_tol=1e-9)
    # achieved = algorithmic bytes per launch / average launch time
    per_launch_s = sum(rl["launch_ms"]) * 1e-3 / rl["launches"]
    assert math.isclose(rl["achieved"], rl["algorithmic_bytes_per_launch"] / per_launch_s / 1e9, rel_tol=1e-9)
    av = rl["alu_view"]
    assert av["peak"] == bench.MFMA_F32_TFLOPS and math.isclose(av["frac"], av["achieved"] / av["peak"])
    assert 0 < rl["chain_hbm_frac"] < 1 and 0 < line["forward_hbm_frac"] < 1
    # memory from the allocator's peaks, beside the analytic figure
    peaks = line["backward_peak_bytes_sparse_dense"]
    assert len(peaks) == len(line["memory_saved_pct"]) == len(line["memory_saved_pct_analytic"])
    for (sp, dn), pct in zip(peaks, line["memory_saved_pct"]):
        assert sp > 0 and dn > 0 and math.isclose(pct, 100.0 * (dn - sp) / dn)
    cb = line["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb["value"] > 0
    assert line["value"] > 0 and line["sparse_backward_ms"] > 0 and line["dense_backward_ms"] > 0


@pytest.mark.gpu
def test_bench_train_mode_short():
    r = _run(["--train", "--train-steps", "20", "--train-batches", "2", "--train-bth", "0.2"])
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["mode"] == "train" and line["steps"] == 20
    for run in ("sparse_bth_0.2", "full_surrogate"):
        assert len(line[run]["ce"]) == 20 and all(np.isfinite(line[run]["ce"]))
        assert line[run]["ce"][-1] < line[run]["ce"][0]  # 20 Adam steps lower the loss
    assert len(line["grad_difference_init"]) == 3


@pytest.mark.gpu
@pytest.mark.parametrize("extra", [[], ["--dw-streams", "1"]])
def test_bench_pipelined_schedule_matches_layerwise(extra):
    """The bench's pipelined schedule (dW layouts and calls on dW streams beside the spike-gradient
    chain) computes the active sets, dW and spike gradients of the layer-by-layer schedule, bit for
    bit (deep workload: five LIF layers)."""
    import torch
    from synth import CONFIGS
    print(f"\n[case] bench schedules, deep, {extra}", flush=True)
    runs = []
    for sched in ("pipelined", "layerwise"):
        args = bench.build_parser().parse_args(["--workload", "deep", "--no-dense", "--no-cpu", "--schedule", sched]
                                               + extra)
        r = bench.Runner(CONFIGS["deep"], args)
        r.prepare(0.2)
        cs = r.step(r.events(), dense=False)
        torch.cuda.synchronize()
        runs.append((r, cs))
    (a, ca), (b, cb) = runs
    assert a.pipelined and not b.pipelined
    for l in range(a.L):
        n = cb[l].nnz()
        assert n > 0 and ca[l].nnz() == n
        assert torch.equal(ca[l].row_ptr, cb[l].row_ptr) and torch.equal(ca[l].col_idx[:n], cb[l].col_idx[:n])
        assert torch.equal(a.dW[l], b.dW[l]), f"dW[{l}]"
        if l < a.L - 1:
            assert torch.equal(a.eps[l][:n], b.eps[l][:n]), f"eps[{l}]"


@pytest.mark.gpu
@pytest.mark.parametrize("extra", [[], ["--conv-csr", "--no-dense"]])
def test_bench_line_on_conv(extra):
    """The conv workload's bench line (pooled-entry chain by default, the conv-CSR chain with
    --conv-csr): the contract's keys, positive timings, the same active-entry counts either way."""
    print(f"\n[case] bench conv {extra}", flush=True)
    r = _run(["--workload", "conv", "--steps", "2", "--warmup", "1", "--no-cpu"] + extra)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "config", "sparse_backward_ms",
              "compaction_ms", "sparse_chain", "nnz", "pooled_active_entries", "memory_saved_pct", "roofline"):
        assert k in line, k
    assert line["config"]["workload"].startswith("conv")
    assert line["value"] > 0 and line["sparse_backward_ms"] > 0 and line["compaction_ms"] > 0
    assert line["nnz"][0] > line["pooled_active_entries"] > 0
    assert ("conv-layer CSR" in line["sparse_chain"]) == ("--conv-csr" in extra)
    rl = line["roofline"]
    assert rl["bound"] == "hbm" and 0 < rl["frac"] < 1 and math.isclose(rl["frac"], rl["achieved"] / rl["peak"])
    # the roofline covers the whole chain; the pooled active set is a secondary figure
    assert math.isclose(rl["launch_ms"], line["sparse_backward_ms"]) and 0 < rl["pooled_active_set"]["frac"] < 1
    assert 0 < line["value_pooled_entries"] < line["value"]
    if "--no-dense" not in extra:
        assert line["dense_backward_ms"] > 0 and line["speedup_vs_dense"] > 1
