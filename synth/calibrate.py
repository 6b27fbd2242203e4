"""Freeze the weight scales of the synthetic workloads into synth/gains.json.

The paper's initialisation U(-sqrt(N), sqrt(N)) (App. E) is not usable as
printed (it would saturate every neuron), so the workloads use
    W_l ~ N(0, sigma_l^2),  sigma_l = kappa / sqrt(m_l),  kappa = 0.4 sqrt(1 - alpha_l^2),
which gives a steady-state membrane standard deviation near 0.4 when m_l
spiking inputs arrive per (t, b) row. m_1 is measured on the generated input
spikes; m_l for deeper layers on the spikes of layer l-1 of a pilot forward
(the oracle's LIF forward on the first PILOT_B samples). The script also records
the active fraction of each layer at the default band.

Run:  python -m synth.calibrate
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from synth.inputs import CONFIGS, _GAINS_PATH, make_spikes, rng_for  # noqa: E402
import oracle  # noqa: E402

PILOT_B = 16
KAPPA_SD = 0.4


def calibrate_conv(name: str) -> dict:
    """Filters: m = mean spiking inputs in a neuron's 3x3xC patch per step (interior neurons)."""
    from oracle import conv as oconv
    from synth.inputs import make_conv_inputs
    cfg = CONFIGS[name]
    H, W, C, F = cfg.conv
    batch = list(range(min(PILOT_B, cfg.B)))
    x = make_spikes(cfg, batch)
    m = 9.0 * C * float((x != 0).mean())
    s = KAPPA_SD * math.sqrt(1.0 - float(cfg.alpha) ** 2) / math.sqrt(m)
    inp = make_conv_inputs(cfg, batch[:4], sigmas=[s, 1.0 / math.sqrt((H // 2) * (W // 2) * F)])
    f = oconv.conv_network_forward(inp.X, inp.Wc, inp.W_out, cfg.alpha, cfg.alpha_out, cfg.theta)
    rho = float(oracle.active_mask(f["V"], cfg.theta, cfg.b_th).mean())
    return {"sigma": [s], "m": [m], "rho_pilot_default_bth": [rho], "pilot_batch": 4, "b_th": cfg.b_th}


def calibrate(name: str) -> dict:
    cfg = CONFIGS[name]
    if cfg.conv:
        return calibrate_conv(name)
    batch = list(range(min(PILOT_B, cfg.B)))
    x = make_spikes(cfg, batch)
    sig, m_list, rho = [], [], []
    for l in range(cfg.n_layers):
        alpha = float(cfg.alpha)
        kappa = KAPPA_SD * math.sqrt(1.0 - alpha * alpha)
        m = float((x != 0).sum()) / (x.shape[0] * x.shape[1])
        s = kappa / math.sqrt(m)
        z = rng_for(cfg.cfg_id, 10 + l + 1).standard_normal((cfg.sizes[l], cfg.sizes[l + 1]))
        W = (z * s).astype(np.float32)
        V, S, _ = oracle.lif_forward(x, W, cfg.alpha, np.float32(cfg.theta))
        r = float(oracle.active_mask(V, cfg.theta, cfg.b_th).mean())
        sig.append(s)
        m_list.append(m)
        rho.append(r)
        x = S
    return {"sigma": sig, "m": m_list, "rho_pilot_default_bth": rho, "pilot_batch": len(batch),
            "b_th": cfg.b_th}


def main(names=None):
    names = names or [n for n in CONFIGS if n != "tiny"]
    out = {}
    if os.path.exists(_GAINS_PATH):
        with open(_GAINS_PATH) as f:
            out = json.load(f)
    for n in names:
        out[n] = calibrate(n)
        print(n, json.dumps(out[n]))
    with open(_GAINS_PATH, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:])
