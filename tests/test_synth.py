"""The seeded generators: determinism, subsets, and the statistics each recipe promises."""
import numpy as np
import pytest

from synth import CONFIGS, make_inputs
from synth.inputs import make_spikes, event_peak_rate


def test_deterministic_and_subset_equals_slice():
    cfg = CONFIGS["audio"]
    a = make_spikes(cfg, [0, 5, 9])
    b = make_spikes(cfg, [5])
    assert np.array_equal(a[:, 1:2], b)
    assert np.array_equal(a, make_spikes(cfg, [0, 5, 9]))


def test_latency_fires_at_most_once():
    cfg = CONFIGS["latency"]
    x = make_spikes(cfg, range(32))
    per_input = x.sum(axis=0)
    assert per_input.max() == 1
    assert abs(per_input.mean() - 0.5) < 0.02
    assert abs(x.sum(axis=2).mean() - 3.92) < 0.1


@pytest.mark.parametrize("name,rate,tol", [("event", 0.010, 0.0015), ("audio", 0.0198, 0.001),
                                           ("stress", 0.02, 0.0005), ("tiny", 0.05, 0.01)])
def test_mean_rates(name, rate, tol):
    cfg = CONFIGS[name]
    x = make_spikes(cfg, range(min(cfg.B, 24)))
    assert abs(x.mean() - rate) < tol


def test_event_layout_is_polarity_grid():
    cfg = CONFIGS["event"]
    x = make_spikes(cfg, [0])[:, 0].reshape(cfg.T, 2, 34, 34)
    # bursts are spatially clustered: neighbouring pixels co-fire far above chance
    a = x[:, :, :, :-1].astype(float)
    b = x[:, :, :, 1:].astype(float)
    p = x.mean()
    assert (a * b).mean() > 3 * p * p
    assert 0.2 < event_peak_rate(cfg.T) < 0.6


def test_inputs_bundle_shapes():
    for name, cfg in CONFIGS.items():
        inp = make_inputs(cfg, [0, 1])
        assert inp.X.shape == (cfg.T, 2, cfg.sizes[0]) and inp.X.dtype == np.uint8
        assert [W.shape for W in inp.Ws] == [(cfg.sizes[l], cfg.sizes[l + 1]) for l in range(cfg.n_layers)]
        assert inp.W_out.shape == (cfg.sizes[-2], cfg.sizes[-1]) and inp.W_out.dtype == np.float32
        assert inp.labels.shape == (2,) and inp.labels.max() < cfg.sizes[-1]
